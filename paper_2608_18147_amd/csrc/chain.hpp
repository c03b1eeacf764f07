// Codebook-chain quantities shared by the refinement and metrics kernels and
// the batched row solver: expected output frequencies and H(Xhat) of a chain
// of distinct-value indices (Sec. 4, Sec. 6), and the local Sec. 6 objective
// of moving one value.
#pragma once
#include "device.hpp"

namespace ecasq {

__device__ __forceinline__ double interval_cost(const Hist& H, int64_t a, int64_t b,
                                                const double2* tab) {
    double C, P;
    cell_at(H, a, b, tab, C, P);
    return C;
}

// Expected frequencies of a chain u_0 < ... < u_{t-1} (Sec. 4: an interior
// value gets U[k,l] + D[l,j]; the first value also takes every entry equal to
// it; the last gets the round-up mass of the last interval), then
// H(Xhat) = sum_q h(f_q / d), summed in index order.
__device__ __forceinline__ double chain_hout(const Hist& H, int32_t t, const int32_t* u, const double2* tab) {
    if (t == 1) return hf(H, H.dd, tab);
    double Hs = 0.0, Uprev = 0.0;
    for (int32_t r = 0; r < t; r++) {
        double Ur = 0.0, Dr = 0.0;
        if (r + 1 < t) ud_at(H, u[r], u[r + 1], Ur, Dr);
        double f;
        if (r == 0) f = H.c0 + Dr;
        else if (r == t - 1) f = Uprev;
        else f = Uprev + Dr;
        Hs = Hs + hf(H, f, tab);
        Uprev = Ur;
    }
    return Hs;
}

// Local Sec. 6 objective of placing u_r at m (neighbours fixed): the MSE of
// the two adjacent intervals plus lambda' times the entropy terms of the
// three values whose expected frequencies change.
__device__ __forceinline__ double refine_local(const Hist& H, int32_t t, const int32_t* u, int32_t r, int64_t m,
                               double lamp, const double2* tab) {
    const int64_t L = u[r - 1], R = u[r + 1];
    const double Cl = interval_cost(H, L, m, tab);
    const double Cr = interval_cost(H, m, R, tab);
    double Ulm, Dlm, Umr, Dmr;
    ud_at(H, L, m, Ulm, Dlm);
    ud_at(H, m, R, Umr, Dmr);
    double fprev, fnext;
    if (r - 1 == 0) {
        fprev = H.c0 + Dlm;
    } else {
        double Ua, Da;
        ud_at(H, u[r - 2], L, Ua, Da);
        fprev = Ua + Dlm;
    }
    const double fcur = Ulm + Dmr;
    if (r + 1 == t - 1) {
        fnext = Umr;
    } else {
        double Ub, Db;
        ud_at(H, R, u[r + 2], Ub, Db);
        fnext = Umr + Db;
    }
    const double Hl = (hf(H, fprev, tab) + hf(H, fcur, tab)) + hf(H, fnext, tab);
    return __builtin_fma(lamp, Hl, Cl + Cr);
}

}  // namespace ecasq
