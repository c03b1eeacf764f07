// Device-side arithmetic of the ECASQ approximate DP (arXiv 2608.18147).
//
// Every function here evaluates one fixed fp64 operation sequence (the
// library is built with -ffp-contract=off, so fma appears only where written)
// so that results are reproducible bit for bit:
//
//   interval (v_a, v_b], a < b, from inclusive prefix sums (App. D):
//     n = N[b]-N[a]  sa = S[b]-S[a]  s2 = S2[b]-S2[a]  w = v_b-v_a
//     tu = fma(-v_a, n, sa)    (= w * U[a,b])
//     td = fma(v_b, n, -sa)    (= w * D[a,b])
//     C  = fma(v_b, tu, fma(v_a, sa, -s2))     (= C_P[a,b])
//   surrogate-entropy term of one interval (Sec. 5, Phi and Phi^first):
//     g = 1/(w*d)  yu = tu*g  yd = td*g (+ c0/d for the first interval)
//     P = fma(max(yu,0), log2c(yu), max(yd,0)*log2c(yd))     (P = -Phi)
//   DP candidate (eq. apx_rec):  fma(-lambda', P, F_prev + C)
//   refinement / output entropy (Sec. 6):
//     U = tu*(1/w)  D = td*(1/w)   h(f) = -(max(y,0)*log2c(y)),  y = f/d
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "log2_table.inc"

namespace ecasq {

// Table-driven log2 (Tang 1990 style).  y = 2^e z with z in [0.7073, 1.4147)
// chosen by subtracting an offset from the high word; the top 8 bits of the
// reduced mantissa select {1/c, log2 c}; r = z/c - 1 (|r| <= 2^-9) feeds the
// degree-6 series of log1p, scaled by RN(1/ln 2).  Finite for every finite y;
// about one ulp for positive normal y.  tab points to the table in LDS.
__device__ __forceinline__ double log2c(double y, const double2* __restrict__ tab) {
    const uint32_t hi = (uint32_t)__double2hiint(y);
    const uint32_t lo = (uint32_t)__double2loint(y);
    const uint32_t tmp = hi - ECASQ_LOG2_OFF_HI;
    const int32_t e = ((int32_t)tmp) >> 20;
    const uint32_t i = (tmp >> 12) & 0xFFu;
    const uint32_t zhi = hi - (tmp & 0xFFF00000u);
    const double z = __hiloint2double((int)zhi, (int)lo);
    const double2 t = tab[i];
    const double r = __builtin_fma(z, t.x, -1.0);
    double q = -1.0 / 6.0;
    q = __builtin_fma(q, r, 1.0 / 5.0);
    q = __builtin_fma(q, r, -0.25);
    q = __builtin_fma(q, r, 1.0 / 3.0);
    q = __builtin_fma(q, r, -0.5);
    q = __builtin_fma(q, r, 1.0);
    const double lp = r * q;
    const double base = (double)e + t.y;
    return __builtin_fma(0x1.71547652b82fep+0, lp, base);
}

// h(y) = -y log2 y for y > 0, 0 otherwise (Sec. 4).
__device__ __forceinline__ double hfun(double y, const double2* __restrict__ tab) {
    return -(__builtin_fmax(y, 0.0) * log2c(y, tab));
}

// C and P (= -Phi, or -Phi^first when `first`) of the interval (v_a, v_b].
__device__ __forceinline__ void cell_terms(double va, double Na, double Sa, double S2a, double vb,
                                           double Nb, double Sb, double S2b, double dd, bool first,
                                           double c0d, const double2* __restrict__ tab, double& C,
                                           double& P) {
    const double n = Nb - Na;
    const double sa = Sb - Sa;
    const double s2 = S2b - S2a;
    const double w = vb - va;
    const double tu = __builtin_fma(-va, n, sa);
    const double td = __builtin_fma(vb, n, -sa);
    C = __builtin_fma(vb, tu, __builtin_fma(va, sa, -s2));
    const double wd = w * dd;
    const double g = 1.0 / wd;
    const double yu = tu * g;
    double yd = td * g;
    if (first) yd = yd + c0d;
    const double lu = log2c(yu, tab);
    const double ld = log2c(yd, tab);
    P = __builtin_fma(__builtin_fmax(yu, 0.0), lu, __builtin_fmax(yd, 0.0) * ld);
}

// U and D of (v_a, v_b] in the refinement (inv) form.
__device__ __forceinline__ void interval_ud(double va, double Na, double Sa, double vb, double Nb,
                                            double Sb, double& U, double& D) {
    const double n = Nb - Na;
    const double sa = Sb - Sa;
    const double w = vb - va;
    const double tu = __builtin_fma(-va, n, sa);
    const double td = __builtin_fma(vb, n, -sa);
    const double inv = 1.0 / w;
    U = tu * inv;
    D = td * inv;
}

// Histogram view passed to the small (one-thread or one-block) kernels.
struct Hist {
    const double* v;
    const double* N;
    const double* S;
    const double* S2;
    int64_t p;
    double dd;   // d as a double
    double c0;   // count of v_0
    double c0d;  // RN(c0 / d)
};

__device__ __forceinline__ void cell_at(const Hist& H, int64_t a, int64_t b,
                                        const double2* __restrict__ tab, double& C, double& P) {
    cell_terms(H.v[a], H.N[a], H.S[a], H.S2[a], H.v[b], H.N[b], H.S[b], H.S2[b], H.dd, a == 0,
               H.c0d, tab, C, P);
}

__device__ __forceinline__ void ud_at(const Hist& H, int64_t a, int64_t b, double& U, double& D) {
    interval_ud(H.v[a], H.N[a], H.S[a], H.v[b], H.N[b], H.S[b], U, D);
}

__device__ __forceinline__ double hf(const Hist& H, double f, const double2* __restrict__ tab) {
    return hfun(f / H.dd, tab);
}

// Copy the log2 table into LDS (call from all threads, then __syncthreads()).
__device__ __forceinline__ void load_log2_table(double2* lds) {
    for (int i = threadIdx.x; i < 256; i += blockDim.x)
        lds[i] = make_double2(kLog2Table[i][0], kLog2Table[i][1]);
}

}  // namespace ecasq
