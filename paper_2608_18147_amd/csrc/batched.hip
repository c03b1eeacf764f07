// Many short vectors in one launch: one wavefront solves one row end to end
// with everything in LDS (sort, exact prefix sums, the lambda search over
// dp_APX solves, recovery, refinement, metrics), several rows per workgroup
// sharing one copy of the log2 table.
//
// Per row the steps are those of the single-vector path (Sec. 2 histogram,
// App. D prefix sums, Sec. 5 eq. apx_base/apx_rec/apx_final, Sec. 3/Sec. 5
// lambda search, Sec. 6 refinement).  Every solve traces its chain back at
// once and keeps it with the solve (two buffers, so that the best feasible
// solve's chain survives the later queries): the sweep over predecessors
// keeps layer values only and recomputes each argmin along the chain; the
// layer-by-layer solver (long rows) keeps the argmins of every layer (s x p
// int16 in LDS).  At these sizes Hirschberg's O(p) bound buys nothing.
//
// Columns sit in lanes (column j = 64c + lane, c < CMAX); the predecessor k is
// uniform and read from LDS as a broadcast.  Column segments entirely at or
// below k are skipped, so only the segment crossing the diagonal carries
// masked lanes.
#include <hip/hip_fp16.h>

#include <initializer_list>

#include "../../include/ecasq.h"
#include "chain.hpp"
#include "device.hpp"
#include "launch.hpp"
#include "wide.hpp"

namespace ecasq {

namespace {

constexpr int kWave = 64;
constexpr int kMaxRows = 4;

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct RowLayout {
    uint32_t keys, v, N, S, S2, F0, F1, last, bp0, bp1, chain, nu, misc, srch, total;
};

__host__ __device__ inline uint32_t up16(uint32_t b) { return (b + 15u) & ~15u; }

// LDS bytes of one row: dpad keys, 4 fp64 arrays of dpad (v, N, S, S2), s+1
// last-column values, two int32 chains, scalars and the search state; the
// layer-by-layer solver (sweep = false) adds two fp64 layer buffers of dpad
// and two (s+1) x dpad int16 argmin tables, the sweep keeps only a chain of
// s+1 in each of the two.
__host__ __device__ inline RowLayout row_layout(int dpad, int s, bool sweep) {
    RowLayout L;
    uint32_t o = 0;
    auto take = [&](uint32_t b) {
        uint32_t at = o;
        o += up16(b);
        return at;
    };
    L.keys = take(4u * dpad);
    L.v = take(8u * dpad);
    L.N = take(8u * dpad);
    L.S = take(8u * dpad);
    L.S2 = take(8u * dpad);
    L.F0 = take(sweep ? 0u : 8u * dpad);
    L.F1 = take(sweep ? 0u : 8u * dpad);
    L.last = take(8u * (s + 1));
    L.bp0 = take(2u * (s + 1) * (sweep ? 1u : (uint32_t)dpad));
    L.bp1 = take(2u * (s + 1) * (sweep ? 1u : (uint32_t)dpad));
    L.chain = take(4u * (s + 1));
    L.nu = take(4u * (s + 1));
    L.misc = take(64);
    L.srch = take(256);  // RowSearch
    L.total = o;
    return L;
}

struct BatchArgs {
    const void* x;
    int64_t n;
    int32_t d, dpad, s, rows_per_block;
    double b;
    int32_t refine_rounds, refine_exhaustive, exact_s, max_passes;
    double* codebooks;
    int32_t* t_out;
    ecasq_info* infos;
};

struct Row {
    const double2* tab;
    double *v, *N, *S, *S2, *F0, *F1, *last;
    int16_t *bp0, *bp1;  // the two argmin buffers (selected, never indexed:
                         // a dynamic index would put the struct in scratch)
    int32_t *chain, *nu;
    double* misc;  // scratch scalars shared by the lanes of the row
    int p, s, dpad, lane;
    double dd, c0, c0d, s2tot;
    int64_t cells;
    int32_t solves;
};

__device__ __forceinline__ int16_t* argmin_buf(const Row& R, int buf) {
    return buf ? R.bp1 : R.bp0;
}

struct Pt {
    double lam, H, M;
    int t, buf;  // buf: argmin buffer holding this solve (-1: closed form)
};

// The budget search of one row, kept in LDS between its solves (written by
// lane 0): A = infeasible point of largest lambda, B = feasible point of
// smallest lambda, L = point of lowest H(I,B), P = the pair's feasible end;
// kind of the query in flight: 0 the first (lambda = 0), 1 the largest
// multiplier, 2 a chord query.
struct RowSearch {
    Pt A, B, L, P;
    double lam, lc, lamF;
    int haveA, haveB, tried40, npass, closed, status, kind, done, buf;
};
static_assert(sizeof(RowSearch) <= 256, "RowSearch fits its LDS slot");

// Values every lane of the wavefront holds alike, moved to scalar registers
// (the compiler cannot prove LDS loads or the wave index uniform).
__device__ __forceinline__ int uniform_i(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ double uniform_d(double x) {
    const int lo = __builtin_amdgcn_readfirstlane(__double2loint(x));
    const int hi = __builtin_amdgcn_readfirstlane(__double2hiint(x));
    return __hiloint2double(hi, lo);
}

__device__ __forceinline__ double readlane_d(double x, int l) {
    const int lo = __builtin_amdgcn_readlane(__double2loint(x), l);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(x), l);
    return __hiloint2double(hi, lo);
}

__device__ __forceinline__ Hist row_hist(const Row& R) {
    Hist H;
    H.v = R.v;
    H.N = R.N;
    H.S = R.S;
    H.S2 = R.S2;
    H.p = R.p;
    H.dd = R.dd;
    H.c0 = R.c0;
    H.c0d = R.c0d;
    return H;
}

// The solve's point from its chain u_0 .. u_{n-1} in R.nu: MSE and H(I,B)
// summed in path order (the same additions as accumulating them along the
// argmins); lane r evaluates the interval (u_r, u_{r+1}] (n <= s <= 32) and
// the sums run over the lanes in order.  The chain is kept in the first
// entries of argmin buffer `buf` (rows 0 and 1 of the table are never
// layers).
__device__ Pt row_chain_point(Row& R, double lam, int n, int buf) {
    const int lane = R.lane;
    const Hist H = row_hist(R);
    const int32_t* u = R.nu;
    double C = 0.0, P = 0.0;
    if (lane + 1 < n) cell_at(H, u[lane], u[lane + 1], R.tab, C, P);
    double mse = 0.0, ph = 0.0;
    for (int r = 0; r + 1 < n; r++) {
        mse = mse + readlane_d(C, r);
        ph = ph - readlane_d(P, r);
    }
    int16_t* keep = argmin_buf(R, buf);
    if (lane < n) keep[lane] = (int16_t)u[lane];
    Pt out;
    out.lam = lam;
    out.M = uniform_d(mse) / R.s2tot;
    out.H = uniform_d(ph);
    out.t = n;
    out.buf = buf;
    R.solves++;
    wave_sync();
    return out;
}

// eq. apx_final on R.last[2..imax]: the lowest i minimising F_i[p-1], or imax
// for exactly min(s, p) values.
__device__ __forceinline__ int row_istar(const Row& R, int imax, int exact_s) {
    int bi = 2;
    double bj = R.last[2];
    for (int i = 3; i <= imax; i++) {
        const double f = R.last[i];
        if (exact_s ? (i == imax) : (f < bj)) {
            bj = f;
            bi = i;
        }
    }
    return bi;
}

// eq. apx_final and the chain traced back through argmin buffer `buf`.
__device__ Pt row_final(Row& R, double lam, int imax, int exact_s, int buf) {
    const int p = R.p, lane = R.lane, dp = R.dpad;
    const int16_t* bp = argmin_buf(R, buf);
    if (lane == 0) {
        const int bi = row_istar(R, imax, exact_s);
        int32_t* u = R.nu;
        u[bi - 1] = p - 1;
        for (int i = bi; i >= 3; i--) u[i - 2] = bp[i * dp + u[i - 1]];
        u[0] = 0;
        R.misc[2] = (double)bi;
    }
    wave_sync();
    const int n = (int)uniform_d(R.misc[2]);
    wave_sync();
    return row_chain_point(R, lam, n, buf);
}

// The same solve as a sweep over predecessors k = 0..p-2 in increasing order
// that updates every layer of every later column from each cell, so C and Phi
// of a cell are evaluated once instead of once per layer.  Column k is final
// when the sweep reaches it (all its predecessors are behind); its layer
// values are broadcast from the lane that holds them.  LG >= imax - 2 layers
// of CMAX columns per lane live in registers, values only: the chain of the
// chosen layer is traced back afterwards, each argmin recomputed for its one
// column from the layer values the lanes still hold (lowest k among equal
// candidates, as the DP's strict '<' in increasing k).  At lambda = 0 every
// candidate is F + C (cell_c), a uniform branch per cell.
template <int CMAX, int LG>
__device__ Pt row_sweep(Row& R, double lam, int exact_s, int buf) {
    const bool zl = lam == 0.0;
    const double lamp = lam * R.s2tot;
    const int p = R.p, lane = R.lane;
    const int imax = R.s < p ? R.s : p;
    const Hist H = row_hist(R);
    double cv[CMAX], cN[CMAX], cS[CMAX], cS2[CMAX], f2[CMAX];
    double best[CMAX][LG];
#pragma unroll
    for (int c = 0; c < CMAX; c++) {
        const int j = c * kWave + lane;
        const int jj = j < p ? j : p - 1;
        cv[c] = R.v[jj];
        cN[c] = R.N[jj];
        cS[c] = R.S[jj];
        cS2[c] = R.S2[jj];
        // layer 2 (eq. apx_base); +inf where j = 0 has no interval
        f2[c] = __builtin_huge_val();
        if (j >= 1 && j < p) {
            double C, P;
            cell_at(H, 0, j, R.tab, C, P);
            f2[c] = __builtin_fma(-lamp, P, 0.0 + C);
        }
#pragma unroll
        for (int l = 0; l < LG; l++) best[c][l] = __builtin_huge_val();
    }
    const double dd = R.dd;
#pragma unroll
    for (int ck = 0; ck < CMAX; ck++) {
        if (ck * kWave > p - 2) break;
        for (int kk = 0; kk < kWave; kk++) {
            const int k = ck * kWave + kk;
            if (k > p - 2) break;
            // F_{i-1}[k] of every layer i = 3 + l, from the lane of column k
            double Fk[LG];
            Fk[0] = readlane_d(f2[ck], kk);
#pragma unroll
            for (int l = 1; l < LG; l++) Fk[l] = readlane_d(best[ck][l - 1], kk);
            const double pv = R.v[k], pN = R.N[k], pS = R.S[k], pS2 = R.S2[k];
            // the costs of (k, j) for this lane's columns from segment ck on
            // (segment ck at kk = 63 takes nothing); with entropy terms, every
            // column's log2 table reads are issued before any is used
            double Q[CMAX];
            if (zl) {
#pragma unroll
                for (int c = ck; c < CMAX; c++)
                    Q[c] = cell_c(pv, pN, pS, pS2, cv[c], cN[c], cS[c], cS2[c]);
            } else {
                double C[CMAX], mu[CMAX], md[CMAX];
                Log2Arg au[CMAX], ad[CMAX];
                double2 tu[CMAX], td[CMAX];
#pragma unroll
                for (int c = ck; c < CMAX; c++) {
                    cell_pre(pv, pN, pS, pS2, cv[c], cN[c], cS[c], cS2[c], dd, false, 0.0, C[c],
                             mu[c], md[c]);
                    au[c] = log2c_arg(mu[c]);
                    ad[c] = log2c_arg(md[c]);
                }
#pragma unroll
                for (int c = ck; c < CMAX; c++) {
                    tu[c] = R.tab[au[c].ir];
                    td[c] = R.tab[ad[c].ir];
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int c = ck; c < CMAX; c++) {
                    const double P = __builtin_fma(mu[c], log2c_fin(au[c], tu[c]),
                                                   md[c] * log2c_fin(ad[c], td[c]));
                    Q[c] = __builtin_fma(-lamp, P, C[c]);
                }
            }
#pragma unroll
            for (int c = ck; c < CMAX; c++) {
                const int j = c * kWave + lane;
                // columns at or below k take nothing from it
                const double q = j > k ? Q[c] : __builtin_huge_val();
#pragma unroll
                for (int l = 0; l < LG; l++) best[c][l] = __builtin_fmin(best[c][l], Fk[l] + q);
            }
        }
    }
    // F_i[p-1] of every layer for eq. apx_final
    const int cl = (p - 1) / kWave, ll = (p - 1) % kWave;
#pragma unroll
    for (int c = 0; c < CMAX; c++) {
        if (c == cl) {
            const double l2 = readlane_d(f2[c], ll);
            if (lane == 0) R.last[2] = l2;
#pragma unroll
            for (int l = 0; l < LG; l++) {
                const double v = readlane_d(best[c][l], ll);
                if (lane == 0 && 3 + l <= imax) R.last[3 + l] = v;
            }
        }
    }
    wave_sync();
    const int bi = uniform_i(row_istar(R, imax, exact_s));
    // traceback: layer i's argmin at the chain's column j from F_{i-1} (layer
    // i-1 = 3 + l held in best[.][l], layer 2 in f2), one (value, k) pair per
    // lane and column segment, then a butterfly over the wavefront
    int jc = p - 1;
    if (lane == 0) {
        R.nu[bi - 1] = p - 1;
        R.nu[0] = 0;
    }
#pragma unroll
    for (int l = LG - 1; l >= -1; l--) {
        const int i = l + 4;
        if (i > bi) continue;
        double bv = __builtin_huge_val();
        int bk = 0x7fffffff;
        const double jv = R.v[jc], jN = R.N[jc], jS = R.S[jc], jS2 = R.S2[jc];
#pragma unroll
        for (int c = 0; c < CMAX; c++) {
            const int k = c * kWave + lane;
            if (k >= i - 2 && k < jc) {
                double Q;
                if (zl) {
                    Q = cell_c(R.v[k], R.N[k], R.S[k], R.S2[k], jv, jN, jS, jS2);
                } else {
                    double C, P;
                    cell_terms(R.v[k], R.N[k], R.S[k], R.S2[k], jv, jN, jS, jS2, dd, false, 0.0,
                               R.tab, C, P);
                    Q = __builtin_fma(-lamp, P, C);
                }
                const double F = l >= 0 ? best[c][l >= 0 ? l : 0] : f2[c];
                const double cand = F + Q;
                if (cand < bv) {
                    bv = cand;
                    bk = k;
                }
            }
        }
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) {
            const double ov = __shfl_xor(bv, off);
            const int ok = __shfl_xor(bk, off);
            if (ov < bv || (ov == bv && ok < bk)) {
                bv = ov;
                bk = ok;
            }
        }
        jc = __builtin_amdgcn_readfirstlane(bk);
        if (lane == 0) R.nu[i - 2] = jc;
    }
    int64_t cells = p - 1;
    for (int i = 3; i <= imax; i++) cells += (int64_t)(p - i + 1) * (p - i + 2) / 2;
    R.cells += cells;
    wave_sync();
    return row_chain_point(R, lam, bi, buf);
}

// One dp_APX solve at lambda (vNMSE units) into argmin buffer `buf`; returns
// the lowest i minimising F_i[p-1] and, along its path, MSE and H(I,B) summed
// in path order (the same additions as accumulating them along the argmins).
template <int CMAX>
__device__ Pt row_solve(Row& R, double lam, int exact_s, int buf) {
    const double lamp = lam * R.s2tot;
    const int p = R.p, lane = R.lane, dp = R.dpad;
    const int imax = R.s < p ? R.s : p;
    int16_t* bp = argmin_buf(R, buf);
    const Hist H = row_hist(R);
    for (int j = 1 + lane; j < p; j += kWave) {
        double C, P;
        cell_at(H, 0, j, R.tab, C, P);
        const double f = __builtin_fma(-lamp, P, 0.0 + C);
        R.F0[j] = f;
        bp[2 * dp + j] = 0;
        if (j == p - 1) R.last[2] = f;
    }
    R.cells += p - 1;
    wave_sync();
    double* Fp = R.F0;
    double* Fc = R.F1;
    // column data of this lane
    double cv[CMAX], cN[CMAX], cS[CMAX], cS2[CMAX];
#pragma unroll
    for (int c = 0; c < CMAX; c++) {
        const int j = c * kWave + lane;
        const int jj = j < p ? j : p - 1;
        cv[c] = R.v[jj];
        cN[c] = R.N[jj];
        cS[c] = R.S[jj];
        cS2[c] = R.S2[jj];
    }
    for (int i = 3; i <= imax; i++) {
        double best[CMAX];
        int32_t bk[CMAX];
#pragma unroll
        for (int c = 0; c < CMAX; c++) {
            best[c] = __builtin_huge_val();
            bk[c] = -1;
        }
        for (int k = i - 2; k <= p - 2; k++) {
            const double pv = R.v[k], pN = R.N[k], pS = R.S[k], pS2 = R.S2[k], pF = Fp[k];
#pragma unroll
            for (int c = 0; c < CMAX; c++) {
                if (c * kWave + kWave - 1 <= k) continue;  // whole segment at or below k
                const int j = c * kWave + lane;
                double C, P;
                cell_terms(pv, pN, pS, pS2, cv[c], cN[c], cS[c], cS2[c], R.dd, false, 0.0, R.tab,
                           C, P);
                const double cand = pF + __builtin_fma(-lamp, P, C);
                const bool lt = (j > k) && (j < p) && cand < best[c];
                bk[c] = lt ? k : bk[c];
                best[c] = lt ? cand : best[c];
            }
        }
#pragma unroll
        for (int c = 0; c < CMAX; c++) {
            const int j = c * kWave + lane;
            if (j >= i - 1 && j < p) {
                Fc[j] = best[c];
                bp[i * dp + j] = (int16_t)bk[c];
                if (j == p - 1) R.last[i] = best[c];
            }
        }
        R.cells += (int64_t)(p - i + 1) * (p - i + 2) / 2;
        wave_sync();
        double* t = Fp;
        Fp = Fc;
        Fc = t;
    }
    return row_final(R, lam, imax, exact_s, buf);
}

// Sec. 6 refinement of the chain in R.chain (t values), one wavefront.
__device__ int row_refine(Row& R, int t, double lamp, double b, int budget, int rounds,
                          int exhaustive) {
    const Hist H = row_hist(R);
    const int lane = R.lane;
    int32_t* u = R.chain;
    int32_t* nu = R.nu;
    int nrun = 0;
    for (int rd = 0; rd < rounds; rd++) {
        bool any = false;
        for (int c = 0; c < 3; c++) {
            for (int r = lane; r < t; r += kWave) nu[r] = u[r];
            wave_sync();
            int moved = 0;
            if (!exhaustive) {
                bool mv = false;
                for (int r = 1 + lane; r <= t - 2; r += kWave) {
                    if (r % 3 != c) continue;
                    const int L = u[r - 1], Rr = u[r + 1];
                    if (Rr - L < 3) continue;
                    int lo = L + 1, hi = Rr - 1;
                    while (lo < hi) {
                        const int mid = lo + (hi - lo) / 2;
                        if (refine_local(H, t, u, r, mid + 1, lamp, R.tab) <
                            refine_local(H, t, u, r, mid, lamp, R.tab))
                            lo = mid + 1;
                        else
                            hi = mid;
                    }
                    if (lo != u[r] && refine_local(H, t, u, r, lo, lamp, R.tab) <
                                          refine_local(H, t, u, r, u[r], lamp, R.tab)) {
                        nu[r] = lo;
                        mv = true;
                    }
                }
                moved = __popcll(__ballot(mv));
            } else {
                for (int r = 1; r <= t - 2; r++) {
                    if (r % 3 != c) continue;
                    const int L = u[r - 1], Rr = u[r + 1];
                    if (Rr - L < 3) continue;
                    double bv = __builtin_huge_val();
                    int bm = -1;
                    for (int m = L + 1 + lane; m < Rr; m += kWave) {
                        const double val = refine_local(H, t, u, r, m, lamp, R.tab);
                        if (val < bv) {
                            bv = val;
                            bm = m;
                        }
                    }
                    for (int off = 32; off > 0; off >>= 1) {
                        const double ov = __shfl_xor(bv, off, kWave);
                        const int om = __shfl_xor(bm, off, kWave);
                        if (om >= 0 && (bm < 0 || ov < bv || (ov == bv && om < bm))) {
                            bv = ov;
                            bm = om;
                        }
                    }
                    if (bm != u[r] && bv < refine_local(H, t, u, r, u[r], lamp, R.tab)) {
                        if (lane == 0) nu[r] = bm;
                        moved++;
                    }
                }
            }
            wave_sync();
            if (moved && budget) {
                if (lane == 0) R.misc[3] = chain_hout(H, t, nu, R.tab) > b ? 1.0 : 0.0;
                wave_sync();
                if (R.misc[3] != 0.0) moved = 0;
            }
            if (moved) {
                for (int r = lane; r < t; r += kWave) u[r] = nu[r];
                any = true;
            }
            wave_sync();
        }
        nrun++;
        if (!any) break;
    }
    return nrun;
}

// File the point q of the query in flight (lane 0).
__device__ void row_search_file(RowSearch* Sr, const Pt& q, double b) {
    auto add = [&](const Pt& x) {
        if (x.H > b) {
            if (!Sr->haveA || x.lam > Sr->A.lam) Sr->A = x;
            Sr->haveA = 1;
        } else {
            if (!Sr->haveB || x.lam < Sr->B.lam) Sr->B = x;
            Sr->haveB = 1;
        }
        if (x.H < Sr->L.H) Sr->L = x;
    };
    if (Sr->kind == 0) {
        Sr->L = q;
        add(q);
        Sr->npass = 1;
    } else if (Sr->kind == 1) {
        add(q);
        Sr->tried40 = 1;
        Sr->npass++;
    } else {
        Sr->npass++;
        if ((q.H == Sr->A.H && q.M == Sr->A.M) || (q.H == Sr->P.H && q.M == Sr->P.M)) {
            Sr->lamF = Sr->lc;
            Sr->done = 1;
        } else {
            add(q);
        }
    }
}

// Decide the next query from the points filed so far, or end the search
// (lane 0).
__device__ void row_search_next(RowSearch* Sr, const Row& R, double b, int max_passes,
                                const double2* __restrict__ tab) {
    if (!Sr->haveA) {  // lambda = 0 is feasible
        Sr->P = Sr->B;
        Sr->lamF = Sr->P.lam;
        Sr->done = 1;
        return;
    }
    Sr->closed = 0;
    if (Sr->haveB) {
        Sr->P = Sr->B;
    } else if (b >= 1.0) {
        double C, P;
        cell_at(row_hist(R), 0, R.p - 1, tab, C, P);
        Sr->P.lam = __builtin_huge_val();
        Sr->P.H = 0.0 - P;
        Sr->P.M = (0.0 + C) / R.s2tot;
        Sr->P.t = 2;
        Sr->P.buf = -1;
        Sr->closed = 1;
    } else {
        if (Sr->tried40 || Sr->npass >= max_passes) {
            Sr->P = Sr->L;  // both solves so far still hold their argmins
            Sr->status = ECASQ_EINFEASIBLE;
            Sr->lamF = Sr->P.lam;
            Sr->done = 1;
            return;
        }
        Sr->kind = 1;
        Sr->lam = 0x1p40;
        Sr->buf = 1;
        return;
    }
    const double lc = (Sr->P.M - Sr->A.M) / (Sr->A.H - Sr->P.H);
    Sr->lc = lc;
    Sr->lamF = Sr->closed ? lc : Sr->P.lam;
    if (!(lc > 0.0) || Sr->npass >= max_passes) {
        Sr->done = 1;
        return;
    }
    Sr->kind = 2;
    Sr->lam = lc;
    Sr->buf = Sr->P.buf == 0 ? 1 : 0;
}

// The unique values of the sorted keys with their counts and exact prefix
// sums (Sec. 2 histogram, App. D prefix sums), one wavefront: lane l takes the
// entries [l E, (l+1) E) in order; its wide sums are combined by an exclusive
// scan over the wavefront (Hillis-Steele, a limb-wise carry add per step),
// then each lane walks its entries from the sum of those before it and writes
// every last occurrence of a value at its rank among the unique values, the
// sums rounded once.  Returns p.
__device__ int row_histogram(Row& R, const uint32_t* keys, int d, int E) {
    const int lane = R.lane;
    const int i0 = lane * E;
    uint64_t s[kSL] = {0}, q[kS2L] = {0};
    int nlast = 0;
    for (int e = 0; e < E; e++) {
        const int i = i0 + e;
        if (i < d) {
            const uint32_t k = keys[i];
            accumulate(s, q, term_of(key_bits(k)));
            nlast += (i == d - 1 || keys[i + 1] != k) ? 1 : 0;
        }
    }
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        uint64_t ts[kSL], tq[kS2L];
#pragma unroll
        for (int l = 0; l < kSL; l++) ts[l] = __shfl_up(s[l], off);
#pragma unroll
        for (int l = 0; l < kS2L; l++) tq[l] = __shfl_up(q[l], off);
        const int tn = __shfl_up(nlast, off);
        if (lane >= off) {
            wide_add_full<kSL>(s, ts);
            wide_add_full<kS2L>(q, tq);
            nlast += tn;
        }
    }
    // inclusive -> exclusive: the sums of the lanes before this one (every
    // lane takes part in the shuffle: a lane reading from an inactive one
    // would not see its value)
#pragma unroll
    for (int l = 0; l < kSL; l++) {
        const uint64_t t = __shfl_up(s[l], 1);
        s[l] = lane ? t : 0ull;
    }
#pragma unroll
    for (int l = 0; l < kS2L; l++) {
        const uint64_t t = __shfl_up(q[l], 1);
        q[l] = lane ? t : 0ull;
    }
    const int p = __builtin_amdgcn_readlane(nlast, kWave - 1);
    int u = __shfl_up(nlast, 1);
    if (lane == 0) u = 0;
    for (int e = 0; e < E; e++) {
        const int i = i0 + e;
        if (i < d) {
            const uint32_t k = keys[i];
            const uint32_t bits = key_bits(k);
            accumulate(s, q, term_of(bits));
            if (i == d - 1 || keys[i + 1] != k) {
                R.v[u] = (double)__uint_as_float(bits);
                R.N[u] = (double)(i + 1);
                R.S[u] = wide_to_double<kSL>(s, true, -149);
                R.S2[u] = wide_to_double<kS2L>(q, false, -298);
                u++;
            }
        }
    }
    return p;
}

template <int DT>
__device__ __forceinline__ uint32_t load_bits(const void* x, int64_t i) {
    if (DT == 0) return reinterpret_cast<const uint32_t*>(x)[i];
    if (DT == 1) return __float_as_uint(__half2float(reinterpret_cast<const __half*>(x)[i]));
    return ((uint32_t)reinterpret_cast<const uint16_t*>(x)[i]) << 16;
}

// LG > 0: DP solves by row_sweep with LG layers in registers; LG = 0: by
// row_solve, layer by layer.
template <int CMAX, int LG>
__device__ __forceinline__ Pt solve_row(Row& R, double lam, int exact_s, int buf) {
    if constexpr (LG > 0)
        return row_sweep<CMAX, LG>(R, lam, exact_s, buf);
    else
        return row_solve<CMAX>(R, lam, exact_s, buf);
}

// Wavefronts per SIMD the register allocation must allow: four for the
// register sweeps of up to 28 layer-column states per lane (a workgroup of
// four rows then takes under a quarter of a CU's LDS), the compiler's choice
// otherwise.
template <int CMAX, int LG>
constexpr int batched_min_waves() {
    return (LG > 0 && CMAX * LG <= 28) ? 4 : 1;
}

template <int DT, int CMAX, int LG>
__global__ __launch_bounds__(256, (batched_min_waves<CMAX, LG>())) void k_batched(BatchArgs A) {
    // the table at a fixed LDS address (a static array) so that the lookups
    // fold it into their offsets; the rows in the dynamic part after it
    __shared__ double2 tab[kLog2Size];
    extern __shared__ __align__(16) char smem[];
    load_log2_table(tab);
    __syncthreads();  // the only block-wide barrier: rows diverge from here on
    const int wave = uniform_i(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t row = (int64_t)blockIdx.x * A.rows_per_block + wave;
    if (wave >= A.rows_per_block || row >= A.n) return;
    const RowLayout L = row_layout(A.dpad, A.s, LG > 0);
    char* base = smem + (size_t)wave * L.total;
    uint32_t* keys = reinterpret_cast<uint32_t*>(base + L.keys);
    Row R;
    R.tab = tab;
    R.v = reinterpret_cast<double*>(base + L.v);
    R.N = reinterpret_cast<double*>(base + L.N);
    R.S = reinterpret_cast<double*>(base + L.S);
    R.S2 = reinterpret_cast<double*>(base + L.S2);
    R.F0 = reinterpret_cast<double*>(base + L.F0);
    R.F1 = reinterpret_cast<double*>(base + L.F1);
    R.last = reinterpret_cast<double*>(base + L.last);
    R.bp0 = reinterpret_cast<int16_t*>(base + L.bp0);
    R.bp1 = reinterpret_cast<int16_t*>(base + L.bp1);
    R.chain = reinterpret_cast<int32_t*>(base + L.chain);
    R.nu = reinterpret_cast<int32_t*>(base + L.nu);
    R.misc = reinterpret_cast<double*>(base + L.misc);
    R.s = A.s;
    R.dpad = A.dpad;
    R.lane = lane;
    R.cells = 0;
    R.solves = 0;
    const int d = A.d, dpad = A.dpad;

    // ingest: order-preserving keys, padding sorts last
    bool bad = false;
    for (int i = lane; i < dpad; i += kWave) {
        uint32_t k = 0xFFFFFFFFu;
        if (i < d) {
            const uint32_t bits = load_bits<DT>(A.x, row * (int64_t)d + i);
            if ((bits & 0x7F800000u) == 0x7F800000u) bad = true;
            k = f32_key(bits);
        }
        keys[i] = k;
    }
    const bool nonfinite = __ballot(bad) != 0ull;
    wave_sync();
    // bitonic sort of dpad keys
    for (int kk = 2; kk <= dpad; kk <<= 1) {
        for (int jj = kk >> 1; jj > 0; jj >>= 1) {
            for (int i = lane; i < dpad; i += kWave) {
                const int pr = i ^ jj;
                if (pr > i) {
                    const uint32_t a = keys[i], c = keys[pr];
                    const bool up = (i & kk) == 0;
                    if ((a > c) == up) {
                        keys[i] = c;
                        keys[pr] = a;
                    }
                }
            }
            wave_sync();
        }
    }
    R.p = uniform_i(row_histogram(R, keys, d, dpad / kWave));
    wave_sync();
    R.dd = (double)d;
    R.c0 = uniform_d(R.N[0]);
    R.c0d = R.c0 / R.dd;
    R.s2tot = uniform_d(R.S2[R.p - 1]);
    const int p = R.p;
    const double b = A.b;

    int status = ECASQ_OK;
    double lamF = 0.0;  // multiplier of the refinement step and of the objective
    int t = 1, passes = 0;
    if (nonfinite) {
        status = ECASQ_ENONFINITE;
        t = 0;
    } else if (p <= 2) {
        t = p;
        if (lane == 0) {
            R.chain[0] = 0;
            if (p == 2) R.chain[1] = 1;
        }
    } else {
        // the budget search with one multiplier per pass (the schedule of the
        // single-vector path at width 1): A = infeasible point of largest
        // lambda, B = feasible point of smallest lambda, Lo = lowest H(I,B);
        // first occurrence wins every tie.  One solve site: lane 0 decides
        // the next query from the state in LDS, every lane solves it, lane 0
        // files the point.
        RowSearch* Sr = reinterpret_cast<RowSearch*>(base + L.srch);
        if (lane == 0) {
            Sr->haveA = Sr->haveB = Sr->tried40 = 0;
            Sr->npass = 0;
            Sr->closed = 0;
            Sr->status = ECASQ_OK;
            Sr->done = 0;
            Sr->lamF = 0.0;
            Sr->kind = 0;
            Sr->lam = 0.0;
            Sr->buf = 0;
        }
        wave_sync();
        for (;;) {
            if (lane == 0 && Sr->npass > 0) row_search_next(Sr, R, b, A.max_passes, tab);
            wave_sync();
            if (uniform_i(Sr->done)) break;
            const double lam = uniform_d(Sr->lam);
            const int qb = uniform_i(Sr->buf);
            const Pt q = solve_row<CMAX, LG>(R, lam, A.exact_s, qb);
            if (lane == 0) row_search_file(Sr, q, b);
            wave_sync();
            if (uniform_i(Sr->done)) break;
        }
        status = uniform_i(Sr->status);
        lamF = uniform_d(Sr->lamF);
        passes = uniform_i(Sr->npass);
        t = uniform_i(Sr->P.t);
        const int pbuf = uniform_i(Sr->P.buf);
        const double plam = uniform_d(Sr->P.lam);
        if (lane == 0) {
            if (t == 2 || pbuf < 0 || !__builtin_isfinite(plam)) {
                R.chain[0] = 0;
                R.chain[1] = p - 1;
            } else {
                const int16_t* kept = argmin_buf(R, pbuf);
                for (int r = 0; r < t; r++) R.chain[r] = kept[r];
            }
        }
        wave_sync();
    }
    int rounds_run = 0;
    if (status != ECASQ_ENONFINITE && A.refine_rounds > 0 && t >= 3 &&
        __builtin_isfinite(lamF))
        rounds_run = row_refine(R, t, lamF * R.s2tot, b, 1, A.refine_rounds,
                                A.refine_exhaustive);
    if (lane == 0) {
        double mse = 0.0, hs = 0.0, ho = 0.0, vn = 0.0;
        if (status != ECASQ_ENONFINITE) {
            const Hist H = row_hist(R);
            for (int r = 0; r + 1 < t; r++) {
                double C, P;
                cell_at(H, R.chain[r], R.chain[r + 1], tab, C, P);
                mse = mse + C;
                hs = hs - P;
            }
            ho = chain_hout(H, t, R.chain, tab);
            vn = R.s2tot > 0.0 ? mse / R.s2tot : 0.0;
            for (int r = 0; r < t; r++) A.codebooks[row * A.s + r] = R.v[R.chain[r]];
            if (p == 2 && hs > b) status = ECASQ_EINFEASIBLE;
        }
        A.t_out[row] = t;
        if (A.infos) {
            // field by field (no stack copy of the struct)
            ecasq_info* inf = A.infos + row;
            inf->t = t;
            inf->p = nonfinite ? 0 : p;
            inf->lambda = lamF;
            inf->mse = mse;
            inf->vnmse = vn;
            inf->entropy = ho;
            inf->entropy_surrogate = hs;
            const double lr = __builtin_isfinite(lamF) ? lamF : 0.0;
            inf->objective = __builtin_fma(lr, ho, vn);
            inf->rate_total = ho + (32.0 * (double)t) / R.dd;
            inf->dp_solves = R.solves;
            inf->refine_rounds_run = rounds_run;
            inf->cells = R.cells;
            inf->status = status;
            inf->search_passes = passes;
        }
    }
}

// The (CMAX, LG) instantiation of k_batched for rows of dpad padded entries
// and s values: the sweep while CMAX x LG register states per lane stay
// within 32 (LG the recursive layers rounded up to 8, 14, 16 or 32), else
// layer by layer (LG = 0).
void batched_config(int dpad, int s, int& cmax, int& lg) {
    const int L = (s < dpad ? s : dpad) - 2;  // recursive layers, at most
    const int c = dpad / kWave;
    auto pick = [&](int c0, std::initializer_list<int> lgs) {
        for (int g : lgs)
            if (g == 0 || L <= g) {
                cmax = c0;
                lg = g;
                return;
            }
    };
    if (c <= 1)
        pick(1, {8, 14, 16, 32});
    else if (c <= 2)
        pick(2, {8, 14, 16, 0});
    else if (c <= 4)
        pick(4, {8, 0});
    else
        pick(8, {0});
}

template <int DT>
hipError_t launch_dt(const BatchArgs& A, int cmax, int lg, unsigned grid, unsigned threads,
                     size_t lds, hipStream_t st) {
    hipError_t e = hipSuccess;
#define ECASQ_LAUNCH(C, G)                                                                  \
    do {                                                                                     \
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_batched<DT, C, G>),        \
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);      \
        if (e != hipSuccess) return e;                                                       \
        k_batched<DT, C, G><<<grid, threads, lds, st>>>(A);                                  \
        return hipGetLastError();                                                            \
    } while (0)
    if (cmax == 1) {
        if (lg == 8) ECASQ_LAUNCH(1, 8);
        if (lg == 14) ECASQ_LAUNCH(1, 14);
        if (lg == 16) ECASQ_LAUNCH(1, 16);
        ECASQ_LAUNCH(1, 32);
    }
    if (cmax == 2) {
        if (lg == 8) ECASQ_LAUNCH(2, 8);
        if (lg == 14) ECASQ_LAUNCH(2, 14);
        if (lg == 16) ECASQ_LAUNCH(2, 16);
        ECASQ_LAUNCH(2, 0);
    }
    if (cmax == 4) {
        if (lg == 8) ECASQ_LAUNCH(4, 8);
        ECASQ_LAUNCH(4, 0);
    }
    ECASQ_LAUNCH(8, 0);
#undef ECASQ_LAUNCH
}

}  // namespace

hipError_t launch_batched(const void* x, int dt, int64_t n, int32_t d, int32_t s, double b,
                          int32_t refine_rounds, int32_t refine_exhaustive, int32_t exact_s,
                          int32_t max_passes, double* codebooks, int32_t* t_out, void* infos,
                          hipStream_t st) {
    int dpad = kWave;
    while (dpad < d) dpad <<= 1;
    int cmax = 0, lg = 0;
    batched_config(dpad, s, cmax, lg);
    const RowLayout L = row_layout(dpad, s, lg > 0);
    // rows per workgroup: as many as fit next to the table in 128 KB of LDS
    const size_t table = sizeof(double2) * kLog2Size;
    int rows = (int)((128 * 1024 - table) / L.total);
    if (rows > kMaxRows) rows = kMaxRows;
    if (rows < 1) return hipErrorInvalidValue;
    BatchArgs A;
    A.x = x;
    A.n = n;
    A.d = d;
    A.dpad = dpad;
    A.s = s;
    A.rows_per_block = rows;
    A.b = b;
    A.refine_rounds = refine_rounds;
    A.refine_exhaustive = refine_exhaustive;
    A.exact_s = exact_s;
    A.max_passes = max_passes;
    A.codebooks = codebooks;
    A.t_out = t_out;
    A.infos = static_cast<ecasq_info*>(infos);
    const size_t lds = (size_t)rows * L.total;  // the table is static
    const unsigned grid = (unsigned)((n + rows - 1) / rows);
    const unsigned threads = (unsigned)(rows * kWave);
    if (dt == 0) return launch_dt<0>(A, cmax, lg, grid, threads, lds, st);
    if (dt == 1) return launch_dt<1>(A, cmax, lg, grid, threads, lds, st);
    return launch_dt<2>(A, cmax, lg, grid, threads, lds, st);
}

}  // namespace ecasq
