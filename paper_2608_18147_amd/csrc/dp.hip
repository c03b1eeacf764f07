// The approximate dynamic program dp_APX of Sec. 5 (eq. apx_base, apx_rec,
// apx_final) and the half-DPs of its Hirschberg recovery.
//
// One layer computes, for every column j,
//     F_i[j] = min_{k < j} F_{i-1}[k] + C[k,j] + lambda' Phi[k,j]
// (forward), or for the backward half of the recovery
//     B_q[j] = min_{k > j} C[j,k] + lambda' Phi[j,k] + B_{q-1}[k].
// The interval cost is evaluated on the fly from prefix sums; nothing of size
// p x p is stored.
//
// Mapping on CDNA4: one lane owns one column j (R columns per lane, strided by
// the block size, so column data sits in VGPRs and loads coalesce).  The
// predecessor index k is uniform across the block: a tile of 256 predecessors
// (v, N, S, S2, F) is staged through LDS and read as broadcasts, so the k loop
// needs no cross-lane reduction at all.  The min over k of one column is split
// into chunks of kc predecessors; each (column block, chunk) pair is one
// workgroup, which balances the triangular work and fills all 256 CUs, and a
// second kernel reduces the per-chunk (value, index) partials in increasing k
// order (lowest k wins ties).  The 256-entry log2 table also lives in LDS.
#include <vector>

#include "device.hpp"
#include "launch.hpp"

namespace ecasq {

namespace {

constexpr int kBlock = 256;
constexpr int kTK = 256;
constexpr int kMaxSplit = 32;

struct LayerArgs {
    const double* v;
    const double* N;
    const double* S;
    const double* S2;
    const double* Fin;  // previous layer, indexed by absolute k
    double* pval;
    int32_t* pidx;
    int64_t kb;   // forward: first predecessor; backward: last predecessor (khi)
    int64_t jlo;  // first column
    int64_t jhi;  // last column (inclusive)
    int64_t nblk;   // column blocks
    int32_t nsplit; // chunks per column block (equal split of its predecessor range)
    double dd;
    double lam;  // lambda' (MSE units)
};

// Predecessor range of block b: forward [kb, jend-1]; backward [j0+1, khi].
// Chunk c of block b's predecessor range [klo, khi], split into nsplit equal
// parts; returns false for an empty chunk.
__device__ __forceinline__ bool chunk_range(int64_t klo, int64_t khi, int32_t nsplit, int64_t c,
                                            int64_t& cs, int64_t& ce) {
    const int64_t len = khi - klo + 1;
    const int64_t kc = (len + nsplit - 1) / nsplit;
    cs = klo + c * kc;
    ce = cs + kc - 1 < khi ? cs + kc - 1 : khi;
    return cs <= khi;
}

template <bool BWD>
__device__ __forceinline__ void block_krange(const LayerArgs& a, int64_t CB, int64_t b,
                                             int64_t& j0, int64_t& jend, int64_t& klo,
                                             int64_t& khi) {
    j0 = a.jlo + b * CB;
    jend = j0 + CB - 1 < a.jhi ? j0 + CB - 1 : a.jhi;
    if (BWD) {
        klo = j0 + 1;
        khi = a.kb;
    } else {
        klo = a.kb;
        khi = jend - 1;
    }
}

// One cell update of column state (cv, cN, cS, cS2 / best, bk) against the
// predecessor (pv, pN, pS, pS2, pF); `ok` masks cells outside the triangle.
template <bool BWD, bool MASKED>
__device__ __forceinline__ void cell_update(double cv, double cN, double cS, double cS2, double pv,
                                            double pN, double pS, double pS2, double pF,
                                            int32_t k, bool ok, double dd, double lam,
                                            const double2* __restrict__ tab, double& best,
                                            int32_t& bk) {
    double C, P;
    if (BWD)
        cell_terms(cv, cN, cS, cS2, pv, pN, pS, pS2, dd, false, 0.0, tab, C, P);
    else
        cell_terms(pv, pN, pS, pS2, cv, cN, cS, cS2, dd, false, 0.0, tab, C, P);
    const double cand = __builtin_fma(-lam, P, pF + C);
    if (MASKED) {
        const bool lt = ok && cand < best;
        bk = lt ? k : bk;
        best = lt ? cand : best;
    } else {
        // strict '<' keeps the lowest k; min() only differs from the select in
        // the sign of an exact zero
        bk = cand < best ? k : bk;
        best = __builtin_fmin(best, cand);
    }
}

// R columns per lane; SMEM: predecessors read through the scalar cache
// (wave-uniform k) instead of being staged through LDS.
template <int R, bool BWD, bool SMEM>
__global__ __launch_bounds__(kBlock) void k_dp_layer(LayerArgs a, const double* __restrict__ gv,
                                                     const double* __restrict__ gN,
                                                     const double* __restrict__ gS,
                                                     const double* __restrict__ gS2,
                                                     const double* __restrict__ gF) {
    __shared__ double2 tab[kLog2Size];
    __shared__ double sv[SMEM ? 1 : kTK], sN[SMEM ? 1 : kTK], sS[SMEM ? 1 : kTK],
        sS2[SMEM ? 1 : kTK], sF[SMEM ? 1 : kTK];
    constexpr int64_t CB = (int64_t)kBlock * R;
    const int tid = threadIdx.x;
    // heaviest column blocks first: high b for forward layers, low b backward
    const int64_t b = BWD ? (int64_t)blockIdx.y : a.nblk - 1 - (int64_t)blockIdx.y;
    const int64_t c = blockIdx.x;
    int64_t j0, jend, klo, khi;
    block_krange<BWD>(a, CB, b, j0, jend, klo, khi);
    int64_t cs, ce;
    if (!chunk_range(klo, khi, a.nsplit, c, cs, ce)) return;  // uniform across the block
    load_log2_table(tab);

    int64_t col[R];
    double cv[R], cN[R], cS[R], cS2[R], best[R];
    int32_t bk[R];
#pragma unroll
    for (int r = 0; r < R; r++) {
        col[r] = j0 + r * kBlock + tid;
        const int64_t jj = col[r] <= jend ? col[r] : jend;
        cv[r] = gv[jj];
        cN[r] = gN[jj];
        cS[r] = gS[jj];
        cS2[r] = gS2[jj];
        best[r] = __builtin_huge_val();
        bk[r] = -1;
    }
    const double lam = a.lam, dd = a.dd;
    if (SMEM) {
        __syncthreads();  // table visible
        // unmasked part: every k below (forward) or above (backward) all columns
        const int64_t us = BWD ? (jend + 1 > cs ? jend + 1 : cs) : cs;
        const int64_t ue = BWD ? ce : (j0 - 1 < ce ? j0 - 1 : ce);
        for (int64_t k = us; k <= ue; k++) {
            const double pv = gv[k], pN = gN[k], pS = gS[k], pS2 = gS2[k], pF = gF[k];
#pragma unroll
            for (int r = 0; r < R; r++)
                cell_update<BWD, false>(cv[r], cN[r], cS[r], cS2[r], pv, pN, pS, pS2, pF,
                                        (int32_t)k, true, dd, lam, tab, best[r], bk[r]);
        }
        // masked part (the diagonal region)
        const int64_t ms = BWD ? cs : (j0 > cs ? j0 : cs);
        const int64_t me = BWD ? (jend < ce ? jend : ce) : ce;
        for (int64_t k = ms; k <= me; k++) {
            const double pv = gv[k], pN = gN[k], pS = gS[k], pS2 = gS2[k], pF = gF[k];
#pragma unroll
            for (int r = 0; r < R; r++)
                cell_update<BWD, true>(cv[r], cN[r], cS[r], cS2[r], pv, pN, pS, pS2, pF,
                                       (int32_t)k, BWD ? (k > col[r]) : (k < col[r]), dd, lam, tab,
                                       best[r], bk[r]);
        }
    } else {
        for (int64_t t0 = cs; t0 <= ce; t0 += kTK) {
            const int nk = (int)(ce - t0 + 1 < kTK ? ce - t0 + 1 : kTK);
            __syncthreads();
            if (tid < nk) {
                const int64_t k = t0 + tid;
                sv[tid] = gv[k];
                sN[tid] = gN[k];
                sS[tid] = gS[k];
                sS2[tid] = gS2[k];
                sF[tid] = gF[k];
            }
            __syncthreads();
            const bool nomask = BWD ? (t0 > jend) : (t0 + nk - 1 < j0);
            if (nomask) {
                for (int kk = 0; kk < nk; kk++) {
#pragma unroll
                    for (int r = 0; r < R; r++)
                        cell_update<BWD, false>(cv[r], cN[r], cS[r], cS2[r], sv[kk], sN[kk],
                                                sS[kk], sS2[kk], sF[kk], (int32_t)(t0 + kk), true,
                                                dd, lam, tab, best[r], bk[r]);
                }
            } else {
                for (int kk = 0; kk < nk; kk++) {
                    const int64_t k = t0 + kk;
#pragma unroll
                    for (int r = 0; r < R; r++)
                        cell_update<BWD, true>(cv[r], cN[r], cS[r], cS2[r], sv[kk], sN[kk],
                                               sS[kk], sS2[kk], sF[kk], (int32_t)k,
                                               BWD ? (k > col[r]) : (k < col[r]), dd, lam, tab,
                                               best[r], bk[r]);
                }
            }
        }
    }
#pragma unroll
    for (int r = 0; r < R; r++) {
        if (col[r] <= jend) {
            const int64_t idx = (b * a.nsplit + c) * CB + r * kBlock + tid;
            a.pval[idx] = best[r];
            a.pidx[idx] = bk[r];
        }
    }
}

struct ReduceArgs {
    LayerArgs L;
    int64_t CB;
    double* Fout;
    // forward main-DP extras (null in the recovery half-DPs)
    const double* Min;
    const double* Pin;
    double* Mout;
    double* Pout;
    int32_t* kstar;
    double* last;  // [3][s+1]: F, MSE, H(I,B) of column p-1 per layer
    int32_t layer;
    int32_t last_stride;
    int64_t p;
    double c0d;
};

template <bool BWD>
__global__ __launch_bounds__(256) void k_dp_reduce(ReduceArgs a) {
    __shared__ double2 tab[kLog2Size];
    load_log2_table(tab);
    __syncthreads();
    const int64_t j = a.L.jlo + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j > a.L.jhi) return;
    const int64_t b = (j - a.L.jlo) / a.CB;
    const int64_t off = (j - a.L.jlo) - b * a.CB;
    int64_t j0, jend, klo, khi;
    block_krange<BWD>(a.L, a.CB, b, j0, jend, klo, khi);
    double best = __builtin_huge_val();
    int32_t bk = -1;
    for (int64_t c = 0; c < a.L.nsplit; c++) {
        int64_t cs, ce;
        if (!chunk_range(klo, khi, a.L.nsplit, c, cs, ce)) break;
        const int64_t idx = (b * a.L.nsplit + c) * a.CB + off;
        const double val = a.L.pval[idx];
        if (val < best) {
            best = val;
            bk = a.L.pidx[idx];
        }
    }
    a.Fout[j] = best;
    if (a.Mout && bk >= 0) {
        double C, P;
        cell_terms(a.L.v[bk], a.L.N[bk], a.L.S[bk], a.L.S2[bk], a.L.v[j], a.L.N[j], a.L.S[j],
                   a.L.S2[j], a.L.dd, bk == 0, a.c0d, tab, C, P);
        const double m = a.Min[bk] + C;
        const double ph = a.Pin[bk] - P;
        a.Mout[j] = m;
        a.Pout[j] = ph;
        if (a.kstar) a.kstar[j] = bk;
        if (j == a.p - 1) {
            a.last[a.layer] = best;
            a.last[a.last_stride + a.layer] = m;
            a.last[2 * a.last_stride + a.layer] = ph;
        }
    }
}

// Forward layer 2 from `lo`: F[j] = C[lo,j] + lambda' Phi'[lo,j] (Phi^first
// when lo == 0), eq. apx_base.  With M non-null also starts the accumulators.
__global__ __launch_bounds__(256) void k_dp_init_fwd(Hist H, int64_t lo, int64_t jl, int64_t jh,
                                                     double lam, double* F, double* M, double* Ph,
                                                     int32_t* kstar, double* last,
                                                     int32_t last_stride) {
    __shared__ double2 tab[kLog2Size];
    load_log2_table(tab);
    __syncthreads();
    const int64_t j = jl + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j > jh) return;
    double C, P;
    cell_at(H, lo, j, tab, C, P);
    const double f = __builtin_fma(-lam, P, 0.0 + C);
    F[j] = f;
    if (M) {
        const double m = 0.0 + C;
        const double ph = 0.0 - P;
        M[j] = m;
        Ph[j] = ph;
        if (kstar) kstar[j] = (int32_t)lo;
        if (j == H.p - 1) {
            last[2] = f;
            last[last_stride + 2] = m;
            last[2 * last_stride + 2] = ph;
        }
    }
}

// Backward layer 2 into `hi`: B[j] = C[j,hi] + lambda' Phi[j,hi].
__global__ __launch_bounds__(256) void k_dp_init_bwd(Hist H, int64_t hi, int64_t jl, int64_t jh,
                                                     double lam, double* B) {
    __shared__ double2 tab[kLog2Size];
    load_log2_table(tab);
    __syncthreads();
    const int64_t j = jl + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j > jh) return;
    double C, P;
    cell_at(H, j, hi, tab, C, P);
    B[j] = __builtin_fma(-lam, P, 0.0 + C);
}

// eq. apx_final: lowest i in [2, imax] minimising F_i[p-1] (or i = imax when
// exactly min(s, p) values are required).  out: J, MSE, H(I,B), i*.
__global__ void k_dp_final(const double* last, int32_t stride, int32_t imax, int32_t exact_s,
                           double* out) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int32_t bi = 2;
    double bj = last[2];
    for (int32_t i = 3; i <= imax; i++) {
        const double f = last[i];
        if (exact_s ? (i == imax) : (f < bj)) {
            bj = f;
            bi = i;
        }
    }
    out[0] = bj;
    out[1] = last[stride + bi];
    out[2] = last[2 * stride + bi];
    out[3] = (double)bi;
}

// Hirschberg split: lowest m in [ml, mh] minimising Fw[m] + Bw[m].
__global__ __launch_bounds__(256) void k_split(const double* Fw, const double* Bw, int64_t ml,
                                               int64_t mh, int64_t* m_out) {
    __shared__ double sv[256];
    __shared__ int64_t si[256];
    const int tid = threadIdx.x;
    double best = __builtin_huge_val();
    int64_t bm = -1;
    for (int64_t m = ml + tid; m <= mh; m += 256) {
        const double tot = Fw[m] + Bw[m];
        if (tot < best) {
            best = tot;
            bm = m;
        }
    }
    sv[tid] = best;
    si[tid] = bm;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (tid < off) {
            const double ov = sv[tid + off];
            const int64_t oi = si[tid + off];
            if (oi >= 0 && (si[tid] < 0 || ov < sv[tid] || (ov == sv[tid] && oi < si[tid]))) {
                sv[tid] = ov;
                si[tid] = oi;
            }
        }
        __syncthreads();
    }
    if (tid == 0) *m_out = si[0];
}

// Chunks per column block: enough workgroups to fill the chip, at least ~1k
// predecessors per chunk, and a multiple of 8 when possible so that the
// round-robin placement of consecutive workgroups on the 8 XCDs gives every
// XCD an equal share of every column block.
int32_t choose_splits(int64_t lenmax) {
    int64_t sp = lenmax / 1024;
    if (sp >= 8) sp = sp / 8 * 8;
    if (sp > kMaxSplit) sp = kMaxSplit;
    return sp < 1 ? 1 : (int32_t)sp;
}

}  // namespace

// Optional timing of the layer kernel: a pair of events on the launch stream
// around every k_dp_layer launch, read back when the solve synchronizes.
namespace {
struct TimedLaunch {
    hipEvent_t a, b;
    int64_t cells;
};
bool g_timing = false;
std::vector<TimedLaunch> g_pending;
std::vector<hipEvent_t> g_pool;
double g_ms = 0.0;
int64_t g_launches = 0, g_cells = 0;

hipEvent_t take_event() {
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}
}  // namespace

void timing_enable(bool on) { g_timing = on; }

void timing_flush() {
    for (auto& t : g_pending) {
        float ms = 0.f;
        if (hipEventSynchronize(t.b) == hipSuccess && hipEventElapsedTime(&ms, t.a, t.b) == hipSuccess) {
            g_ms += ms;
            g_launches++;
            g_cells += t.cells;
        }
        g_pool.push_back(t.a);
        g_pool.push_back(t.b);
    }
    g_pending.clear();
}

void timing_read(double* ms, int64_t* launches, int64_t* cells, bool reset) {
    timing_flush();
    if (ms) *ms = g_ms;
    if (launches) *launches = g_launches;
    if (cells) *cells = g_cells;
    if (reset) {
        g_ms = 0.0;
        g_launches = 0;
        g_cells = 0;
    }
}

int64_t dp_partial_entries(int64_t p) {
    // nblk * nsplit * CB with nsplit <= kMaxSplit and nblk * CB <= p + CB
    const int64_t CB = kBlock * kColsPerLane;
    return (p + CB) * kMaxSplit;
}

#ifndef ECASQ_PRED_SMEM
#define ECASQ_PRED_SMEM 0
#endif

hipError_t launch_dp_layer(const DpLayer& L, hipStream_t st) {
    constexpr int R = kColsPerLane;
    constexpr bool SM = ECASQ_PRED_SMEM != 0;
    const int64_t CB = (int64_t)kBlock * R;
    const int64_t ncol = L.jhi - L.jlo + 1;
    if (ncol <= 0) return hipSuccess;
    const int64_t nblk = (ncol + CB - 1) / CB;
    // longest predecessor range: last block (forward) or first block (backward)
    const int64_t lenmax = L.backward ? (L.kb - L.jlo) : (L.jhi - L.kb);
    const int32_t nsplit = choose_splits(lenmax);
    LayerArgs a;
    a.v = L.H.v;
    a.N = L.H.N;
    a.S = L.H.S;
    a.S2 = L.H.S2;
    a.Fin = L.Fin;
    a.pval = L.pval;
    a.pidx = L.pidx;
    a.kb = L.kb;
    a.jlo = L.jlo;
    a.jhi = L.jhi;
    a.nblk = nblk;
    a.nsplit = nsplit;
    a.dd = L.H.dd;
    a.lam = L.lam;
    dim3 grid((unsigned)nsplit, (unsigned)nblk);
    TimedLaunch tl{nullptr, nullptr, L.cells};
    if (g_timing) {
        tl.a = take_event();
        tl.b = take_event();
        if (tl.a && tl.b) (void)hipEventRecord(tl.a, st);
    }
    if (L.backward)
        k_dp_layer<R, true, SM><<<grid, kBlock, 0, st>>>(a, a.v, a.N, a.S, a.S2, a.Fin);
    else
        k_dp_layer<R, false, SM><<<grid, kBlock, 0, st>>>(a, a.v, a.N, a.S, a.S2, a.Fin);
    if (g_timing && tl.a && tl.b) {
        (void)hipEventRecord(tl.b, st);
        g_pending.push_back(tl);
    }
    ReduceArgs ra;
    ra.L = a;
    ra.CB = CB;
    ra.Fout = L.Fout;
    ra.Min = L.Min;
    ra.Pin = L.Pin;
    ra.Mout = L.Mout;
    ra.Pout = L.Pout;
    ra.kstar = L.kstar;
    ra.last = L.last;
    ra.layer = L.layer;
    ra.last_stride = L.last_stride;
    ra.p = L.H.p;
    ra.c0d = L.H.c0d;
    const unsigned rg = (unsigned)((ncol + 255) / 256);
    if (L.backward)
        k_dp_reduce<true><<<rg, 256, 0, st>>>(ra);
    else
        k_dp_reduce<false><<<rg, 256, 0, st>>>(ra);
    return hipGetLastError();
}

hipError_t launch_dp_init_fwd(const Hist& H, int64_t lo, int64_t jl, int64_t jh, double lam,
                              double* F, double* M, double* Ph, int32_t* kstar, double* last,
                              int32_t last_stride, hipStream_t st) {
    if (jh < jl) return hipSuccess;
    const unsigned g = (unsigned)((jh - jl + 1 + 255) / 256);
    k_dp_init_fwd<<<g, 256, 0, st>>>(H, lo, jl, jh, lam, F, M, Ph, kstar, last, last_stride);
    return hipGetLastError();
}

hipError_t launch_dp_init_bwd(const Hist& H, int64_t hi, int64_t jl, int64_t jh, double lam,
                              double* B, hipStream_t st) {
    if (jh < jl) return hipSuccess;
    const unsigned g = (unsigned)((jh - jl + 1 + 255) / 256);
    k_dp_init_bwd<<<g, 256, 0, st>>>(H, hi, jl, jh, lam, B);
    return hipGetLastError();
}

hipError_t launch_dp_final(const double* last, int32_t stride, int32_t imax, int32_t exact_s,
                           double* out, hipStream_t st) {
    k_dp_final<<<1, 64, 0, st>>>(last, stride, imax, exact_s, out);
    return hipGetLastError();
}

hipError_t launch_split(const double* Fw, const double* Bw, int64_t ml, int64_t mh,
                        int64_t* m_out, hipStream_t st) {
    k_split<<<1, 256, 0, st>>>(Fw, Bw, ml, mh, m_out);
    return hipGetLastError();
}

}  // namespace ecasq
