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
#include <cstring>
#include <vector>

#include "device.hpp"
#include "launch.hpp"

namespace ecasq {

namespace {

constexpr int kBlock = 256;
constexpr int kTK = 256;
constexpr int kMaxLam = kMaxLambdas;
#ifndef ECASQ_MAX_SPLIT
#define ECASQ_MAX_SPLIT 32
#endif
constexpr int kMaxSplit = ECASQ_MAX_SPLIT;  // chunks per column block, at most

struct LayerArgs {
    const double* v;
    const double* N;
    const double* S;
    const double* S2;
    const double* Fin[kMaxLam];  // previous layer per multiplier, indexed by absolute k
    double* pval;                // partials, kMaxLam slices of pstride entries
    int32_t* pidx;
    int64_t pstride;
    int64_t kb;   // forward: first predecessor; backward: last predecessor (khi)
    int64_t jlo;  // first column
    int64_t jhi;  // last column (inclusive)
    int64_t nblk;   // column blocks
    int32_t nsplit; // chunks per column block (equal split of its predecessor range)
    double dd;
    double lam[kMaxLam];  // lambda' (MSE units) per multiplier
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

// Candidate update of one (column, multiplier) state; `ok` masks cells outside
// the triangle.  Strict '<' keeps the lowest k; the unmasked form uses min(),
// which differs from the select only in the sign of an exact zero.
template <bool MASKED>
__device__ __forceinline__ void take(double cand, int32_t k, bool ok, double& best, int32_t& bk) {
    if (MASKED) {
        const bool lt = ok && cand < best;
        bk = lt ? k : bk;
        best = lt ? cand : best;
    } else {
        bk = cand < best ? k : bk;
        best = __builtin_fmin(best, cand);
    }
}

// All cells of one LDS tile of nk predecessors against the lane's R columns.
template <int R, bool BWD, int ML, bool MASKED>
__device__ __forceinline__ void tile_pass(const double* sv, const double* sN, const double* sS,
                                          const double* sS2, const double (*sF)[ML], int64_t t0,
                                          int nk, const int64_t (&col)[R], const double (&cv)[R],
                                          const double (&cN)[R], const double (&cS)[R],
                                          const double (&cS2)[R], double dd,
                                          const double (&lam)[ML], const double2* tab,
                                          double (&best)[R][ML], int32_t (&bk)[R][ML]) {
    for (int kk = 0; kk < nk; kk++) {
        const int64_t k = t0 + kk;
        const double pv = sv[kk], pN = sN[kk], pS = sS[kk], pS2 = sS2[kk];
        double pF[ML];
#pragma unroll
        for (int m = 0; m < ML; m++) pF[m] = sF[kk][m];
#pragma unroll
        for (int r = 0; r < R; r++) {
            double C, P;
            if (BWD)
                cell_terms(cv[r], cN[r], cS[r], cS2[r], pv, pN, pS, pS2, dd, false, 0.0, tab, C,
                           P);
            else
                cell_terms(pv, pN, pS, pS2, cv[r], cN[r], cS[r], cS2[r], dd, false, 0.0, tab, C,
                           P);
            const bool ok = !MASKED || (BWD ? (k > col[r]) : (k < col[r]));
#pragma unroll
            for (int m = 0; m < ML; m++)
                take<MASKED>(pF[m] + __builtin_fma(-lam[m], P, C), (int32_t)k, ok, best[r][m],
                             bk[r][m]);
        }
    }
}

// R columns per lane, ML multipliers per launch (C and Phi of a cell are
// shared by all multipliers); SMEM: predecessors read through the scalar
// cache instead of being staged through LDS (single multiplier only).
template <int R, bool BWD, bool SMEM, int ML>
__global__ __launch_bounds__(kBlock) void k_dp_layer(LayerArgs a, const double* __restrict__ gv,
                                                     const double* __restrict__ gN,
                                                     const double* __restrict__ gS,
                                                     const double* __restrict__ gS2) {
    static_assert(!SMEM || ML == 1, "scalar-cache path is single-multiplier");
    __shared__ double2 tab[kLog2Size];
    __shared__ double sv[SMEM ? 1 : kTK], sN[SMEM ? 1 : kTK], sS[SMEM ? 1 : kTK],
        sS2[SMEM ? 1 : kTK];
    __shared__ double sF[SMEM ? 1 : kTK][ML];
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
    double cv[R], cN[R], cS[R], cS2[R], best[R][ML];
    int32_t bk[R][ML];
#pragma unroll
    for (int r = 0; r < R; r++) {
        col[r] = j0 + r * kBlock + tid;
        const int64_t jj = col[r] <= jend ? col[r] : jend;
        cv[r] = gv[jj];
        cN[r] = gN[jj];
        cS[r] = gS[jj];
        cS2[r] = gS2[jj];
#pragma unroll
        for (int m = 0; m < ML; m++) {
            best[r][m] = __builtin_huge_val();
            bk[r][m] = -1;
        }
    }
    double lam[ML];
#pragma unroll
    for (int m = 0; m < ML; m++) lam[m] = a.lam[m];
    const double dd = a.dd;
    if (SMEM) {
        const double* __restrict__ gF = a.Fin[0];
        __syncthreads();  // table visible
        // unmasked part: every k below (forward) or above (backward) all columns
        const int64_t us = BWD ? (jend + 1 > cs ? jend + 1 : cs) : cs;
        const int64_t ue = BWD ? ce : (j0 - 1 < ce ? j0 - 1 : ce);
        for (int64_t k = us; k <= ue; k++) {
            const double pv = gv[k], pN = gN[k], pS = gS[k], pS2 = gS2[k], pF = gF[k];
#pragma unroll
            for (int r = 0; r < R; r++) {
                double C, P;
                if (BWD)
                    cell_terms(cv[r], cN[r], cS[r], cS2[r], pv, pN, pS, pS2, dd, false, 0.0, tab,
                               C, P);
                else
                    cell_terms(pv, pN, pS, pS2, cv[r], cN[r], cS[r], cS2[r], dd, false, 0.0, tab,
                               C, P);
                take<false>(pF + __builtin_fma(-lam[0], P, C), (int32_t)k, true, best[r][0],
                            bk[r][0]);
            }
        }
        // masked part (the diagonal region)
        const int64_t ms = BWD ? cs : (j0 > cs ? j0 : cs);
        const int64_t me = BWD ? (jend < ce ? jend : ce) : ce;
        for (int64_t k = ms; k <= me; k++) {
            const double pv = gv[k], pN = gN[k], pS = gS[k], pS2 = gS2[k], pF = gF[k];
#pragma unroll
            for (int r = 0; r < R; r++) {
                double C, P;
                if (BWD)
                    cell_terms(cv[r], cN[r], cS[r], cS2[r], pv, pN, pS, pS2, dd, false, 0.0, tab,
                               C, P);
                else
                    cell_terms(pv, pN, pS, pS2, cv[r], cN[r], cS[r], cS2[r], dd, false, 0.0, tab,
                               C, P);
                take<true>(pF + __builtin_fma(-lam[0], P, C), (int32_t)k,
                           BWD ? (k > col[r]) : (k < col[r]), best[r][0], bk[r][0]);
            }
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
#pragma unroll
                for (int m = 0; m < ML; m++) sF[tid][m] = a.Fin[m][k];
            }
            __syncthreads();
            const bool nomask = BWD ? (t0 > jend) : (t0 + nk - 1 < j0);
            if (nomask)
                tile_pass<R, BWD, ML, false>(sv, sN, sS, sS2, sF, t0, nk, col, cv, cN, cS, cS2,
                                             dd, lam, tab, best, bk);
            else
                tile_pass<R, BWD, ML, true>(sv, sN, sS, sS2, sF, t0, nk, col, cv, cN, cS, cS2,
                                            dd, lam, tab, best, bk);
        }
    }
#pragma unroll
    for (int r = 0; r < R; r++) {
        if (col[r] <= jend) {
            const int64_t idx = (b * a.nsplit + c) * CB + r * kBlock + tid;
#pragma unroll
            for (int m = 0; m < ML; m++) {
                a.pval[m * a.pstride + idx] = best[r][m];
                a.pidx[m * a.pstride + idx] = bk[r][m];
            }
        }
    }
}

struct ReduceArgs {
    LayerArgs L;
    int64_t CB;
    double* Fout[kMaxLam];
    // forward main-DP extras (null in the recovery half-DPs)
    const double* Min[kMaxLam];
    const double* Pin[kMaxLam];
    double* Mout[kMaxLam];
    double* Pout[kMaxLam];
    int32_t* kstar[kMaxLam];  // argmin rows per multiplier (may be null)
    double* last;     // per multiplier [3][s+1]: F, MSE, H(I,B) of column p-1 per layer
    int32_t layer;
    int32_t last_stride;
    int64_t p;
    double c0d;
};

// Per (column, multiplier): lexicographic min of the chunk partials in
// increasing k order, then the MSE / H(I,B) accumulators along the argmin.
template <bool BWD>
__global__ __launch_bounds__(256) void k_dp_reduce(ReduceArgs a) {
    __shared__ double2 tab[kLog2Size];
    load_log2_table(tab);
    __syncthreads();
    const int m = blockIdx.y;
    const int64_t j = a.L.jlo + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j > a.L.jhi) return;
    const int64_t b = (j - a.L.jlo) / a.CB;
    const int64_t off = (j - a.L.jlo) - b * a.CB;
    int64_t j0, jend, klo, khi;
    block_krange<BWD>(a.L, a.CB, b, j0, jend, klo, khi);
    const double* pval = a.L.pval + m * a.L.pstride;
    const int32_t* pidx = a.L.pidx + m * a.L.pstride;
    double best = __builtin_huge_val();
    int32_t bk = -1;
    for (int64_t c = 0; c < a.L.nsplit; c++) {
        int64_t cs, ce;
        if (!chunk_range(klo, khi, a.L.nsplit, c, cs, ce)) break;
        const int64_t idx = (b * a.L.nsplit + c) * a.CB + off;
        const double val = pval[idx];
        if (val < best) {
            best = val;
            bk = pidx[idx];
        }
    }
    a.Fout[m][j] = best;
    if (a.Mout[m] && bk >= 0) {
        double C, P;
        cell_terms(a.L.v[bk], a.L.N[bk], a.L.S[bk], a.L.S2[bk], a.L.v[j], a.L.N[j], a.L.S[j],
                   a.L.S2[j], a.L.dd, bk == 0, a.c0d, tab, C, P);
        const double mv = a.Min[m][bk] + C;
        const double ph = a.Pin[m][bk] - P;
        a.Mout[m][j] = mv;
        a.Pout[m][j] = ph;
        if (a.kstar[m]) a.kstar[m][j] = bk;
        if (j == a.p - 1) {
            double* last = a.last + (int64_t)m * 3 * a.last_stride;
            last[a.layer] = best;
            last[a.last_stride + a.layer] = mv;
            last[2 * a.last_stride + a.layer] = ph;
        }
    }
}

// Forward layer 2 from `lo`: F[j] = C[lo,j] + lambda' Phi'[lo,j] (Phi^first
// when lo == 0), eq. apx_base, for every multiplier of I.  With M non-null
// also starts the accumulators.
__global__ __launch_bounds__(256) void k_dp_init_fwd(Hist H, int64_t lo, int64_t jl, int64_t jh,
                                                     DpInit I) {
    __shared__ double2 tab[kLog2Size];
    load_log2_table(tab);
    __syncthreads();
    const int64_t j = jl + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j > jh) return;
    double C, P;
    cell_at(H, lo, j, tab, C, P);
    for (int m = 0; m < I.nlam; m++) {
        if (I.kstar[m]) I.kstar[m][j] = (int32_t)lo;
        const double f = __builtin_fma(-I.lam[m], P, 0.0 + C);
        I.F[m][j] = f;
        if (I.M[m]) {
            const double mv = 0.0 + C;
            const double ph = 0.0 - P;
            I.M[m][j] = mv;
            I.Ph[m][j] = ph;
            if (j == H.p - 1) {
                double* last = I.last + (int64_t)m * 3 * I.last_stride;
                last[2] = f;
                last[I.last_stride + 2] = mv;
                last[2 * I.last_stride + 2] = ph;
            }
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
__global__ void k_dp_final(const double* last_all, int32_t stride, int32_t imax, int32_t exact_s,
                           double* out_all, int32_t nlam) {
    const int m = threadIdx.x;
    if (m >= nlam || blockIdx.x != 0) return;
    const double* last = last_all + (int64_t)m * 3 * stride;
    double* out = out_all + 4 * m;
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
int32_t choose_splits(int64_t lenmax, int64_t cap) {
    int64_t sp = lenmax / 1024;
    if (sp > kMaxSplit) sp = kMaxSplit;
    if (sp > cap) sp = cap;
    if (sp >= 8) sp = sp / 8 * 8;
    return sp < 1 ? 1 : (int32_t)sp;
}

}  // namespace

// Optional timing of the layer kernel: a pair of events on the launch stream
// around every k_dp_layer launch, read back when the solve synchronizes.
namespace {
struct TimedLaunch {
    hipEvent_t a, b;
    int64_t cells;
    int variant;
};
struct TimingTotals {
    double ms = 0.0;
    int64_t launches = 0, cells = 0;
};
bool g_timing = false;
bool g_verbose = false;
std::vector<TimedLaunch> g_pending;
std::vector<hipEvent_t> g_pool;
TimingTotals g_tot[kTimingVariants];
TimedLaunch g_open{nullptr, nullptr, 0, 0};

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

void timing_enable(int mode) {
    g_timing = mode != 0;
    g_verbose = mode == 2;
}

bool timing_verbose() { return g_verbose; }

bool timing_active() { return g_timing; }

void timing_flush() {
    for (auto& t : g_pending) {
        float ms = 0.f;
        if (hipEventSynchronize(t.b) == hipSuccess && hipEventElapsedTime(&ms, t.a, t.b) == hipSuccess) {
            g_tot[t.variant].ms += ms;
            g_tot[t.variant].launches++;
            g_tot[t.variant].cells += t.cells;
        }
        g_pool.push_back(t.a);
        g_pool.push_back(t.b);
    }
    g_pending.clear();
}

void timing_begin(int variant, int64_t cells, hipStream_t st) {
    g_open = TimedLaunch{nullptr, nullptr, cells, variant};
    if (!g_timing) return;
    g_open.a = take_event();
    g_open.b = take_event();
    if (g_open.a && g_open.b) (void)hipEventRecord(g_open.a, st);
}

void timing_end(hipStream_t st) {
    if (!g_timing || !g_open.a || !g_open.b) return;
    (void)hipEventRecord(g_open.b, st);
    g_pending.push_back(g_open);
    g_open = TimedLaunch{nullptr, nullptr, 0, 0};
}

void timing_discard_last() {
    if (g_pending.empty()) return;
    const TimedLaunch& t = g_pending.back();
    (void)hipEventSynchronize(t.b);
    g_pool.push_back(t.a);
    g_pool.push_back(t.b);
    g_pending.pop_back();
}

void timing_read(int variant, double* ms, int64_t* launches, int64_t* cells, bool reset) {
    timing_flush();
    if (variant < 0 || variant >= kTimingVariants) {
        if (ms) *ms = 0.0;
        if (launches) *launches = 0;
        if (cells) *cells = 0;
        return;
    }
    const TimingTotals& t = g_tot[variant];
    if (ms) *ms = t.ms;
    if (launches) *launches = t.launches;
    if (cells) *cells = t.cells;
    if (reset) g_tot[variant] = TimingTotals();
}

int64_t dp_partial_entries(int64_t p) {
    // nblk * nsplit * CB <= (p + CB) * nsplit; at most 2^26 entries per
    // multiplier once p is large (then nblk alone fills the chip)
    const int64_t CB = kBlock * (kColsPerLane > kColsPerLaneMulti ? kColsPerLane
                                                                   : kColsPerLaneMulti);
    int64_t cap = ((int64_t)1 << 26) / (p + CB);
    cap = cap < 1 ? 1 : (cap > kMaxSplit ? kMaxSplit : cap);
    return (p + CB) * cap;
}

#ifndef ECASQ_PRED_SMEM
#define ECASQ_PRED_SMEM 0
#endif

namespace {

template <int R, int ML, bool SM>
hipError_t layer_launch(const DpLayer& L, hipStream_t st) {
    const int64_t CB = (int64_t)kBlock * R;
    const int64_t ncol = L.jhi - L.jlo + 1;
    const int64_t nblk = (ncol + CB - 1) / CB;
    // longest predecessor range: last block (forward) or first block (backward)
    const int64_t lenmax = L.backward ? (L.kb - L.jlo) : (L.jhi - L.kb);
    if (nblk * CB > L.pstride) return hipErrorInvalidValue;
    const int32_t nsplit = choose_splits(lenmax, L.pstride / (nblk * CB));
    LayerArgs a;
    std::memset(&a, 0, sizeof a);
    a.v = L.H.v;
    a.N = L.H.N;
    a.S = L.H.S;
    a.S2 = L.H.S2;
    a.pval = L.pval;
    a.pidx = L.pidx;
    a.pstride = L.pstride;
    a.kb = L.kb;
    a.jlo = L.jlo;
    a.jhi = L.jhi;
    a.nblk = nblk;
    a.nsplit = nsplit;
    a.dd = L.H.dd;
    for (int m = 0; m < ML; m++) {
        a.Fin[m] = L.Fin[m];
        a.lam[m] = L.lam[m];
    }
    dim3 grid((unsigned)nsplit, (unsigned)nblk);
    TimedLaunch tl{nullptr, nullptr, L.cells, ML == 1 ? 0 : 1};
    if (g_timing) {
        tl.a = take_event();
        tl.b = take_event();
        if (tl.a && tl.b) (void)hipEventRecord(tl.a, st);
    }
    if constexpr (ML == 1) {
        if (L.backward)
            k_dp_layer<R, true, SM, 1><<<grid, kBlock, 0, st>>>(a, a.v, a.N, a.S, a.S2);
        else
            k_dp_layer<R, false, SM, 1><<<grid, kBlock, 0, st>>>(a, a.v, a.N, a.S, a.S2);
    } else {
        k_dp_layer<R, false, SM, ML><<<grid, kBlock, 0, st>>>(a, a.v, a.N, a.S, a.S2);
    }
    if (g_timing && tl.a && tl.b) {
        (void)hipEventRecord(tl.b, st);
        g_pending.push_back(tl);
    }
    ReduceArgs ra;
    std::memset(&ra, 0, sizeof ra);
    ra.L = a;
    ra.CB = CB;
    for (int m = 0; m < ML; m++) {
        ra.Fout[m] = L.Fout[m];
        ra.Min[m] = L.Min[m];
        ra.Pin[m] = L.Pin[m];
        ra.Mout[m] = L.Mout[m];
        ra.Pout[m] = L.Pout[m];
        ra.kstar[m] = L.kstar[m];
    }
    ra.last = L.last;
    ra.layer = L.layer;
    ra.last_stride = L.last_stride;
    ra.p = L.H.p;
    ra.c0d = L.H.c0d;
    dim3 rg((unsigned)((ncol + 255) / 256), (unsigned)ML);
    if (L.backward)
        k_dp_reduce<true><<<rg, 256, 0, st>>>(ra);
    else
        k_dp_reduce<false><<<rg, 256, 0, st>>>(ra);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_dp_layer(const DpLayer& L, hipStream_t st) {
    if (L.jhi < L.jlo) return hipSuccess;
    if (L.nlam == 1)
        return layer_launch<kColsPerLane, 1, ECASQ_PRED_SMEM != 0>(L, st);
    if (L.nlam == kMaxLambdas && !L.backward)
        return layer_launch<kColsPerLaneMulti, kMaxLambdas, false>(L, st);
    return hipErrorInvalidValue;
}

hipError_t launch_dp_init_fwd(const Hist& H, int64_t lo, int64_t jl, int64_t jh,
                              const DpInit& I, hipStream_t st) {
    if (jh < jl) return hipSuccess;
    if (I.nlam < 1 || I.nlam > kMaxLambdas) return hipErrorInvalidValue;
    const unsigned g = (unsigned)((jh - jl + 1 + 255) / 256);
    k_dp_init_fwd<<<g, 256, 0, st>>>(H, lo, jl, jh, I);
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
                           int32_t nlam, double* out, hipStream_t st) {
    if (nlam < 1 || nlam > kMaxLambdas) return hipErrorInvalidValue;
    k_dp_final<<<1, 64, 0, st>>>(last, stride, imax, exact_s, out, nlam);
    return hipGetLastError();
}

hipError_t launch_split(const double* Fw, const double* Bw, int64_t ml, int64_t mh,
                        int64_t* m_out, hipStream_t st) {
    k_split<<<1, 256, 0, st>>>(Fw, Bw, ml, mh, m_out);
    return hipGetLastError();
}

}  // namespace ecasq
