// dp_APX (Sec. 5, eq. apx_base / apx_rec / apx_final) for one multiplier as a
// sweep over column blocks that updates every layer from each cell.
//
// The interval cost C[k,j] and the entropy term Phi[k,j] do not depend on the
// layer i, but the layer-by-layer schedule recomputes them for every layer.
// Here the (k, j) triangle is swept once: with F_i[k] final for all layers i
// and all k of the blocks before column block J, one evaluation of C and Phi
// serves the candidates F_{i-1}[k] + C + lambda' Phi of every layer.  The
// price is O(s p) memory (F of every layer: 8 (s+1) p bytes, 0.07 GB at
// p = 2^18, s = 32) instead of O(p) rolling buffers; the values are the same
// bit for bit (same candidate arithmetic; the minimum of a set does not depend
// on the order, up to the sign of an exact zero).
//
// The sweep keeps values only: a layer's update per cell is an add and a min
// (the pair's cost Q = C - lambda' Phi is formed once for all layers).  With
// every F_{i-1} kept, the argmin of any (i, j) is recomputed
// when needed: the traceback of the chosen layer asks for one column per
// layer (t columns of at most p candidates each, a few hundred microseconds,
// against O(s p^2) for tracking the argmin of every cell), taking the lowest k
// among equal candidates exactly as the DP's strict '<' in increasing k does.
// The path's MSE and H(I,B) are then summed along it in path order (the same
// additions the layer-by-layer accumulators perform).
//
// A step of the sweep (blocks of 64 columns, one per wavefront) is one launch
// of k_sweep_step that makes blocks t..t+nb-1 final (nb = ECASQ_SWEEP_NB but
// for the last step), with blocks tp..t-1 made final by the step before:
//   workgroup m    block t+m (m < nb): its costs first, then the final
//                  blocks not yet added to it (t-1, and t..t+m-1 as the
//                  workgroups before it publish them), then the triangle
//                  inside it layer after layer (a layer needs the previous
//                  layer's values of the same block); then it publishes
//                  the block (a flag the later workgroups wait for);
//   the others     blocks J >= t+nb: the contribution of blocks tp..t-1 to
//                  their running minima, kept in F; the next step's
//                  diagonal blocks also take t..t+nb-2 as they are
//                  published, so that its chain starts with one block to add.
// The fixed cost of a launch (dispatch, staging, the running minima read and
// written back) is shared by nb blocks, and the chain inside a launch costs
// one block addition and one triangle per block.
#include <stddef.h>

#include "device.hpp"
#include "launch.hpp"

namespace ecasq {

namespace {

constexpr int kSB = 64;        // columns per block (one wavefront)
constexpr int kTileWaves = 4;  // wavefronts per workgroup
// Wavefronts per column block in the tile role (the block's 64 predecessors
// split between them; their partial minima meet in LDS): 4 below
// ECASQ_SWEEP_SP4_BELOW (column block, layer group) tiles, 2 below
// ECASQ_SWEEP_SP2_BELOW, else 1.  More wavefronts per tile fill the SIMDs of
// the late steps, which have few blocks left, without recomputing C and Phi.
#ifndef ECASQ_SWEEP_SP4_BELOW
#define ECASQ_SWEEP_SP4_BELOW 1792
#endif
#ifndef ECASQ_SWEEP_SP2_BELOW
#define ECASQ_SWEEP_SP2_BELOW 3584
#endif
// diagonal blocks a step makes final (one workgroup each, in a chain within
// the launch; fewer launches share their fixed cost between more blocks)
#ifndef ECASQ_SWEEP_NB
#define ECASQ_SWEEP_NB 16
#endif
// polls of a block's flag before a wait gives up (about a second)
#ifndef ECASQ_SWEEP_SPIN
#define ECASQ_SWEEP_SPIN (1u << 21)
#endif
// widest layer group (register arrays of that many layers per lane)
#ifndef ECASQ_SWEEP_LG_MAX
#define ECASQ_SWEEP_LG_MAX 32
#endif
// tile workgroups keep their column blocks on one XCD from launch to launch
#ifndef ECASQ_SWEEP_XCD
#define ECASQ_SWEEP_XCD 1
#endif
// wavefronts per SIMD the step kernel's registers are sized for (0: the
// compiler's choice).  4 (128 VGPRs) lets the early steps' ~4000 tile
// wavefronts run in one round; it costs a few spilled registers outside the
// predecessor loops.
#ifndef ECASQ_SWEEP_WAVES
#define ECASQ_SWEEP_WAVES 4
#endif
// layer counts per wavefront up to which predecessors are taken in pairs
// (two independent C / Phi chains per iteration; also fewer registers)
#ifndef ECASQ_SWEEP_PAIR_MAX
#define ECASQ_SWEEP_PAIR_MAX 32
#endif
// LDS read pairs the tile loop keeps in flight ahead of their use (0: the
// scheduler's own order)
#ifndef ECASQ_SWEEP_AHEAD
#define ECASQ_SWEEP_AHEAD 2
#endif
// the tile loop issues the four log2 table reads of a predecessor pair
// before it uses any
#ifndef ECASQ_SWEEP_LOG_BATCH
#define ECASQ_SWEEP_LOG_BATCH 1
#endif
#if ECASQ_SWEEP_WAVES > 0
#define ECASQ_STEP_ATTR __attribute__((amdgpu_waves_per_eu(ECASQ_SWEEP_WAVES)))
#else
#define ECASQ_STEP_ATTR
#endif

// Helpers of the step's chain: diagonal block b = t + m takes the blocks
// tp..b-2 it has not yet added (the last step's blocks and this step's
// before b-1) from helper workgroups, kHelpBlocks blocks each, which run side
// by side and leave their partial minima of every layer of block b in a
// buffer of their own.
constexpr int kHelpBlocks = 2;
// (helper_block keeps the costs of exactly two blocks: q0 and q1)
static_assert(kHelpBlocks == 2, "a helper adds two blocks");
constexpr int kHelpMax = ECASQ_SWEEP_NB > 1 ? ECASQ_SWEEP_NB - 1 : 1;  // per diagonal block

// Cost tables Q = C - lambda' Phi (they do not depend on F), formed by the
// workgroups of the chain before they wait for anything and read back into
// registers once: T[k][c] of predecessor 64 kb + k against column 64 b + c
// of a diagonal block b (the last column in place of columns past p - 1; for
// kb = b, +inf unless 64 b + k < the column).  Slot of diagonal workgroup m:
// blocks b-1 and b; slot of its helper h: the helper's blocks.  Then the
// helpers' partial minima, kPLayers layers of 64 columns each.
constexpr int64_t kQTab = (int64_t)kSB * kSB;
constexpr int64_t kQSlot = (int64_t)kHelpBlocks * kQTab;  // two tables per workgroup
constexpr int64_t kPLayers = 256;                         // layers 3..258 include 3..I
constexpr int64_t kPartAt = (int64_t)ECASQ_SWEEP_NB * (1 + kHelpMax) * kQSlot;
constexpr int64_t kQAll = kPartAt + (int64_t)ECASQ_SWEEP_NB * kHelpMax * kPLayers * kSB;

struct SweepArgs {
    Hist H;
    double* F;    // [I+1][ld]: rows 2..I; running minima until a block is final
    double* Q;    // kQAll doubles: the chain's cost tables
    int32_t* K;   // argmins recomputed for inspection (same layout), and scratch
                  // (during the steps: chunk counters of blocks K[0..nblk), the
                  // failure word K[nblk], the helpers' counters after it)
    int64_t ld;
    int32_t I;    // last layer, min(s, p)
    double lamp;  // lambda' (MSE units)
    int64_t nblk;
    const double* lampp;  // device lambda' (replaces lamp when set)
    const int32_t* runp;  // device run flag: 0 skips the solve (null: run)
};

// Every kernel of a solve starts here: false when the run flag says the
// solve is skipped, else lambda' taken from device memory when given.
__device__ __forceinline__ bool sweep_live(SweepArgs& a) {
    if (a.runp && *a.runp == 0) return false;
    if (a.lampp) a.lamp = *a.lampp;
    return true;
}

// Row padding of the staging buffer: the staging stores of a wavefront
// (one row each, the same column) fall in 8 banks instead of one, and rows
// stay 16-byte aligned for the two-value broadcast reads.
constexpr int kSFPad = 2;

// Stage predecessor block [k0, k0+64): v, N, S, S2 and F_{i-1} for the LG
// layers i0..i0+LG-1 (+inf past I).  All kThreads threads of the workgroup
// take part; each issues all its loads before it stores any to LDS.
constexpr int kThreads = kSB * kTileWaves;
template <int LG>
__device__ __forceinline__ void stage_block(const SweepArgs& a, int64_t k0, int32_t i0, double* sv,
                                            double* sN, double* sS, double* sS2,
                                            double (*sF)[LG + kSFPad]) {
    // block [k0, k0+64) lies below a later block, so k0 + 63 < p
    constexpr int R = kSB * LG / kThreads;  // F values per thread
    static_assert(R * kThreads == kSB * LG, "a layer group of 64 columns fills the workgroup");
    // the row stride as a value the compiler cannot carry across calls: the
    // R row addresses are formed here (a few integer operations) instead of
    // being kept for the whole tile loop in registers it does not have
    int64_t ld = a.ld;
    asm volatile("" : "+s"(ld));
    double f[R];
#pragma unroll
    for (int r = 0; r < R; r++) {
        const int x = threadIdx.x + r * kThreads;
        const int kk = x % kSB, l = x / kSB;
        const int32_t i = i0 + l;
        f[r] = i <= a.I ? a.F[(int64_t)(i - 1) * ld + k0 + kk] : __builtin_huge_val();
    }
    if (threadIdx.x < kSB) {
        const int64_t k = k0 + threadIdx.x;
        sv[threadIdx.x] = a.H.v[k];
        sN[threadIdx.x] = a.H.N[k];
        sS[threadIdx.x] = a.H.S[k];
        sS2[threadIdx.x] = a.H.S2[k];
    }
#pragma unroll
    for (int r = 0; r < R; r++) {
        const int x = threadIdx.x + r * kThreads;
        sF[x % kSB][x / kSB] = f[r];
    }
}

// F_{i-1} of the LW layers ic.. of a chunk for blocks u0..u0+n-1 (n <= NU)
// into sF[k][u LW + l] (+inf past I); all kThreads threads take part and
// issue their loads before their stores.
template <int LG, int LW, int NU>
__device__ __forceinline__ void stage_chunk(const SweepArgs& a, int64_t u0, int n, int32_t ic,
                                            double (*sF)[LG + kSFPad]) {
    constexpr int R = (kSB * LW + kThreads - 1) / kThreads;  // values per thread and block
    double f[NU][R];
#pragma unroll
    for (int u = 0; u < NU; u++) {
#pragma unroll
        for (int r = 0; r < R; r++) {
            const int x = threadIdx.x + r * kThreads;
            const int32_t i = ic + x / kSB;
            f[u][r] = u < n && x < kSB * LW && i <= a.I
                          ? a.F[(int64_t)(i - 1) * a.ld + (u0 + u) * kSB + x % kSB]
                          : __builtin_huge_val();
        }
    }
#pragma unroll
    for (int u = 0; u < NU; u++) {
        if (u < n) {
#pragma unroll
            for (int r = 0; r < R; r++) {
                const int x = threadIdx.x + r * kThreads;
                if (x < kSB * LW) sF[x % kSB][u * LW + x / kSB] = f[u][r];
            }
        }
    }
}

// Rows 2..I of F := +inf in columns 0..p-1 (nothing seen yet; also the value
// of every entry outside a layer's valid columns, which makes such
// predecessors lose; columns from p on are never read), row 2 + blockIdx.y.
// Also clears the steps' counters and failure word (K[0..nblk (1 + kHelpMax)]).
__global__ __launch_bounds__(256) void k_sweep_fill(SweepArgs a) {
    if (!sweep_live(a)) return;
    const int64_t p = a.H.p;
    double* row = a.F + (int64_t)(2 + blockIdx.y) * a.ld;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < p;
         j += (int64_t)gridDim.x * blockDim.x)
        row[j] = __builtin_huge_val();
    if (blockIdx.y == 0)
        for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
             x <= a.nblk * (1 + kHelpMax); x += (int64_t)gridDim.x * blockDim.x)
            a.K[x] = 0;
}

// Shared memory of one step workgroup.
template <int LG>
struct StepSmem {
    double2 tab[kLog2Size];
    // v, N, S, S2 of two blocks: a tile's staged predecessor block in [0],
    // the chain roles' two blocks in [0] and [1]
    double hv[2][kSB], hN[2][kSB], hS[2][kSB], hS2[2][kSB];
    double sF[kSB][LG + kSFPad];  // F_{i-1} of the staged block for one layer group
    double pF[kSB];                               // previous layer of block t
    double partV[kTileWaves][kSB];                // per-wave partial minima
};
// the staging rows are read two layers at a time (16-byte LDS reads)
static_assert(offsetof(StepSmem<8>, sF) % 16 == 0 && offsetof(StepSmem<16>, sF) % 16 == 0 &&
                  offsetof(StepSmem<32>, sF) % 16 == 0 && (8 + kSFPad) % 2 == 0,
              "staging rows 16-byte aligned");

// Running minima of LW layers i0.. of column jj (rows past I: +inf).
template <int LW>
__device__ __forceinline__ void load_running(const SweepArgs& a, int64_t jj, int32_t i0,
                                             double (&best)[LW]) {
#pragma unroll
    for (int l = 0; l < LW; l++) {
        const int32_t i = i0 + l;
        best[l] = i <= a.I ? a.F[(int64_t)i * a.ld + jj] : __builtin_huge_val();
    }
}

template <int LW>
__device__ __forceinline__ void store_running(const SweepArgs& a, int64_t j, int32_t i0,
                                              const double (&best)[LW]) {
    if (j >= a.H.p) return;
#pragma unroll
    for (int l = 0; l < LW; l++) {
        const int32_t i = i0 + l;
        if (i <= a.I) a.F[(int64_t)i * a.ld + j] = best[l];
    }
}

// best[l] = min(best[l], F0[l] + Q0, F1[l] + Q1) for the LW layers of two
// staged rows (16-byte aligned), read two layers at a time.  Scheduling
// barriers keep ECASQ_SWEEP_AHEAD read pairs in flight ahead of the adds and
// minima that use them, so that the LDS latency overlaps arithmetic instead
// of stalling the wavefront once per read (left alone, the scheduler waits
// for each read right after issuing it, for want of registers).
template <int LW>
__device__ __forceinline__ void add_min_rows(const double* F0, const double* F1, double Q0,
                                             double Q1, double (&best)[LW]) {
    static_assert(LW % 2 == 0, "layers in pairs");
    constexpr int H = LW / 2;
    constexpr int D = ECASQ_SWEEP_AHEAD < H ? ECASQ_SWEEP_AHEAD : H;
    const double2* r0 = reinterpret_cast<const double2*>(F0);
    const double2* r1 = reinterpret_cast<const double2*>(F1);
    double2 a[H], b[H];
#pragma unroll
    for (int h = 0; h < D; h++) {
        a[h] = r0[h];
        b[h] = r1[h];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int h = 0; h < H; h++) {
        if (h + D < H) {
            a[h + D] = r0[h + D];
            b[h + D] = r1[h + D];
        }
        best[2 * h] = __builtin_fmin(best[2 * h], a[h].x + Q0);
        best[2 * h] = __builtin_fmin(best[2 * h], b[h].x + Q1);
        best[2 * h + 1] = __builtin_fmin(best[2 * h + 1], a[h].y + Q0);
        best[2 * h + 1] = __builtin_fmin(best[2 * h + 1], b[h].y + Q1);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Staged predecessors kb..ke-1 (ke - kb even) against column (cv, cN, cS,
// cS2) for LW layers whose F_{i-1} sit in sF columns lofs..lofs+LW-1.  At
// lambda' = 0 the cost is C alone (cell_c: the same value as the fma with
// a zero multiplier), without the entropy terms.
template <int LG, int LW>
__device__ __forceinline__ void accumulate(const StepSmem<LG>& sm, int lofs, int kb, int ke,
                                           double cv, double cN, double cS, double cS2, double dd,
                                           double lamp, double (&best)[LW]) {
    if constexpr (LW > ECASQ_SWEEP_PAIR_MAX) {
        // many layers per predecessor: enough independent work per iteration
        for (int kk = kb; kk < ke; kk++) {
            double C, P;
            cell_terms(sm.hv[0][kk], sm.hN[0][kk], sm.hS[0][kk], sm.hS2[0][kk], cv, cN, cS, cS2, dd, false,
                       0.0, sm.tab, C, P);
            const double Q = __builtin_fma(-lamp, P, C);
#pragma unroll
            for (int l = 0; l < LW; l++) best[l] = __builtin_fmin(best[l], sm.sF[kk][lofs + l] + Q);
        }
    } else {
    // few layers: two predecessors per iteration, whose C and Phi are
    // independent chains the scheduler can interleave
    for (int kk = kb; kk < ke; kk += 2) {
        const double v0 = sm.hv[0][kk], N0 = sm.hN[0][kk], S0 = sm.hS[0][kk],
                     S20 = sm.hS2[0][kk];
        const double v1 = sm.hv[0][kk + 1], N1 = sm.hN[0][kk + 1], S1 = sm.hS[0][kk + 1],
                     S21 = sm.hS2[0][kk + 1];
        double Q0, Q1;
        if (lamp == 0.0) {  // uniform
            Q0 = cell_c(v0, N0, S0, S20, cv, cN, cS, cS2);
            Q1 = cell_c(v1, N1, S1, S21, cv, cN, cS, cS2);
        } else {
#if ECASQ_SWEEP_LOG_BATCH
            // cell_terms of both predecessors, the four table reads issued
            // together before any is used
            double C0, mu0, md0, C1, mu1, md1;
            cell_pre(v0, N0, S0, S20, cv, cN, cS, cS2, dd, false, 0.0, C0, mu0, md0);
            cell_pre(v1, N1, S1, S21, cv, cN, cS, cS2, dd, false, 0.0, C1, mu1, md1);
            const Log2Arg u0 = log2c_arg(mu0), d0 = log2c_arg(md0);
            const Log2Arg u1 = log2c_arg(mu1), d1 = log2c_arg(md1);
            const double2 tu0 = sm.tab[u0.ir], td0 = sm.tab[d0.ir];
            const double2 tu1 = sm.tab[u1.ir], td1 = sm.tab[d1.ir];
            __builtin_amdgcn_sched_barrier(0);
            const double P0 = __builtin_fma(mu0, log2c_fin(u0, tu0), md0 * log2c_fin(d0, td0));
            const double P1 = __builtin_fma(mu1, log2c_fin(u1, tu1), md1 * log2c_fin(d1, td1));
#else
            double C0, P0, C1, P1;
            cell_terms(v0, N0, S0, S20, cv, cN, cS, cS2, dd, false, 0.0, sm.tab, C0, P0);
            cell_terms(v1, N1, S1, S21, cv, cN, cS, cS2, dd, false, 0.0, sm.tab, C1, P1);
#endif
            Q0 = __builtin_fma(-lamp, P0, C0);
            Q1 = __builtin_fma(-lamp, P1, C1);
        }
#if ECASQ_SWEEP_AHEAD > 0
        add_min_rows<LW>(&sm.sF[kk][lofs], &sm.sF[kk + 1][lofs], Q0, Q1, best);
#else
#pragma unroll
        for (int l = 0; l < LW; l++) {
            best[l] = __builtin_fmin(best[l], sm.sF[kk][lofs + l] + Q0);
            best[l] = __builtin_fmin(best[l], sm.sF[kk + 1][lofs + l] + Q1);
        }
#endif
    }
    }
}

// As accumulate, with the costs Q of predecessors kb..ke-1 (ke - kb even)
// read from Qc[kk * 64] instead of formed here (same update order).
template <int LG, int LW>
__device__ __forceinline__ void accumulate_q(const StepSmem<LG>& sm, int kb, int ke,
                                             const double* __restrict__ Qc, double (&best)[LW]) {
    for (int kk = kb; kk < ke; kk += 2) {
        const double Q0 = Qc[kk * kSB], Q1 = Qc[(kk + 1) * kSB];
#pragma unroll
        for (int l = 0; l < LW; l++) {
            best[l] = __builtin_fmin(best[l], sm.sF[kk][l] + Q0);
            best[l] = __builtin_fmin(best[l], sm.sF[kk + 1][l] + Q1);
        }
    }
}

// v, N, S, S2 of block kb (indices past p - 1 clamped) into LDS; call from
// all threads, then __syncthreads().
__device__ __forceinline__ void stage_hist(const SweepArgs& a, int64_t kb, double* sv, double* sN,
                                           double* sS, double* sS2) {
    if (threadIdx.x < kSB) {
        const int64_t k = kb * kSB + threadIdx.x < a.H.p ? kb * kSB + threadIdx.x : a.H.p - 1;
        sv[threadIdx.x] = a.H.v[k];
        sN[threadIdx.x] = a.H.N[k];
        sS[threadIdx.x] = a.H.S[k];
        sS2[threadIdx.x] = a.H.S2[k];
    }
}

// Cost tables against the columns of block b (cv.. the column of the
// thread's lane, jj its index): T + x kQTab for x = 0..n-1 holds the table of
// the predecessor block whose v, N, S, S2 are staged in sv[x].. (block kb0 +
// x).  A thread takes predecessors wave, wave + 4, ... of each block.  The
// arguments of cell_terms are those of the tiles, so the costs are the same
// bit for bit.
__device__ void form_costs(const SweepArgs& a, int64_t b, int64_t kb0, int n,
                           const double (*sv)[kSB], const double (*sN)[kSB],
                           const double (*sS)[kSB], const double (*sS2)[kSB], int64_t jj,
                           double cv, double cN, double cS, double cS2,
                           const double2* __restrict__ tab, double* __restrict__ T0) {
    const int wave = threadIdx.x / kSB, lane = threadIdx.x % kSB;
    for (int x = 0; x < n; x++) {
        const int64_t kb = kb0 + x;
        double* T = T0 + (int64_t)x * kQTab;
#pragma unroll 2
        for (int k = wave; k < kSB; k += kTileWaves) {
            double q = __builtin_huge_val();
            if (kb < b || kb * kSB + k < jj) {
                if (a.lamp == 0.0) {  // C alone (cell_c), as in the tiles
                    q = cell_c(sv[x][k], sN[x][k], sS[x][k], sS2[x][k], cv, cN, cS, cS2);
                } else {
                    double C, P;
                    cell_terms(sv[x][k], sN[x][k], sS[x][k], sS2[x][k], cv, cN, cS, cS2, a.H.dd,
                               false, 0.0, tab, C, P);
                    q = __builtin_fma(-a.lamp, P, C);
                }
            }
            T[k * kSB + lane] = q;
        }
    }
}

// This wavefront's 16 predecessors' costs from table T (this lane's column).
__device__ __forceinline__ void lane_costs(const double* __restrict__ T,
                                           double (&Q)[kSB / kTileWaves]) {
    constexpr int KW = kSB / kTileWaves;
    const int wave = threadIdx.x / kSB, lane = threadIdx.x % kSB;
#pragma unroll
    for (int q = 0; q < KW; q++) Q[q] = T[(wave * KW + q) * kSB + lane];
}

// Chunk counters of the step's chain: flag[b] counts the chunks of block b
// that are final (a chunk is the LG/4 layers of a layer group that one
// wavefront of the diagonal workgroup holds; chunks are final in order, so
// flag[b] = n means every layer up to the n'th chunk's last); flag[nblk] != 0
// once a wait has given up.  Both live in K (free during the steps) and are
// cleared by k_sweep_fill.
//
// wait_flag: one thread polls flag[b] until it reaches n (device-scope loads,
// which see other XCDs' stores), then an acquire fence makes the chunks'
// values visible to the workgroup, whose threads meet at the barrier.  The
// wait is bounded: after ECASQ_SWEEP_SPIN polls it marks the solve failed and
// returns, and every later wait returns at once, so every wavefront ends;
// k_sweep_pick then reports no codebook.
__device__ __forceinline__ void poll_flag(const SweepArgs& a, int64_t b, int32_t n) {
    int32_t* flag = a.K;
    for (uint32_t r = 0;; r++) {
        if (__hip_atomic_load(flag + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= n) break;
        if ((r & 63) == 0 &&
            __hip_atomic_load(flag + a.nblk, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
            break;
        if (r >= ECASQ_SWEEP_SPIN) {
            __hip_atomic_store(flag + a.nblk, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

__device__ void wait_flag(const SweepArgs& a, int64_t b, int32_t n) {
    if (threadIdx.x == 0) {
        poll_flag(a, b, n);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
}

// As wait_flag for the counters K[b0] (b0 >= 0) and K[h0..h0+nh), all >= n:
// one acquire and one barrier.
__device__ void wait_flags(const SweepArgs& a, int64_t b0, int64_t h0, int nh, int32_t n) {
    if (threadIdx.x == 0) {
        if (b0 >= 0) poll_flag(a, b0, n);
        for (int x = 0; x < nh; x++) poll_flag(a, h0 + x, n);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
}

// flag[b] := n: every wavefront waits for its stores, and after the barrier
// one thread releases them (device scope) and sets the counter.
__device__ void publish_flag(const SweepArgs& a, int64_t b, int32_t n) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __hip_atomic_store(a.K + b, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Stage predecessor block [k0, k0+64) with F_{i-1} of layers i0..i0+LG-1.
template <int LG>
__device__ __forceinline__ void stage_pred(const SweepArgs& a, int64_t k0, int32_t i0,
                                           StepSmem<LG>& sm) {
    stage_block<LG>(a, k0, i0, sm.hv[0], sm.hN[0], sm.hS[0], sm.hS2[0], sm.sF);
}

// Tile role: the column blocks Jw..Jw+per-1 (those in [Jlo, nblk) live) of
// one layer group (its first NL layers; NL < LG only where the layers past
// them exceed I) take the blocks tp..t-1, made final by the last step.  SP
// wavefronts per column block, each taking 64/SP of the predecessors; with
// SP > 1 their partial minima meet in LDS (the staging buffer, free once
// every wavefront is done with it), LG/4 layers at a time, and the wavefront
// that merges a chunk (its partial started from the chunk's running minima)
// writes the result to F.
template <int LG, int NL, int SP>
__device__ void tile_role(const SweepArgs& a, int64_t t, int64_t tp, int64_t Jw, int64_t Jlo,
                          int32_t g, StepSmem<LG>& sm) {
    constexpr int KP = kSB / SP;
    const int32_t i0 = 3 + g * LG;
    const int64_t p = a.H.p;
    const int wave = threadIdx.x / kSB, lane = threadIdx.x % kSB;
    const int part = wave % SP;
    constexpr int64_t per = kTileWaves / SP;  // column blocks per workgroup
    const int64_t J = Jw + wave / SP;  // the same for the SP wavefronts of a column block
    const bool live = J >= Jlo && J < a.nblk;
    if (Jw + per <= Jlo || Jw >= a.nblk || t <= tp) return;  // uniform: nothing to do
    const int64_t j = J * kSB + lane;
    const int64_t jj = live && j < p ? j : p - 1;
    // this column's values and running minima first: their latency overlaps
    // the table and staging loads
    const double cv = a.H.v[jj], cN = a.H.N[jj], cS = a.H.S[jj], cS2 = a.H.S2[jj];
    constexpr int CH = LG / kTileWaves;  // layers per merge chunk (SP > 1)
    double best[NL];
    if constexpr (SP == 1) {
        if (live) load_running<NL>(a, jj, i0, best);
    } else {
        // the wavefront that merges a chunk starts from its running minima
#pragma unroll
        for (int l = 0; l < NL; l++) {
            const int32_t i = i0 + l;
            best[l] = (live && part == (l / CH) % SP && i <= a.I) ? a.F[(int64_t)i * a.ld + jj]
                                                                 : __builtin_huge_val();
        }
    }
    load_log2_table(sm.tab);
    for (int64_t pb = tp; pb < t; pb++) {
        if (pb > tp) __syncthreads();  // every wavefront is done with the last block
        // issue priority 2, 1, 0 over the thirds of the blocks: a SIMD's tile
        // wavefronts otherwise finish one after another (the oldest is issued
        // first) and the last runs alone at a fraction of the issue rate; the
        // chain keeps priority 3
        const int64_t third = (3 * (pb - tp)) / (t - tp);
        if (third == 0)
            __builtin_amdgcn_s_setprio(2);
        else if (third == 1)
            __builtin_amdgcn_s_setprio(1);
        else
            __builtin_amdgcn_s_setprio(0);
        stage_pred<LG>(a, pb * kSB, i0, sm);
        __syncthreads();
        if (live)
            accumulate<LG, NL>(sm, 0, part * KP, part * KP + KP, cv, cN, cS, cS2, a.H.dd, a.lamp,
                               best);
    }
    if constexpr (SP == 1) {
        if (live) store_running<NL>(a, j, i0, best);
    } else {
        // 4 x CH rows of 64 fit the staging buffer
        double (*xb)[kSB] = reinterpret_cast<double (*)[kSB]>(&sm.sF[0][0]);
        const int lead = wave - part;
        __syncthreads();  // the staging buffer is free
#pragma unroll
        for (int c0 = 0; c0 < NL; c0 += CH) {
            const int c = c0 / CH;
#pragma unroll
            for (int l = c0; l < c0 + CH && l < NL; l++) xb[wave * CH + l - c0][lane] = best[l];
            __syncthreads();
            if (live && part == c % SP) {
#pragma unroll
                for (int l = c0; l < c0 + CH && l < NL; l++) {
                    const int32_t i = i0 + l;
                    if (i > a.I) break;
                    double v = xb[lead * CH + l - c0][lane];
#pragma unroll
                    for (int u = 1; u < SP; u++) v = __builtin_fmin(v, xb[(lead + u) * CH + l - c0][lane]);
                    if (j < p) a.F[(int64_t)i * a.ld + j] = v;
                }
            }
            __syncthreads();
        }
    }
}

// Index of the chunk counter of helper h of block b in K.
__device__ __forceinline__ int64_t help_counter(const SweepArgs& a, int64_t b, int h) {
    return a.nblk + 1 + b * kHelpMax + h;
}

// Helpers of diagonal block b = t + m: the blocks tp..b-2 not yet added to
// b, kHelpBlocks per helper.
__device__ __forceinline__ int helpers_of(int64_t t, int64_t tp, int32_t m) {
    const int64_t n = t + m - 1 - tp;
    return n > 0 ? (int)((n + kHelpBlocks - 1) / kHelpBlocks) : 0;
}

// Partial minima of helper h of diagonal workgroup m: kPLayers rows of 64.
__device__ __forceinline__ double* help_partials(const SweepArgs& a, int32_t m, int h) {
    return a.Q + kPartAt + ((int64_t)m * kHelpMax + h) * kPLayers * kSB;
}

// Helper h of diagonal block b = t + m: blocks u0..u1-1 (u0 = tp +
// kHelpBlocks h), chunk by chunk as their chunks become final (waited for):
// each wavefront takes 16 predecessors of each block with their costs in
// registers, the four partial minima meet in LDS and go to the helper's
// buffer, one row per layer; then the helper's counter is published.
template <int LG, int NL>
__device__ void helper_block(const SweepArgs& a, int64_t t, int64_t tp, int32_t m, int h,
                             StepSmem<LG>& sm) {
    constexpr int LW = LG / kTileWaves;   // layers per chunk
    constexpr int KW = kSB / kTileWaves;  // predecessors of a block per wavefront
    const int wave = threadIdx.x / kSB, lane = threadIdx.x % kSB;
    const int64_t p = a.H.p;
    const int64_t b = t + m;
    const int64_t u0 = tp + (int64_t)kHelpBlocks * h;
    const int64_t u1 = min<int64_t>(u0 + kHelpBlocks, b - 1);
    if (u0 >= u1 || a.I < 3) return;  // uniform: nothing to add
    const int nu = (int)(u1 - u0);
    const int64_t jj = min<int64_t>(b * kSB + lane, p - 1);
    double* T = a.Q + ((int64_t)ECASQ_SWEEP_NB + (int64_t)m * kHelpMax + h) * kQSlot;
    double* P = help_partials(a, m, h);
    stage_hist(a, u0, sm.hv[0], sm.hN[0], sm.hS[0], sm.hS2[0]);
    if (nu > 1) stage_hist(a, u0 + 1, sm.hv[1], sm.hN[1], sm.hS[1], sm.hS2[1]);
    const double cv = a.H.v[jj], cN = a.H.N[jj], cS = a.H.S[jj], cS2 = a.H.S2[jj];
    __syncthreads();  // (also the log2 table)
    form_costs(a, b, u0, nu, sm.hv, sm.hN, sm.hS, sm.hS2, jj, cv, cN, cS, cS2, sm.tab, T);
    __syncthreads();  // the tables
    double q0[KW], q1[KW];
    lane_costs(T, q0);
    if (nu > 1) lane_costs(T + kQTab, q1);
    double (*xb)[kSB] = reinterpret_cast<double (*)[kSB]>(&sm.sF[0][0]);
    int32_t cg = 0;  // chunks published
    for (int32_t i0 = 3; i0 <= a.I; i0 += LG) {
#pragma unroll 1
        for (int c = 0; c < kTileWaves; c++) {
            const int32_t ic = i0 + c * LW;  // the chunk's first layer
            if (ic > a.I) break;
            if (u1 - 1 >= t) wait_flag(a, u1 - 1, cg + 1);
            __syncthreads();  // the staging buffer is free
            stage_chunk<LG, LW, kHelpBlocks>(a, u0, nu, ic, sm.sF);
            __syncthreads();
            double pa[LW];
#pragma unroll
            for (int l = 0; l < LW; l++) pa[l] = __builtin_huge_val();
#pragma unroll
            for (int q = 0; q < KW; q++) {
                const int kk = wave * KW + q;
#pragma unroll
                for (int l = 0; l < LW; l++) pa[l] = __builtin_fmin(pa[l], sm.sF[kk][l] + q0[q]);
            }
            if (nu > 1) {
#pragma unroll
                for (int q = 0; q < KW; q++) {
                    const int kk = wave * KW + q;
#pragma unroll
                    for (int l = 0; l < LW; l++)
                        pa[l] = __builtin_fmin(pa[l], sm.sF[kk][LW + l] + q1[q]);
                }
            }
            __syncthreads();  // the staging buffer is free: 4 x LW rows of 64
#pragma unroll
            for (int l = 0; l < LW; l++) xb[wave * LW + l][lane] = pa[l];
            __syncthreads();
            for (int x = threadIdx.x; x < LW * kSB; x += blockDim.x) {
                const int l = x / kSB, c2 = x % kSB;
                P[(int64_t)(ic - 3 + l) * kSB + c2] =
                    __builtin_fmin(__builtin_fmin(xb[l][c2], xb[LW + l][c2]),
                                   __builtin_fmin(xb[2 * LW + l][c2], xb[3 * LW + l][c2]));
            }
            cg++;
            publish_flag(a, help_counter(a, b, h), cg);
        }
        if constexpr (NL < LG) break;  // one group holds every layer (I = NL + 2)
    }
}

// Diagonal role: workgroup m of a step makes block b = t + m final, one chunk
// at a time (chunk c of a layer group: the LW = LG/4 layers that wavefront c
// holds, with their running minima).  It first forms the cost tables of
// block b-1 and of b itself and keeps its 16 predecessors' costs of both in
// registers.  Then per chunk: once that chunk of block b-1 is final and the
// helper has folded the blocks before b-1 into b's running minima (both
// waited for), the holder reads the running minima of the chunk's layers,
// and block b-1's contribution (each wavefront takes 16 of its
// predecessors) is merged into them in LDS; then the chunk's layers inside the
// block in order: each wavefront holds the cost Q of 16 of the block's
// predecessors in registers, the four partial minima meet in LDS and the
// holder merges them; then the chunk is published.  So block b's chunk c
// needs block b-1's chunk c, not all of block b-1.
template <int LG, int NL>
__device__ void diag_block(const SweepArgs& a, int64_t t, int64_t tp, int32_t m,
                           StepSmem<LG>& sm) {
    constexpr int LW = LG / kTileWaves;   // layers per chunk
    constexpr int KW = kSB / kTileWaves;  // predecessors of a block per wavefront
    const int wave = threadIdx.x / kSB, lane = threadIdx.x % kSB;
    const int64_t p = a.H.p;
    const int64_t b = t + m;
    const int64_t j = b * kSB + lane;
    const int64_t jj = j < p ? j : p - 1;
    const bool valid = j < p;
    const int64_t kpd = tp;                 // first block not yet added to b
    const int nh = helpers_of(t, tp, m);    // blocks kpd..b-2 come from the helpers
    // the tables of the costs of (k, j) for block b-1's predecessors k and
    // block b's own (+inf unless k < j), the same for every chunk
    double* T = a.Q + (int64_t)m * kQSlot;  // block b-1's table, then b's own
    const int64_t kb0 = b >= 1 ? b - 1 : b;
    stage_hist(a, kb0, sm.hv[0], sm.hN[0], sm.hS[0], sm.hS2[0]);
    if (b >= 1) stage_hist(a, b, sm.hv[1], sm.hN[1], sm.hS[1], sm.hS2[1]);
    __syncthreads();  // (also the log2 table)
    const int cc = (int)(jj - b * kSB);
    {
        const int o = b >= 1 ? 1 : 0;  // block b's place
        const double cv = sm.hv[o][cc], cN = sm.hN[o][cc], cS = sm.hS[o][cc], cS2 = sm.hS2[o][cc];
        if (a.I >= 3)
            form_costs(a, b, kb0, b >= 1 ? 2 : 1, sm.hv, sm.hN, sm.hS, sm.hS2, jj, cv, cN, cS,
                       cS2, sm.tab, b >= 1 ? T : T + kQTab);
    }
    __syncthreads();  // the tables
    double qP[KW], cQ[KW];
    if (b >= 1) lane_costs(T, qP);
    lane_costs(T + kQTab, cQ);
    // layer 2 (eq. apx_base): the first interval (v_0, v_j]
    if (wave == 0) {
        double f = __builtin_huge_val();
        if (valid && j >= 1) {
            double C, P;
            cell_at(a.H, 0, j, sm.tab, C, P);
            f = __builtin_fma(-a.lamp, P, 0.0 + C);
            a.F[2 * a.ld + j] = f;
        }
        sm.pF[lane] = f;
    }
    __syncthreads();  // layer 2
    double (*xb)[kSB] = reinterpret_cast<double (*)[kSB]>(&sm.sF[0][0]);
    int32_t cg = 0;  // chunks published
    for (int32_t i0 = 3; i0 <= a.I; i0 += LG) {
#pragma unroll 1
        for (int ch = 0; ch < kTileWaves; ch++) {
            const int32_t ic = i0 + ch * LW;  // the chunk's first layer
            if (ic > a.I) break;
            // the helpers' partial minima (usually ready before block b-1's
            // chunk) and the holder's running minima of the chunk's layers,
            // read while the chain waits for block b-1
            if (nh > 0) wait_flags(a, -1, help_counter(a, b, 0), nh, cg + 1);
            double best[LW];
#pragma unroll
            for (int l = 0; l < LW; l++)
                best[l] = wave == ch && ic + l <= a.I ? a.F[(int64_t)(ic + l) * a.ld + jj]
                                                     : __builtin_huge_val();
            if (wave == ch) {
                for (int h = 0; h < nh; h++) {
                    const double* P = help_partials(a, m, h) + (int64_t)(ic - 3) * kSB + lane;
#pragma unroll
                    for (int l = 0; l < LW; l++) best[l] = __builtin_fmin(best[l], P[l * kSB]);
                }
            }
            if (b - 1 >= t) wait_flag(a, b - 1, cg + 1);
            if (b > kpd) {
                // block b-1 for the chunk's layers
                __syncthreads();  // the staging buffer is free
                stage_chunk<LG, LW, 1>(a, b - 1, 1, ic, sm.sF);
                __syncthreads();
                double pa[LW];
#pragma unroll
                for (int l = 0; l < LW; l++) pa[l] = __builtin_huge_val();
#pragma unroll
                for (int q = 0; q < KW; q++) {
                    const int kk = wave * KW + q;
#pragma unroll
                    for (int l = 0; l < LW; l++)
                        pa[l] = __builtin_fmin(pa[l], sm.sF[kk][l] + qP[q]);
                }
                __syncthreads();  // the staging buffer is free: 4 x LW rows of 64
#pragma unroll
                for (int l = 0; l < LW; l++) xb[wave * LW + l][lane] = pa[l];
                __syncthreads();
                if (wave == ch) {
#pragma unroll
                    for (int l = 0; l < LW; l++)
                        best[l] = __builtin_fmin(
                            best[l], __builtin_fmin(__builtin_fmin(xb[l][lane], xb[LW + l][lane]),
                                                    __builtin_fmin(xb[2 * LW + l][lane],
                                                                   xb[3 * LW + l][lane])));
                }
                __syncthreads();
            }
            // the chunk's layers inside the block, in order
#pragma unroll
            for (int q8 = 0; q8 < LW; q8++) {
                const int32_t i = ic + q8;
                if (i > a.I) break;
                // this wavefront's 16 candidates as 4 minima of 4 (short
                // dependency chains), then a tree
                double m4[4];
#pragma unroll
                for (int c4 = 0; c4 < 4; c4++) {
                    m4[c4] = __builtin_huge_val();
#pragma unroll
                    for (int q = 4 * c4; q < 4 * c4 + 4; q++)
                        m4[c4] = __builtin_fmin(m4[c4], sm.pF[wave * KW + q] + cQ[q]);
                }
                sm.partV[wave][lane] =
                    __builtin_fmin(__builtin_fmin(m4[0], m4[1]), __builtin_fmin(m4[2], m4[3]));
                __syncthreads();
                if (wave == ch) {
                    const double v =
                        __builtin_fmin(__builtin_fmin(sm.partV[0][lane], sm.partV[1][lane]),
                                       __builtin_fmin(sm.partV[2][lane], sm.partV[3][lane]));
                    const double bv = __builtin_fmin(best[q8], v);
                    if (valid) a.F[(int64_t)i * a.ld + j] = bv;
                    sm.pF[lane] = valid ? bv : __builtin_huge_val();
                }
                __syncthreads();
            }
            cg++;
            publish_flag(a, b, cg);
        }
        if constexpr (NL < LG) break;  // one group holds every layer (I = NL + 2)
    }
}

// One step of the sweep: workgroups 0..nb-1 make blocks t..t+nb-1 final (a
// chain: each waits for the one before, chunk by chunk), the next nb x
// kHelpMax are their helpers (helper h of block t + m at nb + m kHelpMax + h),
// and the others (tiles, WG index g * nx + wg after them) add blocks tp..t-1,
// the last step's, to the column blocks after this step's.
template <int LG, int NL>
__global__ __launch_bounds__(kSB* kTileWaves) ECASQ_STEP_ATTR void k_sweep_step(
    SweepArgs a, int64_t t, int32_t nb, int64_t tp, int32_t sp, int64_t nx) {
    __shared__ StepSmem<LG> sm;
    if (!sweep_live(a)) return;  // uniform
    const int64_t J1 = t + nb;   // the first column block after the step's
    const int32_t nh = nb * kHelpMax;
    if ((int32_t)blockIdx.x < nb + nh) {
        // the diagonal chain is the step's critical path: let its waves issue
        // ahead of tile waves that share its SIMDs
        __builtin_amdgcn_s_setprio(3);
        load_log2_table(sm.tab);
        if ((int32_t)blockIdx.x < nb) {
            diag_block<LG, NL>(a, t, tp, (int32_t)blockIdx.x, sm);
        } else {
            const int32_t x = (int32_t)blockIdx.x - nb;
            helper_block<LG, NL>(a, t, tp, x / kHelpMax, x % kHelpMax, sm);
        }
    } else {
        const int64_t x = (int64_t)blockIdx.x - nb - nh;
        const int64_t wg = x % nx;
        const int32_t g = (int32_t)(x / nx);
        const int64_t per = kTileWaves / sp;
#if ECASQ_SWEEP_XCD
        // fixed groups of `per` column blocks, group q on the q - q0'th tile
        // workgroup, q0 a multiple of 8: a group keeps its XCD from launch to
        // launch while the chain's workgroups before them are as many
        const int64_t Jw = (((J1 / per) & ~(int64_t)7) + wg) * per;
#else
        const int64_t Jw = J1 + wg * per;
#endif
        if (sp == 4)
            tile_role<LG, NL, 4>(a, t, tp, Jw, J1, g, sm);
        else if (sp == 2)
            tile_role<LG, NL, 2>(a, t, tp, Jw, J1, g, sm);
        else
            tile_role<LG, NL, 1>(a, t, tp, Jw, J1, g, sm);
    }
}

// Traceback state (device): st[0] = i*, the chain u_0..u_{i*-1} at st + 8.
constexpr int kStChain = 8;

// eq. apx_final on the finished table: i* (the lowest argmin over layers, or
// I for exactly s values), u_{i*-1} = p - 1, u_0 = 0, out[0] = J.
// A solve whose steps gave up a wait (failure word set) reports i* = 0: the
// traceback kernels then return at once and the result has t = 0, which the
// callers take as a failed solve.
__global__ __launch_bounds__(64) void k_sweep_pick(SweepArgs a, int32_t exact_s, double* out,
                                                    int32_t* st) {
    if (blockIdx.x != 0 || !sweep_live(a)) return;  // uniform
    const int lane = threadIdx.x;
    const int64_t p = a.H.p;
    if (a.K[a.nblk] != 0) {
        if (lane == 0) {
            st[0] = 0;
            out[0] = __builtin_huge_val();
        }
        return;
    }
    // the lowest i among the least F_i[p-1]: each lane the lowest of its
    // layers 2 + lane, 66 + lane, ..., then (value, i) minima across lanes
    double bj = __builtin_huge_val();
    int32_t bi = 0x7fffffff;
    if (exact_s) {
        bi = a.I;
        bj = a.F[(int64_t)a.I * a.ld + p - 1];
    } else {
        for (int32_t i = 2 + lane; i <= a.I; i += 64) {
            const double f = a.F[(int64_t)i * a.ld + p - 1];
            if (bi == 0x7fffffff || f < bj) {
                bj = f;
                bi = i;
            }
        }
        for (int off = 32; off >= 1; off >>= 1) {
            const double ov = __shfl_xor(bj, off);
            const int32_t oi = __shfl_xor(bi, off);
            if (ov < bj || (ov == bj && oi < bi)) {
                bj = ov;
                bi = oi;
            }
        }
    }
    if (lane == 0) {
        st[0] = bi;
        st[kStChain + bi - 1] = (int32_t)(p - 1);
        st[kStChain] = 0;
        out[0] = bj;
    }
}

// The lowest argmin k of F_{i-1}[k] + C[k,j] + lambda' Phi[k,j] over k in
// [i-2, j-1] for one column j, as (value, k) pairs reduced lexicographically
// (the DP's strict '<' in increasing k keeps the same k).  Part 1: workgroup
// g takes 256 x kTrR consecutive predecessors.
constexpr int kTrT = 256;
constexpr int kTrR = 8;

__device__ __forceinline__ void lexmin(double& v, int32_t& k, double ov, int32_t ok) {
    const bool take = ov < v || (ov == v && ok < k);
    v = take ? ov : v;
    k = take ? ok : k;
}

__global__ __launch_bounds__(kTrT) void k_sweep_trace_part(SweepArgs a, int32_t i,
                                                           const int32_t* __restrict__ st,
                                                           double* __restrict__ pv,
                                                           int32_t* __restrict__ pk) {
    __shared__ double2 tab[kLog2Size];
    __shared__ double rv[kTrT];
    __shared__ int32_t rk[kTrT];
    if (!sweep_live(a) || i > st[0]) return;  // uniform: skipped, or above the chosen layer
    load_log2_table(tab);
    __syncthreads();
    const int64_t j = st[kStChain + i - 1];
    const int64_t klo = i - 2, khi = j - 1;
    const int64_t k0 = klo + (int64_t)blockIdx.x * (kTrT * kTrR);
    double best = __builtin_huge_val();
    int32_t bk = INT32_MAX;
    const double* Fp = a.F + (int64_t)(i - 1) * a.ld;
#pragma unroll
    for (int r = 0; r < kTrR; r++) {
        const int64_t k = k0 + r * kTrT + threadIdx.x;
        if (k <= khi) {
            double C, P;
            cell_at(a.H, k, j, tab, C, P);
            const double cand = Fp[k] + __builtin_fma(-a.lamp, P, C);
            lexmin(best, bk, cand, (int32_t)k);
        }
    }
    rv[threadIdx.x] = best;
    rk[threadIdx.x] = bk;
    __syncthreads();
    for (int off = kTrT / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            double v = rv[threadIdx.x];
            int32_t k = rk[threadIdx.x];
            lexmin(v, k, rv[threadIdx.x + off], rk[threadIdx.x + off]);
            rv[threadIdx.x] = v;
            rk[threadIdx.x] = k;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        pv[blockIdx.x] = rv[0];
        pk[blockIdx.x] = rk[0];
    }
}

// Part 2: the g partials -> u_{i-2}.
__global__ __launch_bounds__(kTrT) void k_sweep_trace_pick(int32_t i, int32_t* __restrict__ st,
                                                           const double* __restrict__ pv,
                                                           const int32_t* __restrict__ pk,
                                                           int32_t g, const int32_t* runp) {
    __shared__ double rv[kTrT];
    __shared__ int32_t rk[kTrT];
    if ((runp && *runp == 0) || i > st[0]) return;
    double best = __builtin_huge_val();
    int32_t bk = INT32_MAX;
    for (int32_t x = threadIdx.x; x < g; x += kTrT) lexmin(best, bk, pv[x], pk[x]);
    rv[threadIdx.x] = best;
    rk[threadIdx.x] = bk;
    __syncthreads();
    for (int off = kTrT / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            double v = rv[threadIdx.x];
            int32_t k = rk[threadIdx.x];
            lexmin(v, k, rv[threadIdx.x + off], rk[threadIdx.x + off]);
            rv[threadIdx.x] = v;
            rk[threadIdx.x] = k;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) st[kStChain + i - 2] = rk[0];
}

// The whole traceback in one workgroup, for small p: layer by layer from i*
// down to 3, the lowest argmin of the chain column's candidates (the same
// (value, k) pairs as the two kernels above, reduced lexicographically: a
// butterfly per wavefront, then across the wavefronts in LDS), the next
// column kept in LDS.  One launch instead of two per layer.
constexpr int kTrOneT = 1024;
constexpr int64_t kTrOneMaxP = 16384;  // at most 16 candidates per thread

__global__ __launch_bounds__(kTrOneT) void k_sweep_trace_one(SweepArgs a, int32_t* __restrict__ st) {
    __shared__ double2 tab[kLog2Size];
    __shared__ double rv[kTrOneT / kSB];
    __shared__ int32_t rk[kTrOneT / kSB];
    __shared__ int32_t jn;
    if (!sweep_live(a)) return;  // uniform
    const int32_t n = st[0];
    if (n < 3) return;  // uniform: no interior value, or a failed solve (0)
    load_log2_table(tab);
    if (threadIdx.x == 0) jn = st[kStChain + n - 1];
    __syncthreads();
    const int lane = threadIdx.x % kSB, wave = threadIdx.x / kSB;
    for (int32_t i = n; i >= 3; i--) {
        const int64_t j = jn;
        const double* Fp = a.F + (int64_t)(i - 1) * a.ld;
        double best = __builtin_huge_val();
        int32_t bk = INT32_MAX;
        for (int64_t k = (i - 2) + (int64_t)threadIdx.x; k < j; k += kTrOneT) {
            double C, P;
            cell_at(a.H, k, j, tab, C, P);
            lexmin(best, bk, Fp[k] + __builtin_fma(-a.lamp, P, C), (int32_t)k);
        }
#pragma unroll
        for (int off = kSB / 2; off > 0; off >>= 1)
            lexmin(best, bk, __shfl_xor(best, off), __shfl_xor(bk, off));
        if (lane == 0) {
            rv[wave] = best;
            rk[wave] = bk;
        }
        __syncthreads();
        if (wave == 0) {
            best = lane < kTrOneT / kSB ? rv[lane] : __builtin_huge_val();
            bk = lane < kTrOneT / kSB ? rk[lane] : INT32_MAX;
#pragma unroll
            for (int off = kSB / 2; off > 0; off >>= 1)
                lexmin(best, bk, __shfl_xor(best, off), __shfl_xor(bk, off));
            if (lane == 0) {
                st[kStChain + i - 2] = bk;
                jn = bk;
            }
        }
        __syncthreads();
    }
}

// The chain's MSE and H(I,B) summed in path order.  One wavefront.
// out: J (already written), MSE, H(I,B), i*.
__global__ __launch_bounds__(kSB) void k_sweep_sums(SweepArgs a, const int32_t* __restrict__ st,
                                                    double* out, int32_t* chain_out) {
    __shared__ double2 tab[kLog2Size];
    __shared__ double cC[256], cP[256];
    if (!sweep_live(a)) return;
    load_log2_table(tab);
    __syncthreads();
    const int lane = threadIdx.x;
    const int32_t n = st[0];
    const int32_t* u = st + kStChain;
    for (int r = lane; r + 1 < n; r += kSB) cell_at(a.H, u[r], u[r + 1], tab, cC[r], cP[r]);
    __syncthreads();
    if (lane == 0) {
        double mse = 0.0, ph = 0.0;
        for (int r = 0; r + 1 < n; r++) {
            mse = mse + cC[r];
            ph = ph - cP[r];
        }
        out[1] = mse;
        out[2] = ph;
        out[3] = (double)n;
    }
    if (chain_out)
        for (int r = lane; r < n; r += kSB) chain_out[r] = u[r];
}

// Argmins of layer i at every valid column (inspection only): one column per
// lane, predecessors in increasing k at wave-uniform addresses.
__global__ __launch_bounds__(256) void k_sweep_argmins(SweepArgs a, int32_t i) {
    __shared__ double2 tab[kLog2Size];
    if (!sweep_live(a)) return;
    load_log2_table(tab);
    __syncthreads();
    const int64_t p = a.H.p;
    const int64_t jfirst = (int64_t)(i - 1) + (int64_t)blockIdx.x * blockDim.x;
    const int64_t j = jfirst + threadIdx.x;
    const int64_t jl = min(jfirst + (int64_t)blockDim.x - 1, p - 1);  // block's last column
    const int64_t jj = j < p ? j : p - 1;
    const double* Fp = a.F + (int64_t)(i - 1) * a.ld;
    double best = __builtin_huge_val();
    int32_t bk = -1;
    for (int64_t k = i - 2; k < jl; k++) {
        double C, P;
        cell_at(a.H, k, jj, tab, C, P);
        const double cand = Fp[k] + __builtin_fma(-a.lamp, P, C);
        const bool lt = k < jj && cand < best;
        bk = lt ? (int32_t)k : bk;
        best = lt ? cand : best;
    }
    if (j < p) a.K[(int64_t)i * a.ld + j] = bk;
}

// Layer 2's argmin is 0 (eq. apx_base) at every valid column.
__global__ __launch_bounds__(256) void k_sweep_argmins2(SweepArgs a) {
    const int64_t j = 1 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j < a.H.p) a.K[2 * a.ld + j] = 0;
}

// Accumulators of layer i for every valid column (inspection only):
// M_i[j] = M_{i-1}[k*] + C[k*, j], Ph_i[j] = Ph_{i-1}[k*] - P[k*, j] with the
// layer-2 start 0 + C[0, j], 0 - P[0, j], as the layer-by-layer DP forms them.
__global__ __launch_bounds__(256) void k_sweep_acc(SweepArgs a, int32_t i, double* M, double* Ph) {
    __shared__ double2 tab[kLog2Size];
    if (!sweep_live(a)) return;
    load_log2_table(tab);
    __syncthreads();
    const int64_t j = (int64_t)(i - 1) + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= a.H.p) return;
    const int32_t bk = a.K[(int64_t)i * a.ld + j];
    if (bk < 0) return;
    double C, P;
    cell_at(a.H, bk, j, tab, C, P);
    const double m0 = i == 2 ? 0.0 : M[(int64_t)(i - 1) * a.ld + bk];
    const double p0 = i == 2 ? 0.0 : Ph[(int64_t)(i - 1) * a.ld + bk];
    M[(int64_t)i * a.ld + j] = m0 + C;
    Ph[(int64_t)i * a.ld + j] = p0 - P;
}

SweepArgs make_args(const SweepSolve& S) {
    SweepArgs a;
    a.H = S.H;
    a.F = S.F;
    a.Q = S.Q;
    a.K = S.K;
    a.ld = S.ld;
    a.I = S.I;
    a.lamp = S.lamp;
    a.nblk = (S.H.p + kSB - 1) / kSB;
    a.lampp = S.lampp;
    a.runp = S.runp;
    return a;
}

// Blocks a step starting at block t makes final.
int32_t step_blocks(int64_t t, int64_t nblk) {
    return (int32_t)(nblk - t < ECASQ_SWEEP_NB ? nblk - t : ECASQ_SWEEP_NB);
}

template <int LG, int NL = LG>
hipError_t sweep_launch(const SweepArgs& a, hipStream_t st) {
    const int32_t ngroups = (a.I - 2 + LG - 1) / LG;
    {
        const int64_t rows = a.I - 1;  // >= 1
        int64_t g = (a.H.p + 255) / 256;
        const int64_t cap = 4096 / rows > 0 ? 4096 / rows : 1;
        if (g > cap) g = cap;
        k_sweep_fill<<<dim3((unsigned)g, (unsigned)rows), 256, 0, st>>>(a);
    }
    // a step makes blocks t..t+nb-1 final; blocks tp..t-1 (the last step's)
    // are final and not yet added to the column blocks after t - 1
    int64_t tp = 0;
    for (int64_t t = 0; t < a.nblk;) {
        const int32_t nb = step_blocks(t, a.nblk);
        const int64_t ntiles = ngroups > 0 ? a.nblk - t - nb : 0;
        const int64_t tiles = ntiles * ngroups;
        const int32_t sp = tiles < ECASQ_SWEEP_SP4_BELOW ? 4 : tiles < ECASQ_SWEEP_SP2_BELOW ? 2 : 1;
        const int64_t per = kTileWaves / sp;  // column blocks per workgroup
#if ECASQ_SWEEP_XCD
        // workgroups of fixed column-block groups (see k_sweep_step), a
        // multiple of 8 per layer group so that every group keeps its XCD
        const int64_t q0 = ((t + nb) / per) & ~(int64_t)7;
        const int64_t nx = ntiles > 0 && tp < t ? ((a.nblk - 1) / per - q0 + 1 + 7) / 8 * 8 : 0;
#else
        const int64_t nx = tp < t ? (ntiles + per - 1) / per : 0;
#endif
        const int64_t nh = (int64_t)nb * kHelpMax;
        const dim3 grid((unsigned)(nb + nh + nx * ngroups)), block(kSB * kTileWaves);
        k_sweep_step<LG, NL><<<grid, block, 0, st>>>(a, t, nb, tp, sp, nx > 0 ? nx : 1);
        tp = t;
        t += nb;
    }
    return hipGetLastError();
}

int32_t trace_groups(int64_t p) { return (int32_t)((p + kTrT * kTrR - 1) / (kTrT * kTrR)); }

size_t trace_scratch_bytes(int64_t p) {
    return (size_t)trace_groups(p) * (sizeof(double) + sizeof(int32_t));
}

// The counters of the steps: a chunk counter per block, the failure word,
// kHelpMax helper counters per block.
size_t counter_bytes(int64_t p) {
    const int64_t nblk = (p + kSB - 1) / kSB;
    return sizeof(int32_t) * (size_t)(nblk * (1 + kHelpMax) + 1);
}

bool sweep_ok(const SweepSolve& S) {
    return S.I >= 2 && S.I <= 255 && S.H.p >= 2 && S.ld >= S.H.p && S.F && S.Q && S.K && S.st &&
           S.kbytes >= counter_bytes(S.H.p) && S.kbytes >= trace_scratch_bytes(S.H.p);
}

// K holds the argmin table of layers 0..I.
bool sweep_argmins_ok(const SweepSolve& S) {
    return sweep_ok(S) && S.kbytes >= sizeof(int32_t) * (size_t)(S.I + 1) * (size_t)S.ld;
}

}  // namespace

size_t sweep_table_bytes(int64_t d, int32_t s) {
    // F (fp64) and K (int32: inspection and traceback scratch), rows 0..s
    return (size_t)(s + 1) * (size_t)d * (sizeof(double) + sizeof(int32_t));
}

size_t sweep_scratch_bytes(int64_t d) {
    const size_t a = counter_bytes(d), b = trace_scratch_bytes(d);
    return a > b ? a : b;
}

size_t sweep_cost_bytes() { return (size_t)kQAll * sizeof(double); }

hipError_t launch_sweep(const SweepSolve& S, int32_t exact_s, double* out, int32_t* chain,
                        hipStream_t st) {
    if (!sweep_ok(S) || !out) return hipErrorInvalidValue;
    const SweepArgs a = make_args(S);
    const int32_t L = a.I - 2;  // recursive layers 3..I
    hipError_t e;
    if (L <= 8)
        e = sweep_launch<8>(a, st);
    else if (L <= 16 || ECASQ_SWEEP_LG_MAX == 16)
        e = sweep_launch<16>(a, st);
    else if (L == 30)  // s = 32: one group without its two layers past I
        e = sweep_launch<32, 30>(a, st);
    else
        e = sweep_launch<32>(a, st);
    if (e != hipSuccess) return e;
    k_sweep_pick<<<1, 64, 0, st>>>(a, exact_s, out, S.st);
    // traceback: layers above i* return at once; small p in one launch
    if (a.H.p <= kTrOneMaxP) {
        k_sweep_trace_one<<<1, kTrOneT, 0, st>>>(a, S.st);
    } else {
        const int32_t g = trace_groups(a.H.p);
        double* pv = reinterpret_cast<double*>(S.K);
        int32_t* pk = reinterpret_cast<int32_t*>(pv + g);
        for (int32_t i = a.I; i >= 3; i--) {
            k_sweep_trace_part<<<(unsigned)g, kTrT, 0, st>>>(a, i, S.st, pv, pk);
            k_sweep_trace_pick<<<1, kTrT, 0, st>>>(i, S.st, pv, pk, g, S.runp);
        }
    }
    k_sweep_sums<<<1, kSB, 0, st>>>(a, S.st, out, chain);
    return hipGetLastError();
}

hipError_t launch_sweep_argmins(const SweepSolve& S, hipStream_t st) {
    if (!sweep_argmins_ok(S)) return hipErrorInvalidValue;
    const SweepArgs a = make_args(S);
    k_sweep_argmins2<<<(unsigned)((a.H.p - 1 + 255) / 256), 256, 0, st>>>(a);
    for (int32_t i = 3; i <= a.I; i++) {
        const int64_t n = a.H.p - (i - 1);
        if (n <= 0) break;
        k_sweep_argmins<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(a, i);
    }
    return hipGetLastError();
}

hipError_t launch_sweep_accumulators(const SweepSolve& S, double* M, double* Ph, hipStream_t st) {
    if (!sweep_argmins_ok(S) || !M || !Ph) return hipErrorInvalidValue;
    const SweepArgs a = make_args(S);
    for (int32_t i = 2; i <= a.I; i++) {
        const int64_t n = a.H.p - (i - 1);
        if (n <= 0) break;
        k_sweep_acc<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(a, i, M, Ph);
    }
    return hipGetLastError();
}

}  // namespace ecasq
