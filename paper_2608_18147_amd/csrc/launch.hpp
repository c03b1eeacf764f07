// Host-side launchers shared by the library's translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "device.hpp"

namespace ecasq {

inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// columns per lane in the DP layer kernel (single multiplier / one pass of
// kMaxLambdas multipliers)
#ifndef ECASQ_COLS_PER_LANE
#define ECASQ_COLS_PER_LANE 2
#endif
#ifndef ECASQ_COLS_PER_LANE_MULTI
#define ECASQ_COLS_PER_LANE_MULTI 1
#endif
constexpr int kColsPerLane = ECASQ_COLS_PER_LANE;
constexpr int kColsPerLaneMulti = ECASQ_COLS_PER_LANE_MULTI;

// multipliers solved together by one sweep of the DP (one search pass)
constexpr int kMaxLambdas = 8;

// ---- prep.hip ----
size_t prep_scratch_bytes(int64_t d);
hipError_t launch_prep(const void* x, int dt, int64_t d, void* scratch, hipStream_t st, double* v,
                       double* N, double* S, double* S2, int64_t* p_dev, uint32_t* flags_dev);

// ---- alphabet.hip ----
// kind 1: uniform grid of m points over [v[0], v[px-1]]; kind 2: the input
// values at ranks floor(k (d-1) / (m-1)); repeats dropped.  Writes the grid and
// the prefix sums at its points; *count = grid size.  2 <= m <= d, px >= 2.
hipError_t launch_alphabet(int32_t kind, int64_t m, int64_t d, const double* v, const double* N,
                           const double* S, const double* S2, int64_t px, double* gv, double* gN,
                           double* gS, double* gS2, int64_t* count, hipStream_t st);

// ---- opt.hip ----
// Optimal lambda-ECASQ (Sec. 4): p x p layers, so p is bounded.
constexpr int64_t kOptMaxP = (int64_t)1 << 16;
// device bytes of the optimal DP's tables for p values and layers 2..imax
// (trace: argmins kept as int32 for launch_opt's Ktrace)
size_t opt_workspace_bytes(int64_t p, int32_t imax, bool trace);
// (k, l, j) candidates, layer-2 entries and final entries of the full DP
int64_t opt_cells(int64_t p, int32_t imax, int32_t exact_s);
// mem: opt_workspace_bytes(p, imax, Ktrace != null) bytes; chain (>= imax
// int32) and res (J' = MSE + lambda' H(Xhat) of the optimum, t) are device
// memory.  full: scan every predecessor (else monotone brackets).  Ftrace /
// Ktrace (optional, (imax+1) p^2 each) receive every layer's values, [i][j][l],
// and argmins of layers >= 3, [i][l][j].
hipError_t launch_opt(const Hist& H, int32_t imax, int32_t exact_s, double lamp, int32_t full,
                      char* mem, int32_t* chain, double* res, double* Ftrace, int32_t* Ktrace,
                      hipStream_t st);

// ---- rans.hip ----
int64_t rans_segments(int64_t d);
size_t rans_bound(int64_t d, int32_t t);      // largest coded stream, bytes
size_t rans_scratch_bytes(int64_t d);
// out: at least rans_bound(d, t) bytes; *total_out (device) = payload bytes;
// *bad (device, zeroed by the caller) counts symbols >= t
hipError_t launch_rans_encode(const uint8_t* sym, int64_t d, int32_t t, uint8_t* out,
                              char* scratch, unsigned long long* total_out, unsigned int* bad,
                              hipStream_t st);
// *bad (device, zeroed by the caller) counts malformed segments
hipError_t launch_rans_decode(const uint8_t* in, int64_t nin, int64_t d, int32_t t, uint8_t* sym,
                              unsigned int* bad, hipStream_t st);

// ---- dp.hip ----
// One DP layer for nlam multipliers (1 or kMaxLambdas); every per-multiplier
// array below holds nlam valid entries.
struct DpLayer {
    Hist H;
    int32_t nlam;
    const double* Fin[kMaxLambdas];
    double* Fout[kMaxLambdas];
    double* pval;     // nlam slices of pstride entries
    int32_t* pidx;
    int64_t pstride;  // >= dp_partial_entries(p)
    int64_t kb;    // forward: first predecessor; backward: last predecessor
    int64_t jlo;   // first column
    int64_t jhi;   // last column (inclusive)
    bool backward;
    double lam[kMaxLambdas];  // lambda' in MSE units
    // forward main-DP accumulators (all null in the recovery half-DPs)
    const double* Min[kMaxLambdas];
    const double* Pin[kMaxLambdas];
    double* Mout[kMaxLambdas];
    double* Pout[kMaxLambdas];
    int32_t* kstar[kMaxLambdas];  // argmin rows per multiplier (null: not recorded)
    double* last;            // nlam blocks of 3 * last_stride doubles
    int32_t layer;
    int32_t last_stride;
    int64_t cells;  // (column, predecessor) cells this launch evaluates, per multiplier
};

// Layer 2 of the forward DP for nlam multipliers.
struct DpInit {
    int32_t nlam;
    double lam[kMaxLambdas];
    double* F[kMaxLambdas];
    double* M[kMaxLambdas];   // null: no accumulators
    double* Ph[kMaxLambdas];
    int32_t* kstar[kMaxLambdas];
    double* last;
    int32_t last_stride;
};
int64_t dp_partial_entries(int64_t p);
void timing_enable(int mode);  // 0 off, 1 timing, 2 timing + a stderr line per DP solve
bool timing_verbose();
void timing_flush();
void timing_read(int variant, double* ms, int64_t* launches, int64_t* cells, bool reset);
// bracket a span of launches on st as one timed unit of `variant` (2: a sweep
// solve, 3: a layer of the optimal DP, 4: a batched launch)
void timing_begin(int variant, int64_t cells, hipStream_t st);
void timing_end(hipStream_t st);
// drop the newest timed unit not yet flushed (a solve that was skipped)
void timing_discard_last();
bool timing_active();
constexpr int kTimingOpt = 3;
constexpr int kTimingBatched = 4;
constexpr int kTimingVariants = 5;
hipError_t launch_dp_layer(const DpLayer& L, hipStream_t st);
hipError_t launch_dp_init_fwd(const Hist& H, int64_t lo, int64_t jl, int64_t jh,
                              const DpInit& I, hipStream_t st);
hipError_t launch_dp_init_bwd(const Hist& H, int64_t hi, int64_t jl, int64_t jh, double lam,
                              double* B, hipStream_t st);
// out: 4 doubles (J, MSE, H(I,B), i*) per multiplier
hipError_t launch_dp_final(const double* last, int32_t stride, int32_t imax, int32_t exact_s,
                           int32_t nlam, double* out, hipStream_t st);
hipError_t launch_split(const double* Fw, const double* Bw, int64_t ml, int64_t mh,
                        int64_t* m_out, hipStream_t st);

// ---- sweep.hip ----
// One dp_APX solve as a sweep over column blocks: F and the argmins of every
// layer in tables of I+1 rows of ld entries (rows 2..I used).
struct SweepSolve {
    Hist H;
    double* F;
    double* Q;     // sweep_cost_bytes(): the next diagonal block's costs
    int32_t* K;    // step counters and traceback scratch; the argmins on request
                   // (launch_sweep_argmins), when it holds (I + 1) x ld int32
    size_t kbytes = 0;  // bytes at K
    int32_t* st;   // traceback state, 264 int32
    int64_t ld;    // >= p
    int32_t I;     // last layer, min(s, p), 2..255
    double lamp;   // lambda' in MSE units (when lampp is null)
    const double* lampp = nullptr;  // device: lambda', read by the kernels
    const int32_t* runp = nullptr;  // device: 0 = skip the whole solve (null: run)
};
size_t sweep_table_bytes(int64_t d, int32_t s);
// Bytes of K that a solve needs for p <= d: the steps' counters and the
// traceback's partials (the argmin table is (s + 1) d int32 on top).
size_t sweep_scratch_bytes(int64_t d);
size_t sweep_cost_bytes();
// The sweep, then eq. apx_final and the traceback (argmins recomputed along
// the chain): out (device, 4 doubles) = J, MSE, H(I,B), i*; chain (device,
// optional, >= i* int32): u_0 = 0 .. u_{i*-1} = p-1.
hipError_t launch_sweep(const SweepSolve& S, int32_t exact_s, double* out, int32_t* chain,
                        hipStream_t st);
// The argmin of every layer and valid column into K (after launch_sweep).
hipError_t launch_sweep_argmins(const SweepSolve& S, hipStream_t st);
// MSE / H(I,B) accumulators of every layer into M, Ph (same layout as F);
// needs the argmins in K.
hipError_t launch_sweep_accumulators(const SweepSolve& S, double* M, double* Ph, hipStream_t st);

// ---- search.hip ----
// The budget search on lambda (Sec. 3 and Sec. 5), kept in device memory and
// advanced by one-thread kernels: after each batch of DP solves the commit
// kernel appends their points and runs the search until it needs more solves
// (todo[0..ntodo), lambda' in todo_lamp, run = 1) or is done (run = 0).
constexpr int kSearchMaxPts = 1024;
struct SearchPt {
    double lam, H, M;
    int32_t t, pad;
};
struct SearchPeek {
    int32_t done, nsol;
    SearchPt last;
};
struct SearchState {
    SearchPeek peek;  // done, nsol and the newest point, for the host's polls
    double b, s2tot, twoH, twoM;
    int32_t max_passes, width, aim, kind, has_chain, s;
    int32_t npts, ncached, nsol, npass, status, done, run;
    int32_t stage, pass_kind, issued, nq, ntodo, nin, force_chord, model, closed, have_A, iA,
        iB, nsol0;
    double lc, lam_final;
    double q[kMaxLambdas], todo[kMaxLambdas], todo_lamp[kMaxLambdas];
    SearchPt A, B;
    SearchPt pts[kSearchMaxPts];
};
struct SearchParams {
    double b, s2tot;
    int32_t max_passes, width, aim, kind, has_chain, s;
    int32_t keep_points;  // 1: keep the points of earlier searches on this input
};
// Start a search: two (device, metrics of the codebook {v_0, v_{p-1}}: MSE at
// [0], H(Xhat) at [2], H(I,B) at [3]).
hipError_t launch_search_begin(SearchState* S, const SearchParams& P, const double* two,
                               hipStream_t st);
// Append the m points solved for the next m entries of todo (a pass's solves
// may come in several commits; the search advances once all are in): res
// (device) holds 4 doubles per point (J, MSE, H, t); chains (device, stride
// S->s, may be null) their codebooks, copied into pchains (kSearchMaxPts x s)
// when S->has_chain.  With gate != 0 the kernel does nothing unless S->run is
// set (a solve that was skipped because the search had ended).
hipError_t launch_search_commit(SearchState* S, const double* res, const int32_t* chains,
                                int32_t m, int32_t* pchains, int32_t gate, hipStream_t st);

// ---- post.hip ----
hipError_t launch_refine(const Hist& H, int32_t t, int32_t* u, double lamp, double b,
                         int32_t budget, int32_t rounds, int32_t exhaustive, int32_t* stats,
                         hipStream_t st);
hipError_t launch_metrics(const Hist& H, int32_t t, const int32_t* u, double lam, double s2tot,
                          double* out, hipStream_t st);
hipError_t launch_gather(const double* v, const int32_t* u, int32_t t, double* codebook,
                         int32_t* rank, hipStream_t st);
hipError_t launch_quantize(const void* x, int dt, int64_t d, const double* codebook, int32_t t,
                           uint64_t seed, uint8_t* symbols, unsigned long long* hist,
                           hipStream_t st);
// the allocation-free rounding's counts: a file-scope device array of 256
// entries, its address on the current device (looked up once per device)
hipError_t quantize_scratch(unsigned long long** out);
// h[0..n) := 0 by a kernel (no memset node, so the call can be captured)
hipError_t launch_zero_counts(unsigned long long* h, int32_t n, hipStream_t st);
hipError_t launch_entropy(const unsigned long long* hist, int32_t t, int64_t d, double* ent,
                          int64_t* hist_out, hipStream_t st);
// time-shared rounding with two codebooks (t0, t1 <= 256) and the entropy of
// its two parts; hist (device, t0 + t1 counters) must start at zero
hipError_t launch_quantize_ts(const void* x, int dt, int64_t d, const double* cb0, int32_t t0,
                              const double* cb1, int32_t t1, double alpha, uint64_t seed,
                              uint8_t* symbols, uint8_t* part, unsigned long long* hist,
                              double* ent, int64_t* hist_out, hipStream_t st);

// ---- batched.hip ----
hipError_t launch_batched(const void* x, int dt, int64_t n, int32_t d, int32_t s, double b,
                          int32_t refine_rounds, int32_t refine_exhaustive, int32_t exact_s,
                          int32_t max_passes, double* codebooks, int32_t* t_out, void* infos,
                          hipStream_t st);

}  // namespace ecasq
