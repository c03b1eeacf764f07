/*
 * ecasq.h - C ABI of libecasq, an MI355X (gfx950) implementation of the
 * approximate dynamic program of Entropy-Constrained Adaptive Stochastic
 * Quantization (ECASQ, arXiv 2608.18147) and the steps around it.
 *
 * Problem (Sec. 1 and Sec. 3): given X in R^d, a maximum codebook size s and
 * an entropy budget b (bits per entry), choose an ordered codebook Q drawn
 * from the input values (P = X) that spans X, has |Q| <= s, and minimises the
 * MSE of unbiased stochastic quantization (SQ, Sec. 2) subject to
 * H(Xhat) <= b.  The library solves the Lagrangian surrogate of Sec. 5
 * (vNMSE + lambda * H(I,B), dp_APX, eq. apx_base / apx_rec / apx_final)
 * exactly, searches lambda for the budget (Sec. 3 and Sec. 5), recovers the
 * codebook, refines it with the three-colour pass of Sec. 6, and rounds the
 * input stochastically (Sec. 2) with Philox4x32-10.
 *
 * By default (ecasq_options.dp_schedule = 1) each DP solve is one sweep over
 * column blocks that keeps F of every layer, O(s d) memory (12 (s+1) d bytes),
 * and the codebook is the argmin traceback of the solve it was found in;
 * `recovery` is then ignored.  The layer-by-layer schedule (dp_schedule = 0)
 * keeps two O(d) layers, as Sec. 5 states the method, and recovers the
 * codebook with Hirschberg's method in O(d) space (recovery = 0) or from
 * stored argmins (recovery = 1).
 *
 * Conventions for every entry point:
 *   - Array arguments named x, codebook*, symbols, hist, t_out, infos_dev and
 *     workspace are DEVICE pointers (HIP memory on the current device); info
 *     is a HOST pointer.  The caller owns all memory; the library never frees
 *     caller memory.
 *   - stream is a hipStream_t passed as void* (NULL = the null stream).  All
 *     device work is ordered on it.  The solve entry points block the calling
 *     thread until their results are in device memory.  The budget search
 *     runs on the device: a one-thread controller kernel picks each next
 *     multiplier and the DP solves read it from device memory, so under the
 *     default settings the host reads back only the number of distinct values
 *     before the search, a done flag between solves and the result at the
 *     end.  Hirschberg recovery (dp_schedule 0), width-8 passes and the
 *     optimal / refinement-aware search points (dp_objective 1, 2) still read
 *     small results back between steps.
 *   - Argument errors are reported before any work is enqueued.  Data errors
 *     (NaN or Inf in x) are detected on the device and returned as
 *     ECASQ_ENONFINITE.
 *   - Ties are broken to the lowest index everywhere (lowest predecessor k,
 *     lowest number of values i, lowest Hirschberg split m); a refinement move
 *     is taken only on a strict improvement.
 *   - All arithmetic of the DP is fp64 and follows one fixed operation order,
 *     so results are reproducible bit for bit across runs.
 */
#ifndef ECASQ_H
#define ECASQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { ECASQ_F32 = 0, ECASQ_F16 = 1, ECASQ_BF16 = 2 } ecasq_dtype;

typedef enum {
    ECASQ_OK = 0,
    ECASQ_EINVAL = -1,      /* bad argument (sizes, null pointers, NaN budget) */
    ECASQ_ENONFINITE = -2,  /* x holds NaN or Inf */
    ECASQ_EINFEASIBLE = -3, /* b below the smallest reachable H(I,B); the
                               lowest-entropy codebook found is still returned */
    ECASQ_ENOMEM = -4,      /* device allocation failed */
    ECASQ_EHIP = -5,        /* a HIP runtime call failed */
    ECASQ_EWORKSPACE = -6   /* caller workspace smaller than ecasq_workspace_size */
} ecasq_status;

typedef struct {
    int32_t refine_rounds;     /* Sec. 6 rounds, upper bound (default 5; 0 = off) */
    int32_t refine_exhaustive; /* 0: binary search of Sec. 6 (default); 1: full scan */
    int32_t exact_s;           /* 0: at most s values (default); 1: exactly min(s, p) */
    int32_t max_search_passes; /* lambda-search passes (default 32) */
    int32_t recovery;          /* dp_schedule 0 only: 0 Hirschberg, O(d) space (default);
                                  1 stored argmins.  Ignored by the default sweep
                                  (dp_schedule 1), which traces its argmins back */
    int32_t search_width;      /* multipliers per search pass: 1 (default) or 8 */
    int32_t dp_schedule;       /* 1: column-block sweep over all layers at once, O(s d)
                                  space (default); 0: layer by layer, O(d) space (see
                                  ecasq_solve_ex) */
    int32_t alphabet;          /* permissible values P (App. D): 0 the distinct input
                                  values, P = X (default); 1 a uniform grid of
                                  alphabet_size points over [min X, max X]; 2 the input
                                  values at alphabet_size evenly spaced ranks */
    int32_t alphabet_size;     /* grid points m, 2 <= m <= d (alphabet 1 and 2) */
    int32_t optimal_scan;      /* optimal DP: 0 monotone brackets (Sec. 4.1, default),
                                  1 every predecessor */
    int32_t dp_objective;      /* budget modes: 0 the search runs on dp_APX and its
                                  H(I,B), then refines (default); 1 on the optimal DP
                                  of ecasq_solve_optimal and H(Xhat); 2 on dp_APX's
                                  codebooks refined at each query's multiplier and
                                  their H(Xhat), returning the feasible one of lowest
                                  vNMSE (1, 2: search_width is 1; no refinement after
                                  the search) */
} ecasq_options;

typedef struct {
    int32_t t;                /* codebook size actually used */
    int32_t p;                /* number of distinct input values */
    double lambda;            /* multiplier of the refinement and of `objective`, vNMSE
                                 units: the final chord slope of the search (budget
                                 mode) or the given lambda */
    double mse;               /* MSE(Q, X) = sum (b_x - x)(x - a_x), Sec. 2 */
    double vnmse;             /* MSE / ||X||^2 */
    double entropy;           /* H(Xhat) from expected frequencies, bits/entry */
    double entropy_surrogate; /* H(I,B) of Sec. 5 */
    double objective;         /* vNMSE + lambda * H(Xhat) */
    double rate_total;        /* H(Xhat) + 32 t / d (App. F.1 rate accounting) */
    int32_t dp_solves;        /* full DP solves (multipliers) run by the search */
    int32_t refine_rounds_run;
    int64_t cells;            /* DP cells evaluated (search + recovery) */
    int32_t status;           /* ecasq_status of the solve */
    int32_t search_passes;    /* passes of the budget search (0 in fixed-lambda mode) */
} ecasq_info;

/* Defaults listed in ecasq_options. */
void ecasq_default_options(ecasq_options *opts);

/*
 * Budget mode (Sec. 3 problem; Sec. 5 lambda tuning; Sec. 6 refinement).
 * x: d entries of type dt in device memory, any order.  s >= 2.  b >= 0.
 * Output codebook: t <= s ascending fp64 values (codebook[0] = min X,
 * codebook[t-1] = max X) in codebook (device, length >= s); codebook_rank
 * (device, length >= s, may be NULL) receives each value's index among the
 * sorted distinct inputs.  Entries past t are left untouched.  info may be NULL.
 * The returned codebook has H(Xhat) <= b whenever the status is ECASQ_OK.
 *
 * Search (Sec. 3 and Sec. 5, supporting-line queries of App. F.7), in passes
 * of w = opts->search_width multipliers that one sweep of the DP solves
 * together (w = 1 is the plain sequential chord search):
 *   pass 1: lambda in {0, 1e-4, 1e-3, 1e-2, 1e-1, 1, 10, 100} (w = 8) or {0};
 *   then A = the point with H(I,B) > b of largest lambda, B = the point with
 *   H(I,B) <= b of smallest lambda (if there is none: the two-value codebook
 *   {min X, max X} when b >= 1, else one solve at lambda = 2^40), and the next
 *   pass is the chord slope lc = (M_B - M_A) / (H_A - H_B) followed, when
 *   w = 8, by A + (B - A) g / 8 for g = 1..7 (lc times 1/4, 1/2, 3/4, 3/2, 2,
 *   3, 4 when B is the two-value codebook);
 *   with w = 1 the pass queries, instead of lc, the slope at H = b of the
 *   curve through A and B on which log(vNMSE) is linear in H,
 *   lq = -(r2 ln 2) M_A 2^(r2 (b - H_A)) with r2 = (log2 M_B - log2 M_A) /
 *   (H_B - H_A) (a table-driven log2 and exp2, so that the query is the same
 *   bit for bit wherever it is computed), while it lies strictly between the
 *   two multipliers and such queries keep finding new points;
 *   the search ends when the solve at lc returns A or B again, or after
 *   max_search_passes passes.
 * The codebook is B, recovered at the multiplier it was found at; the
 * refinement then runs at the final chord slope under the budget guard.
 */
ecasq_status ecasq_solve(const void *x, ecasq_dtype dt, int64_t d, int32_t s,
                         double bits_per_entry, void *stream, double *codebook,
                         int32_t *codebook_rank, ecasq_info *info);

/* ecasq_solve with options and an optional caller workspace (device memory of
 * at least ecasq_workspace_size(d, s, flags) bytes with flags = 1 if
 * opts->recovery == 1, plus 2 if opts->dp_schedule == 1; NULL = allocate
 * internally).
 *
 * Permissible alphabets (App. D with P != X): with opts->alphabet = 1 the
 * candidate values are p_0 = min X, p_k = min X + k ((max X - min X) / (m - 1))
 * (each operation rounded to nearest) for 0 < k < m-1, p_{m-1} = max X; with
 * opts->alphabet = 2 they are the input values at ranks floor(k (d-1) / (m-1))
 * of the sorted input; points equal to their predecessor (or, uniform, not
 * below max X) are dropped.  The interval quantities come from the input's
 * prefix count, sum and sum of squares at the grid points, so the DP costs
 * O(s p^2) in the grid size p <= m; codebook_rank indexes the grid.
 *
 * DP schedules (both compute eq. apx_base / apx_rec / apx_final with the same
 * values and argmins bit for bit):
 *   0  layer by layer with two rolling layers of O(p) memory, as Sec. 5 states
 *      it; the codebook is recovered by Hirschberg's method (recovery 0) or
 *      from stored argmins (recovery 1);
 *   1  one sweep over column blocks in which the interval cost and entropy
 *      term of each cell serve every layer; keeps F of all layers, 8 (s+1) d
 *      bytes, 48 MB of per-launch cost tables and partial minima (any d),
 *      and about d bytes of step counters and traceback scratch
 *      (an int32 argmin table of F's shape only when an inspection call asks
 *      for argmins or accumulators).  The
 *      codebook comes from the argmin traceback of the solve it was found
 *      in, each argmin recomputed from the kept layers (recovery is
 *      ignored). */
ecasq_status ecasq_solve_ex(const void *x, ecasq_dtype dt, int64_t d, int32_t s,
                            double bits_per_entry, const ecasq_options *opts, void *stream,
                            double *codebook, int32_t *codebook_rank, ecasq_info *info,
                            void *workspace, size_t workspace_bytes);

/*
 * Budget mode for nb budgets on one input, in the given order (as
 * ecasq_solve_ex for each).  The histogram is built once and the searches share
 * their DP solves: every solved multiplier's point (H(I,B), vNMSE and, under
 * schedule 1, its codebook) joins a cache that later searches start from, and a
 * multiplier already solved is not solved again.  Each search still returns
 * the lowest-vNMSE supported point with H(I,B) <= b.  budgets: host, nb >= 1
 * values.  codebooks: device, nb x s fp64 (row k holds infos[k].t values);
 * codebook_ranks: device, nb x s int32, may be NULL; infos: host, nb entries,
 * may be NULL (dp_solves, cells and search_passes count budget k's own new
 * solves).  Returns ECASQ_EINFEASIBLE if any budget is infeasible (every row is
 * still written); argument errors as ecasq_solve_ex.
 */
ecasq_status ecasq_solve_budgets(const void *x, ecasq_dtype dt, int64_t d, int32_t s, int32_t nb,
                                 const double *budgets, const ecasq_options *opts, void *stream,
                                 double *codebooks, int32_t *codebook_ranks, ecasq_info *infos);

/* Fixed-multiplier mode: minimise vNMSE + lambda H(I,B) (lambda in vNMSE units,
 * Sec. 3), then refine vNMSE + lambda H(Xhat) without a budget guard. */
ecasq_status ecasq_solve_lagrangian(const void *x, ecasq_dtype dt, int64_t d, int32_t s,
                                    double lambda, const ecasq_options *opts, void *stream,
                                    double *codebook, int32_t *codebook_rank,
                                    ecasq_info *info);

/*
 * Optimal lambda-ECASQ (Sec. 4): the codebook of at most s values (exactly
 * min(s, p) with opts->exact_s) drawn from the permissible values (the
 * distinct input values, or opts->alphabet's grid, App. D) that minimises
 * vNMSE + lambda H(Xhat) exactly, H(Xhat) the entropy of the expected output
 * frequencies; lambda >= 0 in vNMSE units (lambda' = RN(lambda ||X||^2)).
 *
 * The DP runs over states (i, l, j): dp(i,l,j) is the least cost of the values
 * up to v_l with i-1 codebook values ending at v_l plus the MSE of (v_l, v_j],
 *   dp(2,0,j) = C[0,j] + lambda' h((n_0 + D[0,j]) / d),
 *   dp(i,l,j) = C[l,j] + min_k dp(i-1,k,l) + lambda' h((U[k,l] + D[l,j]) / d),
 * answer min over (i, l) of dp(i,l,p-1) + lambda' h(U[l,p-1] / d); lowest
 * index on ties (i, then l, then k).  U/d, D/d and h are evaluated as the
 * approximate DP's cell does (g form, table log2).  One launch per layer, one
 * workgroup per row l; opts->optimal_scan = 0 restricts each column's scan over
 * k to the bracket between the minimisers of the ends of its 64-column segment
 * (the argmin does not increase with j, Lemma quadrangleM: the SMAWK
 * acceleration of Sec. 4.1), 1 scans every k (O(s p^3)).  Where rounding breaks
 * that order between two candidates equal to within rounding, the bracket can
 * return a codebook whose objective exceeds the minimum by a rounding error.
 *
 * Memory: every layer's argmins are kept (no Hirschberg pass): about
 * 24 p^2 + 2 (min(s,p) - 2) p^2 bytes (4 per argmin when p > 32768), allocated
 * on the stream for the call; p <= 65536 (ECASQ_ENOMEM above, or when the
 * allocation fails).  info: dp_solves = 1, cells = the full DP's (k, l, j)
 * candidates plus its layer-2 and final entries, refine_rounds_run = 0 (the
 * refinement options are ignored), objective = vNMSE + lambda H(Xhat) of the
 * codebook.  Errors as ecasq_solve_lagrangian.
 */
ecasq_status ecasq_solve_optimal(const void *x, ecasq_dtype dt, int64_t d, int32_t s,
                                 double lambda, const ecasq_options *opts, void *stream,
                                 double *codebook, int32_t *codebook_rank, ecasq_info *info);

/*
 * Two-way time-sharing (Sec. 7, App. E): the lambda search for b ends at two
 * adjacent supported points, B with H <= b (the codebook ecasq_solve returns
 * before refinement) and A with H > b (the point the final chord starts
 * from); quantizing a share alpha = (b - H_B) / (H_A - H_B) of the entries
 * with A and the rest with B has rate exactly b and the vNMSE of the
 * convexified frontier at b, alpha vNMSE_A + (1 - alpha) vNMSE_B.  H is the
 * search's entropy: H(I,B) with opts->dp_objective = 0, H(Xhat) with 1 (then
 * the time-share is optimal for every b).  Without such a pair (lambda = 0
 * feasible, an infeasible budget, p <= 2) alpha = 0 and both rows hold B.
 * No refinement (the points of the frontier are used as they are).
 *
 * codebooks: device, 2 x s fp64: row 0 = B ("minus", t = infos[0].t values),
 * row 1 = A ("plus"); codebook_ranks: device, 2 x s int32, may be NULL;
 * alpha: host, the share of entries quantized with row 1; infos: host, 2
 * entries (each quantizer's own metrics; lambda = the multiplier it was found
 * at; dp_solves, cells, search_passes of the search), may be NULL.  Returns
 * ECASQ_EINFEASIBLE for an infeasible budget; errors as ecasq_solve_ex.
 */
ecasq_status ecasq_solve_timeshare(const void *x, ecasq_dtype dt, int64_t d, int32_t s,
                                   double bits_per_entry, const ecasq_options *opts,
                                   void *stream, double *codebooks, int32_t *codebook_ranks,
                                   double *alpha, ecasq_info *infos);

/*
 * Time-shared final rounding (Sec. 7): entry i uses codebook1 iff its 53-bit
 * uniform from Philox4x32-10 with counter (j mod 2^32, j / 2^32, 1, 0), j =
 * i / 2, and key (seed mod 2^32, seed / 2^32) is below alpha (words 0 and 1
 * for even i, 2 and 3 for odd i, as in ecasq_quantize; shared randomness: a
 * decoder with the seed knows the partition), else codebook0, and is then
 * rounded exactly as ecasq_quantize rounds (counter word 2 = 0), its symbol
 * indexing its own codebook.  part: device, d bytes (1 = codebook1), may be NULL.
 * The two parts are entropy-coded separately: *empirical_entropy (device) =
 * (n_0 H_0 + n_1 H_1) / d with each part's plug-in entropy over its own
 * entries; hist: device, t0 + t1 int64 counts (codebook0's first), may be NULL.
 * 0 <= alpha <= 1; 1 <= t0, t1 <= 256.
 */
ecasq_status ecasq_quantize_timeshare(const void *x, ecasq_dtype dt, int64_t d,
                                      const double *codebook0, int32_t t0,
                                      const double *codebook1, int32_t t1, double alpha,
                                      uint64_t seed, void *stream, uint8_t *symbols,
                                      uint8_t *part, double *empirical_entropy, int64_t *hist);

/*
 * Entropy coding of symbols in [0, t) with rANS (Duda, arXiv:1311.2540), so
 * that the payload App. F.1 charges at H(Xhat) bits per entry, with a 16-bit
 * descriptor per codebook value, exists as bytes.  Frequencies
 * f_q = max(1, floor(n_q 2^16 / d)) of the symbol counts n_q, made to sum to
 * 2^16 (a surplus to the largest f, lowest q among ties; a deficit one unit at
 * a time from the largest f > 1); 32-bit state in [2^23, 2^31), bytes out;
 * segments of 4096 symbols coded independently (one lane each).  Stream:
 * t little-endian u16 (f_q - 1), then one little-endian u32 per segment (the
 * end of its bytes from the payload start), then the payload; a segment
 * starts with its final encoder state, big-endian.
 *
 * ecasq_encode_bound: the largest stream for d symbols over t values
 * (2 t + 8 ceil(d / 4096) + 2 d bytes; 0 for d outside [1, 2^28] or t outside
 * [1, 256]).  ecasq_encode: symbols and out are device memory, capacity >=
 * the bound; *out_bytes (host) = the stream's length.  ECASQ_EINVAL if a
 * symbol is >= t.  ecasq_decode: in (device, in_bytes) -> d symbols (device);
 * ECASQ_EINVAL for a malformed stream (a segment that overruns its bytes or
 * does not end in the initial state).  Both return after the stream work.
 */
size_t ecasq_encode_bound(int64_t d, int32_t t);
ecasq_status ecasq_encode(const uint8_t *symbols, int64_t d, int32_t t, void *stream,
                          uint8_t *out, size_t capacity, int64_t *out_bytes);
ecasq_status ecasq_decode(const uint8_t *in, int64_t in_bytes, int64_t d, int32_t t,
                          void *stream, uint8_t *symbols);

/*
 * Final stochastic rounding (Sec. 2): symbol i in [0, t) for every entry of x
 * in its original order.  The bracket is q_r < x <= q_{r+1} (x <= q_0 gives
 * r = 0; x > q_{t-1} is clamped to t-1); the entry rounds up iff
 * u < (x - q_r) / (q_{r+1} - q_r) (IEEE fp64), where u = bits 2^-53 and bits
 * = (w_hi 2^32 + w_lo) >> 11 for the output words of Philox4x32-10 with
 * counter (j mod 2^32, j / 2^32, 0, 0), j = i / 2, and key (seed mod 2^32,
 * seed / 2^32): words 0 (lo) and 1 (hi) for even i, 2 and 3 for odd i (one
 * generator call serves two entries).
 * codebook: device, t ascending fp64 values, 1 <= t <= 256.  symbols: device,
 * d bytes.  empirical_entropy: device scalar, plug-in entropy of the symbol
 * histogram in bits/entry.  hist: device, t int64 counts, may be NULL.
 */
ecasq_status ecasq_quantize(const void *x, ecasq_dtype dt, int64_t d, const double *codebook,
                            int32_t t, uint64_t seed, void *stream, uint8_t *symbols,
                            double *empirical_entropy, int64_t *hist);

/*
 * ecasq_quantize for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, outputs and errors as ecasq_quantize, bit for bit the
 * same symbols, counts and entropy, but the symbol counts live in a
 * file-scope device array of 256 64-bit counters (2 KB per device, held
 * until the process ends) instead of memory allocated per call; no
 * hipMalloc, hipFree or memset node is issued (the counts are cleared by a
 * kernel).  t above 256 is rejected with ECASQ_EINVAL.  Every call on one
 * device shares that array: calls that overlap on one device (other streams,
 * other threads) race and must be serialised by the caller.  Returns once
 * the work is enqueued.
 */
ecasq_status ecasq_quantize_noalloc(const void *x, ecasq_dtype dt, int64_t d,
                                    const double *codebook, int32_t t, uint64_t seed,
                                    void *stream, uint8_t *symbols, double *empirical_entropy,
                                    int64_t *hist);

/*
 * Many independent short vectors in one launch (one wavefront per row, several
 * rows per workgroup): x is n rows of d entries, row-major.  Each row is
 * solved as ecasq_solve_ex solves it with the default DP schedule and
 * opts->search_width = 1 and opts->alphabet = 0 (those fields of opts are
 * ignored), except that the search is the plain chord search, without the
 * query aimed at H = b: over many short rows the aimed search needs fewer
 * solves on average but more on its worst rows (on the 4096 x 128 KV-cache
 * rows: 8.0 on average and up to 14, against 8.5 and up to 11), and the
 * launch lasts as long as its slowest rows.  codebooks: device, n x s fp64 (row
 * r's t_out[r] values first, the rest untouched); t_out: device, n int32
 * (0 for a row holding NaN/Inf); infos_dev: device, n ecasq_info, may be NULL
 * (per-row status: ECASQ_OK, ECASQ_EINFEASIBLE or ECASQ_ENONFINITE).
 * 1 <= d <= 512, 2 <= s <= 32.  Returns after the results are in device
 * memory.
 */
ecasq_status ecasq_solve_batched(const void *x, ecasq_dtype dt, int64_t n, int64_t d,
                                 int32_t s, double bits_per_entry, const ecasq_options *opts,
                                 void *stream, double *codebooks, int32_t *t_out,
                                 ecasq_info *infos_dev);

/* Bytes of device workspace a single-vector solve of d entries with at most s
 * values needs; flags: 1 = stored argmins (recovery 1 of schedule 0),
 * 2 = the tables of schedule 1, 4 = a permissible grid (alphabet 1 or 2)
 * (0 when d < 1, s < 2 or flags outside 0..7). */
size_t ecasq_workspace_size(int64_t d, int32_t s, int32_t flags);

/* Static string for a status code. */
const char *ecasq_status_string(ecasq_status st);

/*
 * Inspection entry points used by the parity tests.
 *
 * ecasq_histogram: the sorted distinct values v (ascending, -0 folded into
 * +0), inclusive prefix counts N, and the correctly rounded inclusive prefix
 * sums S = sum c v and S2 = sum c v^2 (App. D prefix quantities).  All outputs
 * are device arrays of length >= d; *p_out (host) receives p.
 *
 * ecasq_dp_trace: forward DP solves of dp_APX (eq. apx_base, apx_rec,
 * apx_final) on the histogram of x at nlam multipliers lambdas[] (host array,
 * vNMSE units, nlam = 1 or 8; with 8 and schedule 0 they run as one search
 * pass does), by DP schedule `schedule` (0 or 1, as in ecasq_options).  For
 * multiplier m and every layer i in [2, min(s,p)] it records, in row
 * (m * (s+1) + i) of device arrays of nlam * (s+1) rows of d entries: F_i[j]
 * (F, fp64), the argmin k*_i[j] (kstar, int32), and the MSE and H(I,B)
 * accumulated along the argmins (M and Ph, fp64; both NULL or both given).
 * Entries outside a layer's valid columns are unspecified.  out (host,
 * 5 * nlam): per multiplier J (MSE units), MSE, H(I,B) of the minimising
 * path, i*, cells.  Schedule 1 keeps values only and recomputes the argmins
 * for the dump (an O(s p^2) pass); with kstar, M and Ph all NULL it returns
 * the values alone.
 */
ecasq_status ecasq_histogram(const void *x, ecasq_dtype dt, int64_t d, void *stream, double *v,
                             double *N, double *S, double *S2, int64_t *p_out);

ecasq_status ecasq_dp_trace(const void *x, ecasq_dtype dt, int64_t d, int32_t s, int32_t nlam,
                            const double *lambdas, int32_t schedule, void *stream, double *F,
                            int32_t *kstar, double *M, double *Ph, double *out);

/*
 * ecasq_opt_trace: the optimal DP of ecasq_solve_optimal with every layer
 * recorded.  F (device fp64) and K (device int32), capacity entries each, at
 * least (min(s,p)+1) p^2 (ECASQ_EINVAL otherwise, checked once p is known):
 * F[i][j][l] = dp(i,l,j) for the layer's valid (l, j) (layers 2..min(s,p)),
 * K[i][l][j] = the minimising k (layers 3..min(s,p)); other entries
 * unspecified.  chain (host, s int32): the codebook's value indices.  out
 * (host, 4 doubles): the optimum's DP value MSE + lambda' H(Xhat) (MSE units),
 * t, p, cells.  p = 1 records nothing.
 */
ecasq_status ecasq_opt_trace(const void *x, ecasq_dtype dt, int64_t d, int32_t s, double lambda,
                             const ecasq_options *opts, void *stream, int64_t capacity,
                             double *F, int32_t *K, int32_t *chain, double *out);

/*
 * Inspection log for the parity tests (process-wide, not thread-safe).
 * ecasq_inspect_enable(on != 0) clears the log and starts recording; 0 clears
 * it and stops.  While on, every budget search (ecasq_solve, _ex, _budgets,
 * _timeshare) appends one point per DP solve it runs, in solve order:
 * lambda (vNMSE units), H (H(I,B), or H(Xhat) with dp_objective 1 and 2),
 * vNMSE and t; points a budget sweep's search reuses from earlier budgets
 * are not repeated.  Every budget result appends the multiplier its codebook
 * was found at, the multiplier of the refinement (info.lambda) and the
 * codebook's value indices before and after refinement.
 * ecasq_inspect_points: copies min(n, cap) points (4 doubles each, host)
 * and returns n; ecasq_inspect_results: copies min(n, cap) results, lams
 * (host, 2 doubles each: found-at, refinement multiplier) and chains (host,
 * 514 int32 each: t_before, the t_before indices in slots 1..256, t_after at
 * slot 257, the t_after indices from slot 258), and returns n.  With out
 * NULL (points) or both arrays NULL (results) the call only returns n;
 * otherwise it clears that part of the log.
 */
void ecasq_inspect_enable(int32_t on);
int32_t ecasq_inspect_points(double *out, int32_t cap);
int32_t ecasq_inspect_results(double *lams, int32_t *chains, int32_t cap);

/*
 * Kernel timing for measurement tools.  While enabled (process-wide), every
 * launch of the DP layer kernel is bracketed by two HIP events recorded on the
 * stream it runs on; the elapsed times are read when the solve synchronizes.
 * Launches are kept apart by variant: 0 = one multiplier per launch (fixed
 * lambda, width-1 search, recovery half-DPs), 1 = the 8 multipliers of a
 * search pass, 2 = a whole solve of DP schedule 1 (all its launches, from
 * the table fill to eq. apx_final, timed as one unit; cells counted as for
 * schedule 0), 3 = one layer of the optimal DP (cells = its (k, l, j)
 * candidates), 4 = one launch of ecasq_solve_batched (cells not counted).
 * ecasq_timing_read returns, for one variant, the summed milliseconds, the
 * number of timed launches and the (column, predecessor) cells those launches
 * evaluated, each cell for every multiplier of its launch (host pointers, any
 * may be NULL); reset != 0 clears that variant's totals.  on = 2 also prints one line per DP solve to stderr (multiplier,
 * H(I,B), vNMSE, values, elapsed time), for long runs.  Not thread-safe.
 */
void ecasq_timing_enable(int32_t on);
void ecasq_timing_read(int32_t variant, double *layer_ms, int64_t *layer_launches,
                       int64_t *layer_cells, int32_t reset);

#ifdef __cplusplus
}
#endif

#endif /* ECASQ_H */
