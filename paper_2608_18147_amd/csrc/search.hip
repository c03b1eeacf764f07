// The budget search on the Lagrange multiplier (Sec. 3: the Lagrangian
// relaxation, a search on lambda for the budget; Sec. 5: keep the lowest-MSE
// solution with H(I,B) <= b; App. F.7: supporting-line queries), kept in device
// memory so that a solve issues its DP solves back to back without reading
// anything back between them.
//
// The state machine follows the search stated in include/ecasq.h step for
// step.  One thread runs it:
//   begin   first pass: lambda = 0 (width 1) or the grid of 8 (width 8);
//   commit  append the points just solved; when a pass is complete, pick A
//           (the infeasible point of largest lambda) and B (the feasible point
//           of smallest lambda, else the two-value codebook {v_0, v_{p-1}} for
//           b >= 1, else one solve at 2^40), and plan the next pass: the chord
//           slope lc = (M_B - M_A) / (H_A - H_B), or with width 1 the aimed
//           query (the slope at H = b of the curve through A and B on which
//           log vNMSE is linear in H) while such queries find new points, and
//           with width 8 seven more multipliers between A and B; stop when the
//           chord query returns A or B again, or after the pass limit.
// A query whose multiplier some point already has reuses that point; the
// machine advances through such queries until it needs a real solve: it then
// lists the multipliers to solve in todo (lambda' = RN(lambda ||X||^2) in
// todo_lamp) and sets run, or it sets done.
#include "device.hpp"
#include "launch.hpp"

namespace ecasq {

namespace {

enum { kStageEval = 0, kStageDecide = 1 };
enum { kPassFirst = 0, kPassNormal = 1, kPassBig = 2 };

constexpr double kBig = 0x1p40;  // the multiplier tried when no point is feasible

__device__ int find_point(const SearchState& S, double lam) {
    for (int x = 0; x < S.npts; x++)
        if (S.pts[x].lam == lam) return x;
    return -1;
}

// What the host polls between solves: done, solves so far, the last point.
__device__ void peek(SearchState& S) {
    S.peek.done = S.done;
    S.peek.nsol = S.nsol;
    if (S.npts > 0) S.peek.last = S.pts[S.npts - 1];
}

__device__ void finish(SearchState& S) {
    // refined points need not lie on a convex curve: the answer is the
    // feasible point of lowest vNMSE found (the first among equals)
    if (S.kind == 2 && S.status == 0) {
        int ib = -1;
        for (int x = 0; x < S.npts; x++)
            if (S.pts[x].H <= S.b && (ib < 0 || S.pts[x].M < S.pts[ib].M)) ib = x;
        if (ib >= 0) {
            S.B = S.pts[ib];
            S.iB = ib;
        }
    }
    S.done = 1;
    S.run = 0;
    S.ntodo = 0;
}

// Run the search until it needs DP solves (run = 1) or ends (done = 1).
__device__ void advance(SearchState& S, const double2* __restrict__ tab) {
    static const double kMul[kMaxLambdas - 1] = {0.25, 0.5, 0.75, 1.5, 2.0, 3.0, 4.0};
    for (int guard = 0; guard < 4 * kSearchMaxPts; guard++) {
        if (S.stage == kStageEval) {
            if (!S.issued) {
                // the multipliers of this pass no point has yet, first
                // occurrences only, in query order
                int m = 0;
                for (int g = 0; g < S.nq; g++) {
                    const double l = S.q[g];
                    bool seen = find_point(S, l) >= 0;
                    for (int h = 0; h < m; h++) seen = seen || S.todo[h] == l;
                    if (!seen) S.todo[m++] = l;
                }
                S.issued = 1;
                if (m > 0) {
                    S.ntodo = m;
                    S.nin = 0;
                    for (int g = 0; g < m; g++) S.todo_lamp[g] = S.todo[g] * S.s2tot;
                    S.run = 1;
                    return;
                }
            }
            // the pass is complete
            S.ntodo = 0;
            S.run = 0;
            if (S.pass_kind == kPassFirst) {
                S.npass = S.nsol > S.nsol0 ? 1 : 0;
            } else if (S.pass_kind == kPassBig) {
                S.npass++;
            } else {
                S.npass++;
                SearchPt C = S.pts[0];
                const int ic = find_point(S, S.q[0]);
                if (ic >= 0) C = S.pts[ic];
                if ((C.H == S.A.H && C.M == S.A.M) || (C.H == S.B.H && C.M == S.B.M)) {
                    if (!S.model) {
                        S.lam_final = S.lc;
                        finish(S);
                        return;
                    }
                    S.force_chord = 1;  // the aimed query found nothing new
                } else {
                    S.force_chord = 0;
                }
            }
            S.stage = kStageDecide;
            continue;
        }
        // decide: A = the infeasible point of largest lambda, B = the
        // feasible point of smallest lambda (the first among equal lambdas)
        int ia = -1, ib = -1;
        for (int x = 0; x < S.npts; x++) {
            if (S.pts[x].H > S.b) {
                if (ia < 0 || S.pts[x].lam > S.pts[ia].lam) ia = x;
            } else {
                if (ib < 0 || S.pts[x].lam < S.pts[ib].lam) ib = x;
            }
        }
        if (ia < 0) {  // lambda = 0 is feasible
            S.B = S.pts[ib];
            S.iB = ib;
            S.have_A = 0;
            S.lam_final = S.B.lam;
            finish(S);
            return;
        }
        S.A = S.pts[ia];
        S.iA = ia;
        S.have_A = 1;
        if (ib >= 0) {
            S.B = S.pts[ib];
            S.iB = ib;
            S.closed = 0;
        } else if (S.b >= 1.0) {
            S.B.lam = __builtin_huge_val();
            S.B.H = S.twoH;
            S.B.M = S.twoM;
            S.B.t = 2;
            S.iB = -1;
            S.closed = 1;
        } else {
            // no feasible point yet: try the largest multiplier once
            if (find_point(S, kBig) >= 0 || S.npass >= S.max_passes) {
                // infeasible budget: the lowest-entropy point found
                int ih = 0;
                for (int x = 1; x < S.npts; x++)
                    if (S.pts[x].H < S.pts[ih].H) ih = x;
                S.B = S.pts[ih];
                S.iB = ih;
                S.have_A = 0;
                S.status = -3;
                S.lam_final = S.B.lam;
                finish(S);
                return;
            }
            S.q[0] = kBig;
            S.nq = 1;
            S.pass_kind = kPassBig;
            S.stage = kStageEval;
            S.issued = 0;
            continue;
        }
        const double lc = (S.B.M - S.A.M) / (S.A.H - S.B.H);
        S.lc = lc;
        S.lam_final = S.closed ? lc : S.B.lam;
        if (!(lc > 0.0) || S.npass >= S.max_passes) {
            finish(S);
            return;
        }
        S.q[0] = lc;
        S.model = 0;
        if (S.width == 1 && S.aim && !S.force_chord && S.A.M > 0.0 && S.B.M > 0.0) {
            const double lq = aim_query(S.b, S.A.H, S.A.M, S.B.H, S.B.M, tab);
            if (__builtin_isfinite(lq) && lq > S.A.lam && lq < S.B.lam) {
                S.q[0] = lq;
                S.model = 1;
            }
        }
        for (int g = 1; g < S.width; g++)
            S.q[g] = S.closed ? lc * kMul[g - 1]
                              : S.A.lam + ((S.B.lam - S.A.lam) * (double)g) / 8.0;
        S.nq = S.width;
        S.pass_kind = kPassNormal;
        S.stage = kStageEval;
        S.issued = 0;
    }
    // every pass adds a point or ends the search, so this is not reached
    S.status = -5;
    finish(S);
}

__global__ __launch_bounds__(64) void k_search_begin(SearchState* __restrict__ Sp, SearchParams P,
                                                     const double* __restrict__ two) {
    __shared__ double2 tab[kLog2Size];
    load_log2_table(tab);
    __syncthreads();
    if (threadIdx.x != 0) return;
    SearchState& S = *Sp;
    static const double kGrid[kMaxLambdas] = {0.0, 1e-4, 1e-3, 1e-2, 1e-1, 1.0, 10.0, 100.0};
    S.b = P.b;
    S.s2tot = P.s2tot;
    S.twoH = P.kind != 0 ? two[2] : two[3];
    S.twoM = (0.0 + two[0]) / P.s2tot;
    S.max_passes = P.max_passes;
    S.width = P.width;
    S.aim = P.aim;
    S.kind = P.kind;
    S.has_chain = P.has_chain;
    S.s = P.s;
    if (!P.keep_points) S.npts = 0;
    S.ncached = S.npts;
    S.nsol = 0;
    S.npass = 0;
    S.status = 0;
    S.done = 0;
    S.run = 0;
    S.force_chord = 0;
    S.model = 0;
    S.closed = 0;
    S.have_A = 0;
    S.iA = S.iB = -1;
    S.lc = 0.0;
    S.lam_final = 0.0;
    S.nsol0 = 0;
    for (int g = 0; g < P.width; g++) S.q[g] = kGrid[g];
    S.nq = P.width;
    S.pass_kind = kPassFirst;
    S.stage = kStageEval;
    S.issued = 0;
    S.ntodo = 0;
    S.nin = 0;
    advance(S, tab);
    peek(S);
}

__global__ __launch_bounds__(64) void k_search_commit(SearchState* __restrict__ Sp,
                                                      const double* __restrict__ res,
                                                      const int32_t* __restrict__ chains,
                                                      int32_t m, int32_t* __restrict__ pchains,
                                                      int32_t gate) {
    __shared__ double2 tab[kLog2Size];
    __shared__ int32_t slot[kMaxLambdas], slot_t[kMaxLambdas];
    SearchState& S = *Sp;
    if (gate && !S.run) return;  // uniform: the solve before this was skipped
    load_log2_table(tab);
    if (threadIdx.x == 0) {
        // points for todo[nin .. nin+m), in query order
        for (int g = 0; g < m; g++) {
            slot[g] = -1;
            slot_t[g] = (int32_t)res[4 * g + 3];
            if (slot_t[g] < 2) S.status = -5;  // a failed solve ends the search
            if (S.npts < kSearchMaxPts && slot_t[g] >= 2) {
                SearchPt& q = S.pts[S.npts];
                q.lam = S.todo[S.nin + g];
                q.H = res[4 * g + 2];
                q.M = res[4 * g + 1] / S.s2tot;
                q.t = slot_t[g];
                q.pad = 0;
                slot[g] = S.npts;
                S.npts++;
            }
            S.nsol++;
        }
        S.nin += m;
    }
    __syncthreads();
    if (S.has_chain && chains && pchains) {
        for (int g = 0; g < m; g++) {
            const int at = slot[g];
            if (at < 0) continue;
            for (int r = threadIdx.x; r < slot_t[g] && r < S.s; r += blockDim.x)
                pchains[(int64_t)at * S.s + r] = chains[(int64_t)g * S.s + r];
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        if (S.status == -5)
            finish(S);
        else if (S.nin >= S.ntodo)
            advance(S, tab);  // the pass's solves are all in
        peek(S);
    }
}

}  // namespace

hipError_t launch_search_begin(SearchState* S, const SearchParams& P, const double* two,
                               hipStream_t st) {
    k_search_begin<<<1, 64, 0, st>>>(S, P, two);
    return hipGetLastError();
}

hipError_t launch_search_commit(SearchState* S, const double* res, const int32_t* chains,
                                int32_t m, int32_t* pchains, int32_t gate, hipStream_t st) {
    k_search_commit<<<1, 64, 0, st>>>(S, res, chains, m, pchains, gate);
    return hipGetLastError();
}

}  // namespace ecasq
