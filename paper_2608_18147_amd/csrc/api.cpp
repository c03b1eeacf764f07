// libecasq host library: argument checks, workspace layout and the launch
// sequence of one ECASQ solve (see include/ecasq.h for the contract).
//
//   prep        sort + weighted histogram + exact prefix sums (Sec. 2, App. D)
//   search      search on lambda in passes of 8 multipliers, each pass one
//               sweep of dp_APX for all 8 (Sec. 3 and Sec. 5; supporting-line
//               queries as in App. F.7)
//   recovery    Hirschberg on the final multiplier (Sec. 5 / Sec. 4.2), or a
//               traceback through stored argmins
//   refinement  three-colour pass (Sec. 6), one kernel
//   metrics     MSE, vNMSE, H(Xhat), H(I,B), objective, total rate
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstddef>
#include <cstring>
#include <vector>

#include "../../include/ecasq.h"
#include "launch.hpp"

using namespace ecasq;

namespace {

// Inspection log (ecasq_inspect_*): every DP solve's point of the budget
// searches and every budget result's codebook before and after refinement.
struct InspectResult {
    double lam_B, lam_final;
    std::vector<int32_t> pre, post;
};
bool g_inspect = false;
std::vector<double> g_ins_pts;  // lambda, H, vNMSE, t per solve
std::vector<InspectResult> g_ins_res;
double g_ins_lamB = 0.0;  // the multiplier the last search's B was found at

#define HIP_TRY(expr)                               \
    do {                                            \
        hipError_t e_ = (expr);                     \
        if (e_ != hipSuccess) return ECASQ_EHIP;    \
    } while (0)

#define ECASQ_TRY(expr)                             \
    do {                                            \
        ecasq_status s_ = (expr);                   \
        if (s_ != ECASQ_OK) return s_;              \
    } while (0)

struct Layout {
    size_t v, N, S, S2, gv, gN, gS, gS2, F0, F1, M0, M1, P0, P1, pval, pidx, last, res, mres,
        small, chain, kstar, prep, swF, swQ, swK, swchain, sstate, schains, two, cres, cchain;
    int64_t pstride;  // partial entries per multiplier
    size_t swKbytes;  // bytes at swK
    size_t total;
};

// Workspace flags: stored argmins of every layer (recovery 1 of the
// layer-by-layer schedule), and the sweep schedule's tables.
constexpr int32_t kWsArgmins = 1;
constexpr int32_t kWsSweep = 2;
constexpr int32_t kWsAlphabet = 4;  // a permissible grid next to the input's histogram
// (internal) schedule 1 with the argmin table of every layer, for the
// inspection call's argmin and accumulator dumps; without it K holds only
// the steps' counters and the traceback's partials
constexpr int32_t kWsSweepArgmins = 8;

Layout layout(int64_t d, int32_t s, int32_t flags) {
    Layout L;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        size_t at = o;
        o += align256(bytes);
        return at;
    };
    const size_t nd = sizeof(double) * (size_t)d;
    L.v = take(nd);
    L.N = take(nd);
    L.S = take(nd);
    L.S2 = take(nd);
    const size_t ng = (flags & kWsAlphabet) ? nd : 0;
    L.gv = take(ng);
    L.gN = take(ng);
    L.gS = take(ng);
    L.gS2 = take(ng);
    const bool sweep = (flags & kWsSweep) != 0;
    // layer-by-layer buffers: kMaxLambdas rows of d per array (one per
    // multiplier of a pass); the sweep keeps whole tables instead
    const size_t ndm = sweep ? 0 : nd * kMaxLambdas;
    L.F0 = take(ndm);
    L.F1 = take(ndm);
    L.M0 = take(ndm);
    L.M1 = take(ndm);
    L.P0 = take(ndm);
    L.P1 = take(ndm);
    L.pstride = sweep ? 0 : dp_partial_entries(d);
    const size_t np = (size_t)L.pstride * kMaxLambdas;
    L.pval = take(sizeof(double) * np);
    L.pidx = take(sizeof(int32_t) * np);
    L.swF = take(sweep ? sizeof(double) * (size_t)(s + 1) * (size_t)d : 0);
    L.swQ = take(sweep ? sweep_cost_bytes() : 0);
    L.swKbytes = !sweep ? 0
                 : (flags & kWsSweepArgmins) ? sizeof(int32_t) * (size_t)(s + 1) * (size_t)d
                                             : sweep_scratch_bytes(d);
    L.swK = take(L.swKbytes);
    L.swchain = take(sizeof(int32_t) * 528);  // chain, then the traceback state
    L.last = take(sizeof(double) * 3 * (size_t)(s + 1) * kMaxLambdas);
    L.res = take(sizeof(double) * 4 * kMaxLambdas);
    L.mres = take(sizeof(double) * 8);
    L.small = take(sizeof(int64_t) * 8);
    L.chain = take(sizeof(int32_t) * (size_t)(s + 8));
    L.kstar = (flags & kWsArgmins) && !sweep ? take(sizeof(int32_t) * (size_t)(s + 1) * (size_t)d)
                                              : 0;
    L.prep = take(prep_scratch_bytes(d));
    // the budget search's state, its points' codebooks and commit inputs
    L.sstate = take(sizeof(SearchState));
    L.schains = take(sizeof(int32_t) * (size_t)kSearchMaxPts * (size_t)s);
    L.two = take(sizeof(double) * 8);
    L.cres = take(sizeof(double) * 4 * kMaxLambdas);
    L.cchain = take(sizeof(int32_t) * (size_t)(s + 8));
    L.total = o;
    return L;
}

struct Point {
    double lam, H, M;
    double mse = 0.0;  // MSE of the point's codebook (points the host scores)
    int32_t t;
    std::vector<int32_t> chain;  // the solve's codebook (sweep schedule only)
};

struct Ctx {
    hipStream_t st;
    char* base;
    Layout L;
    int64_t d;
    int32_t s;
    int64_t p;
    double s2tot;
    Hist H;
    int64_t cells;
    int32_t solves;
    bool own;
    bool sweep;  // dp_APX by the column-block sweep (else layer by layer)
    // search points: 0 dp_APX (H(I,B)), 1 the optimal DP (H(Xhat)), 2 dp_APX's
    // codebook refined at the query's multiplier (H(Xhat))
    int32_t objective = 0;
    int32_t opt_full = 0;   // optimal DP: scan every predecessor
    int32_t refine_rounds = 0, refine_exhaustive = 0, recovery = 0;
    SearchPeek* poll = nullptr;  // pinned host memory (device-resident search)
    hipEvent_t ev[2] = {nullptr, nullptr};

    template <class T>
    T* at(size_t off) const {
        return reinterpret_cast<T*>(base + off);
    }
};

ecasq_status check_x(const void* x, int dt, int64_t d) {
    if (!x || d < 1 || d > ((int64_t)1 << 28)) return ECASQ_EINVAL;
    if (dt < 0 || dt > 2) return ECASQ_EINVAL;
    return ECASQ_OK;
}

ecasq_status ctx_open(Ctx& c, int64_t d, int32_t s, int32_t flags, void* stream, void* ws,
                      size_t ws_bytes) {
    c.st = static_cast<hipStream_t>(stream);
    c.d = d;
    c.s = s;
    c.sweep = (flags & kWsSweep) != 0;
    c.L = layout(d, s, flags);
    c.cells = 0;
    c.solves = 0;
    c.own = ws == nullptr;
    if (ws) {
        if (ws_bytes < c.L.total) return ECASQ_EWORKSPACE;
        c.base = static_cast<char*>(ws);
    } else {
        void* p = nullptr;
        if (hipMallocAsync(&p, c.L.total, c.st) != hipSuccess) return ECASQ_ENOMEM;
        c.base = static_cast<char*>(p);
    }
    return ECASQ_OK;
}

void ctx_close(Ctx& c) {
    if (c.poll || c.ev[0] || c.ev[1]) (void)hipStreamSynchronize(c.st);
    for (auto& e : c.ev)
        if (e) (void)hipEventDestroy(e);
    if (c.poll) (void)hipHostFree(c.poll);
    c.poll = nullptr;
    c.ev[0] = c.ev[1] = nullptr;
    if (c.own && c.base) {
        (void)hipFreeAsync(c.base, c.st);
        (void)hipStreamSynchronize(c.st);
    }
    c.base = nullptr;
}

// Sort, histogram, exact prefix sums; reads p, N[0] and ||X||^2 back.  With a
// permissible grid (alphabet 1 uniform, 2 quantile, of m points), the DP's
// candidates become the grid and p its size (App. D).
ecasq_status ctx_prep(Ctx& c, const void* x, int dt, int32_t alphabet = 0, int64_t m = 0) {
    int64_t* small = c.at<int64_t>(c.L.small);
    uint32_t* flags = reinterpret_cast<uint32_t*>(small + 1);
    HIP_TRY(hipMemsetAsync(small, 0, sizeof(int64_t) * 8, c.st));
    HIP_TRY(launch_prep(x, dt, c.d, c.base + c.L.prep, c.st, c.at<double>(c.L.v),
                        c.at<double>(c.L.N), c.at<double>(c.L.S), c.at<double>(c.L.S2), small,
                        flags));
    // p, the non-finite flag, then S2[p-1] and N[0] (written by the last
    // preparation kernel as doubles): one read
    int64_t hs[4] = {0, 0, 0, 0};
    HIP_TRY(hipMemcpyAsync(hs, small, sizeof hs, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    if ((uint32_t)hs[1] & 1u) return ECASQ_ENONFINITE;
    c.p = hs[0];
    c.H.v = c.at<double>(c.L.v);
    c.H.N = c.at<double>(c.L.N);
    c.H.S = c.at<double>(c.L.S);
    c.H.S2 = c.at<double>(c.L.S2);
    double s2 = 0, c0 = 0;
    std::memcpy(&s2, &hs[2], sizeof s2);
    std::memcpy(&c0, &hs[3], sizeof c0);
    if (alphabet != 0 && c.p >= 2) {
        int64_t* count = small + 5;
        HIP_TRY(launch_alphabet(alphabet, m, c.d, c.H.v, c.H.N, c.H.S, c.H.S2, c.p,
                                c.at<double>(c.L.gv), c.at<double>(c.L.gN), c.at<double>(c.L.gS),
                                c.at<double>(c.L.gS2), count, c.st));
        int64_t np = 0;
        HIP_TRY(hipMemcpyAsync(&np, count, sizeof np, hipMemcpyDeviceToHost, c.st));
        HIP_TRY(hipStreamSynchronize(c.st));
        if (np < 2 || np > m) return ECASQ_EHIP;
        c.p = np;
        c.H.v = c.at<double>(c.L.gv);
        c.H.N = c.at<double>(c.L.gN);
        c.H.S = c.at<double>(c.L.gS);
        c.H.S2 = c.at<double>(c.L.gS2);
        // the grid's first count
        HIP_TRY(hipMemcpyAsync(&c0, c.H.N, sizeof(double), hipMemcpyDeviceToHost, c.st));
        HIP_TRY(hipStreamSynchronize(c.st));
    }
    c.s2tot = s2;
    c.H.p = c.p;
    c.H.dd = (double)c.d;
    c.H.c0 = c0;
    c.H.c0d = c0 / (double)c.d;
    return ECASQ_OK;
}

int64_t tri_cells(int64_t n) { return n * (n + 1) / 2; }

// Optional per-layer dumps of a solve: for multiplier m and layer i, row
// (m * (s + 1) + i) of each array, row stride `stride`; any may be null.
struct Dumps {
    double* F = nullptr;
    int32_t* K = nullptr;
    double* M = nullptr;
    double* P = nullptr;
    int64_t stride = 0;
};

int64_t dp_cells(int64_t p, int32_t imax) {
    int64_t n = p - 1;
    for (int32_t i = 3; i <= imax; i++) n += tri_cells(p - i + 1);
    return n;
}

SweepSolve sweep_args(const Ctx& c) {
    SweepSolve S;
    S.H = c.H;
    S.F = c.at<double>(c.L.swF);
    S.Q = c.at<double>(c.L.swQ);
    S.K = c.at<int32_t>(c.L.swK);
    S.kbytes = c.L.swKbytes;
    S.st = c.at<int32_t>(c.L.swchain) + 256;
    S.ld = c.d;
    S.I = (int32_t)std::min<int64_t>(c.s, c.p);
    S.lamp = 0.0;
    return S;
}

// Enqueue one dp_APX solve by the sweep whose lambda' and run flag the
// kernels read from device memory (the device-resident search); the result
// (J, MSE, H(I,B), t) goes to the res slot and the codebook to the chain slot.
ecasq_status sweep_enqueue(Ctx& c, const double* lampp, const int32_t* runp, int32_t exact_s) {
    SweepSolve S = sweep_args(c);
    S.lampp = lampp;
    S.runp = runp;
    timing_begin(2, dp_cells(c.p, S.I), c.st);
    HIP_TRY(launch_sweep(S, exact_s, c.at<double>(c.L.res), c.at<int32_t>(c.L.swchain), c.st));
    timing_end(c.st);
    return ECASQ_OK;
}

// One dp_APX solve at lam by the column-block sweep: the result, the chain of
// its codebook, and optionally the tables as dumps (row m of a pass).
ecasq_status sweep_solve(Ctx& c, double lam, int32_t exact_s, Point& out, double* J4,
                         const Dumps* dump, int32_t m) {
    const int64_t p = c.p;
    const int32_t imax = (int32_t)std::min<int64_t>(c.s, p);
    SweepSolve S = sweep_args(c);
    S.lamp = lam * c.s2tot;
    double* res = c.at<double>(c.L.res);
    int32_t* ch = c.at<int32_t>(c.L.swchain);
    timing_begin(2, dp_cells(p, imax), c.st);
    HIP_TRY(launch_sweep(S, exact_s, res, ch, c.st));
    timing_end(c.st);
    if (dump) {
        const int32_t ls = c.s + 1;
        const int64_t ds = dump->stride;
        const size_t rows = (size_t)(imax - 1) * (size_t)c.d;
        if (ds != c.d) return ECASQ_EINVAL;
        if (dump->F)
            HIP_TRY(hipMemcpyAsync(dump->F + ((int64_t)m * ls + 2) * ds, S.F + 2 * c.d,
                                   sizeof(double) * rows, hipMemcpyDeviceToDevice, c.st));
        if (dump->K || (dump->M && dump->P)) HIP_TRY(launch_sweep_argmins(S, c.st));
        if (dump->K)
            HIP_TRY(hipMemcpyAsync(dump->K + ((int64_t)m * ls + 2) * ds, S.K + 2 * c.d,
                                   sizeof(int32_t) * rows, hipMemcpyDeviceToDevice, c.st));
        if (dump->M && dump->P)
            HIP_TRY(launch_sweep_accumulators(S, dump->M + (int64_t)m * ls * ds,
                                              dump->P + (int64_t)m * ls * ds, c.st));
    }
    double r[4];
    HIP_TRY(hipMemcpyAsync(r, res, sizeof r, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    const int32_t t = (int32_t)r[3];
    if (t < 2 || t > imax) return ECASQ_EHIP;
    out.chain.assign(t, 0);
    HIP_TRY(hipMemcpyAsync(out.chain.data(), ch, sizeof(int32_t) * t, hipMemcpyDeviceToHost,
                           c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    timing_flush();
    out.lam = lam;
    out.H = r[2];
    out.M = r[1] / c.s2tot;
    out.t = t;
    if (J4) std::memcpy(J4, r, sizeof r);
    c.cells += dp_cells(p, imax);
    c.solves++;
    return ECASQ_OK;
}

// Full dp_APX solves at nlam multipliers lams[] (vNMSE units) in one sweep
// over the layers (nlam must be 1 or kMaxLambdas; the column-block sweep
// solves them one after the other).  J_out (optional): the raw (J, MSE,
// H(I,B), t) of every multiplier.
ecasq_status dp_solve(Ctx& c, const double* lams, int32_t nlam, int32_t exact_s, Point* out,
                      double* J_out, const Dumps* dump) {
    if (nlam != 1 && nlam != kMaxLambdas) return ECASQ_EINVAL;
    const auto t0 = std::chrono::steady_clock::now();
    auto progress = [&](const Point* pts, int32_t n) {
        if (!timing_verbose()) return;
        const double ms =
            std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0)
                .count();
        for (int32_t m = 0; m < n; m++)
            std::fprintf(stderr, "[ecasq] solve %d: lambda=%.6g H(I,B)=%.6f vNMSE=%.6g t=%d (%.1f ms)\n",
                         c.solves - n + m + 1, pts[m].lam, pts[m].H, pts[m].M, pts[m].t, ms);
        std::fflush(stderr);
    };
    if (c.sweep) {
        for (int32_t m = 0; m < nlam; m++) {
            ECASQ_TRY(sweep_solve(c, lams[m], exact_s, out[m], J_out ? J_out + 4 * m : nullptr,
                                  dump, m));
            progress(out + m, 1);
        }
        return ECASQ_OK;
    }
    const int64_t p = c.p;
    const int32_t imax = (int32_t)std::min<int64_t>(c.s, p);
    const int32_t ls = c.s + 1;
    const int64_t d = c.d;
    double* F[2] = {c.at<double>(c.L.F0), c.at<double>(c.L.F1)};
    double* M[2] = {c.at<double>(c.L.M0), c.at<double>(c.L.M1)};
    double* Ph[2] = {c.at<double>(c.L.P0), c.at<double>(c.L.P1)};
    double* last = c.at<double>(c.L.last);
    double* res = c.at<double>(c.L.res);
    const int64_t ds = dump ? dump->stride : 0;
    auto row = [&](auto* base, int32_t m, int32_t i) {
        return base ? base + ((int64_t)m * ls + i) * ds : nullptr;
    };
    // copy columns [j0, p) of layer i (current buffers cur) into the dumps
    auto save = [&](int32_t i, int cur, int64_t j0) -> ecasq_status {
        if (!dump) return ECASQ_OK;
        const size_t nb = sizeof(double) * (size_t)(p - j0);
        for (int32_t m = 0; m < nlam; m++) {
            if (dump->F)
                HIP_TRY(hipMemcpyAsync(row(dump->F, m, i) + j0, F[cur] + m * d + j0, nb,
                                       hipMemcpyDeviceToDevice, c.st));
            if (dump->M)
                HIP_TRY(hipMemcpyAsync(row(dump->M, m, i) + j0, M[cur] + m * d + j0, nb,
                                       hipMemcpyDeviceToDevice, c.st));
            if (dump->P)
                HIP_TRY(hipMemcpyAsync(row(dump->P, m, i) + j0, Ph[cur] + m * d + j0, nb,
                                       hipMemcpyDeviceToDevice, c.st));
        }
        return ECASQ_OK;
    };
    double lamp[kMaxLambdas];
    for (int32_t m = 0; m < nlam; m++) lamp[m] = lams[m] * c.s2tot;
    DpInit I;
    std::memset(&I, 0, sizeof I);
    I.nlam = nlam;
    for (int32_t m = 0; m < nlam; m++) {
        I.lam[m] = lamp[m];
        I.F[m] = F[0] + m * d;
        I.M[m] = M[0] + m * d;
        I.Ph[m] = Ph[0] + m * d;
        I.kstar[m] = dump ? row(dump->K, m, 2) : nullptr;
    }
    I.last = last;
    I.last_stride = ls;
    HIP_TRY(launch_dp_init_fwd(c.H, 0, 1, p - 1, I, c.st));
    ECASQ_TRY(save(2, 0, 1));
    c.cells += (int64_t)nlam * (p - 1);
    int cur = 0;
    for (int32_t i = 3; i <= imax; i++) {
        DpLayer L;
        std::memset(&L, 0, sizeof L);
        L.H = c.H;
        L.nlam = nlam;
        for (int32_t m = 0; m < nlam; m++) {
            L.Fin[m] = F[cur] + m * d;
            L.Fout[m] = F[1 - cur] + m * d;
            L.Min[m] = M[cur] + m * d;
            L.Pin[m] = Ph[cur] + m * d;
            L.Mout[m] = M[1 - cur] + m * d;
            L.Pout[m] = Ph[1 - cur] + m * d;
            L.lam[m] = lamp[m];
            L.kstar[m] = dump ? row(dump->K, m, i) : nullptr;
        }
        L.pval = c.at<double>(c.L.pval);
        L.pidx = c.at<int32_t>(c.L.pidx);
        L.pstride = c.L.pstride;
        L.kb = i - 2;
        L.jlo = i - 1;
        L.jhi = p - 1;
        L.backward = false;
        L.last = last;
        L.layer = i;
        L.last_stride = ls;
        L.cells = tri_cells(p - i + 1);
        HIP_TRY(launch_dp_layer(L, c.st));
        ECASQ_TRY(save(i, 1 - cur, i - 1));
        c.cells += (int64_t)nlam * tri_cells(p - i + 1);
        cur = 1 - cur;
    }
    HIP_TRY(launch_dp_final(last, ls, imax, exact_s, nlam, res, c.st));
    double r[4 * kMaxLambdas];
    HIP_TRY(hipMemcpyAsync(r, res, sizeof(double) * 4 * nlam, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    timing_flush();
    for (int32_t m = 0; m < nlam; m++) {
        out[m].lam = lams[m];
        out[m].H = r[4 * m + 2];
        out[m].M = r[4 * m + 1] / c.s2tot;
        out[m].t = (int32_t)r[4 * m + 3];
    }
    if (J_out) std::memcpy(J_out, r, sizeof(double) * 4 * nlam);
    c.solves += nlam;
    progress(out, nlam);
    return ECASQ_OK;
}

ecasq_status dp_solve1(Ctx& c, double lam, int32_t exact_s, Point& out) {
    return dp_solve(c, &lam, 1, exact_s, &out, nullptr, nullptr);
}


// Optimal lambda-ECASQ at lamp: the codebook (value indices) and the DP's own
// value.  Ftrace / Ktrace: every layer, for the inspection entry point.
ecasq_status opt_solve(Ctx& c, double lam, int32_t exact_s, std::vector<int32_t>& chain,
                       double* J, double* Ftrace, int32_t* Ktrace) {
    if (c.p == 1) {
        chain.assign(1, 0);
        *J = 0.0;
        return ECASQ_OK;
    }
    if (c.p > kOptMaxP) return ECASQ_ENOMEM;
    const int32_t imax = (int32_t)std::min<int64_t>(c.s, c.p);
    const size_t bytes = opt_workspace_bytes(c.p, imax, Ktrace != nullptr);
    void* mem = nullptr;
    if (hipMallocAsync(&mem, bytes, c.st) != hipSuccess) return ECASQ_ENOMEM;
    int32_t* ch = c.at<int32_t>(c.L.chain);
    double* res = c.at<double>(c.L.mres);
    const hipError_t e = launch_opt(c.H, imax, exact_s, lam * c.s2tot, c.opt_full,
                                    static_cast<char*>(mem), ch, res, Ftrace, Ktrace, c.st);
    double r[2] = {0.0, 0.0};
    hipError_t e2 = hipSuccess;
    if (e == hipSuccess) e2 = hipMemcpyAsync(r, res, sizeof r, hipMemcpyDeviceToHost, c.st);
    (void)hipFreeAsync(mem, c.st);
    HIP_TRY(hipStreamSynchronize(c.st));
    HIP_TRY(e);
    HIP_TRY(e2);
    const int32_t t = (int32_t)r[1];
    if (t < 2 || t > imax) return ECASQ_EHIP;
    chain.resize(t);
    HIP_TRY(hipMemcpy(chain.data(), ch, sizeof(int32_t) * t, hipMemcpyDeviceToHost));
    *J = r[0];
    c.cells += opt_cells(c.p, imax, exact_s);
    c.solves += 1;
    return ECASQ_OK;
}


// A search point of the optimal DP: its codebook's H(Xhat) and vNMSE, summed
// over the chain by the metrics kernel.
ecasq_status opt_point(Ctx& c, double lam, int32_t exact_s, Point& out) {
    std::vector<int32_t> chain;
    double J = 0.0;
    ECASQ_TRY(opt_solve(c, lam, exact_s, chain, &J, nullptr, nullptr));
    int32_t* ch = c.at<int32_t>(c.L.chain);
    double* mres = c.at<double>(c.L.mres);
    HIP_TRY(hipMemcpyAsync(ch, chain.data(), sizeof(int32_t) * chain.size(),
                           hipMemcpyHostToDevice, c.st));
    HIP_TRY(launch_metrics(c.H, (int32_t)chain.size(), ch, 0.0, c.s2tot, mres, c.st));
    double m[6];
    HIP_TRY(hipMemcpyAsync(m, mres, sizeof m, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    out.lam = lam;
    out.H = m[2];
    out.M = m[0] / c.s2tot;
    out.mse = m[0];
    out.t = (int32_t)chain.size();
    out.chain = chain;
    if (timing_verbose())
        std::fprintf(stderr, "[ecasq] optimal solve lambda=%.6g H(Xhat)=%.6f vNMSE=%.6g t=%d\n",
                     lam, out.H, out.M, out.t);
    return ECASQ_OK;
}

ecasq_status recover(Ctx& c, int32_t t, double lam, int32_t exact_s, int32_t mode,
                     std::vector<int32_t>& chain);

// A point of the refinement-aware search: dp_APX's codebook at lambda (the
// argmin traceback of the solve), refined at lambda without a budget guard
// (Sec. 6), scored by its own H(Xhat) and vNMSE.
ecasq_status refined_point(Ctx& c, double lam, int32_t exact_s, Point& out) {
    Point P;
    ECASQ_TRY(dp_solve(c, &lam, 1, exact_s, &P, nullptr, nullptr));
    std::vector<int32_t> chain = P.chain;
    if (chain.empty()) ECASQ_TRY(recover(c, P.t, lam, exact_s, c.recovery, chain));
    const int32_t t = (int32_t)chain.size();
    int32_t* ch = c.at<int32_t>(c.L.chain);
    int32_t* stats = ch + c.s + 2;
    double* mres = c.at<double>(c.L.mres);
    HIP_TRY(hipMemcpyAsync(ch, chain.data(), sizeof(int32_t) * t, hipMemcpyHostToDevice, c.st));
    if (t >= 3 && c.refine_rounds > 0) {
        HIP_TRY(hipMemsetAsync(stats, 0, sizeof(int32_t) * 2, c.st));
        HIP_TRY(launch_refine(c.H, t, ch, lam * c.s2tot, HUGE_VAL, 0, c.refine_rounds,
                              c.refine_exhaustive, stats, c.st));
    }
    HIP_TRY(launch_metrics(c.H, t, ch, 0.0, c.s2tot, mres, c.st));
    double m[6];
    HIP_TRY(hipMemcpyAsync(chain.data(), ch, sizeof(int32_t) * t, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipMemcpyAsync(m, mres, sizeof m, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    out.lam = lam;
    out.H = m[2];
    out.M = m[0] / c.s2tot;
    out.mse = m[0];
    out.t = t;
    out.chain = chain;
    return ECASQ_OK;
}

// Result of the budget search: B (the codebook to recover), A (the infeasible
// point the final chord starts from, if any), the multiplier of the
// refinement step and the number of passes.
struct SearchResult {
    Point B;
    Point A;
    bool have_A = false;
    double lam_final;
    int32_t passes;
    ecasq_status status;
};

// Per-context host resources of the device-resident search: a pinned poll
// block and two events (created on first use, released by ctx_close).
ecasq_status search_host_init(Ctx& c) {
    if (c.poll) return ECASQ_OK;
    void* h = nullptr;
    HIP_TRY(hipHostMalloc(&h, 2 * sizeof(SearchPeek), hipHostMallocDefault));
    c.poll = static_cast<SearchPeek*>(h);
    for (auto& e : c.ev) HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    return ECASQ_OK;
}

// The search state's fields before its point list, read back in one copy.
ecasq_status read_state(Ctx& c, SearchState& h) {
    SearchState* S = c.at<SearchState>(c.L.sstate);
    HIP_TRY(hipMemcpyAsync(&h, S, offsetof(SearchState, pts), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    return ECASQ_OK;
}

Point to_point(const SearchPt& q) {
    Point P;
    P.lam = q.lam;
    P.H = q.H;
    P.M = q.M;
    P.t = q.t;
    return P;
}

ecasq_status point_chain(Ctx& c, int32_t at, Point& P) {
    P.chain.assign(P.t, 0);
    HIP_TRY(hipMemcpyAsync(P.chain.data(), c.at<int32_t>(c.L.schains) + (int64_t)at * c.s,
                           sizeof(int32_t) * P.t, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    return ECASQ_OK;
}

void print_point(int32_t n, const SearchPt& q) {
    std::fprintf(stderr, "[ecasq] solve %d: lambda=%.6g H=%.6f vNMSE=%.6g t=%d\n", n, q.lam, q.H,
                 q.M, q.t);
    std::fflush(stderr);
}

// The default configuration (dp_APX by the sweep, one multiplier per pass):
// every solve reads lambda' and a run flag from the search state and is
// followed by the commit kernel, so the host reads back nothing but the done
// flag.  For short solves (fewer than kAheadBlocks column blocks) the host
// keeps one solve queued ahead and polls the done flag of the one before it,
// so solves run back to back; when the search ends, the queued solve and its
// commit find run = 0 and return at once.  Long solves are polled one by one
// (the poll costs nothing next to them, a skipped solve's launches would).
constexpr int64_t kAheadBlocks = 1024;

ecasq_status search_device_loop(Ctx& c, int32_t exact_s, int32_t max_passes) {
    ECASQ_TRY(search_host_init(c));
    SearchState* S = c.at<SearchState>(c.L.sstate);
    double* res = c.at<double>(c.L.res);
    int32_t* ch = c.at<int32_t>(c.L.swchain);
    int32_t* pch = c.at<int32_t>(c.L.schains);
    // the search may end without a solve (every query cached)
    HIP_TRY(hipMemcpyAsync(c.poll, &S->peek, sizeof(SearchPeek), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    if (c.poll[0].done) return ECASQ_OK;
    const int32_t limit = 2 * max_passes + 8;  // each solve adds a point to a finite search
    const int32_t ahead = (c.p + 63) / 64 < kAheadBlocks ? 1 : 0;
    int32_t n = 0;
    for (;;) {
        ECASQ_TRY(sweep_enqueue(c, &S->todo_lamp[0], &S->run, exact_s));
        HIP_TRY(launch_search_commit(S, res, ch, 1, pch, 1, c.st));
        HIP_TRY(hipMemcpyAsync(c.poll + (n & 1), &S->peek, sizeof(SearchPeek),
                               hipMemcpyDeviceToHost, c.st));
        HIP_TRY(hipEventRecord(c.ev[n & 1], c.st));
        n++;
        if (n > ahead) {
            // the solve `ahead` places back and its commit
            const int32_t k = (n - 1 - ahead) & 1;
            HIP_TRY(hipEventSynchronize(c.ev[k]));
            const SearchPeek& pk = c.poll[k];
            if (timing_verbose()) print_point(pk.nsol, pk.last);
            if (pk.done) break;  // a queued solve finds run = 0
        }
        if (n > limit) return ECASQ_EHIP;
    }
    HIP_TRY(hipStreamSynchronize(c.st));
    if (ahead) timing_discard_last();  // the skipped solve
    timing_flush();
    return ECASQ_OK;
}

// One pass's solves driven from the host (the other configurations): the
// state's todo list is read back, each multiplier solved as its kind says,
// and the points committed on the device in query order.
ecasq_status search_host_pass(Ctx& c, const SearchState& h, int32_t exact_s) {
    SearchState* S = c.at<SearchState>(c.L.sstate);
    int32_t* pch = c.at<int32_t>(c.L.schains);
    double* cres = c.at<double>(c.L.cres);
    int32_t* cch = c.at<int32_t>(c.L.cchain);
    const int32_t m = h.ntodo;
    if (c.objective != 0) {
        for (int32_t g = 0; g < m; g++) {
            Point P;
            if (c.objective == 1)
                ECASQ_TRY(opt_point(c, h.todo[g], exact_s, P));
            else
                ECASQ_TRY(refined_point(c, h.todo[g], exact_s, P));
            const double r[4] = {0.0, P.mse, P.H, (double)P.t};
            HIP_TRY(hipMemcpyAsync(cres, r, sizeof r, hipMemcpyHostToDevice, c.st));
            HIP_TRY(hipMemcpyAsync(cch, P.chain.data(), sizeof(int32_t) * P.t,
                                   hipMemcpyHostToDevice, c.st));
            HIP_TRY(launch_search_commit(S, cres, cch, 1, pch, 0, c.st));
        }
        return ECASQ_OK;
    }
    if (c.sweep) {
        for (int32_t g = 0; g < m; g++) {
            Point P;
            ECASQ_TRY(sweep_solve(c, h.todo[g], exact_s, P, nullptr, nullptr, 0));
            HIP_TRY(launch_search_commit(S, c.at<double>(c.L.res), c.at<int32_t>(c.L.swchain), 1,
                                         pch, 0, c.st));
        }
        return ECASQ_OK;
    }
    // layer by layer: one multiplier, or a pass of kMaxLambdas (padded with
    // repeats of the last, which are not counted)
    double todo[kMaxLambdas];
    for (int32_t g = 0; g < m; g++) todo[g] = h.todo[g];
    Point out[kMaxLambdas];
    if (m == 1) {
        ECASQ_TRY(dp_solve(c, todo, 1, exact_s, out, nullptr, nullptr));
    } else {
        for (int32_t g = m; g < kMaxLambdas; g++) todo[g] = todo[m - 1];
        const int64_t cells0 = c.cells;
        const int32_t solves0 = c.solves;
        ECASQ_TRY(dp_solve(c, todo, kMaxLambdas, exact_s, out, nullptr, nullptr));
        c.cells = cells0 + (c.cells - cells0) / kMaxLambdas * m;
        c.solves = solves0 + m;
    }
    HIP_TRY(launch_search_commit(S, c.at<double>(c.L.res), nullptr, m, pch, 0, c.st));
    return ECASQ_OK;
}

// The budget search on lambda (the schedule is stated in include/ecasq.h),
// run by the device state machine of search.hip.  keep: start from the points
// earlier searches on this input solved (a budget sweep), reusing any of
// their multipliers the search queries again.
ecasq_status search(Ctx& c, double b, int32_t exact_s, int32_t max_passes, int32_t width,
                    SearchResult& R, bool keep = false) {
    if (width != 1 && width != kMaxLambdas) return ECASQ_EINVAL;
    if (c.objective != 0) width = 1;
    SearchState* S = c.at<SearchState>(c.L.sstate);
    // the two-value codebook {v_0, v_{p-1}}: B when no point is feasible
    {
        int32_t ends[2] = {0, (int32_t)(c.p - 1)};
        int32_t* ech = c.at<int32_t>(c.L.cchain);
        HIP_TRY(hipMemcpyAsync(ech, ends, sizeof ends, hipMemcpyHostToDevice, c.st));
        HIP_TRY(launch_metrics(c.H, 2, ech, 0.0, c.s2tot, c.at<double>(c.L.two), c.st));
    }
    SearchParams P;
    P.b = b;
    P.s2tot = c.s2tot;
    P.max_passes = max_passes;
    P.width = width;
    P.aim = 1;
    P.kind = c.objective;
    P.has_chain = (c.objective != 0 || c.sweep) ? 1 : 0;
    P.s = c.s;
    P.keep_points = keep ? 1 : 0;
    HIP_TRY(launch_search_begin(S, P, c.at<double>(c.L.two), c.st));
    const int32_t solves0 = c.solves;
    SearchState h;
    if (c.objective == 0 && c.sweep && width == 1) {
        ECASQ_TRY(search_device_loop(c, exact_s, max_passes));
        ECASQ_TRY(read_state(c, h));
        const int32_t imax = (int32_t)std::min<int64_t>(c.s, c.p);
        c.solves += h.nsol;
        c.cells += (int64_t)h.nsol * dp_cells(c.p, imax);
    } else {
        for (int32_t guard = 0;; guard++) {
            ECASQ_TRY(read_state(c, h));
            if (h.done) break;
            if (guard > 4 * kSearchMaxPts || h.ntodo < 1 || h.ntodo > kMaxLambdas)
                return ECASQ_EHIP;
            ECASQ_TRY(search_host_pass(c, h, exact_s));
        }
        if (c.solves - solves0 != h.nsol) return ECASQ_EHIP;
    }
    if (h.status == -5) return ECASQ_EHIP;
    if (g_inspect) {
        const int32_t n0 = h.ncached, n1 = std::min<int32_t>(h.npts, kSearchMaxPts);
        if (n1 > n0) {
            std::vector<SearchPt> q((size_t)(n1 - n0));
            HIP_TRY(hipMemcpyAsync(q.data(), &S->pts[n0], sizeof(SearchPt) * q.size(),
                                   hipMemcpyDeviceToHost, c.st));
            HIP_TRY(hipStreamSynchronize(c.st));
            for (const SearchPt& x : q)
                g_ins_pts.insert(g_ins_pts.end(), {x.lam, x.H, x.M, (double)x.t});
        }
        g_ins_lamB = h.B.lam;
    }
    R.status = h.status == -3 ? ECASQ_EINFEASIBLE : ECASQ_OK;
    R.lam_final = h.lam_final;
    R.passes = h.npass;
    R.B = to_point(h.B);
    if (h.iB >= 0 && P.has_chain) ECASQ_TRY(point_chain(c, h.iB, R.B));
    R.have_A = h.have_A != 0;
    if (R.have_A) {
        R.A = to_point(h.A);
        if (P.has_chain) ECASQ_TRY(point_chain(c, h.iA, R.A));
    }
    return ECASQ_OK;
}

// Hirschberg recovery of the best chain lo = u_0 < ... < u_{n-1} = hi.
ecasq_status hirschberg(Ctx& c, double lamp, int64_t lo, int64_t hi, int32_t n, int32_t* out) {
    if (n == 2) {
        out[0] = (int32_t)lo;
        out[1] = (int32_t)hi;
        return ECASQ_OK;
    }
    if (hi - lo + 1 == n) {
        for (int32_t x = 0; x < n; x++) out[x] = (int32_t)(lo + x);
        return ECASQ_OK;
    }
    const int32_t r = (n - 1) / 2;
    double* Fw[2] = {c.at<double>(c.L.F0), c.at<double>(c.L.F1)};
    double* Bw[2] = {c.at<double>(c.L.M0), c.at<double>(c.L.M1)};
    // forward half: r+1 values starting at lo
    {
        const int64_t jl = lo + 1, jh = hi - (n - 2);
        DpInit I;
        std::memset(&I, 0, sizeof I);
        I.nlam = 1;
        I.lam[0] = lamp;
        I.F[0] = Fw[0];
        HIP_TRY(launch_dp_init_fwd(c.H, lo, jl, jh, I, c.st));
        c.cells += jh - jl + 1;
    }
    int fc = 0;
    for (int32_t q = 3; q <= r + 1; q++) {
        DpLayer L;
        std::memset(&L, 0, sizeof L);
        L.H = c.H;
        L.nlam = 1;
        L.Fin[0] = Fw[fc];
        L.Fout[0] = Fw[1 - fc];
        L.pval = c.at<double>(c.L.pval);
        L.pidx = c.at<int32_t>(c.L.pidx);
        L.pstride = c.L.pstride;
        L.kb = lo + q - 2;
        L.jlo = lo + q - 1;
        L.jhi = hi - (n - q);
        L.backward = false;
        L.lam[0] = lamp;
        for (int64_t j = L.jlo; j <= L.jhi; j++) L.cells += j - L.kb;
        HIP_TRY(launch_dp_layer(L, c.st));
        c.cells += L.cells;
        fc = 1 - fc;
    }
    // backward half: n-r values ending at hi
    {
        const int64_t jl = lo + n - 2, jh = hi - 1;
        HIP_TRY(launch_dp_init_bwd(c.H, hi, jl, jh, lamp, Bw[0], c.st));
        c.cells += jh - jl + 1;
    }
    int bc = 0;
    for (int32_t q = 3; q <= n - r; q++) {
        DpLayer L;
        std::memset(&L, 0, sizeof L);
        L.H = c.H;
        L.nlam = 1;
        L.Fin[0] = Bw[bc];
        L.Fout[0] = Bw[1 - bc];
        L.pval = c.at<double>(c.L.pval);
        L.pidx = c.at<int32_t>(c.L.pidx);
        L.pstride = c.L.pstride;
        L.kb = hi - q + 2;
        L.jlo = lo + n - q;
        L.jhi = hi - q + 1;
        L.backward = true;
        L.lam[0] = lamp;
        for (int64_t j = L.jlo; j <= L.jhi; j++) L.cells += L.kb - j;
        HIP_TRY(launch_dp_layer(L, c.st));
        c.cells += L.cells;
        bc = 1 - bc;
    }
    int64_t* mdev = c.at<int64_t>(c.L.small) + 4;
    HIP_TRY(launch_split(Fw[fc], Bw[bc], lo + r, hi - (n - 1 - r), mdev, c.st));
    int64_t m = -1;
    HIP_TRY(hipMemcpyAsync(&m, mdev, sizeof m, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    timing_flush();
    if (m < lo + r || m > hi - (n - 1 - r)) return ECASQ_EHIP;
    ECASQ_TRY(hirschberg(c, lamp, lo, m, r + 1, out));
    ECASQ_TRY(hirschberg(c, lamp, m, hi, n - r, out + r));
    return ECASQ_OK;
}

// Codebook with t values at lambda (vNMSE units), written to chain (host).
ecasq_status recover(Ctx& c, int32_t t, double lam, int32_t exact_s, int32_t mode,
                     std::vector<int32_t>& chain) {
    chain.assign(t, 0);
    if (c.p == 1) return ECASQ_OK;
    if (t == 2 || !std::isfinite(lam)) {
        chain.assign({0, (int32_t)(c.p - 1)});
        return ECASQ_OK;
    }
    if (mode == 1) {
        int32_t* K = c.at<int32_t>(c.L.kstar);
        Point P;
        Dumps dk;
        dk.K = K;
        dk.stride = c.p;
        ECASQ_TRY(dp_solve(c, &lam, 1, exact_s, &P, nullptr, &dk));
        c.solves--;  // a repeat of a search solve, not a new query
        if (P.t != t) return ECASQ_EHIP;
        chain[t - 1] = (int32_t)(c.p - 1);
        for (int32_t i = t; i >= 3; i--) {
            int32_t k = -1;
            HIP_TRY(hipMemcpyAsync(&k, K + (int64_t)i * c.p + chain[i - 1], sizeof k,
                                   hipMemcpyDeviceToHost, c.st));
            HIP_TRY(hipStreamSynchronize(c.st));
            chain[i - 2] = k;
        }
        chain[0] = 0;
        return ECASQ_OK;
    }
    return hirschberg(c, lam * c.s2tot, 0, c.p - 1, t, chain.data());
}

ecasq_status finish(Ctx& c, std::vector<int32_t>& chain, double lam, double b, bool budget,
                    const ecasq_options& o, double* codebook, int32_t* rank, ecasq_info* info,
                    ecasq_status status, int32_t passes) {
    const int32_t t = (int32_t)chain.size();
    int32_t* ch = c.at<int32_t>(c.L.chain);
    int32_t* stats = ch + c.s + 2;
    HIP_TRY(hipMemcpyAsync(ch, chain.data(), sizeof(int32_t) * t, hipMemcpyHostToDevice, c.st));
    HIP_TRY(hipMemsetAsync(stats, 0, sizeof(int32_t) * 2, c.st));
    if (o.refine_rounds > 0 && std::isfinite(lam) && t >= 3)
        HIP_TRY(launch_refine(c.H, t, ch, lam * c.s2tot, b, budget ? 1 : 0, o.refine_rounds,
                              o.refine_exhaustive, stats, c.st));
    double* mres = c.at<double>(c.L.mres);
    HIP_TRY(launch_metrics(c.H, t, ch, lam, c.s2tot, mres, c.st));
    HIP_TRY(launch_gather(c.H.v, ch, t, codebook, rank, c.st));
    if (g_inspect && budget) {
        InspectResult r;
        r.lam_B = g_ins_lamB;
        r.lam_final = lam;
        r.pre = chain;
        r.post.assign(t, 0);
        HIP_TRY(hipMemcpyAsync(r.post.data(), ch, sizeof(int32_t) * t, hipMemcpyDeviceToHost,
                               c.st));
        HIP_TRY(hipStreamSynchronize(c.st));
        g_ins_res.push_back(std::move(r));
    }
    double m[6];
    int32_t stt[2];
    HIP_TRY(hipMemcpyAsync(m, mres, sizeof m, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipMemcpyAsync(stt, stats, sizeof stt, hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    if (info) {
        std::memset(info, 0, sizeof *info);
        info->t = t;
        info->p = (int32_t)c.p;
        info->lambda = lam;
        info->mse = m[0];
        info->vnmse = m[1];
        info->entropy = m[2];
        info->entropy_surrogate = m[3];
        info->objective = m[4];
        info->rate_total = m[5];
        info->dp_solves = c.solves;
        info->refine_rounds_run = stt[0];
        info->cells = c.cells;
        info->status = status;
        info->search_passes = passes;
    }
    return status;
}

int32_t ws_flags(const ecasq_options& o) {
    return (o.recovery == 1 ? kWsArgmins : 0) | (o.dp_schedule == 1 ? kWsSweep : 0) |
           (o.alphabet != 0 ? kWsAlphabet : 0);
}

ecasq_options defaults() {
    ecasq_options o;
    o.refine_rounds = 5;
    o.refine_exhaustive = 0;
    o.exact_s = 0;
    o.max_search_passes = 32;
    o.search_width = 1;
    o.dp_schedule = 1;
    o.alphabet = 0;
    o.alphabet_size = 0;
    o.optimal_scan = 0;
    o.dp_objective = 0;
    o.recovery = 0;
    return o;
}

bool options_ok(const ecasq_options& o) {
    return o.refine_rounds >= 0 && o.refine_exhaustive >= 0 && o.refine_exhaustive <= 1 &&
           o.exact_s >= 0 && o.exact_s <= 1 && o.max_search_passes >= 1 && o.recovery >= 0 &&
           o.recovery <= 1 && (o.search_width == 1 || o.search_width == kMaxLambdas) &&
           o.dp_schedule >= 0 && o.dp_schedule <= 1 && o.alphabet >= 0 && o.alphabet <= 2 &&
           o.optimal_scan >= 0 && o.optimal_scan <= 1 && o.dp_objective >= 0 &&
           o.dp_objective <= 2;
}

// the grid size of a permissible alphabet must lie in [2, d]
bool alphabet_ok(const ecasq_options& o, int64_t d) {
    return o.alphabet == 0 || (o.alphabet_size >= 2 && o.alphabet_size <= d);
}

ecasq_status solve_budget(const void* x, int dt, int64_t d, int32_t s, double b,
                          const ecasq_options& o, void* stream, double* codebook, int32_t* rank,
                          ecasq_info* info, void* ws, size_t wsb) {
    Ctx c;
    ECASQ_TRY(ctx_open(c, d, s, ws_flags(o), stream, ws, wsb));
    struct Closer {
        Ctx& c;
        ~Closer() { ctx_close(c); }
    } closer{c};
    ECASQ_TRY(ctx_prep(c, x, dt, o.alphabet, o.alphabet_size));
    c.objective = o.dp_objective;
    c.opt_full = o.optimal_scan;
    c.refine_rounds = o.refine_rounds;
    c.refine_exhaustive = o.refine_exhaustive;
    c.recovery = o.recovery;
    std::vector<int32_t> chain;
    ecasq_status status = ECASQ_OK;
    double lam = 0.0;
    int32_t passes = 0;
    if (c.p <= 2) {
        for (int64_t k = 0; k < c.p; k++) chain.push_back((int32_t)k);
    } else {
        SearchResult R;
        ECASQ_TRY(search(c, b, o.exact_s, o.max_search_passes, o.search_width, R));
        status = R.status;
        lam = R.lam_final;
        passes = R.passes;
        if (!R.B.chain.empty())
            chain = R.B.chain;
        else
            ECASQ_TRY(recover(c, R.B.t, R.B.lam, o.exact_s, o.recovery, chain));
    }
    ecasq_options fo = o;
    if (o.dp_objective != 0) fo.refine_rounds = 0;  // the point as the search scored it
    ecasq_info local;
    if (!info) info = &local;
    ecasq_status st = finish(c, chain, lam, b, true, fo, codebook, rank, info, status, passes);
    if (c.p == 2 && (o.dp_objective != 0 ? info->entropy : info->entropy_surrogate) > b) {
        info->status = ECASQ_EINFEASIBLE;
        st = ECASQ_EINFEASIBLE;
    }
    return st;
}

ecasq_status solve_budgets(const void* x, int dt, int64_t d, int32_t s, int32_t nb,
                           const double* budgets, const ecasq_options& o, void* stream,
                           double* codebooks, int32_t* ranks, ecasq_info* infos) {
    Ctx c;
    ECASQ_TRY(ctx_open(c, d, s, ws_flags(o), stream, nullptr, 0));
    struct Closer {
        Ctx& c;
        ~Closer() { ctx_close(c); }
    } closer{c};
    ECASQ_TRY(ctx_prep(c, x, dt, o.alphabet, o.alphabet_size));
    c.objective = o.dp_objective;
    c.opt_full = o.optimal_scan;
    c.refine_rounds = o.refine_rounds;
    c.refine_exhaustive = o.refine_exhaustive;
    c.recovery = o.recovery;
    ecasq_options fo = o;
    if (o.dp_objective != 0) fo.refine_rounds = 0;
    ecasq_status worst = ECASQ_OK;
    for (int32_t k = 0; k < nb; k++) {
        const double b = budgets[k];
        c.cells = 0;
        c.solves = 0;
        std::vector<int32_t> chain;
        ecasq_status status = ECASQ_OK;
        double lam = 0.0;
        int32_t passes = 0;
        if (c.p <= 2) {
            for (int64_t q = 0; q < c.p; q++) chain.push_back((int32_t)q);
        } else {
            SearchResult R;
            ECASQ_TRY(search(c, b, o.exact_s, o.max_search_passes, o.search_width, R, k > 0));
            status = R.status;
            lam = R.lam_final;
            passes = R.passes;
            if (!R.B.chain.empty())
                chain = R.B.chain;
            else
                ECASQ_TRY(recover(c, R.B.t, R.B.lam, o.exact_s, o.recovery, chain));
        }
        ecasq_info* info = infos ? infos + k : nullptr;
        ecasq_info local;
        if (!info) info = &local;
        ecasq_status st = finish(c, chain, lam, b, true, fo, codebooks + (int64_t)k * s,
                                 ranks ? ranks + (int64_t)k * s : nullptr, info, status, passes);
        if (c.p == 2 && (o.dp_objective != 0 ? info->entropy : info->entropy_surrogate) > b) {
            info->status = ECASQ_EINFEASIBLE;
            st = ECASQ_EINFEASIBLE;
        }
        if (st == ECASQ_EINFEASIBLE)
            worst = ECASQ_EINFEASIBLE;
        else if (st != ECASQ_OK)
            return st;
    }
    return worst;
}

// Two-way time-sharing (Sec. 7): the search's final pair B (H <= b) and A
// (H > b) and the share alpha of entries on A with alpha H_A + (1-alpha) H_B = b.
ecasq_status solve_timeshare(const void* x, int dt, int64_t d, int32_t s, double b,
                             const ecasq_options& o, void* stream, double* codebooks,
                             int32_t* ranks, double* alpha_out, ecasq_info* infos) {
    Ctx c;
    ECASQ_TRY(ctx_open(c, d, s, ws_flags(o), stream, nullptr, 0));
    struct Closer {
        Ctx& c;
        ~Closer() { ctx_close(c); }
    } closer{c};
    ECASQ_TRY(ctx_prep(c, x, dt, o.alphabet, o.alphabet_size));
    c.objective = o.dp_objective;
    c.opt_full = o.optimal_scan;
    c.refine_rounds = o.refine_rounds;
    c.refine_exhaustive = o.refine_exhaustive;
    c.recovery = o.recovery;
    std::vector<int32_t> cm, cp;
    ecasq_status status = ECASQ_OK;
    double alpha = 0.0, lam_m = 0.0, lam_p = 0.0;
    int32_t passes = 0;
    if (c.p <= 2) {
        for (int64_t k = 0; k < c.p; k++) cm.push_back((int32_t)k);
        cp = cm;
    } else {
        SearchResult R;
        ECASQ_TRY(search(c, b, o.exact_s, o.max_search_passes, o.search_width, R));
        status = R.status;
        passes = R.passes;
        lam_m = lam_p = R.B.lam;
        if (!R.B.chain.empty())
            cm = R.B.chain;
        else
            ECASQ_TRY(recover(c, R.B.t, R.B.lam, o.exact_s, o.recovery, cm));
        cp = cm;
        if (status == ECASQ_OK && R.have_A) {
            alpha = (b - R.B.H) / (R.A.H - R.B.H);
            lam_p = R.A.lam;
            if (!R.A.chain.empty())
                cp = R.A.chain;
            else
                ECASQ_TRY(recover(c, R.A.t, R.A.lam, o.exact_s, o.recovery, cp));
        }
    }
    ecasq_options fo = o;
    fo.refine_rounds = 0;  // the supported points themselves
    ecasq_info local[2];
    ecasq_info* inf = infos ? infos : local;
    // finish returns the status it is given; only other codes are errors
    ecasq_status e = finish(c, cm, lam_m, b, true, fo, codebooks, ranks, inf, status, passes);
    if (e != status) return e;
    e = finish(c, cp, lam_p, b, true, fo, codebooks + s, ranks ? ranks + s : nullptr, inf + 1,
               status, passes);
    if (e != status) return e;
    if (c.p == 2 && (o.dp_objective != 0 ? inf[0].entropy : inf[0].entropy_surrogate) > b)
        status = ECASQ_EINFEASIBLE;
    inf[0].status = inf[1].status = status;
    if (alpha_out) *alpha_out = alpha;
    return status;
}

}  // namespace

extern "C" {

void ecasq_default_options(ecasq_options* opts) {
    if (opts) *opts = defaults();
}

size_t ecasq_workspace_size(int64_t d, int32_t s, int32_t flags) {
    if (d < 1 || s < 2 || flags < 0 || flags > 7) return 0;
    return layout(d, s, flags).total;
}

const char* ecasq_status_string(ecasq_status st) {
    switch (st) {
        case ECASQ_OK: return "ok";
        case ECASQ_EINVAL: return "invalid argument";
        case ECASQ_ENONFINITE: return "input holds NaN or Inf";
        case ECASQ_EINFEASIBLE: return "entropy budget below the smallest reachable surrogate entropy";
        case ECASQ_ENOMEM: return "device allocation failed";
        case ECASQ_EHIP: return "HIP runtime error";
        case ECASQ_EWORKSPACE: return "workspace too small";
    }
    return "unknown status";
}

ecasq_status ecasq_solve_ex(const void* x, ecasq_dtype dt, int64_t d, int32_t s,
                            double bits_per_entry, const ecasq_options* opts, void* stream,
                            double* codebook, int32_t* codebook_rank, ecasq_info* info,
                            void* workspace, size_t workspace_bytes) {
    ECASQ_TRY(check_x(x, dt, d));
    if (s < 2 || s > 255 || !codebook) return ECASQ_EINVAL;
    if (!(bits_per_entry >= 0.0)) return ECASQ_EINVAL;  // also rejects NaN
    const ecasq_options o = opts ? *opts : defaults();
    if (!options_ok(o) || !alphabet_ok(o, d)) return ECASQ_EINVAL;
    return solve_budget(x, dt, d, s, bits_per_entry, o, stream, codebook, codebook_rank, info,
                        workspace, workspace_bytes);
}

ecasq_status ecasq_solve(const void* x, ecasq_dtype dt, int64_t d, int32_t s,
                         double bits_per_entry, void* stream, double* codebook,
                         int32_t* codebook_rank, ecasq_info* info) {
    return ecasq_solve_ex(x, dt, d, s, bits_per_entry, nullptr, stream, codebook, codebook_rank,
                          info, nullptr, 0);
}

ecasq_status ecasq_solve_budgets(const void* x, ecasq_dtype dt, int64_t d, int32_t s, int32_t nb,
                                 const double* budgets, const ecasq_options* opts, void* stream,
                                 double* codebooks, int32_t* codebook_ranks, ecasq_info* infos) {
    ECASQ_TRY(check_x(x, dt, d));
    if (s < 2 || s > 255 || !codebooks || nb < 1 || !budgets) return ECASQ_EINVAL;
    for (int32_t k = 0; k < nb; k++)
        if (!(budgets[k] >= 0.0)) return ECASQ_EINVAL;  // also rejects NaN
    const ecasq_options o = opts ? *opts : defaults();
    if (!options_ok(o) || !alphabet_ok(o, d)) return ECASQ_EINVAL;
    return solve_budgets(x, dt, d, s, nb, budgets, o, stream, codebooks, codebook_ranks, infos);
}

ecasq_status ecasq_solve_lagrangian(const void* x, ecasq_dtype dt, int64_t d, int32_t s,
                                    double lambda, const ecasq_options* opts, void* stream,
                                    double* codebook, int32_t* codebook_rank, ecasq_info* info) {
    ECASQ_TRY(check_x(x, dt, d));
    if (s < 2 || s > 255 || !codebook || !(lambda >= 0.0) || !std::isfinite(lambda))
        return ECASQ_EINVAL;
    const ecasq_options o = opts ? *opts : defaults();
    if (!options_ok(o) || !alphabet_ok(o, d)) return ECASQ_EINVAL;
    Ctx c;
    ECASQ_TRY(ctx_open(c, d, s, ws_flags(o), stream, nullptr, 0));
    struct Closer {
        Ctx& c;
        ~Closer() { ctx_close(c); }
    } closer{c};
    ECASQ_TRY(ctx_prep(c, x, dt, o.alphabet, o.alphabet_size));
    std::vector<int32_t> chain;
    if (c.p == 1) {
        chain.assign(1, 0);
    } else {
        Point P;
        ECASQ_TRY(dp_solve1(c, lambda, o.exact_s, P));
        if (!P.chain.empty())
            chain = P.chain;
        else
            ECASQ_TRY(recover(c, P.t, lambda, o.exact_s, o.recovery, chain));
    }
    return finish(c, chain, lambda, HUGE_VAL, false, o, codebook, codebook_rank, info, ECASQ_OK,
                  0);
}


ecasq_status ecasq_solve_optimal(const void* x, ecasq_dtype dt, int64_t d, int32_t s,
                                 double lambda, const ecasq_options* opts, void* stream,
                                 double* codebook, int32_t* codebook_rank, ecasq_info* info) {
    ECASQ_TRY(check_x(x, dt, d));
    if (s < 2 || s > 255 || !codebook || !(lambda >= 0.0) || !std::isfinite(lambda))
        return ECASQ_EINVAL;
    const ecasq_options o = opts ? *opts : defaults();
    if (!options_ok(o) || !alphabet_ok(o, d)) return ECASQ_EINVAL;
    Ctx c;
    ECASQ_TRY(ctx_open(c, d, s, o.alphabet != 0 ? kWsAlphabet : 0, stream, nullptr, 0));
    struct Closer {
        Ctx& c;
        ~Closer() { ctx_close(c); }
    } closer{c};
    ECASQ_TRY(ctx_prep(c, x, dt, o.alphabet, o.alphabet_size));
    c.opt_full = o.optimal_scan;
    std::vector<int32_t> chain;
    double J = 0.0;
    ECASQ_TRY(opt_solve(c, lambda, o.exact_s, chain, &J, nullptr, nullptr));
    ecasq_options fo = o;
    fo.refine_rounds = 0;  // the optimum leaves nothing to refine
    return finish(c, chain, lambda, HUGE_VAL, false, fo, codebook, codebook_rank, info, ECASQ_OK,
                  0);
}

ecasq_status ecasq_opt_trace(const void* x, ecasq_dtype dt, int64_t d, int32_t s, double lambda,
                             const ecasq_options* opts, void* stream, int64_t capacity,
                             double* F, int32_t* K, int32_t* chain, double* out) {
    ECASQ_TRY(check_x(x, dt, d));
    if (s < 2 || s > 255 || !F || !K || !chain || !out || !(lambda >= 0.0) ||
        !std::isfinite(lambda))
        return ECASQ_EINVAL;
    const ecasq_options o = opts ? *opts : defaults();
    if (!options_ok(o) || !alphabet_ok(o, d)) return ECASQ_EINVAL;
    Ctx c;
    ECASQ_TRY(ctx_open(c, d, s, o.alphabet != 0 ? kWsAlphabet : 0, stream, nullptr, 0));
    struct Closer {
        Ctx& c;
        ~Closer() { ctx_close(c); }
    } closer{c};
    ECASQ_TRY(ctx_prep(c, x, dt, o.alphabet, o.alphabet_size));
    const int64_t imax = std::min<int64_t>(s, c.p);
    if (c.p > 1 && (imax + 1) * c.p * c.p > capacity) return ECASQ_EINVAL;
    c.opt_full = o.optimal_scan;
    std::vector<int32_t> ch;
    double J = 0.0;
    ECASQ_TRY(opt_solve(c, lambda, o.exact_s, ch, &J, c.p > 1 ? F : nullptr,
                        c.p > 1 ? K : nullptr));
    std::memcpy(chain, ch.data(), sizeof(int32_t) * ch.size());
    out[0] = J;
    out[1] = (double)ch.size();
    out[2] = (double)c.p;
    out[3] = (double)c.cells;
    return ECASQ_OK;
}

ecasq_status ecasq_solve_timeshare(const void* x, ecasq_dtype dt, int64_t d, int32_t s,
                                   double bits_per_entry, const ecasq_options* opts, void* stream,
                                   double* codebooks, int32_t* codebook_ranks, double* alpha,
                                   ecasq_info* infos) {
    ECASQ_TRY(check_x(x, dt, d));
    if (s < 2 || s > 255 || !codebooks || !alpha || !(bits_per_entry >= 0.0)) return ECASQ_EINVAL;
    const ecasq_options o = opts ? *opts : defaults();
    if (!options_ok(o) || !alphabet_ok(o, d)) return ECASQ_EINVAL;
    return solve_timeshare(x, dt, d, s, bits_per_entry, o, stream, codebooks, codebook_ranks,
                           alpha, infos);
}

ecasq_status ecasq_quantize_timeshare(const void* x, ecasq_dtype dt, int64_t d,
                                      const double* codebook0, int32_t t0,
                                      const double* codebook1, int32_t t1, double alpha,
                                      uint64_t seed, void* stream, uint8_t* symbols,
                                      uint8_t* part, double* empirical_entropy, int64_t* hist) {
    ECASQ_TRY(check_x(x, dt, d));
    if (!codebook0 || !codebook1 || t0 < 1 || t0 > 256 || t1 < 1 || t1 > 256 || !symbols ||
        !empirical_entropy || !(alpha >= 0.0 && alpha <= 1.0))
        return ECASQ_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    void* h = nullptr;
    const size_t hb = sizeof(unsigned long long) * 512;
    if (hipMallocAsync(&h, hb, st) != hipSuccess) return ECASQ_ENOMEM;
    unsigned long long* hh = static_cast<unsigned long long*>(h);
    ecasq_status rc = ECASQ_OK;
    if (hipMemsetAsync(hh, 0, hb, st) != hipSuccess ||
        launch_quantize_ts(x, dt, d, codebook0, t0, codebook1, t1, alpha, seed, symbols, part,
                           hh, empirical_entropy, hist, st) != hipSuccess)
        rc = ECASQ_EHIP;
    if (hipFreeAsync(h, st) != hipSuccess) rc = ECASQ_EHIP;
    return rc;
}

size_t ecasq_encode_bound(int64_t d, int32_t t) {
    if (d < 1 || d > ((int64_t)1 << 28) || t < 1 || t > 256) return 0;
    return rans_bound(d, t);
}

ecasq_status ecasq_encode(const uint8_t* symbols, int64_t d, int32_t t, void* stream,
                          uint8_t* out, size_t capacity, int64_t* out_bytes) {
    if (!symbols || !out || !out_bytes || d < 1 || d > ((int64_t)1 << 28) || t < 1 || t > 256)
        return ECASQ_EINVAL;
    if (capacity < rans_bound(d, t)) return ECASQ_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const size_t sb = rans_scratch_bytes(d);
    void* mem = nullptr;
    if (hipMallocAsync(&mem, sb + 512, st) != hipSuccess) return ECASQ_ENOMEM;
    char* base = static_cast<char*>(mem);
    auto* bad = reinterpret_cast<unsigned int*>(base + sb);
    auto* total = reinterpret_cast<unsigned long long*>(base + sb + 256);
    unsigned long long tot = 0;
    unsigned int nbad = 0;
    ecasq_status rc = ECASQ_OK;
    if (hipMemsetAsync(bad, 0, sizeof(unsigned int), st) != hipSuccess ||
        launch_rans_encode(symbols, d, t, out, base, total, bad, st) != hipSuccess ||
        hipMemcpyAsync(&tot, total, sizeof tot, hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipMemcpyAsync(&nbad, bad, sizeof nbad, hipMemcpyDeviceToHost, st) != hipSuccess)
        rc = ECASQ_EHIP;
    if (hipFreeAsync(mem, st) != hipSuccess) rc = ECASQ_EHIP;
    if (hipStreamSynchronize(st) != hipSuccess) rc = ECASQ_EHIP;
    if (rc != ECASQ_OK) return rc;
    if (nbad) return ECASQ_EINVAL;
    *out_bytes = 2 * (int64_t)t + 4 * rans_segments(d) + (int64_t)tot;
    return ECASQ_OK;
}

ecasq_status ecasq_decode(const uint8_t* in, int64_t in_bytes, int64_t d, int32_t t, void* stream,
                          uint8_t* symbols) {
    if (!in || !symbols || d < 1 || d > ((int64_t)1 << 28) || t < 1 || t > 256)
        return ECASQ_EINVAL;
    if (in_bytes < 2 * (int64_t)t + 4 * rans_segments(d)) return ECASQ_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    void* mem = nullptr;
    if (hipMallocAsync(&mem, 256, st) != hipSuccess) return ECASQ_ENOMEM;
    auto* bad = static_cast<unsigned int*>(mem);
    unsigned int nbad = 0;
    ecasq_status rc = ECASQ_OK;
    if (hipMemsetAsync(bad, 0, sizeof(unsigned int), st) != hipSuccess ||
        launch_rans_decode(in, in_bytes, d, t, symbols, bad, st) != hipSuccess ||
        hipMemcpyAsync(&nbad, bad, sizeof nbad, hipMemcpyDeviceToHost, st) != hipSuccess)
        rc = ECASQ_EHIP;
    if (hipFreeAsync(mem, st) != hipSuccess) rc = ECASQ_EHIP;
    if (hipStreamSynchronize(st) != hipSuccess) rc = ECASQ_EHIP;
    if (rc != ECASQ_OK) return rc;
    return nbad ? ECASQ_EINVAL : ECASQ_OK;
}

ecasq_status ecasq_quantize(const void* x, ecasq_dtype dt, int64_t d, const double* codebook,
                            int32_t t, uint64_t seed, void* stream, uint8_t* symbols,
                            double* empirical_entropy, int64_t* hist) {
    ECASQ_TRY(check_x(x, dt, d));
    if (!codebook || t < 1 || t > 256 || !symbols || !empirical_entropy) return ECASQ_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    void* h = nullptr;
    if (hipMallocAsync(&h, sizeof(unsigned long long) * 256, st) != hipSuccess)
        return ECASQ_ENOMEM;
    unsigned long long* hh = static_cast<unsigned long long*>(h);
    ecasq_status rc = ECASQ_OK;
    if (hipMemsetAsync(hh, 0, sizeof(unsigned long long) * 256, st) != hipSuccess ||
        launch_quantize(x, dt, d, codebook, t, seed, symbols, hh, st) != hipSuccess ||
        launch_entropy(hh, t, d, empirical_entropy, hist, st) != hipSuccess)
        rc = ECASQ_EHIP;
    if (hipFreeAsync(h, st) != hipSuccess) rc = ECASQ_EHIP;
    return rc;
}

ecasq_status ecasq_quantize_noalloc(const void* x, ecasq_dtype dt, int64_t d,
                                    const double* codebook, int32_t t, uint64_t seed,
                                    void* stream, uint8_t* symbols, double* empirical_entropy,
                                    int64_t* hist) {
    ECASQ_TRY(check_x(x, dt, d));
    if (!codebook || t < 1 || t > 256 || !symbols || !empirical_entropy) return ECASQ_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    unsigned long long* hh = nullptr;
    HIP_TRY(quantize_scratch(&hh));
    HIP_TRY(launch_zero_counts(hh, t, st));
    HIP_TRY(launch_quantize(x, dt, d, codebook, t, seed, symbols, hh, st));
    HIP_TRY(launch_entropy(hh, t, d, empirical_entropy, hist, st));
    return ECASQ_OK;
}

ecasq_status ecasq_histogram(const void* x, ecasq_dtype dt, int64_t d, void* stream, double* v,
                             double* N, double* S, double* S2, int64_t* p_out) {
    ECASQ_TRY(check_x(x, dt, d));
    if (!v || !N || !S || !S2 || !p_out) return ECASQ_EINVAL;
    Ctx c;
    ECASQ_TRY(ctx_open(c, d, 2, 0, stream, nullptr, 0));
    struct Closer {
        Ctx& c;
        ~Closer() { ctx_close(c); }
    } closer{c};
    ECASQ_TRY(ctx_prep(c, x, dt));
    const size_t nb = sizeof(double) * (size_t)c.p;
    HIP_TRY(hipMemcpyAsync(v, c.H.v, nb, hipMemcpyDeviceToDevice, c.st));
    HIP_TRY(hipMemcpyAsync(N, c.H.N, nb, hipMemcpyDeviceToDevice, c.st));
    HIP_TRY(hipMemcpyAsync(S, c.H.S, nb, hipMemcpyDeviceToDevice, c.st));
    HIP_TRY(hipMemcpyAsync(S2, c.H.S2, nb, hipMemcpyDeviceToDevice, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    *p_out = c.p;
    return ECASQ_OK;
}

ecasq_status ecasq_dp_trace(const void* x, ecasq_dtype dt, int64_t d, int32_t s, int32_t nlam,
                            const double* lambdas, int32_t schedule, void* stream, double* F,
                            int32_t* kstar, double* M, double* Ph, double* out) {
    ECASQ_TRY(check_x(x, dt, d));
    if (s < 2 || s > 255 || !F || !out || !lambdas) return ECASQ_EINVAL;
    if (nlam != 1 && nlam != kMaxLambdas) return ECASQ_EINVAL;
    if (schedule < 0 || schedule > 1 || ((M == nullptr) != (Ph == nullptr))) return ECASQ_EINVAL;
    // argmins may be left out under schedule 1 (values only), not with accumulators
    if (!kstar && (schedule == 0 || M)) return ECASQ_EINVAL;
    for (int32_t m = 0; m < nlam; m++)
        if (!(lambdas[m] >= 0.0) || !std::isfinite(lambdas[m])) return ECASQ_EINVAL;
    Ctx c;
    const int32_t flags = schedule == 1 ? (kWsSweep | (kstar || M ? kWsSweepArgmins : 0)) : 0;
    ECASQ_TRY(ctx_open(c, d, s, flags, stream, nullptr, 0));
    struct Closer {
        Ctx& c;
        ~Closer() { ctx_close(c); }
    } closer{c};
    ECASQ_TRY(ctx_prep(c, x, dt));
    if (c.p < 2) return ECASQ_EINVAL;
    Point P[kMaxLambdas];
    double J[4 * kMaxLambdas];
    Dumps dk;
    dk.F = F;
    dk.K = kstar;
    dk.M = M;
    dk.P = Ph;
    dk.stride = d;
    const int64_t cells0 = c.cells;
    ECASQ_TRY(dp_solve(c, lambdas, nlam, 0, P, J, &dk));
    const double per = (double)((c.cells - cells0) / nlam);
    for (int32_t m = 0; m < nlam; m++) {
        for (int q = 0; q < 4; q++) out[5 * m + q] = J[4 * m + q];
        out[5 * m + 4] = per;
    }
    return ECASQ_OK;
}

void ecasq_inspect_enable(int32_t on) {
    g_inspect = on != 0;
    g_ins_pts.clear();
    g_ins_res.clear();
}

int32_t ecasq_inspect_points(double* out, int32_t cap) {
    const int32_t n = (int32_t)(g_ins_pts.size() / 4);
    if (!out) return n;  // a size query
    std::memcpy(out, g_ins_pts.data(), sizeof(double) * 4 * (size_t)std::max(0, std::min(n, cap)));
    g_ins_pts.clear();
    return n;
}

int32_t ecasq_inspect_results(double* lams, int32_t* chains, int32_t cap) {
    const int32_t n = (int32_t)g_ins_res.size();
    if (!lams && !chains) return n;  // a size query
    for (int32_t k = 0; k < n && k < cap; k++) {
        const InspectResult& r = g_ins_res[k];
        if (lams) {
            lams[2 * k] = r.lam_B;
            lams[2 * k + 1] = r.lam_final;
        }
        if (chains) {
            int32_t* row = chains + (int64_t)k * 2 * 257;
            row[0] = (int32_t)r.pre.size();
            std::memcpy(row + 1, r.pre.data(), sizeof(int32_t) * r.pre.size());
            row[257] = (int32_t)r.post.size();
            std::memcpy(row + 258, r.post.data(), sizeof(int32_t) * r.post.size());
        }
    }
    g_ins_res.clear();
    return n;
}

void ecasq_timing_enable(int32_t on) { timing_enable(on == 2 ? 2 : (on != 0 ? 1 : 0)); }

void ecasq_timing_read(int32_t variant, double* layer_ms, int64_t* layer_launches,
                       int64_t* layer_cells, int32_t reset) {
    timing_read(variant, layer_ms, layer_launches, layer_cells, reset != 0);
}

ecasq_status ecasq_solve_batched(const void* x, ecasq_dtype dt, int64_t n, int64_t d, int32_t s,
                                 double bits_per_entry, const ecasq_options* opts, void* stream,
                                 double* codebooks, int32_t* t_out, ecasq_info* infos_dev) {
    if (!x || n < 1 || d < 1 || d > 512 || s < 2 || s > 32 || !codebooks || !t_out)
        return ECASQ_EINVAL;
    if (dt < 0 || dt > 2 || !(bits_per_entry >= 0.0)) return ECASQ_EINVAL;
    const ecasq_options o = opts ? *opts : defaults();
    if (o.refine_rounds < 0 || o.max_search_passes < 1) return ECASQ_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    timing_begin(kTimingBatched, 0, st);
    HIP_TRY(launch_batched(x, dt, n, (int32_t)d, s, bits_per_entry, o.refine_rounds,
                           o.refine_exhaustive, o.exact_s, o.max_search_passes, codebooks, t_out,
                           infos_dev, st));
    timing_end(st);
    HIP_TRY(hipStreamSynchronize(st));
    timing_flush();
    return ECASQ_OK;
}

}  // extern "C"
