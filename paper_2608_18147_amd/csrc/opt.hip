// Optimal lambda-ECASQ (Sec. 4; App. D closed forms): the DP over states
// (i, l, j) whose entry is the best cost of the values up to v_l with i-1
// codebook values ending at v_l, plus the MSE of (v_l, v_j] with v_l and v_j
// adjacent.  Knowing the neighbours k < l < j of v_l fixes its expected
// frequency U[k,l] + D[l,j], so the output entropy H(Xhat) is exact:
//
//   layer 2 (l = 0):  dp(2,0,j) = C[0,j] + lambda' h(n_0/d + D[0,j]/d)
//   layer i >= 3:     dp(i,l,j) = C[l,j] + min_k dp(i-1,k,l) + lambda' h(U[k,l]/d + D[l,j]/d)
//                     (k = 0 for i = 3, i-3 <= k < l otherwise; l in [i-2, p-2])
//   answer:           min over i, then l, of dp(i,l,p-1) + lambda' h(U[l,p-1]/d)
//
// with the lowest index winning every tie.  Arithmetic: U/d and D/d in the
// g form of the approximate DP's cell (yu = tu * RN(1/(w d)), yd = td * ...),
// e(y) = m log2c(m) with m = max(y, 0), so that lambda' h(y) = -lambda' e(y):
//   layer 2   fma(-lambda', e(yd(0,j) + c0/d), C[0,j])
//   T(k)      fma(-lambda', e(yu(k,l) + yd(l,j)), dp(i-1,k,l))
//   dp        C[l,j] + min_k T(k)
//   final     fma(-lambda', e(yu(l,p-1)), dp(i,l,p-1))
//
// A layer is one launch, one workgroup per row l (heaviest rows first).  The
// predecessor terms of row l, dp(i-1,k,l) and yu(k,l), are contiguous in k
// (layers are stored transposed, D[j][l], and yu once per solve as YU[l][k]),
// so the scan over k reads wave-uniform addresses while the 64 lanes of a
// wavefront hold 64 columns j.
//
// Two scans of k:
//   every predecessor (the definition);
//   monotone brackets (the SMAWK acceleration of Sec. 4.1): for fixed i and l
//   the matrix T(k, j) with its columns reversed is Monge (Lemma
//   quadrangleM), so the lowest minimiser k*(j) does not increase with j.
//   The columns are cut into segments of 64 (one wavefront).  k* of the
//   segment ends is found coarse to fine, each end scanning the bracket
//   left by the ends resolved before it (one wavefront per end, its lanes
//   splitting k); a segment's columns then scan only [k*(its end), k*(the
//   previous end)].  With n_seg = (p - 1 - l) / 64 segments the work per
//   row drops from n_seg (l - k_lo) wavefront-steps to about
//   (1 + log2(n_seg) / 64) (l - k_lo) + a few steps per end.  Where
//   rounding breaks the monotone order of two near-equal candidates, a
//   bracket can miss a minimiser that is better by a rounding error only.
#include "device.hpp"
#include "launch.hpp"

namespace ecasq {

namespace {

constexpr int kOT = 256;   // threads per workgroup of the table kernels
// wavefronts per row of the layer kernel: 4 for the full scan; 2 for the
// monotone brackets (rows with few segments leave fewer of them idle, and
// more rows share a CU)
#ifndef ECASQ_OPT_ROW_WAVES
#define ECASQ_OPT_ROW_WAVES 2
#endif
template <bool FULL>
constexpr int row_waves() { return FULL ? 4 : ECASQ_OPT_ROW_WAVES; }
constexpr int kSeg = 64;   // columns per segment (one wavefront)
constexpr int kMaxSeg = (int)(kOptMaxP / kSeg) + 1;

struct OptLayerArgs {
    Hist H;
    const double* YU;  // [l][k] = yu(k, l), k < l
    const double* Dp;  // layer i-1: Dp[l * p + k] = dp(i-1, k, l)
    double* Dc;        // layer i:   Dc[j * p + l] = dp(i, l, j)
    void* K;           // layer i argmins, [l][j], int16 (p <= 32768) or int32
    double* fin;       // layer i final values, per l
    double lamp;       // lambda' (MSE units)
    int64_t p;
    int32_t i;
    int32_t wide;
};

__device__ __forceinline__ double elog(double y, const double2* __restrict__ tab) {
    const double m = __builtin_fmax(y, 0.0);
    return m * log2c(m, tab);
}

// C[a,b], yu = U[a,b]/d and yd = D[a,b]/d of (v_a, v_b] (App. D closed forms).
__device__ __forceinline__ void interval_y(const Hist& H, int64_t a, int64_t b, double& C,
                                           double& yu, double& yd) {
    const double va = H.v[a], vb = H.v[b];
    const double n = H.N[b] - H.N[a];
    const double sa = H.S[b] - H.S[a];
    const double s2 = H.S2[b] - H.S2[a];
    const double w = vb - va;
    const double tu = __builtin_fma(-va, n, sa);
    const double td = __builtin_fma(vb, n, -sa);
    C = __builtin_fma(vb, tu, __builtin_fma(va, sa, -s2));
    const double g = recip_rn(w * H.dd);
    yu = tu * g;
    yd = td * g;
}

// Candidates k = k0..k1 in increasing order; strict '<' keeps the lowest k.
// A and Y are read at wave-uniform addresses, eight predecessors per step.
__device__ __forceinline__ void scan(const double* __restrict__ A, const double* __restrict__ Y,
                                     int64_t k0, int64_t k1, double yd, double lamp,
                                     const double2* __restrict__ tab, double& best,
                                     int32_t& kb) {
    int64_t k = k0;
    for (; k + 7 <= k1; k += 8) {
        double a8[8], y8[8];
#pragma unroll
        for (int u = 0; u < 8; u++) {
            a8[u] = A[k + u];
            y8[u] = Y[k + u];
        }
#pragma unroll
        for (int u = 0; u < 8; u++) {
            const double T = __builtin_fma(-lamp, elog(y8[u] + yd, tab), a8[u]);
            const bool lt = T < best;
            kb = lt ? (int32_t)(k + u) : kb;
            best = lt ? T : best;
        }
    }
    for (; k <= k1; k++) {
        const double T = __builtin_fma(-lamp, elog(Y[k] + yd, tab), A[k]);
        const bool lt = T < best;
        kb = lt ? (int32_t)k : kb;
        best = lt ? T : best;
    }
}

// Candidates k = k0, k0 + 64, ... <= k1 (one lane's share of a wavefront's
// scan), strict '<' keeping the lowest k of this lane.
__device__ __forceinline__ void scan_strided(const double* __restrict__ A,
                                             const double* __restrict__ Y, int64_t k0,
                                             int64_t k1, double yd, double lamp,
                                             const double2* __restrict__ tab, double& best,
                                             int32_t& kb) {
    int64_t k = k0;
    for (; k + 3 * kSeg <= k1; k += 4 * kSeg) {
        double a4[4], y4[4];
#pragma unroll
        for (int u = 0; u < 4; u++) {
            a4[u] = A[k + u * kSeg];
            y4[u] = Y[k + u * kSeg];
        }
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const double T = __builtin_fma(-lamp, elog(y4[u] + yd, tab), a4[u]);
            const bool lt = T < best;
            kb = lt ? (int32_t)(k + u * kSeg) : kb;
            best = lt ? T : best;
        }
    }
    for (; k <= k1; k += kSeg) {
        const double T = __builtin_fma(-lamp, elog(Y[k] + yd, tab), A[k]);
        const bool lt = T < best;
        kb = lt ? (int32_t)k : kb;
        best = lt ? T : best;
    }
}

__device__ __forceinline__ void emit(const OptLayerArgs& a, int64_t l, int64_t j, double C,
                                     double yu, double best, int32_t kb,
                                     const double2* __restrict__ tab) {
    const int64_t p = a.p;
    const double v = C + best;
    a.Dc[j * p + l] = v;
    if (a.wide)
        static_cast<int32_t*>(a.K)[l * p + j] = kb;
    else
        static_cast<int16_t*>(a.K)[l * p + j] = (int16_t)kb;
    if (j == p - 1) a.fin[l] = __builtin_fma(-a.lamp, elog(yu, tab), v);
}

__global__ __launch_bounds__(kOT) void k_opt_yu(Hist H, double* __restrict__ YU) {
    const int64_t p = H.p;
    const int64_t l = (int64_t)blockIdx.x + 1;
    for (int64_t k = threadIdx.x; k < l; k += kOT) {
        double C, yu, yd;
        interval_y(H, k, l, C, yu, yd);
        YU[l * p + k] = yu;
    }
}

__global__ __launch_bounds__(kOT) void k_opt_layer2(Hist H, double* __restrict__ Dc,
                                                    double* __restrict__ fin, double lamp) {
    __shared__ double2 tab[kLog2Size];
    load_log2_table(tab);
    __syncthreads();
    const int64_t p = H.p;
    const int64_t j = 1 + (int64_t)blockIdx.x * kOT + threadIdx.x;
    if (j >= p) return;
    double C, yu, yd;
    interval_y(H, 0, j, C, yu, yd);
    const double v = __builtin_fma(-lamp, elog(yd + H.c0d, tab), C);
    Dc[j * p] = v;
    if (j == p - 1) fin[0] = __builtin_fma(-lamp, elog(yu, tab), v);
}

template <bool FULL>
__global__ __launch_bounds__(row_waves<FULL>() * 64) void k_opt_layer(OptLayerArgs a) {
    constexpr int kRW = row_waves<FULL>();
    constexpr int kRT = kRW * 64;  // threads of the row's workgroup
    __shared__ double2 tab[kLog2Size];
    __shared__ int32_t kst[FULL ? 1 : kMaxSeg + 1];
    const int tid = threadIdx.x, lane = tid & (kSeg - 1), w = tid >> 6;
    const int64_t p = a.p;
    const int64_t l = p - 2 - (int64_t)blockIdx.x;  // heaviest rows first
    load_log2_table(tab);
    __syncthreads();
    const int64_t klo = a.i == 3 ? 0 : a.i - 3;
    const int64_t khi = a.i == 3 ? 0 : l - 1;
    const double* A = a.Dp + l * p;
    const double* Y = a.YU + l * p;
    if (FULL) {
        for (int64_t j0 = l + 1; j0 < p; j0 += kRT) {
            const int64_t j = j0 + tid;
            const bool ok = j < p;
            double C = 0.0, yu = 0.0, yd = 0.0;
            if (ok) interval_y(a.H, l, j, C, yu, yd);
            double best = HUGE_VAL;
            int32_t kb = -1;
            scan(A, Y, klo, khi, yd, a.lamp, tab, best, kb);
            if (ok) emit(a, l, j, C, yu, best, kb, tab);
        }
        return;
    }
    const int64_t nseg = (p - 1 - l + kSeg - 1) / kSeg;
    // k* at the segment ends e_q = min(l + 64 (q+1), p-1), kept as kst[q+1]
    // with kst[0] = k_hi.  They do not increase with q, so they are resolved
    // coarse to fine: at stride S the ends r = S, 3S, 5S, ... (r = q+1) scan
    // only [k*(r+S), k*(r-S)] (k_lo past the last end), both resolved at a
    // coarser stride.  One wavefront per end (the stride's ends dealt to the
    // four in turn): its lanes split k and a butterfly over (T, k) keeps the
    // lowest k of the minimum, as a scan in increasing k with strict '<' does.
    int64_t S = 1;
    while (S <= nseg) S <<= 1;
    if (tid == 0) kst[0] = (int32_t)khi;
    __syncthreads();
    for (S >>= 1; S >= 1; S >>= 1) {
        const int64_t nends = (nseg / S + 1) / 2;  // odd multiples of S up to nseg
        for (int64_t m = w; m < nends; m += kRW) {
            const int64_t r = (2 * m + 1) * S;
            const int64_t kB = kst[r - S];
            const int64_t kA = r + S <= nseg ? (int64_t)kst[r + S] : klo;
            const int64_t e = min(l + kSeg * r, p - 1);
            double C, yu, yd;
            interval_y(a.H, l, e, C, yu, yd);
            double best = HUGE_VAL;
            int32_t kb = -1;
            scan_strided(A, Y, kA + lane, kB, yd, a.lamp, tab, best, kb);
#pragma unroll
            for (int off = kSeg / 2; off > 0; off >>= 1) {
                const double ob = __shfl_xor(best, off);
                const int32_t okb = __shfl_xor(kb, off);
                if (ob < best || (ob == best && okb < kb)) {
                    best = ob;
                    kb = okb;
                }
            }
            // no finite candidate (not reached for finite inputs): keep the
            // bracket's low end so later brackets stay inside [k_lo, k_hi]
            if (lane == 0) kst[r] = kb < 0 ? (int32_t)kA : kb;
        }
        __syncthreads();
    }
    // each segment's columns scan between the minimisers of its end and of
    // the previous segment's end
    for (int64_t q = w; q < nseg; q += kRW) {
        const int64_t k0 = kst[q + 1], k1 = kst[q];
        const int64_t j = l + 1 + kSeg * q + lane;
        const bool ok = j < p;
        double C = 0.0, yu = 0.0, yd = 0.0;
        if (ok) interval_y(a.H, l, j, C, yu, yd);
        double best = HUGE_VAL;
        int32_t kb = -1;
        scan(A, Y, k0, k1, yd, a.lamp, tab, best, kb);
        if (ok) emit(a, l, j, C, yu, best, kb, tab);
    }
}

// The answer over the final values of every layer (or layer imax only),
// lowest (i, l) among ties, and the traceback through the stored argmins.
constexpr int kFT = 1024;

__global__ __launch_bounds__(kFT) void k_opt_final(const double* __restrict__ fin, int64_t p,
                                                   int32_t imax, int32_t exact_s,
                                                   const void* __restrict__ K, int32_t wide,
                                                   int32_t* __restrict__ chain,
                                                   double* __restrict__ res) {
    __shared__ double sb[kFT];
    __shared__ int64_t sp[kFT];
    const int tid = threadIdx.x;
    double best = HUGE_VAL;
    int64_t bpos = INT64_MAX;
    for (int32_t i = exact_s ? imax : 2; i <= imax; i++) {
        const int64_t lo = i == 2 ? 0 : i - 2, hi = i == 2 ? 0 : p - 2;
        for (int64_t l = lo + tid; l <= hi; l += kFT) {
            const double f = fin[(int64_t)i * p + l];
            if (f < best) {
                best = f;
                bpos = (int64_t)i * p + l;
            }
        }
    }
    sb[tid] = best;
    sp[tid] = bpos;
    __syncthreads();
    for (int off = kFT / 2; off > 0; off >>= 1) {
        if (tid < off) {
            const double o = sb[tid + off];
            const int64_t op = sp[tid + off];
            if (o < sb[tid] || (o == sb[tid] && op < sp[tid])) {
                sb[tid] = o;
                sp[tid] = op;
            }
        }
        __syncthreads();
    }
    if (tid != 0) return;
    const int64_t pos = sp[0];
    if (pos == INT64_MAX) {  // no finite final value: reported as t = 0
        res[0] = sb[0];
        res[1] = 0.0;
        return;
    }
    const int32_t t = (int32_t)(pos / p);
    int64_t l = pos % p, j = p - 1;
    chain[t - 1] = (int32_t)(p - 1);
    chain[t - 2] = (int32_t)l;
    const int64_t pp = p * p;
    for (int32_t i = t; i >= 3; i--) {
        const int64_t at = (int64_t)(i - 3) * pp + l * p + j;
        const int64_t k = wide ? static_cast<const int32_t*>(K)[at]
                               : static_cast<const int16_t*>(K)[at];
        chain[i - 3] = (int32_t)k;
        j = l;
        l = k;
    }
    res[0] = sb[0];
    res[1] = (double)t;
}

struct OptLayout {
    size_t YU, D0, D1, fin, K, total;
    int32_t wide;
};

OptLayout opt_layout(int64_t p, int32_t imax, bool wide) {
    OptLayout L;
    const size_t pp = (size_t)p * (size_t)p;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align256(bytes);
        return at;
    };
    L.wide = (wide || p > 32768) ? 1 : 0;
    L.YU = take(sizeof(double) * pp);
    L.D0 = take(sizeof(double) * pp);
    L.D1 = take(sizeof(double) * pp);
    L.fin = take(sizeof(double) * (size_t)(imax + 1) * (size_t)p);
    L.K = take((L.wide ? 4 : 2) * pp * (size_t)(imax > 2 ? imax - 2 : 0));
    L.total = o;
    return L;
}

}  // namespace

size_t opt_workspace_bytes(int64_t p, int32_t imax, bool trace) {
    return opt_layout(p, imax, trace).total;
}

int64_t opt_cells(int64_t p, int32_t imax, int32_t exact_s) {
    int64_t cells = p - 1;  // layer 2
    for (int64_t i = 2; i <= imax; i++) {
        if (i >= 3) {
            for (int64_t l = i - 2; l <= p - 2; l++) {
                const int64_t nk = i == 3 ? 1 : l - (i - 3);
                cells += nk * (p - 1 - l);
            }
        }
        if (!exact_s || i == imax) cells += i == 2 ? 1 : p - 1 - (i - 2);
    }
    return cells;
}

hipError_t launch_opt(const Hist& H, int32_t imax, int32_t exact_s, double lamp, int32_t full,
                      char* mem, int32_t* chain, double* res, double* Ftrace, int32_t* Ktrace,
                      hipStream_t st) {
    const int64_t p = H.p;
    if (p < 2 || p > kOptMaxP || imax < 2 || imax > p) return hipErrorInvalidValue;
    const OptLayout L = opt_layout(p, imax, Ktrace != nullptr);
    const size_t pp = (size_t)p * (size_t)p;
    double* YU = reinterpret_cast<double*>(mem + L.YU);
    double* D[2] = {reinterpret_cast<double*>(mem + L.D0), reinterpret_cast<double*>(mem + L.D1)};
    double* fin = reinterpret_cast<double*>(mem + L.fin);
    char* K = mem + L.K;
    const size_t ksz = L.wide ? 4 : 2;
    k_opt_yu<<<dim3((unsigned)(p - 1)), dim3(kOT), 0, st>>>(H, YU);
    k_opt_layer2<<<dim3((unsigned)((p - 1 + kOT - 1) / kOT)), dim3(kOT), 0, st>>>(
        H, D[0], fin + 2 * p, lamp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (Ftrace) {
        e = hipMemcpyAsync(Ftrace + 2 * pp, D[0], sizeof(double) * pp, hipMemcpyDeviceToDevice, st);
        if (e != hipSuccess) return e;
    }
    for (int32_t i = 3; i <= imax; i++) {
        OptLayerArgs a;
        a.H = H;
        a.YU = YU;
        a.Dp = D[(i - 3) & 1];
        a.Dc = D[(i - 2) & 1];
        a.K = K + (size_t)(i - 3) * pp * ksz;
        a.fin = fin + (size_t)i * (size_t)p;
        a.lamp = lamp;
        a.p = p;
        a.i = i;
        a.wide = L.wide;
        const unsigned rows = (unsigned)(p - 1 - (i - 2));
        int64_t cells = 0;
        if (timing_active()) {
            for (int64_t l = i - 2; l <= p - 2; l++)
                cells += (i == 3 ? 1 : l - (i - 3)) * (p - 1 - l);
        }
        timing_begin(kTimingOpt, cells, st);
        if (full)
            k_opt_layer<true><<<dim3(rows), dim3(row_waves<true>() * 64), 0, st>>>(a);
        else
            k_opt_layer<false><<<dim3(rows), dim3(row_waves<false>() * 64), 0, st>>>(a);
        timing_end(st);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (Ftrace) {
            e = hipMemcpyAsync(Ftrace + (size_t)i * pp, a.Dc, sizeof(double) * pp,
                               hipMemcpyDeviceToDevice, st);
            if (e != hipSuccess) return e;
        }
        if (Ktrace) {
            e = hipMemcpyAsync(Ktrace + (size_t)i * pp, a.K, sizeof(int32_t) * pp,
                               hipMemcpyDeviceToDevice, st);
            if (e != hipSuccess) return e;
        }
    }
    k_opt_final<<<dim3(1), dim3(kFT), 0, st>>>(fin, p, imax, exact_s, K, L.wide, chain, res);
    return hipGetLastError();
}

}  // namespace ecasq
