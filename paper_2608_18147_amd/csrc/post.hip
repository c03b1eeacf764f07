// Steps after the DP: three-colour refinement (Sec. 6), solution metrics,
// codebook gather, and the final unbiased stochastic rounding (Sec. 2) with
// a plug-in entropy of the symbol histogram.
#include <hip/hip_fp16.h>

#include <mutex>

#include "chain.hpp"
#include "device.hpp"
#include "launch.hpp"

namespace ecasq {

namespace {

constexpr int kMaxT = 256;

// The whole refinement in one block: rounds of colour substeps 0, 1, 2.  All
// movers of a colour are independent (their objectives share no frequency)
// and are searched in parallel, one thread each; a substep whose result
// violates the budget (budget mode) is undone; refinement stops after a round
// without a committed move.  stats: rounds run, moves committed.
__global__ __launch_bounds__(256) void k_refine(Hist H, int32_t t, int32_t* __restrict__ ug,
                                                double lamp, double b, int32_t budget,
                                                int32_t rounds, int32_t exhaustive,
                                                int32_t* __restrict__ stats) {
    __shared__ double2 tab[kLog2Size];
    __shared__ int32_t u[kMaxT], nu[kMaxT];
    __shared__ int32_t moved_s, commit_s;
    __shared__ double redv[256];
    __shared__ int64_t redi[256];
    const int tid = threadIdx.x;
    load_log2_table(tab);
    for (int r = tid; r < t; r += blockDim.x) u[r] = ug[r];
    __syncthreads();
    int32_t nrun = 0, nmoves = 0;
    for (int32_t rd = 0; rd < rounds; rd++) {
        int any = 0;
        for (int32_t c = 0; c < 3; c++) {
            for (int r = tid; r < t; r += blockDim.x) nu[r] = u[r];
            if (tid == 0) moved_s = 0;
            __syncthreads();
            if (!exhaustive) {
                for (int32_t r = 1 + tid; r <= t - 2; r += blockDim.x) {
                    if (r % 3 != c) continue;
                    const int64_t L = u[r - 1], R = u[r + 1];
                    if (R - L < 3) continue;
                    int64_t lo = L + 1, hi = R - 1;
                    while (lo < hi) {
                        const int64_t mid = lo + (hi - lo) / 2;
                        if (refine_local(H, t, u, r, mid + 1, lamp, tab) <
                            refine_local(H, t, u, r, mid, lamp, tab))
                            lo = mid + 1;
                        else
                            hi = mid;
                    }
                    if (lo != u[r] && refine_local(H, t, u, r, lo, lamp, tab) <
                                          refine_local(H, t, u, r, u[r], lamp, tab)) {
                        nu[r] = (int32_t)lo;
                        atomicAdd(&moved_s, 1);
                    }
                }
            } else {
                for (int32_t r = 1; r <= t - 2; r++) {
                    if (r % 3 != c) continue;
                    const int64_t L = u[r - 1], R = u[r + 1];
                    if (R - L < 3) continue;
                    double bv = __builtin_huge_val();
                    int64_t bm = -1;
                    for (int64_t m = L + 1 + tid; m < R; m += blockDim.x) {
                        const double val = refine_local(H, t, u, r, m, lamp, tab);
                        if (val < bv) {
                            bv = val;
                            bm = m;
                        }
                    }
                    redv[tid] = bv;
                    redi[tid] = bm;
                    __syncthreads();
                    for (int off = blockDim.x / 2; off > 0; off >>= 1) {
                        if (tid < off) {
                            const double ov = redv[tid + off];
                            const int64_t oi = redi[tid + off];
                            if (oi >= 0 && (redi[tid] < 0 || ov < redv[tid] ||
                                            (ov == redv[tid] && oi < redi[tid]))) {
                                redv[tid] = ov;
                                redi[tid] = oi;
                            }
                        }
                        __syncthreads();
                    }
                    if (tid == 0) {
                        const int64_t m = redi[0];
                        if (m != u[r] &&
                            redv[0] < refine_local(H, t, u, r, u[r], lamp, tab)) {
                            nu[r] = (int32_t)m;
                            moved_s += 1;
                        }
                    }
                    __syncthreads();
                }
            }
            __syncthreads();
            if (tid == 0) {
                int32_t moved = moved_s;
                if (moved && budget && chain_hout(H, t, nu, tab) > b) moved = 0;
                commit_s = moved;
            }
            __syncthreads();
            const int32_t moved = commit_s;
            if (moved) {
                for (int r = tid; r < t; r += blockDim.x) u[r] = nu[r];
                any = 1;
                nmoves += moved;
            }
            __syncthreads();
        }
        nrun++;
        if (!any) break;
    }
    for (int r = tid; r < t; r += blockDim.x) ug[r] = u[r];
    if (tid == 0) {
        stats[0] = nrun;
        stats[1] = nmoves;
    }
}

// out: MSE, vNMSE, H(Xhat), H(I,B), vNMSE + lambda H(Xhat), H(Xhat) + 32t/d.
// The interval terms and the values' entropy terms are formed one per
// thread; one thread then sums them in index order (the sums of the chain
// walk in chain_hout and of the path accumulators, bit for bit).
__global__ void k_metrics(Hist H, int32_t t, const int32_t* __restrict__ u, double lam,
                          double s2tot, double* __restrict__ out) {
    __shared__ double2 tab[kLog2Size];
    __shared__ double sC[kMaxT], sP[kMaxT], sU[kMaxT], sD[kMaxT], sh[kMaxT];
    load_log2_table(tab);
    __syncthreads();
    for (int32_t r = threadIdx.x; r + 1 < t; r += blockDim.x) {
        double C, P, U, D;
        cell_at(H, u[r], u[r + 1], tab, C, P);
        ud_at(H, u[r], u[r + 1], U, D);
        sC[r] = C;
        sP[r] = P;
        sU[r] = U;
        sD[r] = D;
    }
    __syncthreads();
    // expected frequency of value q (as chain_hout forms it), then h(f / d)
    for (int32_t q = threadIdx.x; q < t; q += blockDim.x) {
        double f;
        if (t == 1) f = H.dd;
        else if (q == 0) f = H.c0 + sD[0];
        else if (q == t - 1) f = sU[t - 2];
        else f = sU[q - 1] + sD[q];
        sh[q] = hf(H, f, tab);
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    double mse = 0.0, hs = 0.0;
    for (int32_t r = 0; r + 1 < t; r++) {
        mse = mse + sC[r];
        hs = hs - sP[r];
    }
    double ho = sh[0];
    if (t > 1) {
        ho = 0.0;
        for (int32_t q = 0; q < t; q++) ho = ho + sh[q];
    }
    const double vn = s2tot > 0.0 ? mse / s2tot : 0.0;
    const double lr = __builtin_isfinite(lam) ? lam : 0.0;
    out[0] = mse;
    out[1] = vn;
    out[2] = ho;
    out[3] = hs;
    out[4] = __builtin_fma(lr, ho, vn);
    out[5] = ho + (32.0 * (double)t) / H.dd;
}

__global__ void k_gather(const double* __restrict__ v, const int32_t* __restrict__ u, int32_t t,
                         double* __restrict__ codebook, int32_t* __restrict__ rank) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= t) return;
    codebook[r] = v[u[r]];
    if (rank) rank[r] = u[r];
}

// Philox4x32-10 (Salmon et al., SC'11): ten rounds of two 32x32->64 products
// mixed with the other words and the round key; the key advances by the two
// Weyl increments between rounds.
__device__ __forceinline__ void philox4x32_10(uint32_t (&c)[4], uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int rnd = 0; rnd < 10; rnd++) {
        if (rnd) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        // each 32 x 32 -> 64 product in one instruction (hi and lo halves)
        const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        const uint32_t n0 = hi1 ^ c[1] ^ k0;
        const uint32_t n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
}

template <int DT>
__device__ __forceinline__ double load_x(const void* x, int64_t i) {
    if (DT == 0) return (double)reinterpret_cast<const float*>(x)[i];
    if (DT == 1) return (double)__half2float(reinterpret_cast<const __half*>(x)[i]);
    const uint32_t bits = ((uint32_t)reinterpret_cast<const uint16_t*>(x)[i]) << 16;
    return (double)__uint_as_float(bits);
}

// The rounding's codebook in LDS: the values q_0 .. q_{t-1}; in s, the
// search's copy, q_0 .. q_{t-2} followed by +inf (so the search needs no
// bound: no x is below +inf, and a bracket never starts at q_{t-1}); each
// interval's width D_r = q_{r+1} - q_r and, where 1/D_r is a normal number,
// R_r = RN(1/D_r) (NaN otherwise, which sends every entry of that interval to
// the exact division).
struct RoundBook {
    double q[kMaxT], s[2 * kMaxT], D[kMaxT], R[kMaxT];
};

__device__ __forceinline__ void load_book(RoundBook& B, const double* __restrict__ cb, int32_t t) {
    for (int r = threadIdx.x; r < kMaxT; r += blockDim.x) B.q[r] = r < t ? cb[r] : 0.0;
    for (int r = threadIdx.x; r < 2 * kMaxT; r += blockDim.x)
        B.s[r] = r <= t - 2 ? cb[r] : __builtin_huge_val();
    __syncthreads();
    for (int r = threadIdx.x; r + 1 < t; r += blockDim.x) {
        const double D = B.q[r + 1] - B.q[r];
        B.D[r] = D;
        B.R[r] = (D >= 0x1p-1000 && D <= 0x1p+1000) ? 1.0 / D : __builtin_nan("");
    }
}

__device__ __forceinline__ int32_t search_step(int32_t t) {
    return t >= 3 ? (int32_t)(1u << (31 - __builtin_clz((uint32_t)(t - 2)))) : 0;
}

// Symbol of x under the codebook (t >= 2) and the 53-bit uniform u: the
// bracket r (the largest r <= t-2 with q_r < x, else 0, by a search over
// powers of two from the largest power h <= t-2: indices up to 2h - 1 <
// 2 kMaxT), then up iff u < RN((x - q_r) / D_r).  The quotient is
// first taken as RN(N R_r) (N = x - q_r): within 0.4 2^-50 of the exact RN
// quotient, relative, for quotients in [2^-900, 2^900], so u below or above
// it by more than 2^-50 (relative) decides the comparison, and N = +-0 means
// a quotient of +-0, which u never is below.  Only u inside that band, or a
// quotient outside that range (NaN included), takes the IEEE division.
__device__ __forceinline__ uint32_t round_one(const RoundBook& B, int32_t h,
                                              double xv, double u) {
    int32_t lo = 0;
    for (int32_t step = h; step > 0; step >>= 1) {
        const int32_t m = lo + step;
        lo = B.s[m] < xv ? m : lo;
    }
    const double N = xv - B.q[lo];
    const double qa = N * B.R[lo];
    const double aq = __builtin_fabs(qa);
    const double m = aq * 0x1p-50;
    bool up = u < qa - m;  // false when N = +-0 (qa is then +-0 or NaN)
    const bool sure = N == 0.0 || (aq >= 0x1p-900 && aq <= 0x1p+900 && (up || u > qa + m));
    if (!sure) up = u < N / B.D[lo];
    return (uint32_t)lo + (up ? 1u : 0u);
}

__device__ __forceinline__ double uniform53(uint32_t lo, uint32_t hi) {
    const uint64_t bits = ((((uint64_t)hi) << 32) | lo) >> 11;
    return (double)bits * 0x1p-53;
}

// Final stochastic rounding (Sec. 2), two entries per thread: entries 2j and
// 2j+1 take words (0, 1) and (2, 3) of Philox4x32-10 at counter (j_lo, j_hi,
// 0, 0) with key (k0, k1).  Symbol counts gather in LDS per workgroup.
template <int DT>
__global__ __launch_bounds__(256) void k_quantize(const void* __restrict__ x, int64_t d,
                                                  const double* __restrict__ cb, int32_t t,
                                                  uint32_t k0, uint32_t k1,
                                                  uint8_t* __restrict__ symbols,
                                                  unsigned long long* __restrict__ hist) {
    __shared__ RoundBook B;
    __shared__ unsigned int lh[kMaxT];
    for (int r = threadIdx.x; r < kMaxT; r += blockDim.x) lh[r] = 0u;
    load_book(B, cb, t);
    __syncthreads();
    const int32_t h = search_step(t);
    const int64_t npair = (d + 1) / 2;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < npair;
         j += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i0 = 2 * j;
        const bool two = i0 + 1 < d;
        uint32_t s0 = 0, s1 = 0;
        if (t > 1) {
            const double x0 = load_x<DT>(x, i0);
            const double x1 = two ? load_x<DT>(x, i0 + 1) : 0.0;
            uint32_t c[4] = {(uint32_t)j, (uint32_t)((uint64_t)j >> 32), 0u, 0u};
            philox4x32_10(c, k0, k1);
            s0 = round_one(B, h, x0, uniform53(c[0], c[1]));
            s1 = round_one(B, h, x1, uniform53(c[2], c[3]));
        }
        symbols[i0] = (uint8_t)s0;
        atomicAdd(&lh[s0], 1u);
        if (two) {
            symbols[i0 + 1] = (uint8_t)s1;
            atomicAdd(&lh[s1], 1u);
        }
    }
    __syncthreads();
    for (int r = threadIdx.x; r < t; r += blockDim.x)
        if (lh[r]) atomicAdd(&hist[r], (unsigned long long)lh[r]);
}

// Time-shared rounding (Sec. 7): entry i takes the second codebook iff its
// partition uniform, from Philox counter (j_lo, j_hi, 1, 0) with j = i / 2
// (words (0, 1) for even i, (2, 3) for odd), is below alpha, and is then
// rounded with its codebook exactly as k_quantize rounds it (counter (j_lo,
// j_hi, 0, 0)).  hist: the first codebook's t0 counts, then the second's t1;
// part[i] = 1 for the second.
template <int DT>
__global__ __launch_bounds__(256) void k_quantize_ts(
    const void* __restrict__ x, int64_t d, const double* __restrict__ cb0, int32_t t0,
    const double* __restrict__ cb1, int32_t t1, double alpha, uint32_t k0, uint32_t k1,
    uint8_t* __restrict__ symbols, uint8_t* __restrict__ part,
    unsigned long long* __restrict__ hist) {
    __shared__ RoundBook B[2];
    __shared__ unsigned int lh[2][kMaxT];
    for (int r = threadIdx.x; r < kMaxT; r += blockDim.x) {
        lh[0][r] = 0u;
        lh[1][r] = 0u;
    }
    load_book(B[0], cb0, t0);
    load_book(B[1], cb1, t1);
    __syncthreads();
    const int32_t h0 = search_step(t0), h1 = search_step(t1);
    const int64_t npair = (d + 1) / 2;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < npair;
         j += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i0 = 2 * j;
        const bool two = i0 + 1 < d;
        uint32_t w[4] = {(uint32_t)j, (uint32_t)((uint64_t)j >> 32), 1u, 0u};
        philox4x32_10(w, k0, k1);
        uint32_t c[4] = {(uint32_t)j, (uint32_t)((uint64_t)j >> 32), 0u, 0u};
        philox4x32_10(c, k0, k1);
#pragma unroll
        for (int e = 0; e < 2; e++) {
            const int64_t i = i0 + e;
            if (e == 1 && !two) break;
            const int pw = uniform53(w[2 * e], w[2 * e + 1]) < alpha ? 1 : 0;
            const int32_t t = pw ? t1 : t0;
            uint32_t sym = 0;
            if (t > 1)
                sym = round_one(B[pw], pw ? h1 : h0, load_x<DT>(x, i),
                                uniform53(c[2 * e], c[2 * e + 1]));
            symbols[i] = (uint8_t)sym;
            if (part) part[i] = (uint8_t)pw;
            atomicAdd(&lh[pw][sym], 1u);
        }
    }
    __syncthreads();
    for (int r = threadIdx.x; r < t0; r += blockDim.x)
        if (lh[0][r]) atomicAdd(&hist[r], (unsigned long long)lh[0][r]);
    for (int r = threadIdx.x; r < t1; r += blockDim.x)
        if (lh[1][r]) atomicAdd(&hist[t0 + r], (unsigned long long)lh[1][r]);
}

// Sum over a 256-thread workgroup (a butterfly per wavefront, then the four
// wavefront sums in order); every thread gets the total.
__device__ __forceinline__ double block_sum(double v, double* red) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    __syncthreads();  // red is free
    if (threadIdx.x % 64 == 0) red[threadIdx.x / 64] = v;
    __syncthreads();
    return ((red[0] + red[1]) + red[2]) + red[3];
}

// Plug-in entropy of one symbol histogram (t <= 256 counts, one per thread):
// H = sum of h(n_r / n) over the nonzero counts, n = the counts' total
// (d for the plain rounding, the part's size for a time-shared part).
__device__ __forceinline__ double plugin_entropy(const unsigned long long* __restrict__ hist,
                                                 int32_t t, double n, int64_t* hist_out,
                                                 const double2* __restrict__ tab, double* red) {
    const int r = threadIdx.x;
    double h = 0.0;
    if (r < t) {
        const unsigned long long c = hist[r];
        if (hist_out) hist_out[r] = (int64_t)c;
        if (c) h = hfun((double)c / n, tab);
    }
    return block_sum(h, red);
}

// Entropy of a time-shared rounding: each part's plug-in entropy over its own
// entries, weighted by its size: (n_0 H_0 + n_1 H_1) / d.
__global__ __launch_bounds__(256) void k_entropy_ts(const unsigned long long* __restrict__ hist,
                                                    int32_t t0, int32_t t1, int64_t d,
                                                    double* __restrict__ ent,
                                                    int64_t* __restrict__ hist_out) {
    __shared__ double2 tab[kLog2Size];
    __shared__ double red[4];
    load_log2_table(tab);
    __syncthreads();
    double total = 0.0;
    int32_t base = 0;
    for (int w = 0; w < 2; w++) {
        const int32_t t = w ? t1 : t0;
        const int r = threadIdx.x;
        const double nr = r < t ? (double)hist[base + r] : 0.0;  // counts < 2^53: exact
        const double n = block_sum(nr, red);
        if (n > 0.0) {
            const double H = plugin_entropy(hist + base, t, n, hist_out ? hist_out + base : nullptr,
                                            tab, red);
            total = total + n * H;
        } else if (hist_out && r < t) {
            hist_out[base + r] = 0;
        }
        base += t;
    }
    if (threadIdx.x == 0) *ent = total / (double)d;
}

__global__ __launch_bounds__(256) void k_entropy(const unsigned long long* __restrict__ hist,
                                                 int32_t t, int64_t d, double* __restrict__ ent,
                                                 int64_t* __restrict__ hist_out) {
    __shared__ double2 tab[kLog2Size];
    __shared__ double red[4];
    load_log2_table(tab);
    __syncthreads();
    const double H = plugin_entropy(hist, t, (double)d, hist_out, tab, red);
    if (threadIdx.x == 0) *ent = H;
}

// Symbol counts of the allocation-free rounding entry point: one array per
// device, alive until the process ends, shared by every such call on that
// device (calls that overlap on one device race on it).
static __device__ __align__(256) unsigned long long scratch[kMaxT];

__global__ void k_zero_counts(unsigned long long* __restrict__ h, int32_t n) {
    for (int32_t r = threadIdx.x; r < n; r += blockDim.x) h[r] = 0ull;
}

}  // namespace

// Device address of `scratch` on the current device, looked up once per
// device (the host-side name is not a device address).
hipError_t quantize_scratch(unsigned long long** out) {
    constexpr int kMaxDev = 64;
    static std::mutex mu;
    static unsigned long long* ptr[kMaxDev] = {};
    static hipError_t err[kMaxDev] = {};
    static bool done[kMaxDev] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!done[dev]) {
        void* p = nullptr;
        err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        ptr[dev] = static_cast<unsigned long long*>(p);
        done[dev] = true;
    }
    if (err[dev] != hipSuccess) return err[dev];
    *out = ptr[dev];
    return hipSuccess;
}

hipError_t launch_zero_counts(unsigned long long* h, int32_t n, hipStream_t st) {
    k_zero_counts<<<1, 256, 0, st>>>(h, n);
    return hipGetLastError();
}

hipError_t launch_refine(const Hist& H, int32_t t, int32_t* u, double lamp, double b,
                         int32_t budget, int32_t rounds, int32_t exhaustive, int32_t* stats,
                         hipStream_t st) {
    k_refine<<<1, 256, 0, st>>>(H, t, u, lamp, b, budget, rounds, exhaustive, stats);
    return hipGetLastError();
}

hipError_t launch_metrics(const Hist& H, int32_t t, const int32_t* u, double lam, double s2tot,
                          double* out, hipStream_t st) {
    if (t < 1 || t > kMaxT) return hipErrorInvalidValue;
    k_metrics<<<1, 256, 0, st>>>(H, t, u, lam, s2tot, out);
    return hipGetLastError();
}

hipError_t launch_gather(const double* v, const int32_t* u, int32_t t, double* codebook,
                         int32_t* rank, hipStream_t st) {
    k_gather<<<(t + 63) / 64, 64, 0, st>>>(v, u, t, codebook, rank);
    return hipGetLastError();
}

hipError_t launch_quantize(const void* x, int dt, int64_t d, const double* codebook, int32_t t,
                           uint64_t seed, uint8_t* symbols, unsigned long long* hist,
                           hipStream_t st) {
    int64_t g = ((d + 1) / 2 + 255) / 256;  // a thread per pair of entries
    if (g > 4096) g = 4096;
    if (g < 1) g = 1;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    if (dt == 0)
        k_quantize<0><<<(unsigned)g, 256, 0, st>>>(x, d, codebook, t, k0, k1, symbols, hist);
    else if (dt == 1)
        k_quantize<1><<<(unsigned)g, 256, 0, st>>>(x, d, codebook, t, k0, k1, symbols, hist);
    else
        k_quantize<2><<<(unsigned)g, 256, 0, st>>>(x, d, codebook, t, k0, k1, symbols, hist);
    return hipGetLastError();
}

hipError_t launch_entropy(const unsigned long long* hist, int32_t t, int64_t d, double* ent,
                          int64_t* hist_out, hipStream_t st) {
    k_entropy<<<1, 256, 0, st>>>(hist, t, d, ent, hist_out);
    return hipGetLastError();
}

hipError_t launch_quantize_ts(const void* x, int dt, int64_t d, const double* cb0, int32_t t0,
                              const double* cb1, int32_t t1, double alpha, uint64_t seed,
                              uint8_t* symbols, uint8_t* part, unsigned long long* hist,
                              double* ent, int64_t* hist_out, hipStream_t st) {
    int64_t g = ((d + 1) / 2 + 255) / 256;  // a thread per pair of entries
    if (g > 4096) g = 4096;
    if (g < 1) g = 1;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    if (dt == 0)
        k_quantize_ts<0><<<(unsigned)g, 256, 0, st>>>(x, d, cb0, t0, cb1, t1, alpha, k0, k1,
                                                      symbols, part, hist);
    else if (dt == 1)
        k_quantize_ts<1><<<(unsigned)g, 256, 0, st>>>(x, d, cb0, t0, cb1, t1, alpha, k0, k1,
                                                      symbols, part, hist);
    else
        k_quantize_ts<2><<<(unsigned)g, 256, 0, st>>>(x, d, cb0, t0, cb1, t1, alpha, k0, k1,
                                                      symbols, part, hist);
    k_entropy_ts<<<1, 256, 0, st>>>(hist, t0, t1, d, ent, hist_out);
    return hipGetLastError();
}

}  // namespace ecasq
