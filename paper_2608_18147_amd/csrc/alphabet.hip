// Permissible alphabets P != X (App. D): the DP's candidate values are a grid
// over [min X, max X] instead of the distinct input values, and the interval
// quantities come from the input's prefix count, sum and sum of squares at the
// grid points (the entries <= p).  With min X and max X as the first and last
// grid points, every later step (DP, search, refinement, metrics, rounding)
// runs unchanged on the grid.
//
//   uniform  p_k = min X + k * ((max X - min X) / (m - 1)) for 0 < k < m-1,
//            each operation rounded to nearest, p_0 = min X, p_{m-1} = max X;
//   quantile p_k = the input value at rank floor(k (d - 1) / (m - 1)).
// A point equal to its predecessor (or, for the uniform grid, an inner point
// not below max X) is dropped.  One workgroup walks the grid in tiles of 1024 points,
// a tile-wide scan of the kept flags placing the survivors.
#include "device.hpp"
#include "launch.hpp"

namespace ecasq {

namespace {

constexpr int kAT = 1024;

// Last index i with v[i] <= q (v ascending, v[0] <= q).
__device__ __forceinline__ int64_t last_le(const double* v, int64_t n, double q) {
    int64_t lo = 0, hi = n - 1;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo + 1) / 2;
        if (v[mid] <= q)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// First index i with N[i] > r (N ascending integer counts, N[n-1] > r).
__device__ __forceinline__ int64_t first_gt(const double* N, int64_t n, double r) {
    int64_t lo = 0, hi = n - 1;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (N[mid] > r)
            hi = mid;
        else
            lo = mid + 1;
    }
    return lo;
}

struct AlphaArgs {
    const double *v, *N, *S, *S2;  // distinct input values and their prefix sums
    int64_t px;                    // number of distinct input values (>= 2)
    int64_t d;
    int64_t m;                     // requested grid size (2 <= m <= d)
    int32_t kind;                  // 1 uniform, 2 quantile
    double *gv, *gN, *gS, *gS2;    // the grid and the prefix sums at its points
    int64_t* count;                // number of grid points kept
};

// Grid point k: its value and the index of the last input value <= it.
__device__ __forceinline__ void point(const AlphaArgs& a, int64_t k, double& q, int64_t& idx) {
    if (a.kind == 1) {
        const double lo = a.v[0], hi = a.v[a.px - 1];
        if (k == 0) {
            q = lo;
            idx = 0;
            return;
        }
        if (k == a.m - 1) {
            q = hi;
            idx = a.px - 1;
            return;
        }
        const double step = (hi - lo) / (double)(a.m - 1);
        q = lo + (double)k * step;
        idx = last_le(a.v, a.px, q);
    } else {
        const int64_t r = (k * (a.d - 1)) / (a.m - 1);
        idx = first_gt(a.N, a.px, (double)r);
        q = a.v[idx];
    }
}

__global__ __launch_bounds__(kAT) void k_alphabet(AlphaArgs a) {
    __shared__ int32_t scan[kAT];
    __shared__ int64_t base;
    const int tid = threadIdx.x;
    if (tid == 0) base = 0;
    const double hi = a.v[a.px - 1];
    for (int64_t t0 = 0; t0 < a.m; t0 += kAT) {
        const int64_t k = t0 + tid;
        double q = 0.0;
        int64_t idx = 0;
        int32_t keep = 0;
        if (k < a.m) {
            point(a, k, q, idx);
            if (k == 0 || (a.kind == 1 && k == a.m - 1)) {
                keep = 1;
            } else {
                // the points rise with k, so the predecessor is the largest
                // point kept so far or a repeat of it
                double qp;
                int64_t ip;
                point(a, k - 1, qp, ip);
                keep = a.kind == 1 ? (q > qp && q < hi) : (idx > ip);
            }
        }
        // inclusive scan of the kept flags (Hillis-Steele)
        scan[tid] = keep;
        __syncthreads();
        for (int off = 1; off < kAT; off <<= 1) {
            const int32_t add = tid >= off ? scan[tid - off] : 0;
            __syncthreads();
            scan[tid] += add;
            __syncthreads();
        }
        if (keep) {
            const int64_t o = base + scan[tid] - 1;
            a.gv[o] = q;
            a.gN[o] = a.N[idx];
            a.gS[o] = a.S[idx];
            a.gS2[o] = a.S2[idx];
        }
        __syncthreads();
        if (tid == 0) base += scan[kAT - 1];
        __syncthreads();
    }
    if (tid == 0) *a.count = base;
}

}  // namespace

hipError_t launch_alphabet(int32_t kind, int64_t m, int64_t d, const double* v, const double* N,
                           const double* S, const double* S2, int64_t px, double* gv, double* gN,
                           double* gS, double* gS2, int64_t* count, hipStream_t st) {
    if ((kind != 1 && kind != 2) || m < 2 || m > d || px < 2) return hipErrorInvalidValue;
    AlphaArgs a{v, N, S, S2, px, d, m, kind, gv, gN, gS, gS2, count};
    k_alphabet<<<1, kAT, 0, st>>>(a);
    return hipGetLastError();
}

}  // namespace ecasq
