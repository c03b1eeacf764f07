// Input preparation on the device: ingest, radix sort, weighted histogram and
// exact prefix sums (the O(d) steps before the DP).
//
// The paper sorts a copy of X and works on its weighted histogram (Sec. 2) and
// evaluates interval costs from prefix counts and sums N, S, S2 (App. D).  Here
// the prefix sums are exact: every fp32 value is an integer multiple of 2^-149,
// so S and S2 are accumulated as wide two's-complement integers (5 and 10
// 64-bit limbs) and rounded to fp64 once, to nearest even.  The result does not
// depend on the summation order, which lets the scan run in parallel and still
// match a sequential exact sum bit for bit.
#include <hip/hip_fp16.h>

#include "device.hpp"
#include "launch.hpp"
#include "wide.hpp"

namespace ecasq {

namespace {

constexpr int kSortBlock = 1024;  // threads per sort workgroup (>= 256 digits)
constexpr int kSortItems = 4;
constexpr int kSortTile = kSortBlock * kSortItems;

constexpr int kRec = 16;  // u64 words per chunk record: S, S2, run ends
constexpr int kChunk = 8;
constexpr int kScanBlock = 256;

template <int DT>
__global__ __launch_bounds__(256) void k_ingest(const void* __restrict__ x, int64_t d,
                                                uint32_t* __restrict__ keys,
                                                uint32_t* __restrict__ flags) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < d;
         i += (int64_t)gridDim.x * blockDim.x) {
        uint32_t bits;
        if (DT == 0) {
            bits = reinterpret_cast<const uint32_t*>(x)[i];
        } else if (DT == 1) {
            bits = __float_as_uint(__half2float(reinterpret_cast<const __half*>(x)[i]));
        } else {
            bits = ((uint32_t)reinterpret_cast<const uint16_t*>(x)[i]) << 16;
        }
        if ((bits & 0x7F800000u) == 0x7F800000u) {
            atomicOr(flags, 1u);
            bits = 0u;
        }
        keys[i] = f32_key(bits);
    }
}

__global__ __launch_bounds__(kSortBlock) void k_radix_hist(const uint32_t* __restrict__ keys,
                                                           int64_t n, int shift,
                                                           uint32_t* __restrict__ hist, int nblk) {
    __shared__ uint32_t cnt[256];
    const int tid = threadIdx.x;
    if (tid < 256) cnt[tid] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int it = 0; it < kSortItems; it++) {
        const int64_t idx = base + (int64_t)it * kSortBlock + tid;
        if (idx < n) atomicAdd(&cnt[(keys[idx] >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 256) hist[(int64_t)tid * nblk + blockIdx.x] = cnt[tid];
}

// Exclusive scan of m uint32 values in place, one block of 1024 threads, in
// tiles of 8192 values staged through LDS (coalesced loads and stores):
// each thread scans 8 consecutive values of the tile, the thread totals are
// scanned by wavefront shuffles and then across the 16 wavefronts, and a
// carry takes each tile's total to the next.
__global__ __launch_bounds__(1024) void k_scan_u32(uint32_t* __restrict__ a, int64_t m) {
    constexpr int V = 8, T = 1024 * V;
    __shared__ uint32_t buf[T];
    __shared__ uint32_t part[16];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    uint32_t carry = 0;
    for (int64_t base = 0; base < m; base += T) {
        const int n = m - base < T ? (int)(m - base) : T;
        for (int i = tid; i < T; i += 1024) buf[i] = i < n ? a[base + i] : 0u;
        __syncthreads();
        uint32_t v[V], s = 0;
#pragma unroll
        for (int u = 0; u < V; u++) {
            v[u] = buf[tid * V + u];
            s += v[u];
        }
        // every lane takes part in every shuffle
        uint32_t x = s;
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t y = __shfl_up(x, off);
            if (lane >= off) x += y;
        }
        if (lane == 63) part[wave] = x;
        __syncthreads();
        uint32_t wpre = 0, total = 0;
        for (int w = 0; w < 16; w++) {
            wpre += w < wave ? part[w] : 0u;
            total += part[w];
        }
        uint32_t run = carry + wpre + x - s;  // exclusive
#pragma unroll
        for (int u = 0; u < V; u++) {
            buf[tid * V + u] = run;
            run += v[u];
        }
        __syncthreads();
        for (int i = tid; i < n; i += 1024) a[base + i] = buf[i];
        carry += total;
        __syncthreads();  // buf and part are reused by the next tile
    }
}

// Stable scatter of one 8-bit digit.  Items are taken in index order
// (tile, then item slot, then thread); equal digits keep that order.
__global__ __launch_bounds__(kSortBlock) void k_radix_scatter(const uint32_t* __restrict__ kin,
                                                              uint32_t* __restrict__ kout,
                                                              int64_t n, int shift,
                                                              const uint32_t* __restrict__ hist,
                                                              int nblk) {
    __shared__ uint32_t base[256];
    __shared__ uint32_t wcnt[kSortBlock / 64][256];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    if (tid < 256) {
        base[tid] = hist[(int64_t)tid * nblk + blockIdx.x];
        for (int w = 0; w < kSortBlock / 64; w++) wcnt[w][tid] = 0;
    }
    __syncthreads();
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t tile = (int64_t)blockIdx.x * kSortTile;
    for (int it = 0; it < kSortItems; it++) {
        const int64_t idx = tile + (int64_t)it * kSortBlock + tid;
        const bool valid = idx < n;
        const uint32_t key = valid ? kin[idx] : 0u;
        const uint32_t dig = (key >> shift) & 255u;
        uint64_t peers = __ballot(valid);
        for (int bit = 0; bit < 8; bit++) {
            const bool set = (dig >> bit) & 1u;
            const uint64_t bal = __ballot(set);
            peers &= set ? bal : ~bal;
        }
        const uint32_t rank = __popcll(peers & lt_mask);
        if (valid && rank == 0) wcnt[wave][dig] = __popcll(peers);
        __syncthreads();
        if (valid) {
            uint32_t pos = base[dig] + rank;
            for (int w = 0; w < wave; w++) pos += wcnt[w][dig];
            kout[pos] = key;
        }
        __syncthreads();
        if (tid < 256) {
            uint32_t tot = 0;
            for (int w = 0; w < kSortBlock / 64; w++) {
                tot += wcnt[w][tid];
                wcnt[w][tid] = 0;
            }
            base[tid] += tot;
        }
        __syncthreads();
    }
}

// Per-chunk totals: S (5 words), S2 (10 words), number of run ends (1 word).
__global__ __launch_bounds__(kScanBlock) void k_scan_local(const uint32_t* __restrict__ keys,
                                                           int64_t d, int64_t nchunk,
                                                           uint64_t* __restrict__ rec) {
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= nchunk) return;
    uint64_t s[kSL] = {0}, q[kS2L] = {0};
    uint64_t ends = 0;
    const int64_t i0 = c * kChunk;
    for (int e = 0; e < kChunk; e++) {
        const int64_t i = i0 + e;
        if (i >= d) break;
        const uint32_t k = keys[i];
        accumulate(s, q, term_of(key_bits(k)));
        if (i == d - 1 || keys[i + 1] != k) ends++;
    }
    uint64_t* r = rec + c * kRec;
#pragma unroll
    for (int l = 0; l < kSL; l++) r[l] = s[l];
#pragma unroll
    for (int l = 0; l < kS2L; l++) r[kSL + l] = q[l];
    r[kRec - 1] = ends;
}

__device__ __forceinline__ void rec_add(uint64_t* a, const uint64_t* b) {
    wide_add_full<kSL>(a, b);
    wide_add_full<kS2L>(a + kSL, b + kSL);
    a[kRec - 1] += b[kRec - 1];
}

// Exclusive scan of each run of kScanBlock chunk records in place, one
// workgroup per run (record c at thread c mod kScanBlock), and the run's
// total to tot[run].  The records hold exact integers, so the order of the
// additions does not change any sum.
__global__ __launch_bounds__(kScanBlock) void k_scan_runs(uint64_t* __restrict__ rec,
                                                          int64_t nchunk,
                                                          uint64_t* __restrict__ tot) {
    __shared__ uint64_t part[kScanBlock][kRec + 1];  // padded: lanes spread over the banks
    const int tid = threadIdx.x;
    const int64_t c = (int64_t)blockIdx.x * kScanBlock + tid;
    const bool live = c < nchunk;
    for (int l = 0; l < kRec; l++) part[tid][l] = live ? rec[c * kRec + l] : 0ull;
    __syncthreads();
    for (int off = 1; off < kScanBlock; off <<= 1) {
        uint64_t t[kRec];
        const bool on = tid >= off;
        for (int l = 0; l < kRec; l++) t[l] = on ? part[tid - off][l] : 0ull;
        __syncthreads();
        if (on) rec_add(part[tid], t);
        __syncthreads();
    }
    if (live)
        for (int l = 0; l < kRec; l++) rec[c * kRec + l] = tid ? part[tid - 1][l] : 0ull;
    if (tid == kScanBlock - 1)
        for (int l = 0; l < kRec; l++) tot[(int64_t)blockIdx.x * kRec + l] = part[tid][l];
}

// Exclusive scan of the chunk records in place (one block); writes the number
// of distinct values to *p_out.
__global__ __launch_bounds__(kScanBlock) void k_scan_records(uint64_t* __restrict__ rec,
                                                             int64_t nchunk,
                                                             int64_t* __restrict__ p_out) {
    __shared__ uint64_t part[kScanBlock][kRec + 1];  // padded: lanes spread over the banks
    const int tid = threadIdx.x;
    const int64_t per = (nchunk + kScanBlock - 1) / kScanBlock;
    const int64_t lo = tid * per;
    const int64_t hi = lo + per < nchunk ? lo + per : nchunk;
    uint64_t acc[kRec] = {0};
    for (int64_t c = lo; c < hi; c++) rec_add(acc, rec + c * kRec);
    for (int l = 0; l < kRec; l++) part[tid][l] = acc[l];
    __syncthreads();
    for (int off = 1; off < kScanBlock; off <<= 1) {
        uint64_t t[kRec];
        const bool on = tid >= off;
        for (int l = 0; l < kRec; l++) t[l] = on ? part[tid - off][l] : 0ull;
        __syncthreads();
        if (on) rec_add(part[tid], t);
        __syncthreads();
    }
    uint64_t run[kRec];
    for (int l = 0; l < kRec; l++) run[l] = tid ? part[tid - 1][l] : 0ull;
    if (tid == kScanBlock - 1) *p_out = (int64_t)part[tid][kRec - 1];
    for (int64_t c = lo; c < hi; c++) {
        uint64_t cur[kRec];
        for (int l = 0; l < kRec; l++) cur[l] = rec[c * kRec + l];
        for (int l = 0; l < kRec; l++) rec[c * kRec + l] = run[l];
        rec_add(run, cur);
    }
}

// Walk each chunk from its exclusive prefix (its run's, from tot, plus its
// own within the run) and write the histogram entry of every run end: v[u], N[u] (inclusive count), S[u], S2[u] (rounded once).
__global__ __launch_bounds__(kScanBlock) void k_scan_emit(const uint32_t* __restrict__ keys,
                                                          int64_t d, int64_t nchunk,
                                                          const uint64_t* __restrict__ rec,
                                                          const uint64_t* __restrict__ tot,
                                                          double* __restrict__ v,
                                                          double* __restrict__ N,
                                                          double* __restrict__ S,
                                                          double* __restrict__ S2) {
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= nchunk) return;
    // the chunk's exclusive prefix: its run's prefix plus its place in the run
    uint64_t r[kRec];
#pragma unroll
    for (int l = 0; l < kRec; l++) r[l] = tot[(c / kScanBlock) * kRec + l];
    rec_add(r, rec + c * kRec);
    uint64_t s[kSL], q[kS2L];
#pragma unroll
    for (int l = 0; l < kSL; l++) s[l] = r[l];
#pragma unroll
    for (int l = 0; l < kS2L; l++) q[l] = r[kSL + l];
    int64_t u = (int64_t)r[kRec - 1];
    const int64_t i0 = c * kChunk;
    for (int e = 0; e < kChunk; e++) {
        const int64_t i = i0 + e;
        if (i >= d) break;
        const uint32_t k = keys[i];
        const uint32_t bits = key_bits(k);
        accumulate(s, q, term_of(bits));
        if (i == d - 1 || keys[i + 1] != k) {
            v[u] = (double)__uint_as_float(bits);
            N[u] = (double)(i + 1);
            S[u] = wide_to_double<kSL>(s, true, -149);
            S2[u] = wide_to_double<kS2L>(q, false, -298);
            u++;
        }
    }
}

// ||X||^2 = S2[p-1] and the count of the smallest value N[0] beside p in
// the host-read slots (one read after preparation instead of two).
__global__ void k_prep_tail(const int64_t* __restrict__ p, const double* __restrict__ N,
                            const double* __restrict__ S2, double* __restrict__ out) {
    if (threadIdx.x != 0) return;
    const int64_t n = p[0];
    out[0] = n >= 1 ? S2[n - 1] : 0.0;
    out[1] = n >= 1 ? N[0] : 0.0;
}

}  // namespace

size_t prep_scratch_bytes(int64_t d) {
    const int64_t nblk = (d + kSortTile - 1) / kSortTile;
    const int64_t nchunk = (d + kChunk - 1) / kChunk;
    size_t b = 0;
    b += align256(sizeof(uint32_t) * d) * 2;           // keys, ping-pong
    b += align256(sizeof(uint32_t) * 256 * nblk);      // digit histogram
    b += align256(sizeof(uint64_t) * kRec * nchunk);   // chunk records
    b += align256(sizeof(uint64_t) * kRec * ((nchunk + kScanBlock - 1) / kScanBlock));  // runs
    b += align256(sizeof(uint32_t) * 4);               // flags
    return b;
}

hipError_t launch_prep(const void* x, int dt, int64_t d, void* scratch, hipStream_t st, double* v,
                       double* N, double* S, double* S2, int64_t* p_dev, uint32_t* flags_dev) {
    const int64_t nblk = (d + kSortTile - 1) / kSortTile;
    const int64_t nchunk = (d + kChunk - 1) / kChunk;
    char* w = static_cast<char*>(scratch);
    uint32_t* k0 = reinterpret_cast<uint32_t*>(w);
    w += align256(sizeof(uint32_t) * d);
    uint32_t* k1 = reinterpret_cast<uint32_t*>(w);
    w += align256(sizeof(uint32_t) * d);
    uint32_t* hist = reinterpret_cast<uint32_t*>(w);
    w += align256(sizeof(uint32_t) * 256 * nblk);
    uint64_t* rec = reinterpret_cast<uint64_t*>(w);
    w += align256(sizeof(uint64_t) * kRec * nchunk);
    uint64_t* tot = reinterpret_cast<uint64_t*>(w);

    const int ig = (int)((d + 255) / 256 < 65536 ? (d + 255) / 256 : 65536);
    if (dt == 0) k_ingest<0><<<ig, 256, 0, st>>>(x, d, k0, flags_dev);
    else if (dt == 1) k_ingest<1><<<ig, 256, 0, st>>>(x, d, k0, flags_dev);
    else k_ingest<2><<<ig, 256, 0, st>>>(x, d, k0, flags_dev);
    for (int pass = 0; pass < 4; pass++) {
        const int shift = 8 * pass;
        k_radix_hist<<<(unsigned)nblk, kSortBlock, 0, st>>>(k0, d, shift, hist, (int)nblk);
        k_scan_u32<<<1, 1024, 0, st>>>(hist, 256 * nblk);
        k_radix_scatter<<<(unsigned)nblk, kSortBlock, 0, st>>>(k0, k1, d, shift, hist, (int)nblk);
        uint32_t* t = k0;
        k0 = k1;
        k1 = t;
    }
    const unsigned sg = (unsigned)((nchunk + kScanBlock - 1) / kScanBlock);
    // chunk totals; each run of kScanBlock chunks scanned by a workgroup;
    // the run totals scanned by one; then every chunk walked from its prefix
    k_scan_local<<<sg, kScanBlock, 0, st>>>(k0, d, nchunk, rec);
    k_scan_runs<<<sg, kScanBlock, 0, st>>>(rec, nchunk, tot);
    k_scan_records<<<1, kScanBlock, 0, st>>>(tot, (int64_t)sg, p_dev);
    k_scan_emit<<<sg, kScanBlock, 0, st>>>(k0, d, nchunk, rec, tot, v, N, S, S2);
    k_prep_tail<<<1, 64, 0, st>>>(p_dev, N, S2, reinterpret_cast<double*>(p_dev + 2));
    return hipGetLastError();
}

}  // namespace ecasq
