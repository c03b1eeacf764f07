// Entropy coding of the final symbols with rANS (Duda, arXiv:1311.2540), so
// that the rate the paper charges (App. F.1: the payload at about H(Xhat)
// bits per entry plus a 16-bit descriptor per codebook value) is realised as
// bytes.
//
//   frequencies  f_q = max(1, floor(n_q M / d)), M = 2^16; a surplus goes to
//                the largest f (lowest q among ties), a deficit is taken one
//                unit at a time from the largest f > 1; c_q = f_0 + .. + f_{q-1}
//   state        x in [L, 256 L), L = 2^23, bytes out
//   encode       a segment's symbols in reverse: while x >= 2^15 f_q emit
//                x's low byte, x >>= 8; x = floor(x/f_q) 2^16 + x mod f_q + c_q;
//                finally emit x's four bytes, low first; the segment's stream
//                is the emitted bytes in reverse order
//   decode       x = 4 bytes big-endian; slot = x mod 2^16, q: c_q <= slot <
//                c_q + f_q, x = f_q (x >> 16) + slot - c_q, refill bytes while
//                x < L; every segment ends at x = L
//   stream       t u16 (f_q - 1, little-endian), one u32 per segment of 4096
//                symbols (its end, counted from the payload start), payload
//
// Segments are coded independently, one lane each: encoding writes a
// segment's bytes backwards into a private slot of the scratch buffer, a scan
// of the lengths places them, and a copy packs them.
#include "device.hpp"
#include "launch.hpp"

namespace ecasq {

namespace {

constexpr int kRSeg = 4096;
constexpr uint32_t kRL = 1u << 23;
constexpr uint32_t kRM = 1u << 16;
constexpr int64_t kRSegCap = 2 * kRSeg + 16;  // 2 bytes per symbol at most, plus the state

__global__ __launch_bounds__(256) void k_sym_hist(const uint8_t* __restrict__ sym, int64_t d,
                                                  int32_t t, unsigned long long* __restrict__ hist,
                                                  unsigned int* __restrict__ bad) {
    __shared__ unsigned int lh[256];
    lh[threadIdx.x] = 0u;
    __syncthreads();
    unsigned int nbad = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < d;
         i += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t q = sym[i];
        atomicAdd(&lh[q], 1u);
        nbad += q >= (uint32_t)t ? 1u : 0u;
    }
    __syncthreads();
    if (lh[threadIdx.x]) atomicAdd(&hist[threadIdx.x], (unsigned long long)lh[threadIdx.x]);
    if (nbad) atomicAdd(bad, nbad);
}

// f and c of the t symbols (fc[0..t) and fc[256..256+t)), and the stream's
// frequency header.  One thread: t <= 256.
__global__ void k_rans_freqs(const unsigned long long* __restrict__ hist, int32_t t, int64_t d,
                             uint32_t* __restrict__ fc, uint8_t* __restrict__ head) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int64_t sum = 0;
    for (int32_t q = 0; q < t; q++) {
        const uint64_t v = (hist[q] * (uint64_t)kRM) / (uint64_t)d;
        fc[q] = v > 0 ? (uint32_t)v : 1u;
        sum += fc[q];
    }
    int64_t diff = (int64_t)kRM - sum;
    if (diff > 0) {
        int32_t j = 0;
        for (int32_t q = 1; q < t; q++)
            if (fc[q] > fc[j]) j = q;
        fc[j] += (uint32_t)diff;
    }
    while (diff < 0) {
        int32_t j = -1;
        for (int32_t q = 0; q < t; q++)
            if (fc[q] > 1u && (j < 0 || fc[q] > fc[j])) j = q;
        fc[j] -= 1u;
        diff += 1;
    }
    uint32_t c = 0;
    for (int32_t q = 0; q < t; q++) {
        fc[256 + q] = c;
        c += fc[q];
        const uint32_t m1 = fc[q] - 1u;
        head[2 * q] = (uint8_t)(m1 & 0xFFu);
        head[2 * q + 1] = (uint8_t)(m1 >> 8);
    }
}

__global__ __launch_bounds__(64) void k_rans_encode(const uint8_t* __restrict__ sym, int64_t d,
                                                    const uint32_t* __restrict__ fc, int32_t t,
                                                    uint8_t* __restrict__ scratch,
                                                    uint32_t* __restrict__ lens, int64_t nseg) {
    __shared__ uint32_t sf[256], sc[256];
    for (int q = threadIdx.x; q < 256; q += blockDim.x) {
        sf[q] = q < t ? fc[q] : 1u;  // symbols >= t are reported by the histogram
        sc[q] = q < t ? fc[256 + q] : 0u;
    }
    __syncthreads();
    const int64_t seg = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (seg >= nseg) return;
    const int64_t a = seg * kRSeg;
    const int64_t n = min((int64_t)kRSeg, d - a);
    uint8_t* reg = scratch + seg * kRSegCap;
    int64_t w = kRSegCap;
    uint32_t x = kRL;
    for (int64_t i = n - 1; i >= 0; i--) {
        const uint32_t q = sym[a + i];
        const uint32_t f = sf[q], c = sc[q];
        const uint32_t xmax = (1u << 15) * f;
        while (x >= xmax) {
            reg[--w] = (uint8_t)(x & 0xFFu);
            x >>= 8;
        }
        x = ((x / f) << 16) + (x % f) + c;
    }
    for (int k = 0; k < 4; k++) reg[--w] = (uint8_t)((x >> (8 * k)) & 0xFFu);
    lens[seg] = (uint32_t)(kRSegCap - w);
}

// Inclusive scan of the segment lengths into the stream's end table
// (little-endian u32, byte by byte: the table need not be aligned); *total =
// the payload size.  One workgroup.
constexpr int kRScan = 1024;

__global__ __launch_bounds__(kRScan) void k_rans_offsets(const uint32_t* __restrict__ lens,
                                                         int64_t nseg, uint8_t* __restrict__ ends,
                                                         uint32_t* __restrict__ starts,
                                                         unsigned long long* __restrict__ total) {
    __shared__ uint32_t sc[kRScan];
    __shared__ uint32_t carry;
    if (threadIdx.x == 0) carry = 0u;
    __syncthreads();
    for (int64_t b0 = 0; b0 < nseg; b0 += kRScan) {
        const int64_t k = b0 + threadIdx.x;
        const uint32_t v = k < nseg ? lens[k] : 0u;
        sc[threadIdx.x] = v;
        __syncthreads();
        for (int off = 1; off < kRScan; off <<= 1) {
            const uint32_t add = (int)threadIdx.x >= off ? sc[threadIdx.x - off] : 0u;
            __syncthreads();
            sc[threadIdx.x] += add;
            __syncthreads();
        }
        if (k < nseg) {
            const uint32_t e = carry + sc[threadIdx.x];
            starts[k] = e - v;
            for (int q = 0; q < 4; q++) ends[4 * k + q] = (uint8_t)((e >> (8 * q)) & 0xFFu);
        }
        __syncthreads();
        if (threadIdx.x == 0) carry += sc[kRScan - 1];
        __syncthreads();
    }
    if (threadIdx.x == 0) *total = carry;
}

__global__ __launch_bounds__(256) void k_rans_pack(const uint8_t* __restrict__ scratch,
                                                   const uint32_t* __restrict__ lens,
                                                   const uint32_t* __restrict__ starts,
                                                   uint8_t* __restrict__ payload) {
    const int64_t seg = blockIdx.x;
    const uint32_t n = lens[seg];
    const uint8_t* src = scratch + seg * kRSegCap + (kRSegCap - n);
    uint8_t* dst = payload + starts[seg];
    for (uint32_t i = threadIdx.x; i < n; i += blockDim.x) dst[i] = src[i];
}

// One lane per segment.  bad: set when a segment runs past its bytes or does
// not end in the initial state.
__global__ __launch_bounds__(64) void k_rans_decode(const uint8_t* __restrict__ in, int64_t nin,
                                                    int64_t d, int32_t t, int64_t nseg,
                                                    uint8_t* __restrict__ sym,
                                                    unsigned int* __restrict__ bad) {
    __shared__ uint32_t sf[256], sc[256];
    if (threadIdx.x == 0) {
        uint32_t c = 0;
        for (int32_t q = 0; q < t; q++) {
            sf[q] = ((uint32_t)in[2 * q] | ((uint32_t)in[2 * q + 1] << 8)) + 1u;
            sc[q] = c;
            c += sf[q];
        }
        if (c != kRM) atomicAdd(bad, 1u);
    }
    __syncthreads();
    const int64_t seg = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (seg >= nseg) return;
    const uint8_t* ends = in + 2 * t;
    auto end_at = [&](int64_t k) {
        return (int64_t)((uint32_t)ends[4 * k] | ((uint32_t)ends[4 * k + 1] << 8) |
                         ((uint32_t)ends[4 * k + 2] << 16) | ((uint32_t)ends[4 * k + 3] << 24));
    };
    const int64_t pay = 2 * (int64_t)t + 4 * nseg;
    const int64_t lo = pay + (seg == 0 ? 0 : end_at(seg - 1));
    const int64_t hi = pay + end_at(seg);
    if (lo + 4 > hi || hi > nin) {
        atomicAdd(bad, 1u);
        return;
    }
    const int64_t a = seg * kRSeg;
    const int64_t n = min((int64_t)kRSeg, d - a);
    int64_t pos = lo;
    uint32_t x = ((uint32_t)in[pos] << 24) | ((uint32_t)in[pos + 1] << 16) |
                 ((uint32_t)in[pos + 2] << 8) | (uint32_t)in[pos + 3];
    pos += 4;
    bool ok = true;
    for (int64_t i = 0; i < n; i++) {
        const uint32_t slot = x & (kRM - 1u);
        int32_t lo_q = 0, hi_q = t - 1;  // largest q with c_q <= slot
        while (lo_q < hi_q) {
            const int32_t mid = (lo_q + hi_q + 1) >> 1;
            if (sc[mid] <= slot) lo_q = mid;
            else hi_q = mid - 1;
        }
        const uint32_t q = (uint32_t)lo_q;
        x = sf[q] * (x >> 16) + slot - sc[q];
        while (x < kRL) {
            if (pos >= hi) {
                ok = false;
                break;
            }
            x = (x << 8) | in[pos++];
        }
        if (!ok) break;
        sym[a + i] = (uint8_t)q;
    }
    if (!ok || x != kRL || pos != hi) atomicAdd(bad, 1u);
}

}  // namespace

int64_t rans_segments(int64_t d) { return (d + kRSeg - 1) / kRSeg; }

size_t rans_bound(int64_t d, int32_t t) {
    const int64_t nseg = rans_segments(d);
    return (size_t)(2 * (int64_t)t + 8 * nseg + 2 * d);
}

size_t rans_scratch_bytes(int64_t d) {
    const int64_t nseg = rans_segments(d);
    return align256(sizeof(unsigned long long) * 256) + align256(sizeof(uint32_t) * 512) +
           align256(sizeof(uint32_t) * 4) + 2 * align256(sizeof(uint32_t) * (size_t)nseg) +
           align256(sizeof(unsigned long long)) + (size_t)nseg * kRSegCap;
}

hipError_t launch_rans_encode(const uint8_t* sym, int64_t d, int32_t t, uint8_t* out,
                              char* scratch, unsigned long long* total_out, unsigned int* bad,
                              hipStream_t st) {
    const int64_t nseg = rans_segments(d);
    char* p = scratch;
    auto take = [&](size_t b) {
        char* r = p;
        p += align256(b);
        return r;
    };
    auto* hist = reinterpret_cast<unsigned long long*>(take(sizeof(unsigned long long) * 256));
    auto* fc = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * 512));
    (void)take(sizeof(uint32_t) * 4);
    auto* lens = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * (size_t)nseg));
    auto* starts = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * (size_t)nseg));
    (void)take(sizeof(unsigned long long));
    auto* regions = reinterpret_cast<uint8_t*>(p);
    hipError_t e = hipMemsetAsync(hist, 0, sizeof(unsigned long long) * 256, st);
    if (e != hipSuccess) return e;
    int64_t g = (d + 255) / 256;
    if (g > 1024) g = 1024;
    k_sym_hist<<<(unsigned)g, 256, 0, st>>>(sym, d, t, hist, bad);
    k_rans_freqs<<<1, 64, 0, st>>>(hist, t, d, fc, out);
    k_rans_encode<<<(unsigned)((nseg + 63) / 64), 64, 0, st>>>(sym, d, fc, t, regions, lens, nseg);
    k_rans_offsets<<<1, kRScan, 0, st>>>(lens, nseg, out + 2 * t, starts, total_out);
    k_rans_pack<<<(unsigned)nseg, 256, 0, st>>>(regions, lens, starts,
                                                out + 2 * (int64_t)t + 4 * nseg);
    return hipGetLastError();
}

hipError_t launch_rans_decode(const uint8_t* in, int64_t nin, int64_t d, int32_t t, uint8_t* sym,
                              unsigned int* bad, hipStream_t st) {
    const int64_t nseg = rans_segments(d);
    k_rans_decode<<<(unsigned)((nseg + 63) / 64), 64, 0, st>>>(in, nin, d, t, nseg, sym, bad);
    return hipGetLastError();
}

}  // namespace ecasq
