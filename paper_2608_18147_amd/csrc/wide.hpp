// Order-preserving keys of binary32 values and exact wide-integer prefix
// sums, shared by the single-vector prep kernels and the batched row solver.
//
// Every fp32 value (and so every fp16 / bf16 value) is an integer multiple of
// 2^-149: |x| = M * 2^(sh - 149) with M < 2^24.  Sums of x (S) and of x^2 (S2)
// are therefore exact two's-complement integers of 5 and 10 64-bit limbs,
// rounded to fp64 once, to nearest even.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ecasq {

constexpr int kSL = 5;    // limbs of the signed S accumulator
constexpr int kS2L = 10;  // limbs of the S2 accumulator

// Order-preserving map from binary32 bits (finite) to uint32; -0 becomes +0.
__device__ __forceinline__ uint32_t f32_key(uint32_t bits) {
    if (bits == 0x80000000u) bits = 0u;
    return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}

__device__ __forceinline__ uint32_t key_bits(uint32_t k) {
    return (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
}

// ---- wide integers ---------------------------------------------------------

// a += (neg ? -X : X) mod 2^(64L), where X = (hi:lo) << (64*word).
template <int L>
__device__ __forceinline__ void wide_add(uint64_t (&a)[L], int word, uint64_t lo, uint64_t hi,
                                         bool neg) {
    uint64_t carry = neg ? 1ull : 0ull;
#pragma unroll
    for (int l = 0; l < L; l++) {
        uint64_t x = (l == word) ? lo : ((l == word + 1) ? hi : 0ull);
        if (neg) x = ~x;
        const uint64_t t = a[l] + x;
        const uint64_t c1 = t < x;
        const uint64_t t2 = t + carry;
        const uint64_t c2 = t2 < carry;
        a[l] = t2;
        carry = c1 | c2;
    }
}

template <int L>
__device__ __forceinline__ void wide_add_full(uint64_t* a, const uint64_t* b) {
    uint64_t carry = 0;
#pragma unroll
    for (int l = 0; l < L; l++) {
        const uint64_t t = a[l] + b[l];
        const uint64_t c1 = t < b[l];
        const uint64_t t2 = t + carry;
        const uint64_t c2 = t2 < carry;
        a[l] = t2;
        carry = c1 | c2;
    }
}

// Round the integer a (two's complement if is_signed) times 2^scale to the
// nearest double, ties to even.  Requires the result to be a normal double.
template <int L>
__device__ __forceinline__ double wide_to_double(const uint64_t (&a)[L], bool is_signed, int scale) {
    uint64_t m[L];
    const bool neg = is_signed && (a[L - 1] >> 63);
    uint64_t carry = 1;
#pragma unroll
    for (int l = 0; l < L; l++) {
        if (neg) {
            const uint64_t t = ~a[l] + carry;
            carry = (carry && t == 0) ? 1ull : 0ull;
            m[l] = t;
        } else {
            m[l] = a[l];
        }
    }
    int h = -1;
#pragma unroll
    for (int l = 0; l < L; l++)
        if (m[l] != 0) h = l;
    if (h < 0) return 0.0;
    uint64_t top = 0, below = 0, rest = 0;
    int lz = 0;
#pragma unroll
    for (int l = 0; l < L; l++) {
        if (l == h) {
            lz = __clzll(m[l]);
            top = m[l] << lz;
        }
    }
#pragma unroll
    for (int l = 0; l < L; l++) {
        if (l == h - 1) {
            if (lz) top |= m[l] >> (64 - lz);
            below = lz ? (m[l] << lz) : m[l];
        }
        if (l < h - 1) rest |= m[l];
    }
    const bool sticky = (below | rest) != 0;
    uint64_t mant = top >> 11;
    const uint32_t rem = (uint32_t)(top & 0x7FFu);
    const bool up = rem > 0x400u || (rem == 0x400u && (sticky || (mant & 1ull)));
    mant += up ? 1ull : 0ull;
    const int e2 = 64 * h + (63 - lz) - 52 + scale;
    const double r = ldexp((double)mant, e2);
    return neg ? -r : r;
}

struct Term {
    uint32_t M;   // integer mantissa (<= 2^24)
    int sh;       // |x| = M * 2^(sh - 149)
    bool neg;
};

__device__ __forceinline__ Term term_of(uint32_t bits) {
    const uint32_t ex = (bits >> 23) & 0xFFu;
    const uint32_t mf = bits & 0x7FFFFFu;
    Term t;
    t.M = ex ? (mf | 0x800000u) : mf;
    t.sh = ex ? (int)ex - 1 : 0;
    t.neg = (bits >> 31) != 0;
    return t;
}

__device__ __forceinline__ void accumulate(uint64_t (&s)[kSL], uint64_t (&q)[kS2L], const Term& t) {
    {
        const int b = t.sh & 63;
        const uint64_t M = t.M;
        const uint64_t lo = M << b;
        const uint64_t hi = b ? (M >> (64 - b)) : 0ull;
        wide_add<kSL>(s, t.sh >> 6, lo, hi, t.neg);
    }
    {
        const int sh2 = 2 * t.sh;
        const int b = sh2 & 63;
        const uint64_t M2 = (uint64_t)t.M * (uint64_t)t.M;
        const uint64_t lo = M2 << b;
        const uint64_t hi = b ? (M2 >> (64 - b)) : 0ull;
        wide_add<kS2L>(q, sh2 >> 6, lo, hi, false);
    }
}

}  // namespace ecasq
