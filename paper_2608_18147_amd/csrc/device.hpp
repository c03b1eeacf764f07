// Device-side arithmetic of the ECASQ approximate DP (arXiv 2608.18147).
//
// Every function here evaluates one fixed fp64 operation sequence (the
// library is built with -ffp-contract=off, so fma appears only where written)
// so that results are reproducible bit for bit:
//
//   interval (v_a, v_b], a < b, from inclusive prefix sums (App. D):
//     n = N[b]-N[a]  sa = S[b]-S[a]  s2 = S2[b]-S2[a]  w = v_b-v_a
//     tu = fma(-v_a, n, sa)    (= w * U[a,b])
//     td = fma(v_b, n, -sa)    (= w * D[a,b])
//     C  = fma(v_b, tu, fma(v_a, sa, -s2))     (= C_P[a,b])
//   surrogate-entropy term of one interval (Sec. 5, Phi and Phi^first):
//     g = 1/(w*d)  yu = tu*g  yd = td*g (+ c0/d for the first interval)
//     mu = max(yu,0)  md = max(yd,0)
//     P = fma(mu, log2c(mu), md*log2c(md))                    (P = -Phi)
//   DP candidate (eq. apx_rec):  F_prev + Q,  Q = fma(-lambda', P, C)
//   refinement / output entropy (Sec. 6):
//     U = tu*(1/w)  D = td*(1/w)   h(f) = -(m*log2c(m)),  m = max(f/d, 0)
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "exp2_table.inc"
#include "log2_table.inc"

namespace ecasq {

constexpr int kLog2Bits = ECASQ_LOG2_BITS;
constexpr int kLog2Size = 1 << kLog2Bits;

// Table-driven log2 (Tang 1990 style).  e comes from y's high word minus an
// offset, so that z = ldexp(y, -e) lies in [0.7073, 1.4146) for positive
// normal y; the top 10 bits of the reduced mantissa select {1/c, log2 c};
// r = z/c - 1 (|r| <= 2^-11) feeds the degree-5 series of log1p with
// RN(1/ln 2) folded into its coefficients, c_k = RN(RN(1/ln 2) RN(+-1/k)).  Finite for every y >= 0 (callers pass max(y, 0)); about one ulp
// for positive normal y.
// tab points to the table in LDS.
//
// Evaluation order on the device: u = (OFF_HI + 0xFFFFF) - hi gives
// -e = u >> 20 (arithmetic) in one subtraction and, in bits 10..19, the
// complement 1023 - i of the table index, so the LDS copy of the table is
// stored in reverse; e + lc is formed as lc - (double)(-e), the same IEEE sum.
// log2c in two parts, for callers that issue several table reads before
// using any: the reduction and the table index, then the series.
struct Log2Arg {
    double z;   // ldexp(y, -e)
    int32_t ne; // -e
    uint32_t ir; // mirrored table index
};

__device__ __forceinline__ Log2Arg log2c_arg(double y) {
    const uint32_t hi = (uint32_t)__double2hiint(y);
    const int32_t u = (int32_t)((ECASQ_LOG2_OFF_HI + 0xFFFFFu) - hi);
    Log2Arg r;
    r.ne = u >> 20;  // -e
    r.ir = ((uint32_t)u >> (20 - kLog2Bits)) & (kLog2Size - 1);
    r.z = __builtin_ldexp(y, r.ne);
    return r;
}

__device__ __forceinline__ double log2c_fin(const Log2Arg& a, double2 t) {
    const double r = __builtin_fma(a.z, t.x, -1.0);
    constexpr double K = 0x1.71547652b82fep+0;
    double q = K * (1.0 / 5.0);
    q = __builtin_fma(q, r, K * -0.25);
    q = __builtin_fma(q, r, K * (1.0 / 3.0));
    q = __builtin_fma(q, r, K * -0.5);
    q = __builtin_fma(q, r, K * 1.0);
    const double base = t.y - (double)a.ne;
    return __builtin_fma(r, q, base);
}

__device__ __forceinline__ double log2c(double y, const double2* __restrict__ tab) {
    const Log2Arg a = log2c_arg(y);
    return log2c_fin(a, tab[a.ir]);
}

// Table-driven base-2 exponential (Tang 1989 style): y = k/64 + r with
// k = RN(64 y) (64 y is exact) and r = (64 y - k) / 64 (exact, |r| <= 1/128);
// 2^y = 2^floor(k/64) * T[k mod 64] * 2^r with T[i] = RN(2^(i/64)) and
// 2^r - 1 = r (C1 + C2 r + ... + C5 r^4), C_k = RN(ln(2)^k / k!).  About one
// ulp for |y| < 1000; NaN stays NaN, y <= -1100 gives 0, y >= 1100 gives +inf.
__device__ __forceinline__ double exp2c(double y) {
    if (y != y) return y;
    if (!(y > -1100.0)) return 0.0;
    if (!(y < 1100.0)) return __builtin_huge_val();
    const double y64 = y * 64.0;
    const double kd = __builtin_rint(y64);
    const double r = (y64 - kd) * 0x1p-6;
    const int64_t k = (int64_t)kd;
    const int32_t i = (int32_t)(k & 63);
    const int32_t e = (int32_t)((k - i) / 64);
    double q = kExp2Coef[4];
    q = __builtin_fma(q, r, kExp2Coef[3]);
    q = __builtin_fma(q, r, kExp2Coef[2]);
    q = __builtin_fma(q, r, kExp2Coef[1]);
    q = __builtin_fma(q, r, kExp2Coef[0]);
    const double pm1 = q * r;
    const double t = kExp2Table[i];
    return __builtin_ldexp(__builtin_fma(t, pm1, t), e);
}

// The budget search's aimed multiplier (one multiplier per pass): the slope
// at H = b of the curve through the bracketing points A (H_A > b) and B on
// which log vNMSE is linear in H, in base 2:
//   r2 = (log2 M_B - log2 M_A) / (H_B - H_A),  M_b = M_A 2^(r2 (b - H_A)),
//   lq = -(r2 ln 2) M_b.
__device__ __forceinline__ double aim_query(double b, double HA, double MA, double HB, double MB,
                                            const double2* __restrict__ tab) {
    const double r2 = (log2c(MB, tab) - log2c(MA, tab)) / (HB - HA);
    const double mb = MA * exp2c(r2 * (b - HA));
    return -(r2 * 0x1.62e42fefa39efp-1) * mb;
}

// 1/x rounded to nearest for positive x with |log2 x| < 700: the hardware
// reciprocal refined by two Newton steps and one residual correction.  These
// are the same operations, in the same order, as the IEEE double division
// 1.0/x on this target when no operand scaling is needed (true in this range),
// so the result equals 1.0/x bit for bit.
__device__ __forceinline__ double recip_rn(double x) {
    double r = __builtin_amdgcn_rcp(x);
    double e = __builtin_fma(-x, r, 1.0);
    r = __builtin_fma(r, e, r);
    e = __builtin_fma(-x, r, 1.0);
    r = __builtin_fma(r, e, r);
    e = __builtin_fma(-x, r, 1.0);
    return __builtin_fma(e, r, r);
}

// h(y) = -y log2 y for y > 0, 0 otherwise (Sec. 4).
__device__ __forceinline__ double hfun(double y, const double2* __restrict__ tab) {
    const double m = __builtin_fmax(y, 0.0);
    return -(m * log2c(m, tab));
}

// C and the clamped scaled frequencies mu = max(yu, 0), md = max(yd, 0) of
// the interval (v_a, v_b]: everything of cell_terms before the logarithms.
__device__ __forceinline__ void cell_pre(double va, double Na, double Sa, double S2a, double vb,
                                         double Nb, double Sb, double S2b, double dd, bool first,
                                         double c0d, double& C, double& mu, double& md) {
    const double n = Nb - Na;
    const double sa = Sb - Sa;
    const double s2 = S2b - S2a;
    const double w = vb - va;
    const double tu = __builtin_fma(-va, n, sa);
    const double td = __builtin_fma(vb, n, -sa);
    C = __builtin_fma(vb, tu, __builtin_fma(va, sa, -s2));
    const double wd = w * dd;  // in [2^-148, 2^157] for fp32 inputs and d <= 2^28
    const double g = recip_rn(wd);
    const double yu = tu * g;
    double yd = td * g;
    if (first) yd = yd + c0d;
    mu = __builtin_fmax(yu, 0.0);
    md = __builtin_fmax(yd, 0.0);
}

// C and P (= -Phi, or -Phi^first when `first`) of the interval (v_a, v_b].
__device__ __forceinline__ void cell_terms(double va, double Na, double Sa, double S2a, double vb,
                                           double Nb, double Sb, double S2b, double dd, bool first,
                                           double c0d, const double2* __restrict__ tab, double& C,
                                           double& P) {
    double mu, md;
    cell_pre(va, Na, Sa, S2a, vb, Nb, Sb, S2b, dd, first, c0d, C, mu, md);
    P = __builtin_fma(mu, log2c(mu, tab), md * log2c(md, tab));
}

// C alone, by the operations cell_terms uses for it.  At lambda' = 0 the DP
// candidate fma(-lambda', P, C) is C bit for bit: the product is a zero (P is
// finite), and C is never -0 (v_b is never -0 and t_u > 0 when v_b = 0), so
// a solve at lambda = 0 needs no entropy terms.
__device__ __forceinline__ double cell_c(double va, double Na, double Sa, double S2a, double vb,
                                         double Nb, double Sb, double S2b) {
    const double n = Nb - Na;
    const double sa = Sb - Sa;
    const double s2 = S2b - S2a;
    const double tu = __builtin_fma(-va, n, sa);
    return __builtin_fma(vb, tu, __builtin_fma(va, sa, -s2));
}

// U and D of (v_a, v_b] in the refinement (inv) form.
__device__ __forceinline__ void interval_ud(double va, double Na, double Sa, double vb, double Nb,
                                            double Sb, double& U, double& D) {
    const double n = Nb - Na;
    const double sa = Sb - Sa;
    const double w = vb - va;
    const double tu = __builtin_fma(-va, n, sa);
    const double td = __builtin_fma(vb, n, -sa);
    const double inv = 1.0 / w;
    U = tu * inv;
    D = td * inv;
}

// Histogram view passed to the small (one-thread or one-block) kernels.
struct Hist {
    const double* v;
    const double* N;
    const double* S;
    const double* S2;
    int64_t p;
    double dd;   // d as a double
    double c0;   // count of v_0
    double c0d;  // RN(c0 / d)
};

__device__ __forceinline__ void cell_at(const Hist& H, int64_t a, int64_t b,
                                        const double2* __restrict__ tab, double& C, double& P) {
    cell_terms(H.v[a], H.N[a], H.S[a], H.S2[a], H.v[b], H.N[b], H.S[b], H.S2[b], H.dd, a == 0,
               H.c0d, tab, C, P);
}

__device__ __forceinline__ void ud_at(const Hist& H, int64_t a, int64_t b, double& U, double& D) {
    interval_ud(H.v[a], H.N[a], H.S[a], H.v[b], H.N[b], H.S[b], U, D);
}

__device__ __forceinline__ double hf(const Hist& H, double f, const double2* __restrict__ tab) {
    return hfun(f / H.dd, tab);
}

// Copy the log2 table into LDS in reverse order (see log2c); call from all
// threads, then __syncthreads().
__device__ __forceinline__ void load_log2_table(double2* lds) {
    for (int i = threadIdx.x; i < kLog2Size; i += blockDim.x)
        lds[kLog2Size - 1 - i] = make_double2(kLog2Table[i][0], kLog2Table[i][1]);
}

}  // namespace ecasq
