/*
 * ECASQ approximate-DP oracle (plain C, fp64, slow, obviously correct).
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load this library.  It shares no code with
 * the GPU library; the two meet only through the canonical arithmetic stated
 * below, which each side implements on its own.
 *
 * What it computes (paper: arXiv 2608.18147):
 *   - interval quantities C, U, D from prefix sums        (App. D, closed forms)
 *   - Phi and Phi^first surrogate-entropy terms           (Sec. 5, def. of Phi)
 *   - dp_APX base, recurrence and final minimum           (Sec. 5, eq. apx_base,
 *                                                          apx_rec, apx_final)
 *   - Hirschberg recovery of the codebook in O(p) space   (Sec. 5, last paragraph
 *                                                          before Lemma 4; Sec. 4.2)
 *   - a backpointer traceback, used as a cross-check
 *   - the lambda search for a budget b                    (Sec. 3 Lagrangian;
 *                                                          Sec. 5 budget tuning;
 *                                                          App. F.7 slope queries)
 *   - the three-colour refinement                         (Sec. 6)
 *
 * Canonical arithmetic (both sides evaluate exactly this, -ffp-contract=off,
 * fma only where written):
 *   interval (v_a, v_b], a < b:
 *     n  = N[b]-N[a]   sa = S[b]-S[a]   s2 = S2[b]-S2[a]   w = v_b - v_a
 *     tu = fma(-v_a, n, sa)        td = fma(v_b, n, -sa)
 *     C  = fma(v_b, tu, fma(v_a, sa, -s2))
 *   DP cell entropy (g form):
 *     g = 1/(w*d)   yu = tu*g   yd = td*g  (+ c0/d if a == 0, first interval)
 *     mu = max(yu,0)   md = max(yd,0)
 *     P = fma(mu, log2c(mu), md*log2c(md))                      (P = -Phi)
 *     Q    = fma(-lambda', P, C)                                  (the cell's cost)
 *     cand = F_prev + Q
 *   refinement / output-entropy (inv form):
 *     U = tu*(1/w)   D = td*(1/w)   h(f) = -(m*log2c(m)), m = max(f/d, 0)
 *   log2c: table-driven, see log2c() below.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OFF_HI 0x3FE6A200u /* entry 599 is centred on 1.0 */
#define TBITS 10
#define TSIZE (1 << TBITS)

/* log2(1 + r) ~ r * (c1 + c2 r + ... + c5 r^4) with c_k = RN(RN(1/ln 2) * RN((-1)^(k+1) / k)),
 * the degree-5 Taylor series of log1p scaled by 1/ln 2 (|r| <= 2^-11). */
#define L2K 0x1.71547652b82fep+0
#define L2C1 (L2K * 1.0)
#define L2C2 (L2K * -0.5)
#define L2C3 (L2K * (1.0 / 3.0))
#define L2C4 (L2K * -0.25)
#define L2C5 (L2K * (1.0 / 5.0))

static double g_invc[TSIZE];
static double g_lc[TSIZE];

void orc_set_log2_table(const double *invc, const double *lc)
{
    memcpy(g_invc, invc, sizeof g_invc);
    memcpy(g_lc, lc, sizeof g_lc);
}

/* Canonical base-2 logarithm.  For a positive normal y it returns log2(y) to
 * about one ulp; for y = 0 or a subnormal y it returns some finite value (its
 * callers multiply by y).  Steps: e = (high word of y minus an offset) >> 20
 * and z = ldexp(y, -e), so z lies in [~0.7073, ~1.4147) for positive normal y;
 * table entry i (top 10 bits of the reduced mantissa) gives invc ~ 1/z and
 * lc = log2(1/invc);
 * r = z*invc - 1 with |r| <= 2^-11; log2(1+r) from the degree-5 Taylor series of
 * log1p with RN(1/ln 2) folded into its coefficients. */
static double log2c(double y)
{
    uint64_t bits;
    memcpy(&bits, &y, 8);
    uint32_t hi = (uint32_t)(bits >> 32);
    uint32_t tmp = hi - OFF_HI;
    int32_t e = ((int32_t)tmp) >> 20;
    uint32_t i = (tmp >> (20 - TBITS)) & (TSIZE - 1);
    double z = ldexp(y, -e);
    double r = fma(z, g_invc[i], -1.0);
    double q = L2C5;
    q = fma(q, r, L2C4);
    q = fma(q, r, L2C3);
    q = fma(q, r, L2C2);
    q = fma(q, r, L2C1);
    double base = (double)e + g_lc[i];
    return fma(r, q, base);
}

double orc_log2c(double y) { return log2c(y); }

/* Canonical base-2 exponential (Tang 1989, table-driven).  y = k/64 + r with
 * k = RN(64 y) (64 y is exact) and r = (64 y - k) / 64, exact, |r| <= 1/128;
 * 2^y = 2^floor(k/64) * T[k mod 64] * 2^r with T[i] = RN(2^(i/64)) and
 * 2^r - 1 = r * (C1 + C2 r + C3 r^2 + C4 r^3 + C5 r^4), C_k = RN(ln(2)^k / k!)
 * (the Taylor series of e^(r ln 2), truncation below 2^-60 here).  About one
 * ulp for |y| < 1000; NaN stays NaN, y <= -1100 gives 0, y >= 1100 gives +inf. */
static double g_exp2t[64];
static double g_exp2k[5];

void orc_set_exp2_table(const double *t, const double *c)
{
    memcpy(g_exp2t, t, sizeof g_exp2t);
    memcpy(g_exp2k, c, sizeof g_exp2k);
}

static double exp2c(double y)
{
    if (y != y) return y;
    if (!(y > -1100.0)) return 0.0;
    if (!(y < 1100.0)) return INFINITY;
    double y64 = y * 64.0;
    double kd = rint(y64);
    double r = (y64 - kd) * 0x1p-6;
    int64_t k = (int64_t)kd;
    int32_t i = (int32_t)(k & 63);
    int32_t e = (int32_t)((k - i) / 64);
    double q = g_exp2k[4];
    q = fma(q, r, g_exp2k[3]);
    q = fma(q, r, g_exp2k[2]);
    q = fma(q, r, g_exp2k[1]);
    q = fma(q, r, g_exp2k[0]);
    double pm1 = q * r;
    double m = fma(g_exp2t[i], pm1, g_exp2t[i]);
    return ldexp(m, e);
}

double orc_exp2c(double y) { return exp2c(y); }

/* The width-1 search's aimed multiplier (see orc_search): the slope at H = b
 * of the curve through A and B on which log vNMSE is linear in H, in base 2:
 *   r2 = (log2 M_B - log2 M_A) / (H_B - H_A),  M_b = M_A 2^(r2 (b - H_A)),
 *   lq = -(r2 ln 2) M_b. */
static double aim_query(double b, double HA, double MA, double HB, double MB)
{
    double r2 = (log2c(MB) - log2c(MA)) / (HB - HA);
    double mb = MA * exp2c(r2 * (b - HA));
    return -(r2 * 0x1.62e42fefa39efp-1) * mb;
}

double orc_aim_query(double b, double HA, double MA, double HB, double MB)
{
    return aim_query(b, HA, MA, HB, MB);
}

/* h(y) = -y log2 y for y > 0, 0 otherwise (Sec. 4, definition of h). */
static double hfun(double y)
{
    double m = fmax(y, 0.0);
    return -(m * log2c(m));
}

double orc_h(double y) { return hfun(y); }

typedef struct {
    const double *v;  /* sorted unique values v_0 < ... < v_{p-1} */
    const double *N;  /* inclusive prefix counts (exact in fp64) */
    const double *S;  /* inclusive prefix sums of c*v, correctly rounded */
    const double *S2; /* inclusive prefix sums of c*v^2, correctly rounded */
    int64_t p;
    double dd;  /* d as a double */
    double c0;  /* count of v_0 */
    double c0d; /* RN(c0 / d) */
    double s2tot; /* ||X||^2 = S2[p-1] */
} hist_t;

/* C[a,b] and the DP-form P = -Phi (Phi^first when a == 0) of the interval
 * (v_a, v_b].  App. D closed forms; Sec. 5 definition of Phi and Phi^first. */
static void cell_terms(const hist_t *H, int64_t a, int64_t b, double *C, double *P)
{
    double va = H->v[a], vb = H->v[b];
    double n = H->N[b] - H->N[a];
    double sa = H->S[b] - H->S[a];
    double s2 = H->S2[b] - H->S2[a];
    double w = vb - va;
    double tu = fma(-va, n, sa);
    double td = fma(vb, n, -sa);
    *C = fma(vb, tu, fma(va, sa, -s2));
    double wd = w * H->dd;
    double g = 1.0 / wd;
    double yu = tu * g;
    double yd = td * g;
    if (a == 0)
        yd = yd + H->c0d;
    double mu = fmax(yu, 0.0);
    double md = fmax(yd, 0.0);
    *P = fma(mu, log2c(mu), md * log2c(md));
}

/* U[a,b] and D[a,b] of (v_a, v_b] in the inv form (App. D closed forms). */
static void interval_ud(const hist_t *H, int64_t a, int64_t b, double *U, double *D)
{
    double va = H->v[a], vb = H->v[b];
    double n = H->N[b] - H->N[a];
    double sa = H->S[b] - H->S[a];
    double w = vb - va;
    double tu = fma(-va, n, sa);
    double td = fma(vb, n, -sa);
    double inv = 1.0 / w;
    *U = tu * inv;
    *D = td * inv;
}

static double interval_c(const hist_t *H, int64_t a, int64_t b)
{
    double C, P;
    cell_terms(H, a, b, &C, &P);
    return C;
}

static double hf(const hist_t *H, double f) { return hfun(f / H->dd); }

/* Interval quantities of (v_a, v_b] for tests: C, U, D (inv form), P (DP form). */
void orc_interval(const double *v, const double *N, const double *S, const double *S2,
                  int64_t p, int64_t d, int64_t a, int64_t b, double *out)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    double C, P, U, D;
    cell_terms(&H, a, b, &C, &P);
    interval_ud(&H, a, b, &U, &D);
    out[0] = C; out[1] = U; out[2] = D; out[3] = P;
}

/* ------------------------------------------------------------------------- */
/* Approximate DP, forward, O(p) rolling layers (Sec. 5).                      */

typedef struct {
    double J;    /* min_i F_i[p-1], MSE units */
    double mse;  /* MSE of the minimising path (accumulated along argmins) */
    double phi;  /* H(I,B) of that path, bits */
    int32_t t;   /* number of values i* */
    int64_t cells;
} dp_result;

/*
 * F_2[j]   = C[0,j] + lambda' Phi^first[0,j]                      (eq. apx_base)
 * F_i[j]   = min_{i-2 <= k < j} F_{i-1}[k] + C[k,j] + lambda' Phi[k,j]  (eq. apx_rec)
 * answer   = min_{2 <= i <= min(s,p)} F_i[p-1]                       (eq. apx_final)
 * Ties: lowest k, lowest i.  mse/phi are carried along the chosen k.
 * bp (optional, (s+1)*p int32): bp[i*p+j] = argmin k of layer i.
 * fdump (optional, (s+1)*p doubles): F_i[j] for every layer.
 */
int orc_dp_forward(const double *v, const double *N, const double *S, const double *S2,
                   int64_t p, int64_t d, int32_t s, int32_t exact_s, double lamp,
                   double *out /* J, mse, phi, t, cells */, int32_t *bp, double *fdump,
                   double *lastF /* optional [s+1] */)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    dp_result R = {0.0, 0.0, 0.0, 1, 0};
    if (p == 1) {
        out[0] = 0.0; out[1] = 0.0; out[2] = 0.0; out[3] = 1; out[4] = 0;
        return 0;
    }
    int32_t imax = (int32_t)((int64_t)s < p ? s : p);
    double *F0 = malloc(sizeof(double) * p), *F1 = malloc(sizeof(double) * p);
    double *M0 = malloc(sizeof(double) * p), *M1 = malloc(sizeof(double) * p);
    double *P0 = malloc(sizeof(double) * p), *P1 = malloc(sizeof(double) * p);
    if (!F0 || !F1 || !M0 || !M1 || !P0 || !P1)
        return -4;
    double bestJ = INFINITY, bestM = 0, bestP = 0;
    int32_t bestI = 2;
    /* layer 2 */
    F0[0] = INFINITY; M0[0] = 0; P0[0] = 0;
    for (int64_t j = 1; j < p; j++) {
        double C, P;
        cell_terms(&H, 0, j, &C, &P);
        F0[j] = fma(-lamp, P, 0.0 + C);
        M0[j] = 0.0 + C;
        P0[j] = 0.0 - P;
        if (bp) bp[2 * p + j] = 0;
    }
    R.cells += p - 1;
    if (fdump) memcpy(fdump + 2 * p, F0, sizeof(double) * p);
    if (lastF) lastF[2] = F0[p - 1];
    bestJ = F0[p - 1]; bestM = M0[p - 1]; bestP = P0[p - 1]; bestI = 2;
    for (int32_t i = 3; i <= imax; i++) {
        int64_t klo = i - 2, jlo = i - 1;
        for (int64_t j = 0; j < jlo; j++) { F1[j] = INFINITY; M1[j] = 0; P1[j] = 0; }
#pragma omp parallel for schedule(dynamic, 64)
        for (int64_t j = jlo; j < p; j++) {
            double best = INFINITY;
            int64_t bk = -1;
            for (int64_t k = klo; k < j; k++) {
                double C, P;
                cell_terms(&H, k, j, &C, &P);
                double cand = F0[k] + fma(-lamp, P, C);
                if (cand < best) { best = cand; bk = k; }
            }
            F1[j] = best;
            if (bk >= 0) {
                double C, P;
                cell_terms(&H, bk, j, &C, &P);
                M1[j] = M0[bk] + C;
                P1[j] = P0[bk] - P;
            } else {
                M1[j] = 0; P1[j] = 0;
            }
            if (bp) bp[(int64_t)i * p + j] = (int32_t)bk;
        }
        for (int64_t j = jlo; j < p; j++) R.cells += j - klo;
        if (fdump) memcpy(fdump + (int64_t)i * p, F1, sizeof(double) * p);
        if (lastF) lastF[i] = F1[p - 1];
        if (exact_s ? (i == imax) : (F1[p - 1] < bestJ)) {
            bestJ = F1[p - 1]; bestM = M1[p - 1]; bestP = P1[p - 1]; bestI = i;
        }
        double *t;
        t = F0; F0 = F1; F1 = t;
        t = M0; M0 = M1; M1 = t;
        t = P0; P0 = P1; P1 = t;
    }
    free(F0); free(F1); free(M0); free(M1); free(P0); free(P1);
    out[0] = bestJ; out[1] = bestM; out[2] = bestP; out[3] = bestI; out[4] = (double)R.cells;
    return 0;
}

/* Sampled columns of one layer: for each j in cols (j >= layer - 1), eq. apx_base
 * (layer 2: the interval (v_0, v_j] with the first-interval entropy term) or
 * eq. apx_rec (layer >= 3: min over layer-2 <= k < j of
 * Fprev[k] + C[k,j] + lambda' Phi[k,j], lowest k on ties), and the MSE and
 * H(I,B) accumulators carried from the argmin.  Fprev, Mprev, Pprev: the full
 * previous layer (unused for layer 2).  Lets a caller check any column of any
 * layer from the layer before it without running the whole DP.              */
void orc_dp_columns(const double *v, const double *N, const double *S, const double *S2,
                    int64_t p, int64_t d, int32_t layer, double lamp, const double *Fprev,
                    const double *Mprev, const double *Pprev, int64_t ncols, const int64_t *cols,
                    double *F, int32_t *K, double *M, double *Ph)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t x = 0; x < ncols; x++) {
        int64_t j = cols[x];
        double C, P;
        if (layer == 2) {
            cell_terms(&H, 0, j, &C, &P);
            F[x] = fma(-lamp, P, 0.0 + C);
            K[x] = 0;
            M[x] = 0.0 + C;
            Ph[x] = 0.0 - P;
            continue;
        }
        double best = INFINITY;
        int64_t bk = -1;
        for (int64_t k = layer - 2; k < j; k++) {
            cell_terms(&H, k, j, &C, &P);
            double cand = Fprev[k] + fma(-lamp, P, C);
            if (cand < best) { best = cand; bk = k; }
        }
        F[x] = best;
        K[x] = (int32_t)bk;
        if (bk >= 0) {
            cell_terms(&H, bk, j, &C, &P);
            M[x] = Mprev[bk] + C;
            Ph[x] = Pprev[bk] - P;
        } else {
            M[x] = 0.0;
            Ph[x] = 0.0;
        }
    }
}

/* Traceback through stored argmins (cross-check for Hirschberg). */
void orc_traceback(const int32_t *bp, int64_t p, int32_t t, int32_t *chain)
{
    chain[t - 1] = (int32_t)(p - 1);
    for (int32_t i = t; i >= 3; i--)
        chain[i - 2] = bp[(int64_t)i * p + chain[i - 1]];
    chain[0] = 0;
}

/* ------------------------------------------------------------------------- */
/* Hirschberg recovery (Sec. 5, specialised from Sec. 4.2): find the best chain
 * lo = u_0 < ... < u_{n-1} = hi by a forward half-DP over r+1 values from lo,
 * a backward half-DP over n-r values to hi, a split at the lowest m minimising
 * Fw[m] + Bw[m], and recursion on both halves.  r = floor((n-1)/2).            */

static int64_t g_hb_cells;

static void hb_forward(const hist_t *H, double lamp, int64_t lo, int64_t hi, int n, int q_end,
                       double *F /* indexed by j - lo */)
{
    int64_t len = hi - lo + 1;
    double *G = malloc(sizeof(double) * len);
    for (int64_t x = 0; x < len; x++) F[x] = INFINITY;
    F[0] = 0.0;
    for (int q = 2; q <= q_end; q++) {
        int64_t jl = lo + q - 1, jh = hi - (n - q);
        int64_t kl = lo + q - 2;
        /* at q = 2 the only finite predecessor is lo itself */
        for (int64_t x = 0; x < len; x++) G[x] = INFINITY;
#pragma omp parallel for schedule(dynamic, 64)
        for (int64_t j = jl; j <= jh; j++) {
            double best = INFINITY;
            int64_t ke = (q == 2) ? lo : j - 1;
            for (int64_t k = kl; k <= ke; k++) {
                double C, P;
                cell_terms(H, k, j, &C, &P);
                double cand = F[k - lo] + fma(-lamp, P, C);
                if (cand < best) best = cand;
            }
            G[j - lo] = best;
        }
        for (int64_t j = jl; j <= jh; j++) g_hb_cells += (q == 2) ? 1 : j - kl;
        memcpy(F, G, sizeof(double) * len);
    }
    free(G);
}

static void hb_backward(const hist_t *H, double lamp, int64_t lo, int64_t hi, int n, int q_end,
                        double *B /* indexed by j - lo */)
{
    int64_t len = hi - lo + 1;
    double *G = malloc(sizeof(double) * len);
    for (int64_t x = 0; x < len; x++) B[x] = INFINITY;
    B[len - 1] = 0.0;
    for (int q = 2; q <= q_end; q++) {
        int64_t jl = lo + (n - q), jh = hi - q + 1;
        int64_t kh = hi - q + 2;
        for (int64_t x = 0; x < len; x++) G[x] = INFINITY;
#pragma omp parallel for schedule(dynamic, 64)
        for (int64_t j = jl; j <= jh; j++) {
            double best = INFINITY;
            int64_t ks = (q == 2) ? hi : j + 1; /* at q = 2 only hi is finite */
            for (int64_t k = ks; k <= kh; k++) {
                double C, P;
                cell_terms(H, j, k, &C, &P);
                double cand = B[k - lo] + fma(-lamp, P, C);
                if (cand < best) best = cand;
            }
            G[j - lo] = best;
        }
        for (int64_t j = jl; j <= jh; j++) g_hb_cells += (q == 2) ? 1 : kh - j;
        memcpy(B, G, sizeof(double) * len);
    }
    free(G);
}

static void hb_solve(const hist_t *H, double lamp, int64_t lo, int64_t hi, int n, int32_t *out)
{
    if (n == 2) { out[0] = (int32_t)lo; out[1] = (int32_t)hi; return; }
    if (hi - lo + 1 == n) {
        for (int x = 0; x < n; x++) out[x] = (int32_t)(lo + x);
        return;
    }
    int r = (n - 1) / 2;
    int64_t len = hi - lo + 1;
    double *Fw = malloc(sizeof(double) * len), *Bw = malloc(sizeof(double) * len);
    hb_forward(H, lamp, lo, hi, n, r + 1, Fw);
    hb_backward(H, lamp, lo, hi, n, n - r, Bw);
    int64_t m = -1;
    double best = INFINITY;
    for (int64_t x = lo + r; x <= hi - (n - 1 - r); x++) {
        double tot = Fw[x - lo] + Bw[x - lo];
        if (tot < best) { best = tot; m = x; }
    }
    free(Fw); free(Bw);
    hb_solve(H, lamp, lo, m, r + 1, out);
    hb_solve(H, lamp, m, hi, n - r, out + r);
}

int orc_hirschberg(const double *v, const double *N, const double *S, const double *S2,
                   int64_t p, int64_t d, int32_t t, double lamp, int32_t *chain, int64_t *cells)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    g_hb_cells = 0;
    if (t == 1) { chain[0] = 0; if (cells) *cells = 0; return 0; }
    hb_solve(&H, lamp, 0, p - 1, t, chain);
    if (cells) *cells = g_hb_cells;
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Metrics of a chain of unique indices u_0 = 0 < ... < u_{t-1} = p-1.        */

/* Expected frequency of every value (Sec. 4: f = U[k,l] + D[l,j]; the first
 * value also takes every entry equal to it, the last takes the round-up mass
 * of the last interval). */
static void chain_freqs(const hist_t *H, int32_t t, const int32_t *u, double *f)
{
    if (t == 1) { f[0] = H->dd; return; }
    double Uprev = 0;
    for (int32_t r = 0; r < t; r++) {
        double Ur = 0, Dr = 0;
        if (r + 1 < t) interval_ud(H, u[r], u[r + 1], &Ur, &Dr);
        if (r == 0) f[0] = H->c0 + Dr;
        else if (r == t - 1) f[r] = Uprev;
        else f[r] = Uprev + Dr;
        Uprev = Ur;
    }
}

static double chain_hout(const hist_t *H, int32_t t, const int32_t *u)
{
    double *f = malloc(sizeof(double) * t);
    chain_freqs(H, t, u, f);
    double Hs = 0.0;
    for (int32_t r = 0; r < t; r++) Hs = Hs + hf(H, f[r]);
    free(f);
    return Hs;
}

/* out: mse, vnmse, H(Xhat), H(I,B), J = vNMSE + lambda*H(Xhat), R_tot */
void orc_chain_metrics(const double *v, const double *N, const double *S, const double *S2,
                       int64_t p, int64_t d, int32_t t, const int32_t *u, double lam, double *out)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    double mse = 0.0, hs = 0.0;
    for (int32_t r = 0; r + 1 < t; r++) {
        double C, P;
        cell_terms(&H, u[r], u[r + 1], &C, &P);
        mse = mse + C;
        hs = hs - P;
    }
    double ho = chain_hout(&H, t, u);
    double vn = H.s2tot > 0 ? mse / H.s2tot : 0.0;
    double lr = isfinite(lam) ? lam : 0.0;
    out[0] = mse;
    out[1] = vn;
    out[2] = ho;
    out[3] = hs;
    out[4] = fma(lr, ho, vn);
    out[5] = ho + (32.0 * (double)t) / H.dd;
}

/* ------------------------------------------------------------------------- */
/* Three-colour refinement (Sec. 6).                                           */

/* Local objective of moving u_r to m with u_{r-1}, u_{r+1} (and u_{r-2},
 * u_{r+2}) fixed: the two interval MSEs plus lambda' times the entropy terms of
 * the three values whose expected frequencies change. */
static double refine_local(const hist_t *H, int32_t t, const int32_t *u, int32_t r, int64_t m,
                           double lamp)
{
    int64_t L = u[r - 1], R = u[r + 1];
    double Cl = interval_c(H, L, m), Cr = interval_c(H, m, R);
    double Ulm, Dlm, Umr, Dmr;
    interval_ud(H, L, m, &Ulm, &Dlm);
    interval_ud(H, m, R, &Umr, &Dmr);
    double fprev, fnext;
    if (r - 1 == 0) {
        fprev = H->c0 + Dlm;
    } else {
        double Ua, Da;
        interval_ud(H, u[r - 2], L, &Ua, &Da);
        fprev = Ua + Dlm;
    }
    double fcur = Ulm + Dmr;
    if (r + 1 == t - 1) {
        fnext = Umr;
    } else {
        double Ub, Db;
        interval_ud(H, R, u[r + 2], &Ub, &Db);
        fnext = Umr + Db;
    }
    double Hl = (hf(H, fprev) + hf(H, fcur)) + hf(H, fnext);
    return fma(lamp, Hl, Cl + Cr);
}

/* Exported for the tests that pin it: the local objective of mover r at m. */
double orc_refine_local(const double *v, const double *N, const double *S, const double *S2,
                        int64_t p, int64_t d, int32_t t, const int32_t *u, int32_t r, int64_t m,
                        double lamp)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    return refine_local(&H, t, u, r, m, lamp);
}

/* The position a mover r (1 <= r <= t-2) searches out in the open range
 * (u_{r-1}, u_{r+1}) (Sec. 6): the lowest minimiser of the local objective
 * (exhaustive), or the paper's binary search, which keeps the half whose
 * forward difference points downhill: lo = L+1, hi = R-1; while lo < hi,
 * mid = lo + (hi-lo)/2 and lo = mid+1 if L_r(mid+1) < L_r(mid), else hi = mid.
 * Returns u_r itself when the range holds only u_r. */
static int64_t refine_search(const hist_t *H, int32_t t, const int32_t *u, int32_t r,
                             double lamp, int32_t exhaustive)
{
    int64_t L = u[r - 1], R = u[r + 1];
    if (R - L < 3) return u[r];
    if (exhaustive) {
        double bv = INFINITY;
        int64_t m = -1;
        for (int64_t x = L + 1; x < R; x++) {
            double val = refine_local(H, t, u, r, x, lamp);
            if (val < bv) { bv = val; m = x; }
        }
        return m;
    }
    int64_t lo = L + 1, hi = R - 1;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (refine_local(H, t, u, r, mid + 1, lamp) < refine_local(H, t, u, r, mid, lamp))
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

int64_t orc_refine_search(const double *v, const double *N, const double *S, const double *S2,
                          int64_t p, int64_t d, int32_t t, const int32_t *u, int32_t r,
                          double lamp, int32_t exhaustive)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    return refine_search(&H, t, u, r, lamp, exhaustive);
}

/* One colour substep (Sec. 6): every mover r = c (mod 3), 1 <= r <= t-2,
 * searched against the chain u as it stands; a mover whose found position
 * strictly lowers its local objective moves there.  The new chain goes to nu
 * (u itself is not changed); returns the number of movers that moved.  Movers
 * of one colour are three apart, so the frequencies each of them changes
 * (its own and its two neighbours') are disjoint. */
static int32_t refine_substep(const hist_t *H, int32_t t, const int32_t *u, int32_t c,
                              double lamp, int32_t exhaustive, int32_t *nu)
{
    int32_t moved = 0;
    memcpy(nu, u, sizeof(int32_t) * t);
    for (int32_t r = 1; r <= t - 2; r++) {
        if (r % 3 != c) continue;
        int64_t m = refine_search(H, t, u, r, lamp, exhaustive);
        if (m != u[r] &&
            refine_local(H, t, u, r, m, lamp) < refine_local(H, t, u, r, u[r], lamp)) {
            nu[r] = (int32_t)m;
            moved++;
        }
    }
    return moved;
}

int32_t orc_refine_substep(const double *v, const double *N, const double *S, const double *S2,
                           int64_t p, int64_t d, int32_t t, const int32_t *u, int32_t c,
                           double lamp, int32_t exhaustive, int32_t *nu)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    if (t < 3) { memcpy(nu, u, sizeof(int32_t) * t); return 0; }
    return refine_substep(&H, t, u, c, lamp, exhaustive, nu);
}

/* Refines u in place: rounds of the substeps of colours 0, 1, 2 (Sec. 6),
 * stopping after a round in which nothing moved or after `rounds` rounds.
 * In budget mode a substep whose result has H(Xhat) > b is undone.  Returns
 * the number of rounds run. */
int orc_refine(const double *v, const double *N, const double *S, const double *S2, int64_t p,
               int64_t d, int32_t t, int32_t *u, double lamp, double b, int32_t budget_mode,
               int32_t rounds, int32_t exhaustive, int32_t *moves_out)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    int32_t nrun = 0, nmoves = 0;
    if (t < 3) { if (moves_out) *moves_out = 0; return 0; }
    int32_t *nu = malloc(sizeof(int32_t) * t);
    for (int32_t rd = 0; rd < rounds; rd++) {
        int any = 0;
        for (int32_t c = 0; c < 3; c++) {
            int32_t moved = refine_substep(&H, t, u, c, lamp, exhaustive, nu);
            if (moved && budget_mode && chain_hout(&H, t, nu) > b)
                moved = 0;
            if (moved) {
                memcpy(u, nu, sizeof(int32_t) * t);
                any = 1;
                nmoves += moved;
            }
        }
        nrun++;
        if (!any) break;
    }
    free(nu);
    if (moves_out) *moves_out = nmoves;
    return nrun;
}

/* ------------------------------------------------------------------------- */
/* Lambda search for a budget b (Sec. 3: search on lambda; Sec. 5: keep the
 * lowest-MSE solution with H(I,B) <= b), in passes of `width` multipliers
 * (width 8 or 1; lambda in vNMSE units; each query is one full DP solve at
 * lambda' = RN(lambda * ||X||^2)):
 *
 *   pass 1: lambda in {0, 1e-4, 1e-3, 1e-2, 1e-1, 1, 10, 100} (width 8) or
 *   {0} (width 1);
 *   then, with A = the infeasible point (H(I,B) > b) of largest lambda and
 *   B = the feasible point of smallest lambda (or, if none, the two-value
 *   codebook {v_0, v_{p-1}} when b >= 1, else the solve at lambda = 2^40):
 *     lc = (M_B - M_A) / (H_A - H_B), the slope of the chord AB (App. F.7
 *     supporting-line query);
 *     next pass: lc and width-1 more multipliers, la + (lb - la) g / 8 for
 *     g = 1..7 (or lc times 1/4, 1/2, 3/4, 3/2, 2, 3, 4 when B is the
 *     two-value codebook);
 *     width 1 with aim != 0 queries, instead of lc, the slope at H = b of the
 *     curve through A and B on which log(vNMSE) is linear in H:
 *       r2 = (log2 M_B - log2 M_A) / (H_B - H_A),  M_b = M_A 2^(r2 (b - H_A)),
 *       lq = -(r2 ln 2) M_b   (canonical log2c and exp2c, ln 2 rounded),
 *     when it lies strictly between la and lb and the previous such query found
 *     a new point; otherwise it queries lc;
 *   stop when the answer at lc is A or B again (H and M bit for bit): no DP
 *   solution lies below the chord, A and B are adjacent supported points.
 *
 * Width 1 is the plain sequential chord search.  Returns B, the multiplier at
 * which B was found (used to recover it) and the final chord slope lc (the
 * multiplier of the refinement step).  A query whose lambda equals that of a
 * point already solved reuses the point (no solve); a point's lambda is the
 * multiplier of its first query.
 *
 * cache (optional): points solved before, 4 doubles each (lambda, H(I,B),
 * vNMSE, t), *ncache of them; they join the point set from the start (grid
 * multipliers among them are not solved again), and the points this search
 * solves are appended (up to cap).  Searches for several budgets on one input
 * share their solves this way.
 * traj (optional, 4 doubles per solve): lambda, H(I,B), vNMSE, t.
 * replay (optional, nreplay points of 4 doubles as traj): instead of solving,
 * the n-th solve the search asks for takes the n-th replay point, whose
 * lambda must equal the query bit for bit; the search then returns -2 at the
 * first query that differs or runs past the list (a recorded trajectory is
 * checked against the decisions this search takes on its points).
 * out: lambda_B, H_B, M_B, t_B, solves, cells, status (0 ok, -3 infeasible),
 *      lambda_final, passes
 */
#define SEARCH_M 8
#define MAX_PTS 1024

typedef struct {
    double lam, H, M;
    int32_t t;
} point_t;

int orc_opt_dp(const double *v, const double *N, const double *S, const double *S2, int64_t p,
               int64_t d, int32_t s, int32_t exact_s, double lamp, int32_t *chain, double *out,
               int32_t *Kdump, double *Fdump);

/* One point of the search on the optimal DP (Sec. 4): r[1] = MSE and
 * r[2] = H(Xhat) of the optimal codebook at lamp (from its chain, as the
 * metrics sum them), r[3] = t, r[4] = cells. */
static void opt_point(const double *v, const double *N, const double *S, const double *S2,
                      int64_t p, int64_t d, int32_t s, int32_t exact_s, double lamp, double *r)
{
    int32_t *chain = malloc(sizeof(int32_t) * (size_t)(s > 2 ? s : 2));
    double o[3], m[6];
    orc_opt_dp(v, N, S, S2, p, d, s, exact_s, lamp, chain, o, NULL, NULL);
    orc_chain_metrics(v, N, S, S2, p, d, (int32_t)o[1], chain, 0.0, m);
    r[0] = o[0]; r[1] = m[0]; r[2] = m[2]; r[3] = o[1]; r[4] = o[2];
    free(chain);
}

/* One point of the refinement-aware search: the approximate DP's codebook at
 * lamp (the traceback of its argmins), refined at lamp without a budget guard
 * (Sec. 6), scored by its own MSE (r[1]) and H(Xhat) (r[2]); r[3] = t,
 * r[4] = the DP's cells. */
static void refined_point(const double *v, const double *N, const double *S, const double *S2,
                          int64_t p, int64_t d, int32_t s, int32_t exact_s, double lamp,
                          int32_t rounds, int32_t exhaustive, double *r)
{
    double o[5], m[6];
    int32_t *bp = malloc(sizeof(int32_t) * (size_t)(s + 1) * (size_t)p);
    int32_t *chain = malloc(sizeof(int32_t) * (size_t)(s > 2 ? s : 2));
    orc_dp_forward(v, N, S, S2, p, d, s, exact_s, lamp, o, bp, NULL, NULL);
    int32_t t = (int32_t)o[3];
    orc_traceback(bp, p, t, chain);
    if (t >= 3 && rounds > 0)
        orc_refine(v, N, S, S2, p, d, t, chain, lamp, INFINITY, 0, rounds, exhaustive, NULL);
    orc_chain_metrics(v, N, S, S2, p, d, t, chain, 0.0, m);
    r[0] = 0.0; r[1] = m[0]; r[2] = m[2]; r[3] = t; r[4] = o[4];
    free(bp);
    free(chain);
}

int orc_search(const double *v, const double *N, const double *S, const double *S2, int64_t p,
               int64_t d, int32_t s, double b, int32_t exact_s, int32_t max_passes, int32_t width,
               int32_t aim, int32_t dp_kind, int32_t refine_rounds, int32_t refine_exhaustive,
               double *cache, int32_t *ncache, int32_t cache_cap, double *traj,
               int32_t traj_cap, const double *replay, int32_t nreplay, double *out)
{
    if (width != 1 && width != SEARCH_M) return -1;
    if (dp_kind != 0 && width != 1) return -1;
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    double r[5];
    int32_t nsol = 0, npass = 0;
    double cells = 0;
    point_t *pts = malloc(sizeof(point_t) * MAX_PTS);
    int32_t npts = 0;
    if (cache && ncache) {
        for (int32_t x = 0; x < *ncache && npts < MAX_PTS; x++) {
            pts[npts].lam = cache[4 * x]; pts[npts].H = cache[4 * x + 1];
            pts[npts].M = cache[4 * x + 2]; pts[npts].t = (int32_t)cache[4 * x + 3];
            npts++;
        }
    }
    int32_t ncached = npts;
    if (p <= 2) {
        /* every value is used; nothing to search */
        out[0] = 0.0; out[1] = 0.0; out[2] = 0.0; out[3] = (double)p; out[4] = 0; out[5] = 0;
        out[6] = 0; out[7] = 0.0; out[8] = 0;
        out[9] = out[10] = out[11] = out[12] = NAN;
        if (p == 2) {
            double C, P;
            cell_terms(&H, 0, 1, &C, &P);
            out[1] = 0.0 - P;
            out[2] = (0.0 + C) / H.s2tot;
            if (dp_kind != 0) {
                int32_t two[2] = {0, 1};
                double m[6];
                orc_chain_metrics(v, N, S, S2, p, d, 2, two, 0.0, m);
                out[1] = m[2];
            }
            if (out[1] > b) out[6] = -3;
        }
        free(pts);
        return 0;
    }
    /* evaluate one multiplier: reuse a solved point of the same lambda, else a
       full DP solve */
#define EVAL(lam_)                                                                            \
    do {                                                                                      \
        double l_ = (lam_);                                                                   \
        int hit_ = 0;                                                                         \
        for (int x_ = 0; x_ < npts; x_++) if (pts[x_].lam == l_) { hit_ = 1; break; }          \
        if (!hit_) {                                                                          \
            double M_;                                                                        \
            if (replay) {                                                                     \
                if (nsol >= nreplay || replay[4 * nsol] != l_) goto replay_mismatch;          \
                r[2] = replay[4 * nsol + 1]; M_ = replay[4 * nsol + 2];                       \
                r[3] = replay[4 * nsol + 3]; r[4] = 0;                                        \
            } else {                                                                          \
                if (dp_kind == 1)                                                             \
                    opt_point(v, N, S, S2, p, d, s, exact_s, l_ * H.s2tot, r);                \
                else if (dp_kind == 2)                                                        \
                    refined_point(v, N, S, S2, p, d, s, exact_s, l_ * H.s2tot, refine_rounds, \
                                  refine_exhaustive, r);                                      \
                else                                                                          \
                    orc_dp_forward(v, N, S, S2, p, d, s, exact_s, l_ * H.s2tot, r, NULL, NULL, \
                                   NULL);                                                     \
                M_ = r[1] / H.s2tot;                                                          \
            }                                                                                 \
            if (npts < MAX_PTS) {                                                             \
                pts[npts].lam = l_; pts[npts].H = r[2]; pts[npts].M = M_;                     \
                pts[npts].t = (int32_t)r[3]; npts++;                                           \
            }                                                                                 \
            cells += r[4];                                                                    \
            if (traj && nsol < traj_cap) {                                                    \
                traj[4 * nsol] = l_; traj[4 * nsol + 1] = r[2];                               \
                traj[4 * nsol + 2] = M_; traj[4 * nsol + 3] = r[3];                           \
            }                                                                                 \
            nsol++;                                                                           \
        }                                                                                     \
    } while (0)
/* the point of a query (after EVAL) */
#define POINT_OF(lam_, dst_)                                                                  \
    do {                                                                                      \
        for (int x_ = 0; x_ < npts; x_++) if (pts[x_].lam == (lam_)) { dst_ = pts[x_]; break; } \
    } while (0)

    static const double grid[SEARCH_M] = {0.0, 1e-4, 1e-3, 1e-2, 1e-1, 1.0, 10.0, 100.0};
    {
        int32_t before = nsol;
        for (int g = 0; g < width; g++) EVAL(grid[g]);
        npass = nsol > before ? 1 : 0;
    }
    int32_t status = 0;
    point_t A, B;
    double lam_final = 0.0;
    int have_A = 0, have_B = 0, closed = 0, force_chord = 0;
    for (;;) {
        /* A: infeasible point of largest lambda; B: feasible point of smallest
           lambda (first occurrence wins among equal lambdas) */
        int ia = -1, ib = -1;
        for (int x = 0; x < npts; x++) {
            if (pts[x].H > b) {
                if (ia < 0 || pts[x].lam > pts[ia].lam) ia = x;
            } else {
                if (ib < 0 || pts[x].lam < pts[ib].lam) ib = x;
            }
        }
        if (ia < 0) { /* lambda = 0 is feasible */
            B = pts[ib]; have_B = 1; have_A = 0; lam_final = B.lam;
            break;
        }
        A = pts[ia];
        have_A = 1;
        if (ib >= 0) {
            B = pts[ib]; closed = 0;
        } else if (b >= 1.0) {
            double C, P;
            cell_terms(&H, 0, p - 1, &C, &P);
            B.lam = INFINITY; B.H = 0.0 - P; B.M = (0.0 + C) / H.s2tot; B.t = 2; closed = 1;
            if (dp_kind != 0) { /* H(Xhat) of {v_0, v_{p-1}} */
                int32_t two[2] = {0, (int32_t)(p - 1)};
                double m[6];
                orc_chain_metrics(v, N, S, S2, p, d, 2, two, 0.0, m);
                B.H = m[2];
            }
        } else {
            /* no feasible point yet: try the largest multiplier once */
            int tried = 0;
            for (int x = 0; x < npts; x++) if (pts[x].lam == 0x1p40) tried = 1;
            if (tried || npass >= max_passes) {
                /* infeasible budget: return the lowest-entropy point found */
                int ih = 0;
                for (int x = 1; x < npts; x++) if (pts[x].H < pts[ih].H) ih = x;
                B = pts[ih]; have_B = 1; have_A = 0; status = -3; lam_final = B.lam;
                break;
            }
            EVAL(0x1p40);
            npass++;
            continue;
        }
        have_B = 1;
        double lc = (B.M - A.M) / (A.H - B.H);
        lam_final = closed ? lc : B.lam;
        if (!(lc > 0.0) || npass >= max_passes) break;
        double q[SEARCH_M];
        q[0] = lc;
        /* width 1: aim at H = b first (the tangent slope at b of the curve
           through A and B on which log M is linear in H) while that finds new
           points; the chord query certifies the end */
        int model = 0;
        if (width == 1 && aim && !force_chord && A.M > 0.0 && B.M > 0.0) {
            double lq = aim_query(b, A.H, A.M, B.H, B.M);
            if (isfinite(lq) && lq > A.lam && lq < B.lam) {
                q[0] = lq;
                model = 1;
            }
        }
        for (int g = 1; g < width; g++) {
            if (closed) {
                static const double mul[SEARCH_M - 1] = {0.25, 0.5, 0.75, 1.5, 2.0, 3.0, 4.0};
                q[g] = lc * mul[g - 1];
            } else {
                q[g] = A.lam + ((B.lam - A.lam) * (double)g) / 8.0;
            }
        }
        for (int g = 0; g < width; g++) EVAL(q[g]);
        npass++;
        point_t Cq = pts[0];
        POINT_OF(q[0], Cq);
        if ((Cq.H == A.H && Cq.M == A.M) || (Cq.H == B.H && Cq.M == B.M)) {
            if (!model) {
                lam_final = lc;
                break;
            }
            force_chord = 1; /* the aimed query found nothing new */
        } else {
            force_chord = 0;
        }
    }
#undef EVAL
#undef POINT_OF
    (void)have_B;
    if (cache && ncache) {
        for (int32_t x = ncached; x < npts && *ncache < cache_cap; x++) {
            double *c = cache + 4 * (*ncache);
            c[0] = pts[x].lam; c[1] = pts[x].H; c[2] = pts[x].M; c[3] = (double)pts[x].t;
            (*ncache)++;
        }
    }
    out[0] = B.lam; out[1] = B.H; out[2] = B.M; out[3] = B.t; out[4] = nsol; out[5] = cells;
    out[6] = status; out[7] = lam_final; out[8] = npass;
    /* refined points need not lie on a convex curve: the answer is the
       feasible point of lowest vNMSE found (the first among equals) */
    if (dp_kind == 2 && status == 0) {
        int ib = -1;
        for (int x = 0; x < npts; x++)
            if (pts[x].H <= b && (ib < 0 || pts[x].M < pts[ib].M)) ib = x;
        if (ib >= 0) {
            out[0] = pts[ib].lam; out[1] = pts[ib].H; out[2] = pts[ib].M; out[3] = pts[ib].t;
        }
    }
    /* A: the infeasible point the final chord starts from (NaN if none) */
    out[9] = have_A ? A.lam : NAN; out[10] = have_A ? A.H : NAN;
    out[11] = have_A ? A.M : NAN; out[12] = have_A ? (double)A.t : NAN;
    free(pts);
    return 0;
replay_mismatch:
    out[4] = nsol;
    free(pts);
    return -2;
}

/* ------------------------------------------------------------------------- */
/* Optimal lambda-ECASQ (Sec. 4; App. D for the closed forms).                */
/*
 * State (i, l, j): the best cost of the values up to v_l using i-1 codebook
 * values that end at v_l, plus the MSE of (v_l, v_j] with v_l and v_j
 * adjacent in the codebook.  The expected frequency of v_l is then known:
 * U[k,l] + D[l,j], with k the codebook value before v_l.
 *
 *   layer 2 (l = 0):  dp(2,0,j) = C[0,j] + lambda' h(n_0/d + D[0,j]/d)
 *   layer i >= 3:     dp(i,l,j) = C[l,j] + min_k dp(i-1,k,l) + lambda' h(U[k,l]/d + D[l,j]/d)
 *                     k = 0 for i = 3, i-3 <= k < l for i >= 4, l in [i-2, p-2]
 *   answer:           min over i <= min(s,p) (i = min(s,p) with exact_s), then
 *                     over l, of dp(i,l,p-1) + lambda' h(U[l,p-1]/d)
 *
 * Every minimum takes the lowest index among ties (i, then l, then k).
 * Canonical arithmetic: U/d and D/d in the DP's g form (yu, yd of the apx
 * cell), e(y) = m log2c(m) with m = max(y, 0) (so lambda' h = -lambda' e):
 *   layer 2:  fma(-lambda', e(yd(0,j) + c0/d), C[0,j])
 *   T(k)   =  fma(-lambda', e(yu(k,l) + yd(l,j)), dp(i-1,k,l))
 *   dp     =  C[l,j] + min_k T(k)
 *   final  =  fma(-lambda', e(yu(l,p-1)), dp(i,l,p-1))
 * The minimum is over every admissible k (the definition; the SMAWK
 * acceleration of Sec. 4.1 finds the same minimiser when the matrix is Monge).
 */

/* yu = U[a,b]/d and yd = D[a,b]/d of (v_a, v_b] in the g form, and C[a,b]. */
static void interval_y(const hist_t *H, int64_t a, int64_t b, double *C, double *yu, double *yd)
{
    double va = H->v[a], vb = H->v[b];
    double n = H->N[b] - H->N[a];
    double sa = H->S[b] - H->S[a];
    double s2 = H->S2[b] - H->S2[a];
    double w = vb - va;
    double tu = fma(-va, n, sa);
    double td = fma(vb, n, -sa);
    *C = fma(vb, tu, fma(va, sa, -s2));
    double g = 1.0 / (w * H->dd);
    *yu = tu * g;
    *yd = td * g;
}

static double elog(double y)
{
    double m = fmax(y, 0.0);
    return m * log2c(m);
}

/* out: J' = MSE + lambda' H(Xhat) of the optimum (lambda' units), t, cells
 * (admissible (k, l, j) triples plus layer-2 and final entries).
 * chain (capacity s): the codebook's value indices.  Kdump (optional):
 * (min(s,p)+1) x p x p int32 argmins, -1 where undefined.  Fdump (optional):
 * the same shape of dp values (+inf where undefined). */
int orc_opt_dp(const double *v, const double *N, const double *S, const double *S2, int64_t p,
               int64_t d, int32_t s, int32_t exact_s, double lamp, int32_t *chain, double *out,
               int32_t *Kdump, double *Fdump)
{
    hist_t H = {v, N, S, S2, p, (double)d, N[0], N[0] / (double)d, S2[p - 1]};
    if (p == 1) {
        chain[0] = 0;
        out[0] = 0.0; out[1] = 1; out[2] = 0;
        return 0;
    }
    int64_t imax = s < p ? s : p;
    size_t pp = (size_t)p * (size_t)p;
    double *prev = malloc(sizeof(double) * pp);
    double *cur = malloc(sizeof(double) * pp);
    int32_t *K = malloc(sizeof(int32_t) * pp * (size_t)(imax + 1));
    if (!prev || !cur || !K) { free(prev); free(cur); free(K); return -4; }
    for (size_t q = 0; q < pp * (size_t)(imax + 1); q++) K[q] = -1;
    int64_t cells = 0;
    double best = INFINITY;
    int64_t bi = -1, bl = -1;
    for (size_t q = 0; q < pp; q++) cur[q] = INFINITY;
    for (int64_t j = 1; j < p; j++) {
        double C, yu, yd;
        interval_y(&H, 0, j, &C, &yu, &yd);
        cur[j] = fma(-lamp, elog(yd + H.c0d), C);
        cells++;
    }
    for (int64_t i = 2; i <= imax; i++) {
        if (i >= 3) {
            double *t = prev; prev = cur; cur = t;
            for (size_t q = 0; q < pp; q++) cur[q] = INFINITY;
            /* the rows l are independent given layer i-1 */
#pragma omp parallel for schedule(dynamic, 4) reduction(+ : cells)
            for (int64_t l = i - 2; l <= p - 2; l++) {
                int64_t klo = i == 3 ? 0 : i - 3;
                int64_t khi = i == 3 ? 0 : l - 1;
                double *yuk = malloc(sizeof(double) * (size_t)(khi + 1));
                for (int64_t k = klo; k <= khi; k++) {
                    double Ck, ydk;
                    interval_y(&H, k, l, &Ck, &yuk[k], &ydk);
                }
                for (int64_t j = l + 1; j < p; j++) {
                    double C, yu, yd;
                    interval_y(&H, l, j, &C, &yu, &yd);
                    double bt = INFINITY;
                    int32_t kb = -1;
                    for (int64_t k = klo; k <= khi; k++) {
                        double T = fma(-lamp, elog(yuk[k] + yd), prev[k * p + l]);
                        if (T < bt) { bt = T; kb = (int32_t)k; }
                        cells++;
                    }
                    cur[l * p + j] = C + bt;
                    K[(size_t)i * pp + (size_t)(l * p + j)] = kb;
                }
                free(yuk);
            }
        }
        if (Fdump) memcpy(Fdump + (size_t)i * pp, cur, sizeof(double) * pp);
        if (exact_s && i != imax) continue;
        int64_t lo = i == 2 ? 0 : i - 2, hi = i == 2 ? 0 : p - 2;
        for (int64_t l = lo; l <= hi; l++) {
            double C, yu, yd;
            interval_y(&H, l, p - 1, &C, &yu, &yd);
            double f = fma(-lamp, elog(yu), cur[l * p + p - 1]);
            cells++;
            if (f < best) { best = f; bi = i; bl = l; }
        }
    }
    int32_t t = (int32_t)bi;
    chain[t - 1] = (int32_t)(p - 1);
    chain[t - 2] = (int32_t)bl;
    int64_t l = bl, j = p - 1;
    for (int64_t i = bi; i >= 3; i--) {
        int32_t k = K[(size_t)i * pp + (size_t)(l * p + j)];
        chain[i - 3] = k;
        j = l;
        l = k;
    }
    if (Kdump) memcpy(Kdump, K, sizeof(int32_t) * pp * (size_t)(imax + 1));
    out[0] = best;
    out[1] = t;
    out[2] = (double)cells;
    free(prev); free(cur); free(K);
    return 0;
}
