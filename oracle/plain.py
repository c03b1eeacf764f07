"""Plain definitions of the ECASQ quantities, written out per entry.

TEST INFRASTRUCTURE ONLY: the product path never imports this module.

Everything here follows the paper's definitions directly, with no prefix sums
and no canonical operation order, so it can pin the C oracle (which uses the
closed forms) from outside:

  * SQ rounding, MSE and vNMSE                      (Sec. 2, Preliminaries)
  * expected frequencies f_q and H(Xhat)            (Sec. 1 and Sec. 3)
  * the surrogate H(I,B) with its interval index I  (Sec. 5, incl. its footnote
    on x = q_1)
  * brute force over every spanning Q drawn from the input values or from a
    permissible set P (App. D)
  * the classic ASQ DP, eq. (1)                     (Sec. 2)
  * the optimal DP over (l, j) states               (Sec. 4, App. D with L = {0},
                                                    R = {p-1})

Exact rational arithmetic (fractions.Fraction) is used where the inputs are
small; entropies are returned as floats from exact frequencies.
"""
from fractions import Fraction
from itertools import combinations
import math

import numpy as np


def h(y):
    """h(y) = -y log2 y for y > 0, else 0 (Sec. 4)."""
    y = float(y)
    return -y * math.log2(y) if y > 0 else 0.0


def _hist(x):
    xs = [Fraction(float(a)) for a in np.asarray(x, dtype=np.float64).ravel()]
    return xs


def sq_probs(x, Q):
    """For each entry: (a_x, b_x, Pr[round up]) under SQ with codebook Q.

    a_x = max{q <= x}, b_x = min{q >= x}; up with probability (x-a)/(b-a)
    (Sec. 2).  Q must span x.
    """
    Qs = sorted(Fraction(float(q)) for q in Q)
    out = []
    for xv in _hist(x):
        lo = max(q for q in Qs if q <= xv)
        hi = min(q for q in Qs if q >= xv)
        pu = Fraction(0) if lo == hi else (xv - lo) / (hi - lo)
        out.append((xv, lo, hi, pu))
    return Qs, out


def mse(x, Q):
    """MSE(Q, X) = sum_x (b_x - x)(x - a_x) (Sec. 2), exact."""
    _, rows = sq_probs(x, Q)
    return sum((hi - xv) * (xv - lo) for xv, lo, hi, _ in rows)


def norm2(x):
    return sum(v * v for v in _hist(x))


def vnmse(x, Q):
    """vNMSE = MSE / ||X||^2 (Sec. 2)."""
    return mse(x, Q) / norm2(x)


def freqs(x, Q):
    """Expected frequency f_q = sum_x Pr[xhat = q] (Sec. 3), exact."""
    Qs, rows = sq_probs(x, Q)
    f = {q: Fraction(0) for q in Qs}
    for xv, lo, hi, pu in rows:
        if lo == hi:
            f[lo] += 1
        else:
            f[hi] += pu
            f[lo] += 1 - pu
    return Qs, [f[q] for q in Qs]


def entropy_out(x, Q):
    """H(Xhat) = sum_q h(f_q / d) (Sec. 3)."""
    d = len(_hist(x))
    _, f = freqs(x, Q)
    return sum(h(fq / d) for fq in f)


def entropy_surrogate(x, Q):
    """H(I,B) of Sec. 5: I is the interval index with q_I < x <= q_{I+1}
    (x = q_1 gets I = 1), B the round-up bit; the pair is drawn over a uniform
    coordinate and the rounding."""
    Qs = sorted(Fraction(float(q)) for q in Q)
    xs = _hist(x)
    d = len(xs)
    if len(Qs) == 1:
        return 0.0
    mass = {}
    for xv in xs:
        if xv <= Qs[0]:
            i = 0
        else:
            i = max(k for k in range(len(Qs) - 1) if Qs[k] < xv)
        pu = (xv - Qs[i]) / (Qs[i + 1] - Qs[i])
        mass[(i, 1)] = mass.get((i, 1), 0) + pu
        mass[(i, 0)] = mass.get((i, 0), 0) + (1 - pu)
    return sum(h(m / d) for m in mass.values())


def objective(x, Q, lam, which="out"):
    """vNMSE + lambda * H, with H = H(Xhat) ('out') or H(I,B) ('sur')."""
    H = entropy_out(x, Q) if which == "out" else entropy_surrogate(x, Q)
    return float(vnmse(x, Q)) + lam * H


def spanning_codebooks(x, s, P=None):
    """Every Q drawn from the permissible values P (default: the distinct input
    values, P = X) with |Q| <= s that spans X: here P's first and last values
    are min X and max X, which every Q then contains (Sec. 2 and Sec. 4;
    App. D with L = {first}, R = {last})."""
    if P is None:
        v = sorted(set(float(a) for a in np.asarray(x, dtype=np.float64).ravel()))
    else:
        v = sorted(set(float(a) for a in P))
        xf = np.asarray(x, dtype=np.float64)
        assert v[0] == xf.min() and v[-1] == xf.max()
    if len(v) == 1:
        yield (v[0],)
        return
    inner = v[1:-1]
    for m in range(0, min(s, len(v)) - 1):
        for comb in combinations(inner, m):
            yield (v[0],) + comb + (v[-1],)


def brute_force(x, s, lam, which="sur", P=None):
    """min over spanning Q (drawn from P, default X) of vNMSE + lambda * H.
    Returns (J, Q)."""
    best = None
    for Q in spanning_codebooks(x, s, P):
        J = objective(x, Q, lam, which)
        if best is None or J < best[0]:
            best = (J, Q)
    return best


def brute_force_budget(x, s, b, which="out"):
    """min MSE over spanning Q with H <= b.  Returns (MSE, Q) or (inf, None)."""
    best = (math.inf, None)
    for Q in spanning_codebooks(x, s):
        H = entropy_out(x, Q) if which == "out" else entropy_surrogate(x, Q)
        if H <= b + 1e-12:
            m = float(mse(x, Q))
            if m < best[0]:
                best = (m, Q)
    return best


def weighted_hist(x):
    v, c = np.unique(np.asarray(x, dtype=np.float64).ravel() + 0.0, return_counts=True)
    return [Fraction(float(a)) for a in v], [int(a) for a in c]


def asq_dp(x, s):
    """Classic ASQ DP, eq. (1) of Sec. 2, on the weighted histogram.

    C[k,j] = sum over entries in [v_k, v_j] of (v_j - x)(x - v_k);
    dp(2, j) = C[0, j]; dp(i, j) = min_{k<j} dp(i-1, k) + C[k, j].
    Returns the minimum MSE with at most s values (exact)."""
    v, c = weighted_hist(x)
    p = len(v)
    if p == 1:
        return Fraction(0)

    def C(k, j):
        return sum(c[l] * (v[j] - v[l]) * (v[l] - v[k]) for l in range(k, j + 1))

    dp = [None] * p
    for j in range(1, p):
        dp[j] = C(0, j)
    best = dp[p - 1]
    for i in range(3, min(s, p) + 1):
        nd = [None] * p
        for j in range(i - 1, p):
            nd[j] = min(dp[k] + C(k, j) for k in range(i - 2, j) if dp[k] is not None)
        dp = nd
        best = min(best, dp[p - 1])
    return best


def optimal_dp(x, s, lam):
    """Optimal lambda-ECASQ DP over states (l, j) (Sec. 4; App. D with P = X,
    L = {0}, R = {p-1}), in float64 from per-entry sums.

      dp(2, 0, j) = C[0,j] + lam' h((n_0 + D[0,j]) / d)
      dp(i, l, j) = C[l,j] + min_{k<l} dp(i-1, k, l) + lam' h((U[k,l] + D[l,j]) / d)
      answer      = min_i min_{l<p-1} dp(i, l, p-1) + lam' h(U[l,p-1] / d)

    lam is in vNMSE units (lam' = lam ||X||^2).  Returns (J in vNMSE units,
    Q as a tuple of values)."""
    v, c = weighted_hist(x)
    p = len(v)
    d = sum(c)
    nx = float(sum(ci * vi * vi for vi, ci in zip(v, c)))
    if p == 1:
        return 0.0, (float(v[0]),)
    lp = lam * nx
    vf = [float(a) for a in v]
    # plain per-entry interval sums over the half-open (v_a, v_b]
    Cm = np.zeros((p, p))
    Um = np.zeros((p, p))
    Dm = np.zeros((p, p))
    for a in range(p):
        for b in range(a + 1, p):
            w = vf[b] - vf[a]
            cs = us = ds = 0.0
            for l in range(a + 1, b + 1):
                cs += c[l] * (vf[b] - vf[l]) * (vf[l] - vf[a])
                us += c[l] * (vf[l] - vf[a]) / w
                ds += c[l] * (vf[b] - vf[l]) / w
            Cm[a, b], Um[a, b], Dm[a, b] = cs, us, ds
    hv = np.vectorize(h)
    INF = math.inf
    # layer 2: only l = 0
    cur = np.full((p, p), INF)
    back = {}
    for j in range(1, p):
        cur[0, j] = Cm[0, j] + lp * h((c[0] + Dm[0, j]) / d)
    layers = {2: cur.copy()}
    for i in range(3, min(s, p) + 1):
        nxt = np.full((p, p), INF)
        for l in range(1, p - 1):
            prev = cur[:l, l]  # dp(i-1, k, l), k < l
            if not np.isfinite(prev).any():
                continue
            js = np.arange(l + 1, p)
            # T[k, j] = prev[k] + lp h((U[k,l] + D[l,j]) / d)
            y = (Um[:l, l][:, None] + Dm[l, js][None, :]) / d
            T = prev[:, None] + lp * hv(y)
            kbest = np.argmin(T, axis=0)
            nxt[l, js] = Cm[l, js] + T[kbest, np.arange(len(js))]
            for jj, j in enumerate(js):
                back[(i, l, j)] = int(kbest[jj])
        cur = nxt
        layers[i] = cur.copy()
    best = (INF, None)
    for i, L in layers.items():
        for l in range(0, p - 1):
            val = L[l, p - 1] + lp * h(Um[l, p - 1] / d)
            if val < best[0]:
                best = (val, (i, l))
    J, (i, l) = best
    # trace back the values
    idx = [p - 1, l]
    j = p - 1
    while i > 2:
        k = back[(i, l, j)]
        idx.append(k)
        j, l, i = l, k, i - 1
    idx = sorted(set(idx))
    return J / nx, tuple(vf[k] for k in idx)


# --------------------------------------------------------------------------
# Three-colour refinement (Sec. 6) on the plain objective.


def _interval_mse(xs, lo, hi):
    """Sum over the entries in (lo, hi] of (hi - x)(x - lo), exact."""
    return sum((hi - xv) * (xv - lo) for xv in xs if lo < xv <= hi)


def refine_local(x, Q, r, lam_p):
    """What moving q_r (0 < r < t-1) changes in MSE + lam' H(Xhat), per entry:
    the MSE of the entries in (q_{r-1}, q_{r+1}] plus lam' times h(f/d) of the
    three values whose expected frequencies depend on q_r (q_{r-1}, q_r,
    q_{r+1}), with f from the per-entry rounding probabilities (Sec. 3).
    lam' is in MSE units.  Exact (a Fraction) when lam' = 0."""
    xs = _hist(x)
    Qs, f = freqs(x, Q)
    d = len(xs)
    m = _interval_mse(xs, Qs[r - 1], Qs[r]) + _interval_mse(xs, Qs[r], Qs[r + 1])
    if lam_p == 0:
        return m
    return float(m) + lam_p * ((h(f[r - 1] / d) + h(f[r] / d)) + h(f[r + 1] / d))


class NearTie(Exception):
    """A decision of the plain refinement fell within rounding of a tie."""


def _less(a, b, tol):
    """a < b, raising NearTie when the two are within tol of each other but
    not exactly equal Fractions (then rounding could decide either way)."""
    if isinstance(a, Fraction) and isinstance(b, Fraction):
        return a < b
    if abs(a - b) <= tol:
        raise NearTie()
    return a < b


def refine_search(x, v, chain, r, lam_p, exhaustive=False, tol=0.0):
    """The position (a unique index) mover r's search finds in the open range
    (u_{r-1}, u_{r+1}) (Sec. 6): the lowest minimiser of refine_local
    (exhaustive), or the binary search on the sign of its forward difference
    (lo = L+1, hi = R-1; while lo < hi: mid = lo + (hi-lo)//2, lo = mid+1 if
    L(mid+1) < L(mid), else hi = mid)."""
    L, R = chain[r - 1], chain[r + 1]
    if R - L < 3:
        return chain[r]

    def val(m):
        Q = [v[k] for k in chain]
        Q[r] = v[m]
        return refine_local(x, Q, r, lam_p)

    if exhaustive:
        best, bm = None, None
        for m in range(L + 1, R):
            cur = val(m)
            if best is None or _less(cur, best, tol):
                best, bm = cur, m
        return bm
    lo, hi = L + 1, R - 1
    while lo < hi:
        mid = lo + (hi - lo) // 2
        if _less(val(mid + 1), val(mid), tol):
            lo = mid + 1
        else:
            hi = mid
    return lo


def refine(x, v, chain, lam_p, b=math.inf, budget=False, rounds=5, exhaustive=False, tol=0.0):
    """Sec. 6 on the plain objective: rounds of the colour substeps c = 0, 1, 2;
    in a substep every mover r = c (mod 3), 1 <= r <= t-2, searched against
    the chain as it stands, moves to the found position if that strictly lowers
    refine_local; with the budget guard the substep is undone if the new
    codebook's H(Xhat) exceeds b.  Stops after a round without a move or after
    `rounds` rounds.  Returns (chain, rounds run); raises NearTie when a
    decision is within tol of a tie (or the guard within tol of b)."""
    u = list(int(a) for a in chain)
    t = len(u)
    nrun = 0
    if t < 3:
        return u, 0
    for _ in range(rounds):
        any_move = False
        for c in range(3):
            nu = list(u)
            moved = 0
            for r in range(1, t - 1):
                if r % 3 != c:
                    continue
                m = refine_search(x, v, u, r, lam_p, exhaustive, tol)
                if m == u[r]:
                    continue
                Qm = [v[k] for k in u]
                Qm[r] = v[m]
                Q0 = [v[k] for k in u]
                if _less(refine_local(x, Qm, r, lam_p), refine_local(x, Q0, r, lam_p), tol):
                    nu[r] = m
                    moved += 1
            if moved and budget:
                Hn = entropy_out(x, [v[k] for k in nu])
                if abs(Hn - b) <= 1e-12:
                    raise NearTie()
                if Hn > b:
                    moved = 0
            if moved:
                u = nu
                any_move = True
        nrun += 1
        if not any_move:
            break
    return u, nrun
