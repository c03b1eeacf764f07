"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test names the passage it checks.  None of them compares the oracle with
itself: the references are printed values (tests/golden), brute force over all
codebooks, textbook recurrences, closed forms, exact rational arithmetic,
mpmath, math.fsum and published Philox test vectors.
"""
import math
from fractions import Fraction

import mpmath
import numpy as np
import pytest

from oracle import native, pipeline, plain
from oracle.log2_table import build_table
from oracle.philox import philox4x32_10
from tests.conftest import golden


def fr(s):
    return Fraction(s)


# --------------------------------------------------------------------------
# Printed examples


def test_worked_entropy_example():
    """Sec. 3: X=<0,1,10>, Q={0,10} gives H ~ 0.948 bits/entry."""
    g = golden("worked_example.txt")
    x = [float(a) for a in g["x"].split()]
    Q = [float(a) for a in g["Q"].split()]
    Qs, f = plain.freqs(x, Q)
    assert [fq / len(x) for fq in f] == [fr(a) for a in g["f_over_d"].split()]
    H = plain.entropy_out(x, Q)
    assert round(H, int(g["H_out_digits"])) == float(g["H_out"])
    assert plain.mse(x, Q) == 9
    # the C oracle's closed forms give the same numbers
    Hh = pipeline.prepare(np.array(x, dtype=np.float32))
    m = pipeline.chain_metrics(Hh, np.array([0, 2], dtype=np.int32), 0.0)
    assert m["mse"] == 9.0
    assert abs(m["entropy"] - H) < 1e-15
    # one interval: the surrogate equals the true entropy
    assert abs(m["entropy_surrogate"] - H) < 1e-15
    assert abs(m["vnmse"] - 9 / 101) < 1e-16


def test_app_e1_quantizers_and_thresholds():
    """App. E.1: table of A, B, C and the multiplier thresholds."""
    g = golden("app_e1_lagrange.txt")
    x = [0.0] * 4 + [2.0] * 4
    dig = int(g["H_digits"])
    for name in "ABC":
        Q = [float(a) for a in g[name].split()]
        _, f = plain.freqs(x, Q)
        assert [fq / len(x) for fq in f] == [fr(a) for a in g[name + "_dist"].split()]
        assert round(plain.entropy_out(x, Q), dig) == float(g[name + "_H"])
        assert plain.vnmse(x, Q) == fr(g[name + "_vnmse"])
    HA = plain.entropy_out(x, [0, 4])
    HB = plain.entropy_out(x, [0, 3])
    assert round(HB, 6) == float(g["B_H_6"]) and round(HA, 6) == float(g["A_H_6"])
    lam_bc = 0.5 / (1 - HB)
    lam_ba = 0.5 / (HB - HA)
    assert lam_bc > float(g["B_over_C_lambda_above"])
    assert lam_ba < float(g["B_over_A_lambda_below"])
    # lambda is in vNMSE units: the crossings happen exactly there
    J = lambda Q, lam: plain.objective(x, Q, lam, "out")
    assert J([0, 3], lam_bc * 1.001) < J([0, 2], lam_bc * 1.001)
    assert J([0, 3], lam_bc * 0.999) > J([0, 2], lam_bc * 0.999)
    assert J([0, 3], lam_ba * 0.999) < J([0, 4], lam_ba * 0.999)
    # no lambda makes B the Lagrangian optimum
    for lam in np.linspace(0, 20, 401):
        assert min(J([0, 4], lam), J([0, 2], lam)) <= J([0, 3], lam) + 1e-15
    # time-sharing A and C at b = 0.95
    b = float(g["b_ts"])
    alpha = (b - HA) / (1 - HA)
    dts = int(g["ts_digits"])
    assert round(alpha, dts) == float(g["alpha_ts"])
    assert round((1 - alpha) * 1.0, dts) == float(g["vnmse_ts"])


def test_app_e2_nonadjacent_and_solvers():
    """App. E.2: with 0,1,2 each d/3, s=3, b=3/2 the adjacent solution is {0,2}."""
    g = golden("app_e2_nonadjacent.txt")
    x = [0.0] * 3 + [1.0] * 3 + [2.0] * 3
    assert abs(plain.entropy_out(x, [0, 1, 2]) - math.log2(3)) < 1e-15
    _, f = plain.freqs(x, [0, 2])
    assert [fq / len(x) for fq in f] == [fr(a) for a in g["Q2_dist"].split()]
    assert plain.entropy_out(x, [0, 2]) == float(g["Q2_H"])
    assert plain.vnmse(x, [0, 2]) == fr(g["Q2_vnmse"])
    # the non-adjacent rule's entropy as printed
    Hn = sum(plain.h(fr(a)) for a in g["nonadj_dist"].split())
    assert round(Hn, int(g["nonadj_H_digits"])) == float(g["nonadj_H"])
    alpha = (1.5 - 1) / (math.log2(3) - 1)
    assert round(alpha, int(g["alpha_digits"])) == float(g["alpha"])
    assert round((1 - alpha) / 5, int(g["ts_vnmse_digits"])) == float(g["ts_vnmse"])
    # exact optimum and both of our solvers return {0, 2} at b = 3/2
    s, b = int(g["s"]), float(g["b"])
    m, Q = plain.brute_force_budget(x, s, b, "out")
    assert Q == (0.0, 2.0) and m == 3.0
    r = pipeline.solve(np.array(x, dtype=np.float32), s, b)
    assert list(r.codebook) == [0.0, 2.0]
    assert r.entropy == 1.0


# --------------------------------------------------------------------------
# Canonical log2, exact prefix sums


def test_log2c_accuracy():
    """The canonical log2 stays within 2.5 ulp of the true value (mpmath)."""
    L = native.lib()
    rng = np.random.default_rng(5)
    ys = np.concatenate([rng.uniform(0, 1, 4000), 10 ** rng.uniform(-300, 300, 4000),
                         1 + rng.uniform(-2e-2, 2e-2, 4000), 1 + rng.uniform(-1e-9, 1e-9, 500)])
    mpmath.mp.prec = 120
    worst = 0.0
    for y in ys:
        got = L.orc_log2c(float(y))
        ref = mpmath.log(mpmath.mpf(float(y)), 2)
        worst = max(worst, float(abs((mpmath.mpf(got) - ref) / math.ulp(float(ref)))))
    assert worst <= 2.5
    for k in range(-1000, 1000, 37):
        assert L.orc_log2c(2.0 ** k) == k
    assert L.orc_log2c(1.0) == 0.0


def test_log2_table_correctly_rounded():
    """Each table entry is the correctly rounded log2 (checked at 400 bits)."""
    invc, lc = build_table()
    mpmath.mp.prec = 400
    for ic, l in zip(invc, lc):
        exact = -mpmath.log(mpmath.mpf(ic), 2)
        err = abs(mpmath.mpf(l) - exact)
        assert err <= mpmath.mpf(math.ulp(l)) / 2


def test_h_zero_and_negative():
    """h(y) = 0 for y <= 0 and -y log2 y otherwise (Sec. 4)."""
    L = native.lib()
    assert L.orc_h(0.0) == 0.0 and L.orc_h(-1e-300) == 0.0 and L.orc_h(-3.0) == 0.0
    assert L.orc_h(1.0) == 0.0
    assert abs(L.orc_h(0.25) - 0.5) < 1e-16


def test_exact_prefix_sums_against_fsum():
    """S and S2 equal the correctly rounded exact sums (math.fsum is exact)."""
    rng = np.random.default_rng(2)
    x = np.concatenate([rng.standard_normal(300) * 10.0 ** rng.integers(-30, 30, 300),
                        rng.standard_normal(50)]).astype(np.float32)
    x = np.concatenate([x, x[:40]])  # duplicates
    v, c = pipeline.histogram(x)
    N, S, S2 = pipeline.exact_prefix(v, c)
    for k in range(0, len(v), 7):
        terms = [float(v[i]) for i in range(k + 1) for _ in range(int(c[i]))]
        assert S[k] == math.fsum(terms)
        assert S2[k] == math.fsum(float(Fraction(t) ** 2) for t in terms) or \
            S2[k] == float(sum(Fraction(t) ** 2 for t in terms))
        assert N[k] == len(terms)


# --------------------------------------------------------------------------
# Closed forms


def test_unit_grid_closed_forms():
    """X = 0..w with unit weights: C[0,w] = (w^3-w)/6, U = (w+1)/2, D = (w-1)/2
    (App. D definitions of C_P, U_P, D_P on the half-open interval)."""
    for w in (1, 2, 3, 7, 30, 100):
        x = np.arange(w + 1, dtype=np.float32)
        H = pipeline.prepare(x)
        C, U, D, P = pipeline.interval(H, 0, w)
        assert C == (w ** 3 - w) / 6
        assert U == (w + 1) / 2 and D == (w - 1) / 2


def test_s2_closed_form():
    """s = 2 forces Q = {min, max}: MSE = sum (max-x)(x-min), H(I,B) = H(Xhat)."""
    rng = np.random.default_rng(3)
    for _ in range(5):
        x = rng.standard_normal(200).astype(np.float32)
        r = pipeline.solve_lagrangian(x, 2, 0.3)
        xs = [Fraction(float(a)) for a in x]
        lo, hi = min(xs), max(xs)
        m = sum((hi - a) * (a - lo) for a in xs)
        assert r.t == 2 and list(r.codebook) == [float(lo), float(hi)]
        assert abs(r.mse - float(m)) <= 1e-12 * float(m)
        assert abs(r.entropy - r.entropy_surrogate) < 1e-14
        assert abs(r.entropy - plain.entropy_out(x, [float(lo), float(hi)])) < 1e-13


def test_frequency_identity_and_expected_frequency():
    """For unbiased SQ, MSE = sum_q f_q q^2 - ||X||^2 (App. E.3 lemma), and the
    interior frequency is U[k,l] + D[l,j] with sum f = d (Sec. 4)."""
    rng = np.random.default_rng(4)
    x = np.round(rng.standard_normal(40) * 4).astype(np.float32)
    v = sorted(set(float(a) for a in x))
    Q = [v[0], v[3], v[7], v[-1]]
    Qs, f = plain.freqs(x, Q)
    assert sum(f) == len(x)
    assert plain.mse(x, Q) == sum(fq * q * q for fq, q in zip(f, Qs)) - plain.norm2(x)
    H = pipeline.prepare(x)
    idx = [v.index(q) for q in Q]
    _, U01, D01, _ = pipeline.interval(H, idx[0], idx[1])
    _, U12, D12, _ = pipeline.interval(H, idx[1], idx[2])
    assert abs((U01 + D12) - float(f[1])) < 1e-12


def test_monotone_round_masses():
    """U(k,l) is non-increasing in k and D(l,j) non-decreasing in j (App. B)."""
    rng = np.random.default_rng(6)
    x = rng.standard_normal(60).astype(np.float32)
    H = pipeline.prepare(x)
    l = 30
    Us = [pipeline.interval(H, k, l)[1] for k in range(l)]
    Ds = [pipeline.interval(H, l, j)[2] for j in range(l + 1, H.p)]
    assert all(a >= b - 1e-12 for a, b in zip(Us, Us[1:]))
    assert all(a <= b + 1e-12 for a, b in zip(Ds, Ds[1:]))


# --------------------------------------------------------------------------
# The DPs against brute force


def _tiny_inputs(n, seed):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        d = int(rng.integers(2, 11))
        if rng.random() < 0.5:
            x = rng.integers(-5, 6, size=d).astype(np.float32) * np.float32(rng.choice([0.5, 1, 3]))
        else:
            x = rng.standard_normal(d).astype(np.float32)
        s = int(rng.integers(2, 6))
        lam = 0.0 if rng.random() < 0.15 else float(10 ** rng.uniform(-3, 1))
        if np.all(x == 0) or len(set(x.tolist())) < 2:
            continue
        yield x, s, lam


def test_apx_dp_equals_brute_force():
    """eq. apx_base/apx_rec/apx_final minimise vNMSE + lambda H(I,B) over all
    spanning Q with |Q| <= s; Hirschberg and the backpointer traceback recover a
    minimiser."""
    for x, s, lam in _tiny_inputs(120, 11):
        H = pipeline.prepare(x)
        r = pipeline.dp_forward(H, s, lam * H.s2tot, backpointers=True)
        Jb, _ = plain.brute_force(x, s, lam, "sur")
        assert abs(r["J"] / H.s2tot - Jb) <= 1e-12 * max(1.0, Jb)
        ch, _ = pipeline.hirschberg(H, r["t"], lam * H.s2tot)
        m = pipeline.chain_metrics(H, ch, lam)
        assert abs(m["vnmse"] + lam * m["entropy_surrogate"] - Jb) <= 1e-12 * max(1.0, Jb)
        assert list(ch) == list(r["chain_bp"])
        # carried accumulators describe the chosen path
        assert abs(r["mse"] - m["mse"]) <= 1e-12 * max(1.0, m["mse"])
        assert abs(r["phi"] - m["entropy_surrogate"]) <= 1e-12


def test_apx_dp_on_permissible_grids_equals_brute_force():
    """App. D with P != X: on a uniform grid over [min X, max X] and on a
    quantile grid, the DP over the grid's prefix quantities minimises
    vNMSE + lambda H(I,B) over every spanning Q drawn from the grid."""
    for x, s, lam in _tiny_inputs(60, 21):
        for alphabet in (("uniform", 7), ("uniform", 3), ("quantile", 5)):
            H = pipeline.prepare(x, alphabet)
            if H.p < 2:
                continue
            assert H.v[0] == float(np.min(x)) and H.v[-1] == float(np.max(x))
            assert np.all(np.diff(H.v) > 0)
            r = pipeline.dp_forward(H, s, lam * H.s2tot, backpointers=True)
            Jb, _ = plain.brute_force(x, s, lam, "sur", P=list(H.v))
            assert abs(r["J"] / H.s2tot - Jb) <= 1e-12 * max(1.0, Jb), alphabet
            m = pipeline.chain_metrics(H, r["chain_bp"], lam)
            assert abs(m["vnmse"] + lam * m["entropy_surrogate"] - Jb) <= 1e-12 * max(1.0, Jb)
            # expected output frequencies from the grid's prefix quantities
            Q = [float(H.v[k]) for k in r["chain_bp"]]
            assert abs(m["entropy"] - plain.entropy_out(x, Q)) <= 1e-12


def test_permissible_grids():
    """Grid construction: endpoints min X and max X, strictly increasing, the
    uniform grid's interior points min X + k step, the quantile grid drawn from
    X at ranks floor(k (d - 1) / (m - 1)); prefix counts and sums at the grid
    points equal the plain counts and sums of the entries <= p."""
    rng = np.random.default_rng(22)
    x = np.round(rng.standard_normal(500) * 4).astype(np.float32) / np.float32(4)
    xs = np.sort(x.astype(np.float64))
    Hu = pipeline.prepare(x, ("uniform", 11))
    step = (xs[-1] - xs[0]) / 10.0
    assert list(Hu.v) == [xs[0]] + [xs[0] + k * step for k in range(1, 10)] + [xs[-1]]
    Hq = pipeline.prepare(x, ("quantile", 9))
    want = []
    for k in range(9):
        q = xs[(k * 499) // 8]
        if not want or q > want[-1]:
            want.append(q)
    assert list(Hq.v) == want
    for H in (Hu, Hq):
        for k, pk in enumerate(H.v):
            sel = xs[xs <= pk]
            assert H.N[k] == len(sel)
            assert abs(H.S[k] - math.fsum(sel)) <= 1e-12 * max(1.0, abs(math.fsum(sel)))
            assert abs(H.S2[k] - math.fsum(sel * sel)) <= 1e-12 * math.fsum(sel * sel)
    # a grid finer than the data's spacing (fp64 has 29 more bits than the
    # fp32 data, so its points stay distinct)
    y = np.array([1.0, 1.0 + 2.0 ** -23], dtype=np.float32)
    Hy = pipeline.prepare(y, ("uniform", 1000))
    assert len(Hy.v) == 1000 and np.all(np.diff(Hy.v) > 0) and Hy.v[-1] == np.float64(y[1])
    assert list(Hy.N) == [1.0] * 999 + [2.0]


def test_optimal_dp_equals_brute_force_and_sandwich():
    """Sec. 4 optimal DP = brute-force min of vNMSE + lambda H(Xhat); and
    J_opt <= J_apx <= J_opt + lambda (from H(Xhat) <= H(I,B) <= H(Xhat)+1)."""
    for x, s, lam in _tiny_inputs(80, 12):
        Jo, _ = plain.optimal_dp(x, s, lam)
        Jbo, _ = plain.brute_force(x, s, lam, "out")
        assert abs(Jo - Jbo) <= 1e-12 * max(1.0, Jbo)
        H = pipeline.prepare(x)
        Ja = pipeline.dp_forward(H, s, lam * H.s2tot)["J"] / H.s2tot
        assert Jbo <= Ja + 1e-12 and Ja <= Jbo + lam + 1e-12


def test_native_optimal_dp_equals_brute_force():
    """The C optimal DP (Sec. 4, states (i, l, j), the full minimum over k):
    its optimum equals the brute-force minimum of vNMSE + lambda H(Xhat) over
    every spanning codebook, its own value matches its codebook's objective, and
    the independent per-entry implementation agrees; exactly s values with
    exact_s; on permissible grids (App. D) the minimum over grid codebooks."""
    for x, s, lam in _tiny_inputs(120, 31):
        H = pipeline.prepare(x)
        r = pipeline.solve_optimal(x, s, lam)
        Jb, Qb = plain.brute_force(x, s, lam, "out")
        assert abs(r.objective - Jb) <= 1e-12 * max(1.0, Jb), (x, s, lam)
        assert abs(r.dp_value / H.s2tot - r.objective) <= 1e-12 * max(1.0, Jb)
        Jo, Qo = plain.optimal_dp(x, s, lam)
        assert abs(Jo - Jb) <= 1e-12 * max(1.0, Jb)
        assert r.t <= s and r.codebook[0] == H.v[0] and r.codebook[-1] == H.v[-1]
        if s <= H.p:
            re = pipeline.solve_optimal(x, s, lam, exact_s=True)
            cands = [Q for Q in plain.spanning_codebooks(x, s) if len(Q) == s]
            Je = min(plain.objective(x, Q, lam, "out") for Q in cands)
            assert re.t == s and abs(re.objective - Je) <= 1e-12 * max(1.0, Je)
    for x, s, lam in _tiny_inputs(40, 32):
        for alpha in (("uniform", 9), ("quantile", 4)):
            H = pipeline.prepare(x, alpha)
            r = pipeline.solve_optimal(x, s, lam, alphabet=alpha)
            Jb, _ = plain.brute_force(x, s, lam, "out", P=list(H.v))
            assert abs(r.objective - Jb) <= 1e-12 * max(1.0, Jb), (x, s, lam, alpha)


def test_optimal_dp_special_cases():
    """lambda = 0 is ASQ (Sec. 3: the minimum MSE with at most s values, the
    textbook DP eq. (1)); a prohibitive lambda keeps two values; p = 1 and
    p = 2."""
    rng = np.random.default_rng(33)
    for _ in range(10):
        x = rng.standard_normal(int(rng.integers(20, 60))).astype(np.float32)
        s = int(rng.integers(2, 8))
        H = pipeline.prepare(x)
        r = pipeline.solve_optimal(x, s, 0.0)
        a = float(plain.asq_dp(x, s))
        assert abs(r.mse - a) <= 1e-12 * max(1.0, a)
        assert pipeline.solve_optimal(x, s, 1e6).t == 2
    r = pipeline.solve_optimal(np.full(7, 2.5, dtype=np.float32), 4, 0.1)
    assert r.t == 1 and r.mse == 0.0
    x2 = np.array([1, 1, 3], dtype=np.float32)
    r = pipeline.solve_optimal(x2, 4, 0.1)
    assert r.t == 2 and r.mse == 0.0 and list(r.codebook) == [1.0, 3.0]


def test_optimal_argmins_monotone_lemma_quadrangle():
    """Lemma quadrangleM (Sec. 4.1): for fixed i and l the matrix of
    T(k, j) is Monge with its columns reversed, so the lowest minimiser k*(j)
    does not increase with j.  Checked on every (i, l) of random inputs: where
    k*(j+1) > k*(j), the two candidates must tie to rounding."""
    rng = np.random.default_rng(34)
    viol = checked = 0
    for trial in range(6):
        d = int(rng.integers(40, 90))
        x = (rng.standard_normal(d) * (1 + 3 * (trial % 2))).astype(np.float32)
        H = pipeline.prepare(x)
        s = 7
        lam = float(10 ** rng.uniform(-3, 0))
        lamp = lam * H.s2tot
        r = pipeline.opt_dp(H, s, lamp, dump=True)
        K, F = r["K"], r["F"]
        p = H.p

        def T(i, k, l, j):  # the candidate in plain float arithmetic
            U = pipeline.interval(H, k, l)[1]
            D = pipeline.interval(H, l, j)[2]
            return F[i - 1, k, l] + lamp * plain.h((U + D) / H.d)

        for i in range(4, min(s, p) + 1):
            for l in range(i - 2, p - 1):
                ks = K[i, l, l + 1:p]
                checked += len(ks)
                for jj in range(len(ks) - 1):
                    if ks[jj + 1] > ks[jj]:
                        viol += 1
                        j = l + 1 + jj
                        # the minimiser at j + 1 and the monotone one tie to rounding
                        a, b = T(i, ks[jj + 1], l, j + 1), T(i, ks[jj], l, j + 1)
                        assert abs(a - b) <= 1e-12 * max(1.0, abs(a)), (trial, i, l, j)
    assert checked > 20000 and viol <= 3, (checked, viol)


def _lower_hull_at(points, b):
    """min M over mixtures of (H, M) points with H <= b: the lower convex
    envelope up to the lowest-M point, flat after it."""
    mstar = min(m for _, m in points)
    hstar = min(h for h, m in points if m == mstar)
    if b >= hstar:
        return mstar
    pts = sorted(set(pt for pt in points if pt[0] <= hstar))
    hull = []
    for pt in pts:
        while len(hull) >= 2:
            (x1, y1), (x2, y2) = hull[-2], hull[-1]
            if (x2 - x1) * (pt[1] - y1) - (y2 - y1) * (pt[0] - x1) <= 0:
                hull.pop()
            else:
                break
        hull.append(pt)
    if b >= hull[-1][0]:
        return min(y for _, y in hull)
    for (x1, y1), (x2, y2) in zip(hull, hull[1:]):
        if x1 <= b <= x2:
            return y1 + (y2 - y1) * (b - x1) / (x2 - x1)
    return math.inf


def test_timesharing_reaches_the_convex_frontier():
    """Sec. 7 / App. E: the two-way time-share of the search's final pair has
    rate b and the vNMSE of the lower convex envelope of every spanning
    codebook's (H, vNMSE) at b, so no single codebook with H <= b does
    better; with the optimal DP the entropy is H(Xhat) (the paper's optimality
    for every b), with the approximate DP it is H(I,B)."""
    checked = mixed = 0
    for x, s, _ in _tiny_inputs(40, 41):
        if len(set(x.tolist())) < 4:
            continue
        for dp, which in (("optimal", "out"), ("approx", "sur")):
            pts = []
            for Q in plain.spanning_codebooks(x, s):
                Hq = (plain.entropy_out(x, Q) if which == "out"
                      else plain.entropy_surrogate(x, Q))
                pts.append((float(Hq), float(plain.vnmse(x, Q))))
            hmin, hmax = min(p[0] for p in pts), max(p[0] for p in pts)
            for frac in (0.2, 0.45, 0.7, 0.9):
                b = hmin + frac * (hmax - hmin)
                if b < 1.0 and hmin > b:
                    continue
                r = pipeline.solve_timeshare(x, s, b, dp=dp)
                if r["status"] != 0:
                    continue
                hull = _lower_hull_at(pts, b)
                assert r["M_mix"] <= hull + 1e-12, (x, s, b, dp)
                assert hull <= r["M_mix"] + 1e-12, (x, s, b, dp)
                single = min(m for hq, m in pts if hq <= b + 1e-12)
                assert r["M_mix"] <= single + 1e-12
                if r["alpha"] > 0.0:
                    mixed += 1
                    assert abs(r["H_mix"] - b) <= 1e-12
                    assert 0.0 < r["alpha"] < 1.0 and r["HB"] <= b < r["HA"]
                    # the pair is the codebooks' own (H, vNMSE)
                    pl, mi = r["plus"], r["minus"]
                    Hp = pl.entropy if dp == "optimal" else pl.entropy_surrogate
                    Hm = mi.entropy if dp == "optimal" else mi.entropy_surrogate
                    assert abs(Hp - r["HA"]) <= 1e-12 and abs(Hm - r["HB"]) <= 1e-12
                    assert abs(pl.vnmse - r["MA"]) <= 1e-12 and abs(mi.vnmse - r["MB"]) <= 1e-12
                checked += 1
    assert checked > 100 and mixed > 40, (checked, mixed)


def test_refinement_aware_search():
    """Search on the true H(Xhat) of refined codebooks: the answer is
    feasible (H(Xhat) <= b, recomputed exactly), no better than the brute-force
    optimum under the same budget, the lowest-vNMSE feasible point among the
    search's solves, and each solve's point is the refined codebook's own
    (H(Xhat), vNMSE)."""
    n = 0
    for x, s, _ in _tiny_inputs(60, 43):
        if len(set(x.tolist())) < 4:
            continue
        H = pipeline.prepare(x)
        for b in (1.1, 1.5, 2.0):
            r = pipeline.solve(x, s, b, dp="refined", recovery="backpointers", width=1)
            if r.status != 0:
                continue
            Hout = float(plain.entropy_out(x, list(r.codebook)))
            assert Hout <= b + 1e-12 and abs(Hout - r.entropy) <= 1e-12
            m_opt, _ = plain.brute_force_budget(x, s, b, "out")
            assert float(m_opt) / float(plain.norm2(x)) <= r.vnmse * (1 + 1e-12) + 1e-15
            sr = pipeline.search(H, s, b, width=1, dp="refined")
            feas = [row for row in sr["traj"] if row[1] <= b]
            if feas:
                assert min(row[2] for row in feas) == r.vnmse or abs(
                    min(row[2] for row in feas) - r.vnmse) <= 1e-15
            for lam, hh, mm, t in sr["traj"][:3]:
                rr = pipeline.dp_forward(H, s, lam * H.s2tot, backpointers=True)
                ch = rr["chain_bp"]
                if len(ch) >= 3:
                    ch, _, _ = pipeline.refine(H, ch, lam * H.s2tot)
                m = pipeline.chain_metrics(H, ch, 0.0)
                assert m["entropy"] == hh and m["mse"] / H.s2tot == mm and len(ch) == t
            n += 1
    assert n > 60, n


def test_timeshared_rounding():
    """Time-shared rounding: alpha = 0 and alpha = 1 reduce to the plain
    rounding with one codebook; the share of entries on the second codebook
    is alpha (binomial); every entry stays unbiased; the entropy is the
    size-weighted plug-in entropy of the two parts."""
    rng = np.random.default_rng(42)
    x = rng.standard_normal(20000).astype(np.float32)
    lo, hi = float(x.min()), float(x.max())
    cm = np.array([lo, -0.5, 0.7, hi])
    cp = np.array([lo, -1.0, 0.0, 1.0, hi])
    sym0, _, _ = pipeline.quantize(x, cm, 7)[:3]
    s0, part0, h0, e0 = pipeline.quantize_timeshare(x, cm, cp, 0.0, 7)
    assert not part0.any() and np.array_equal(s0, sym0)
    assert abs(e0 - pipeline.quantize(x, cm, 7)[2]) <= 1e-15
    s1, part1, _, _ = pipeline.quantize_timeshare(x, cm, cp, 1.0, 7)
    assert part1.all() and np.array_equal(s1, pipeline.quantize(x, cp, 7)[0])
    alpha = 0.37
    s, part, hist, ent = pipeline.quantize_timeshare(x, cm, cp, alpha, 9)
    n = len(x)
    z = (part.sum() - alpha * n) / math.sqrt(n * alpha * (1 - alpha))
    assert abs(z) < 5
    assert hist.sum() == n and hist[:4].sum() == n - part.sum()
    e_m = pipeline._plugin_entropy(s[part == 0], 4)[1]
    e_p = pipeline._plugin_entropy(s[part == 1], 5)[1]
    assert abs(ent - ((n - part.sum()) * e_m + part.sum() * e_p) / n) <= 1e-12
    # unbiased: the mean reconstruction over seeds tends to x
    xs = x[:200]
    acc = np.zeros(len(xs))
    seeds = 300
    for sd in range(seeds):
        sy, pt, _, _ = pipeline.quantize_timeshare(xs, cm, cp, alpha, 1000 + sd)
        acc += np.where(pt == 1, cp[np.minimum(sy, 4)], cm[np.minimum(sy, 3)])
    err = acc / seeds - xs.astype(np.float64)
    assert abs(err.mean()) < 0.02 and np.abs(err).max() < 0.35


def test_entropy_sandwich_per_codebook():
    """eq. apx_entropy_sandwich: H(Xhat) <= H(I,B) <= H(Xhat) + 1 for every Q."""
    rng = np.random.default_rng(7)
    for _ in range(40):
        x = rng.integers(-4, 5, size=int(rng.integers(2, 12))).astype(np.float32)
        for Q in list(plain.spanning_codebooks(x, 5))[:20]:
            a, b = plain.entropy_out(x, Q), plain.entropy_surrogate(x, Q)
            assert a <= b + 1e-12 and b <= a + 1 + 1e-12


def test_lambda_zero_is_asq():
    """lambda = 0 reduces to ASQ (Sec. 3): the approx DP equals the textbook
    DP eq. (1) and the brute-force minimum MSE."""
    for x, s, _ in _tiny_inputs(60, 13):
        H = pipeline.prepare(x)
        r = pipeline.dp_forward(H, s, 0.0)
        a = plain.asq_dp(x, s)
        bf = min(plain.mse(x, Q) for Q in plain.spanning_codebooks(x, s))
        assert a == bf
        assert abs(r["J"] - float(a)) <= 1e-12 * max(1.0, float(a)) + 1e-13 * H.s2tot


def test_lemma4_on_brute_force():
    """Lemma 4: the minimum-MSE Q with H(I,B) <= b has H(Xhat) <= b and MSE no
    larger than OPT(b - 1)."""
    rng = np.random.default_rng(8)
    for _ in range(25):
        x = rng.integers(-5, 6, size=int(rng.integers(4, 10))).astype(np.float32)
        if len(set(x.tolist())) < 3:
            continue
        for b in (1.2, 1.6, 2.0, 2.5):
            m_apx, Q = plain.brute_force_budget(x, 5, b, "sur")
            if Q is None:
                continue
            assert plain.entropy_out(x, Q) <= b + 1e-12
            m_opt, _ = plain.brute_force_budget(x, 5, b - 1, "out")
            assert m_apx <= m_opt + 1e-9


def test_mse_monotone_in_s_and_b():
    """The exact constrained optimum is non-increasing in s and in b; the
    budget solver's MSE is non-increasing in b (it returns hull vertices)."""
    rng = np.random.default_rng(9)
    x = rng.integers(-6, 7, size=9).astype(np.float32)
    prev = math.inf
    for s in (2, 3, 4, 5):
        m, _ = plain.brute_force_budget(x, s, 2.0, "out")
        assert m <= prev + 1e-12
        prev = m
    prev = math.inf
    for b in (1.0, 1.5, 2.0, 2.5, 3.0):
        m, _ = plain.brute_force_budget(x, 5, b, "out")
        assert m <= prev + 1e-12
        prev = m
    y = np.random.default_rng(10).standard_normal(400).astype(np.float32)
    prev = math.inf
    for b in (1.0, 1.5, 2.0, 2.5, 3.0, 3.5):
        r = pipeline.solve(y, 12, b, refine_rounds=0)
        assert r.entropy_surrogate <= b
        assert r.mse <= prev * (1 + 1e-12)
        prev = r.mse


# --------------------------------------------------------------------------
# Search, recovery, refinement


def test_search_matches_dense_lambda_grid():
    """The slope search returns the best feasible supported point: among DP
    solutions over a dense lambda grid, none with H(I,B) <= b has lower vNMSE."""
    rng = np.random.default_rng(14)
    x = rng.standard_normal(120).astype(np.float32)
    s = 8
    H = pipeline.prepare(x)
    pts = []
    for lam in np.concatenate([[0.0], np.logspace(-4, 2, 1500)]):
        r = pipeline.dp_forward(H, s, lam * H.s2tot)
        pts.append((r["phi"], r["mse"] / H.s2tot))
    for b in (1.3, 1.8, 2.2, 2.9):
        best = min(m for hh, m in pts if hh <= b)
        found = []
        for width, aim in ((1, True), (1, False), (8, True)):
            sr = pipeline.search(H, s, b, width=width, aim=aim)
            assert sr["status"] == 0 and sr["H"] <= b
            assert sr["M"] <= best * (1 + 1e-12)
            # A and B adjacent on the lower hull: the final slope lies between
            # the multipliers A and B were found at
            assert sr["lam_final"] <= sr["lam"] or sr["lam"] == 0.0
            found.append((sr["H"], sr["M"], sr["t"]))
        # every schedule (aimed or plain sequential, passes of 8) ends at the
        # same supported point
        assert found[0] == found[1] == found[2]


def test_budget_sweep_shares_solves():
    """Several budgets on one input with a shared lambda cache: each budget's
    codebook and metrics equal those of its own search (the search ends at the
    same hull vertex however it starts), with fewer DP solves in total."""
    x = inputs_student(1000, 4)
    budgets = (1.0, 2.0, 3.0, 4.0)
    for width in (1, 8):
        shared = pipeline.solve_budgets(x, 12, budgets, refine_rounds=2, width=width)
        alone = [pipeline.solve(x, 12, b, refine_rounds=2, width=width) for b in budgets]
        for r, a in zip(shared, alone):
            assert r.t == a.t and list(r.rank) == list(a.rank)
            assert r.lam == a.lam and r.status == a.status
            for k in ("mse", "entropy", "entropy_surrogate", "objective"):
                assert getattr(r, k) == getattr(a, k)
        assert sum(r.dp_solves for r in shared) < sum(a.dp_solves for a in alone)


def inputs_student(d, seed):
    rng = np.random.default_rng(seed)
    return rng.standard_t(3, d).astype(np.float32)


def test_dp_columns_match_full_layers():
    """The sampled-column recomputation (used to check full-size GPU layers)
    equals the full forward DP layer by layer, and its accumulators at the last
    column equal the MSE and H(I,B) the DP reports for its chosen layer."""
    rng = np.random.default_rng(17)
    x = rng.standard_normal(400).astype(np.float32)
    s, lam = 9, 0.03
    H = pipeline.prepare(x)
    p = H.p
    lamp = lam * H.s2tot
    r = pipeline.dp_forward(H, s, lamp, backpointers=True, dump=True)
    F2, K2, M, Ph = pipeline.dp_columns(H, 2, lamp, cols=np.arange(1, p))
    np.testing.assert_array_equal(F2, r["F"][2, 1:p])
    Mfull = np.zeros(p)
    Pfull = np.zeros(p)
    Mfull[1:], Pfull[1:] = M, Ph
    Ffull = r["F"][2].copy()
    accs = {2: (Mfull.copy(), Pfull.copy())}
    for i in range(3, s + 1):
        cols = np.arange(i - 1, p)
        F, K, M, Ph = pipeline.dp_columns(H, i, lamp, Ffull, Mfull, Pfull, cols)
        np.testing.assert_array_equal(F, r["F"][i, i - 1:p])
        np.testing.assert_array_equal(K, r["bp"][i, i - 1:p])
        Ffull = r["F"][i].copy()
        Mfull = np.zeros(p)
        Pfull = np.zeros(p)
        Mfull[i - 1:], Pfull[i - 1:] = M, Ph
        accs[i] = (Mfull.copy(), Pfull.copy())
    t = r["t"]
    assert accs[t][0][p - 1] == r["mse"] and accs[t][1][p - 1] == r["phi"]
    # the accumulators equal the interval sums along the traced-back chain
    m = pipeline.chain_metrics(H, r["chain_bp"], lam)
    assert abs(accs[t][0][p - 1] - m["mse"]) <= 1e-12 * m["mse"]


def test_hirschberg_matches_backpointers_at_scale():
    """Hirschberg recovery (Sec. 5) equals the stored-argmin traceback and its
    recomputed cost equals the DP optimum."""
    rng = np.random.default_rng(15)
    for d, s, lam in ((700, 12, 0.05), (1500, 20, 0.01), (900, 7, 0.0)):
        x = rng.standard_normal(d).astype(np.float32)
        H = pipeline.prepare(x)
        r = pipeline.dp_forward(H, s, lam * H.s2tot, backpointers=True)
        ch, _ = pipeline.hirschberg(H, r["t"], lam * H.s2tot)
        assert list(ch) == list(r["chain_bp"])
        m = pipeline.chain_metrics(H, ch, lam)
        J = m["mse"] + lam * H.s2tot * m["entropy_surrogate"]
        assert abs(J - r["J"]) <= 1e-12 * abs(r["J"])


def test_refinement_never_worsens_and_colours_separate():
    """Sec. 6: each committed colour substep lowers vNMSE + lambda H(Xhat);
    moves inside one colour class are independent (their objective changes add
    up exactly), which is what allows updating them in parallel."""
    rng = np.random.default_rng(16)
    x = np.round(rng.standard_normal(300) * 8).astype(np.float32)
    lam = 0.02
    H = pipeline.prepare(x)
    r = pipeline.dp_forward(H, 10, lam * H.s2tot, backpointers=True)
    chain = r["chain_bp"]
    base = pipeline.chain_metrics(H, chain, lam)["objective"]
    for rounds in (1, 2, 5):
        u, _, _ = pipeline.refine(H, chain, lam * H.s2tot, rounds=rounds)
        assert pipeline.chain_metrics(H, u, lam)["objective"] <= base + 1e-15
    # additivity, checked with the plain (exact-frequency) objective
    xs = [float(a) for a in x]
    vals = [float(a) for a in H.v]
    Q0 = [vals[k] for k in chain]
    J0 = plain.objective(xs, Q0, lam, "out")
    t = len(chain)
    for c in range(3):
        movers = [r_ for r_ in range(1, t - 1) if r_ % 3 == c]
        deltas, newQ = [], list(Q0)
        for r_ in movers:
            lo, hi = chain[r_ - 1], chain[r_ + 1]
            if hi - lo < 3:
                continue
            m = lo + 1 if chain[r_] != lo + 1 else lo + 2
            Q1 = list(Q0)
            Q1[r_] = vals[m]
            deltas.append(plain.objective(xs, Q1, lam, "out") - J0)
            newQ[r_] = vals[m]
        Jall = plain.objective(xs, newQ, lam, "out")
        assert abs((Jall - J0) - sum(deltas)) < 1e-12


def test_refinement_two_colours_would_not_separate():
    """Why three colours: moving q_r and q_{r+2} together changes f_{r+1}
    through both, so their objective changes do not add up."""
    x = [float(a) for a in range(0, 13)]
    Q0 = [0.0, 3.0, 6.0, 9.0, 12.0]
    lam = 0.5
    J0 = plain.objective(x, Q0, lam, "out")
    d1 = plain.objective(x, [0.0, 4.0, 6.0, 9.0, 12.0], lam, "out") - J0
    d3 = plain.objective(x, [0.0, 3.0, 6.0, 11.0, 12.0], lam, "out") - J0
    both = plain.objective(x, [0.0, 4.0, 6.0, 11.0, 12.0], lam, "out") - J0
    assert abs(both - (d1 + d3)) > 1e-6


# --------------------------------------------------------------------------
# Final rounding


def test_philox_known_answers():
    """Philox4x32-10 test vectors published with Random123 (Salmon et al., SC'11)."""
    cases = [
        ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
        ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
        ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
         (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
    ]
    for ctr, key, want in cases:
        a = [np.array([c], dtype=np.uint64) for c in ctr]
        got = philox4x32_10(*a, np.array([key[0]], dtype=np.uint64),
                            np.array([key[1]], dtype=np.uint64))
        assert tuple(int(g[0]) for g in got) == want


def test_uniforms_are_uniform():
    u = pipeline.uniforms(200000, 12345)
    assert u.min() >= 0 and u.max() < 1
    hist, _ = np.histogram(u, bins=50, range=(0, 1))
    chi2 = ((hist - 4000) ** 2 / 4000).sum()
    assert chi2 < 100  # 49 dof, p ~ 1e-5


def test_uniforms_stream_layout():
    """Entries 2j and 2j+1 take words (0, 1) and (2, 3) of the generator at
    counter (j, 0, stream, 0); an odd count ends on an even entry."""
    seed = 0x1234_5678_9ABC_DEF0
    for stream in (0, 1):
        u = pipeline.uniforms(7, seed, stream)
        assert len(u) == 7
        for j in range(4):
            a = [np.array([v], dtype=np.uint64) for v in (j, 0, stream, 0)]
            w = [int(g[0]) for g in philox4x32_10(*a, np.array([seed & 0xFFFFFFFF], dtype=np.uint64),
                                                  np.array([seed >> 32], dtype=np.uint64))]
            for e in range(2):
                if 2 * j + e < 7:
                    bits = ((w[2 * e + 1] << 32) | w[2 * e]) >> 11
                    assert u[2 * j + e] == bits * 2.0 ** -53


def test_uniform_pairs_are_independent():
    """The two entries that share a generator call are jointly uniform: a
    10 x 10 chi-square on (u_2j, u_2j+1), and the two streams against each
    other."""
    n = 400000
    for a, b in ((pipeline.uniforms(n, 99)[0::2], pipeline.uniforms(n, 99)[1::2]),
                 (pipeline.uniforms(n, 99, 0), pipeline.uniforms(n, 99, 1))):
        h, _, _ = np.histogram2d(a, b, bins=10, range=[[0, 1], [0, 1]])
        e = len(a) / 100.0
        assert ((h - e) ** 2 / e).sum() < 160  # 99 dof, p ~ 1e-4


def test_quantize_is_unbiased():
    """E[xhat] = x for SQ (Sec. 2): mean over K seeds within 5 sigma per entry,
    and the empirical MSE matches sum (b-x)(x-a)."""
    x = np.random.default_rng(17).standard_normal(300).astype(np.float32)
    q = np.array([x.min(), -0.7, 0.0, 0.4, 1.3, x.max()], dtype=np.float64)
    K = 400
    acc = np.zeros(len(x))
    sq = np.zeros(len(x))
    for seed in range(K):
        sym, hist, _ = pipeline.quantize(x, q, seed)
        xh = q[sym]
        acc += xh
        sq += (xh - x.astype(np.float64)) ** 2
    xf = x.astype(np.float64)
    r = np.clip(np.searchsorted(q, xf, side="left") - 1, 0, len(q) - 2)
    var = (q[r + 1] - xf) * (xf - q[r])
    z = (acc / K - xf) / np.sqrt(np.maximum(var, 1e-30) / K)
    assert np.all(np.abs(z[var > 0]) < 5.5)
    assert abs(sq.sum() / K - var.sum()) < 0.05 * var.sum()


def test_quantize_edges():
    """x = q_0 maps to symbol 0; x = q_{r+1} maps to r+1; t = 1 maps to 0."""
    q = np.array([-1.0, 0.0, 2.0])
    sym, hist, ent = pipeline.quantize(np.array([-1.0, 0.0, 2.0], dtype=np.float32), q, 0)
    assert list(sym) == [0, 1, 2] and list(hist) == [1, 1, 1]
    assert abs(ent - math.log2(3)) < 1e-15
    sym, hist, ent = pipeline.quantize(np.array([5.0, 5.0], dtype=np.float32), np.array([5.0]), 0)
    assert list(sym) == [0, 0] and ent == 0.0
