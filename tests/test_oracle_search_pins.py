"""Pins of the oracle's canonical exp2 and of the budget search's aimed query
and trajectory replay (Sec. 3 and Sec. 5: the search on lambda for a budget)."""
import math

import mpmath
import numpy as np
import pytest

from oracle import native, pipeline
from oracle.log2_table import build_exp2_table


def _ulps(a, b):
    return abs(a - b) / math.ulp(b)


def test_exp2_table_and_coefficients():
    """T[i] = RN(2^(i/64)) and C_k = RN(ln(2)^k / k!): checked against an
    exact integer test of the rounding (T) and a 400-bit evaluation (C)."""
    T, C = build_exp2_table()
    for i, t in enumerate(T):
        # t is RN(2^(i/64)) iff 2^(i/64) lies within half an ulp of t:
        # (t - u/2)^64 < 2^i < (t + u/2)^64, compared in exact integers
        m, e = math.frexp(t)  # t = m 2^e, m in [0.5, 1)
        M = int(m * 2 ** 53)  # t = M 2^(e-53)
        lo, hi = (2 * M - 1), (2 * M + 1)  # (t -+ u/2) = (2M -+ 1) 2^(e-54)
        sh = 64 * (e - 54)
        if sh >= 0:
            assert lo ** 64 * 2 ** sh < 2 ** i < hi ** 64 * 2 ** sh
        else:
            assert lo ** 64 < 2 ** (i - sh) < hi ** 64
    mpmath.mp.prec = 400
    for k, c in enumerate(C, start=1):
        exact = mpmath.log(2) ** k / mpmath.factorial(k)
        assert abs(mpmath.mpf(c) - exact) <= mpmath.mpf(math.ulp(c)) / 2


def test_exp2c_against_mpmath():
    """exp2c within 2 ulp of 2^y (mpmath, 200 bits) over |y| < 1000, exact at
    integers, monotone across the table's breakpoints."""
    L = native.lib()
    mpmath.mp.prec = 200
    rng = np.random.default_rng(5)
    ys = np.concatenate([rng.uniform(-60, 60, 3000), rng.uniform(-1000, 1000, 500),
                         rng.uniform(-1 / 64, 1 / 64, 500), np.arange(-64, 65) / 64.0 + 1e-9])
    for y in ys:
        got = L.orc_exp2c(float(y))
        want = float(mpmath.power(2, mpmath.mpf(float(y))))
        assert _ulps(got, want) <= 2.0, (y, got, want)
    for k in range(-1020, 1020, 7):
        assert L.orc_exp2c(float(k)) == math.ldexp(1.0, k)
    prev = 0.0
    for y in np.linspace(-3, 3, 20001):
        v = L.orc_exp2c(float(y))
        assert v >= prev
        prev = v
    assert L.orc_exp2c(-2000.0) == 0.0 and L.orc_exp2c(2000.0) == math.inf
    assert math.isnan(L.orc_exp2c(math.nan))


def test_aimed_query_is_the_tangent_slope():
    """The aimed multiplier is -dM/dH at H = b of M(H) = M_A (M_B/M_A)^((H-H_A)/(H_B-H_A)),
    the curve through A and B on which log vNMSE is linear in H: checked
    against that formula in 200-bit arithmetic to 1e-12 relative."""
    L = native.lib()
    mpmath.mp.prec = 200
    rng = np.random.default_rng(6)
    for _ in range(500):
        HB = float(rng.uniform(0.2, 4.0))
        HA = HB + float(rng.uniform(0.05, 2.0))
        MA = float(10 ** rng.uniform(-6, -1))
        MB = MA * float(10 ** rng.uniform(0.05, 3))
        b = float(rng.uniform(HB, HA))
        got = L.orc_aim_query(b, HA, MA, HB, MB)
        rho = (mpmath.log(MB) - mpmath.log(MA)) / (mpmath.mpf(HB) - HA)
        mb = MA * mpmath.exp(rho * (mpmath.mpf(b) - HA))
        want = float(-rho * mb)
        assert want > 0 and abs(got - want) <= 1e-12 * want


@pytest.mark.parametrize("width", [1, 8])
def test_replayed_search_takes_the_same_decisions(width):
    """A search re-run on its own recorded trajectory (points standing in for
    the solves) returns the same result; a trajectory with one multiplier
    changed, or cut short, is refused."""
    x = np.random.default_rng(7).standard_normal(600).astype(np.float32)
    H = pipeline.prepare(x)
    for b in (0.8, 1.7, 2.6):
        r = pipeline.search(H, 12, b, width=width)
        rr = pipeline.search(H, 12, b, width=width, replay=r["traj"])
        for k in ("lam", "H", "M", "t", "solves", "status", "lam_final", "passes"):
            assert rr[k] == r[k] or (isinstance(r[k], float) and math.isnan(r[k])), k
        assert np.array_equal(rr["traj"], r["traj"])
        bad = r["traj"].copy()
        bad[-1, 0] = np.nextafter(bad[-1, 0], np.inf)
        with pytest.raises(pipeline.ReplayMismatch):
            pipeline.search(H, 12, b, width=width, replay=bad)
        if len(r["traj"]) > 1:
            with pytest.raises(pipeline.ReplayMismatch):
                pipeline.search(H, 12, b, width=width, replay=r["traj"][:-1])
