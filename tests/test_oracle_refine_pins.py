"""Pins of the oracle's three-colour refinement (Sec. 6) against the plain
per-entry definitions in oracle/plain.py.

The refinement moves one codebook value q_r inside the open range between its
neighbours so as to lower vNMSE + lambda H(Xhat).  Moving q_r changes the MSE
of the entries between q_{r-1} and q_{r+1} and the expected frequencies of
q_{r-1}, q_r and q_{r+1} only, so the oracle evaluates a local objective built
from the App. D closed forms.  These tests check that local objective value
by value against the per-entry MSE and frequencies (Sec. 2, Sec. 3), the
exhaustive search against the plain lowest argmin, the binary search against
the same search run on the plain objective (including inputs with exact ties,
where '<' and '<=' part ways), one colour substep against the sum of its
movers' plain objective changes, and whole refinements (rounds, colours,
strict acceptance, the budget guard) against a plain re-implementation.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import pipeline, plain


def _tiny_cases(seed, n, exact=False):
    """Tiny inputs (d <= 10, with duplicates), a random spanning chain of at
    least 3 values, and a multiplier.  exact=True: small integers and lambda = 0,
    where both sides compute the MSE exactly and ties are real."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        d = int(rng.integers(5, 11))
        if exact:
            x = rng.integers(-4, 5, size=d).astype(np.float32)
            lam = 0.0
        else:
            x = (rng.standard_normal(d) * rng.choice([0.3, 1.0, 5.0])).astype(np.float32)
            if rng.random() < 0.5:  # duplicates
                x[rng.integers(0, d, size=3)] = x[0]
            lam = float(10 ** rng.uniform(-3, 0.5))
        H = pipeline.prepare(x)
        p = H.p
        if p < 4:
            continue
        t = int(rng.integers(3, min(p, 6) + 1))
        inner = np.sort(rng.choice(np.arange(1, p - 1), size=t - 2, replace=False))
        chain = np.array([0, *inner, p - 1], dtype=np.int32)
        out.append((x, H, chain, lam))
    return out


def _tol(H, lamp):
    """Rounding of the closed forms: a few ulps of ||X||^2 (the prefix-sum
    cancellation) plus a few of lambda' times the entropy terms."""
    return 1e-11 * (H.s2tot + lamp)


def _Q(H, chain, r=None, m=None):
    Q = [float(H.v[k]) for k in chain]
    if r is not None:
        Q[r] = float(H.v[m])
    return Q


def test_local_objective_is_the_plain_definition():
    """Sec. 6 local objective, value by value: for every mover r and every m
    in (u_{r-1}, u_{r+1}) the oracle's L_r(m) equals the per-entry MSE of
    (q_{r-1}, q_{r+1}] plus lambda' (h(f_{r-1}/d) + h(f_r/d) + h(f_{r+1}/d))
    with the frequencies counted entry by entry; the first and last values'
    frequencies (the first takes every entry equal to it) included."""
    n_checked = 0
    for x, H, chain, lam in _tiny_cases(101, 60) + _tiny_cases(102, 20, exact=True):
        lamp = lam * H.s2tot
        tol = _tol(H, lamp)
        xs = [float(a) for a in x]
        t = len(chain)
        for r in range(1, t - 1):
            for m in range(chain[r - 1] + 1, chain[r + 1]):
                got = pipeline.refine_local(H, chain, r, m, lamp)
                want = plain.refine_local(xs, _Q(H, chain, r, m), r, lamp)
                assert abs(got - float(want)) <= tol, (xs, list(chain), r, m, lam)
                n_checked += 1
    assert n_checked > 300


def test_local_objective_differences_are_global_differences():
    """Moving q_r changes nothing outside the local objective: L_r(m) - L_r(m')
    equals ||X||^2 times the change of the whole plain objective
    vNMSE + lambda H(Xhat) (Sec. 6 works on that objective)."""
    for x, H, chain, lam in _tiny_cases(103, 40):
        lamp = lam * H.s2tot
        xs = [float(a) for a in x]
        t = len(chain)
        for r in range(1, t - 1):
            J0 = plain.objective(xs, _Q(H, chain), lam, "out")
            L0 = pipeline.refine_local(H, chain, r, int(chain[r]), lamp)
            for m in range(chain[r - 1] + 1, chain[r + 1]):
                Jm = plain.objective(xs, _Q(H, chain, r, m), lam, "out")
                Lm = pipeline.refine_local(H, chain, r, m, lamp)
                assert abs((Lm - L0) - H.s2tot * (Jm - J0)) <= 2 * _tol(H, lamp)


def _search_cases():
    return _tiny_cases(104, 80) + _tiny_cases(105, 60, exact=True)


@pytest.mark.parametrize("exhaustive", [True, False])
def test_search_is_the_plain_search(exhaustive):
    """The exhaustive search returns the lowest minimiser of the plain local
    objective; the binary search returns what the same binary search (lo =
    L+1, hi = R-1, step right iff L(mid+1) < L(mid)) returns on the plain
    objective.  Cases whose plain decisions fall within rounding of a tie are
    skipped; with integer inputs at lambda = 0 both sides are exact and ties
    are decided, not skipped."""
    decided = ties = 0
    for x, H, chain, lam in _search_cases():
        lamp = lam * H.s2tot
        xs = [float(a) for a in x]
        v = [float(a) for a in H.v]
        for r in range(1, len(chain) - 1):
            try:
                want = plain.refine_search(xs, v, list(chain), r, lamp, exhaustive, _tol(H, lamp))
            except plain.NearTie:
                continue
            got = pipeline.refine_search(H, chain, r, lamp, exhaustive)
            assert got == want, (xs, list(chain), r, lam, exhaustive)
            decided += 1
            if lam == 0.0:
                L, R = chain[r - 1], chain[r + 1]
                vals = [plain.refine_local(xs, _Q(H, chain, r, m), r, 0.0) for m in range(L + 1, R)]
                ties += len(vals) != len(set(vals))
    assert decided > 150 and ties > 5


@pytest.mark.parametrize("n", [5, 7, 9, 11])
def test_binary_search_on_a_symmetric_tie(n):
    """Equally spaced values 0..n with one entry each and the chain (0, u, n):
    the local objective of the middle value is symmetric about n/2, so for odd
    n the two middle positions tie exactly.  The paper's search steps right
    only on a strict decrease, so it stops at the lower of the two; the
    exhaustive search also returns the lower one; and a mover already at the
    upper one does not move (the move must be a strict improvement)."""
    x = np.arange(n + 1, dtype=np.float32)
    H = pipeline.prepare(x)
    xs = [float(a) for a in x]
    v = [float(a) for a in H.v]
    lo_mid, hi_mid = (n - 1) // 2, (n + 1) // 2
    vals = {m: plain.refine_local(xs, [0.0, v[m], float(n)], 1, 0.0) for m in range(1, n)}
    assert vals[lo_mid] == vals[hi_mid] == min(vals.values())
    for u1 in range(1, n):
        chain = np.array([0, u1, n], dtype=np.int32)
        for exh in (False, True):
            want = plain.refine_search(xs, v, list(chain), 1, 0.0, exh)
            assert want == lo_mid
            assert pipeline.refine_search(H, chain, 1, 0.0, exh) == want
        u, _, moves = pipeline.refine(H, chain, 0.0, rounds=5)
        assert list(u) == [0, lo_mid if u1 != hi_mid else hi_mid, n]
        assert moves == (0 if u1 in (lo_mid, hi_mid) else 1)


def test_substep_change_is_the_sum_of_mover_changes():
    """One colour substep (Sec. 6): the chain it returns equals the plain
    substep, and its change of vNMSE + lambda H(Xhat) equals the sum of the
    changes each of its movers makes alone (movers three apart change disjoint
    frequencies)."""
    checked = 0
    for x, H, chain, lam in _tiny_cases(106, 80) + _tiny_cases(107, 40, exact=True):
        lamp = lam * H.s2tot
        xs = [float(a) for a in x]
        v = [float(a) for a in H.v]
        t = len(chain)
        for c in range(3):
            nu, moved = pipeline.refine_substep(H, chain, c, lamp)
            assert all(nu[r] == chain[r] for r in range(t) if not (1 <= r <= t - 2 and r % 3 == c))
            want = list(chain)
            try:
                for r in range(1, t - 1):
                    if r % 3 != c:
                        continue
                    m = plain.refine_search(xs, v, list(chain), r, lamp, False, _tol(H, lamp))
                    if m != chain[r] and plain._less(
                            plain.refine_local(xs, _Q(H, chain, r, m), r, lamp),
                            plain.refine_local(xs, _Q(H, chain), r, lamp), _tol(H, lamp)):
                        want[r] = m
            except plain.NearTie:
                continue
            assert list(nu) == want and moved == sum(a != b for a, b in zip(want, chain))
            J0 = plain.objective(xs, _Q(H, chain), lam, "out")
            deltas = 0.0
            for r in range(1, t - 1):
                if nu[r] != chain[r]:
                    deltas += plain.objective(xs, _Q(H, chain, r, int(nu[r])), lam, "out") - J0
            Jn = plain.objective(xs, [v[k] for k in nu], lam, "out")
            assert abs((Jn - J0) - deltas) <= 1e-12 * (1 + abs(J0))
            checked += moved > 0
    assert checked > 20


@pytest.mark.parametrize("exhaustive", [False, True])
@pytest.mark.parametrize("budget", [False, True])
def test_refinement_equals_the_plain_refinement(exhaustive, budget):
    """Whole refinements (up to 5 rounds of colours 0, 1, 2, strict acceptance,
    stop after a round without a move, and with the budget guard the substep
    undone when H(Xhat) exceeds b) equal the plain re-implementation on the
    plain objective, chain and rounds run."""
    agree = moved = 0
    rng = np.random.default_rng(108 + 2 * exhaustive + budget)
    for x, H, chain, lam in _tiny_cases(109, 50) + _tiny_cases(110, 25, exact=True):
        lamp = lam * H.s2tot
        xs = [float(a) for a in x]
        v = [float(a) for a in H.v]
        b = math.inf
        if budget:
            H0 = plain.entropy_out(xs, _Q(H, chain))
            b = H0 + float(rng.uniform(-0.3, 0.3))
        try:
            want, nrun = plain.refine(xs, v, list(chain), lamp, b, budget, 5, exhaustive,
                                      _tol(H, lamp))
        except plain.NearTie:
            continue
        got, n, _ = pipeline.refine(H, chain, lamp, b, budget, 5, exhaustive)
        assert list(got) == want and n == nrun, (xs, list(chain), lam, b)
        agree += 1
        moved += want != list(chain)
    assert agree > 50 and moved > 15
