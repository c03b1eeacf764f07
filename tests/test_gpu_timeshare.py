"""GPU parity of the budget search over the optimal DP and of two-way
time-sharing (Sec. 7, App. E) against the CPU oracle, through the C ABI.

Codebooks, time-share weights and partitions must match the oracle exactly;
objectives and entropies within 1e-9 relative.
"""
import math
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import pipeline
from paper_2608_18147_amd import ecasq, inputs

pytestmark = pytest.mark.gpu

REL = 1e-9


def _say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def _dev(x):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda")


def _close(a, b, rel=REL):
    if math.isinf(a) or math.isinf(b):
        return a == b
    return abs(a - b) <= rel * max(abs(a), abs(b), 1e-300)


def _compare(g, r, passes=True):
    cb, rk, info = g
    assert info["t"] == r.t and info["p"] == r.p
    np.testing.assert_array_equal(rk.cpu().numpy(), r.rank)
    np.testing.assert_array_equal(cb.cpu().numpy(), r.codebook)
    assert info["lambda"] == r.lam or (math.isinf(info["lambda"]) and math.isinf(r.lam))
    for k in ("mse", "vnmse", "entropy", "entropy_surrogate", "objective", "rate_total"):
        assert _close(info[k], getattr(r, k)), (k, info[k], getattr(r, k))
    assert info["dp_solves"] == r.dp_solves
    assert info["refine_rounds_run"] == r.refine_rounds
    assert info["cells"] == r.cells
    assert info["status"] == r.status
    if passes:
        assert info["search_passes"] == r.passes


def _rounded(d, seed):
    return (np.round(inputs.normal(d, seed) * 6.0) / 6.0).astype(np.float32)


OPT_BUDGET_CASES = [
    ("normal_300_b2", lambda: inputs.normal(300, 31), 8, 2.0, {}),
    ("lognormal_500_b1.5", lambda: inputs.lognormal_signed(500, 32), 10, 1.5, {}),
    ("student_400_b2.5", lambda: inputs.student_t(400, 33), 12, 2.5, {}),
    ("dups_b1.2", lambda: _rounded(3000, 34), 10, 1.2, {}),
    ("b_above_max", lambda: inputs.normal(200, 35), 6, 9.0, {}),
    ("b_below_one", lambda: inputs.normal(200, 36), 6, 0.4, {}),
    ("exact_s", lambda: inputs.normal(300, 37), 7, 2.2, dict(exact_s=1)),
    ("uniform_grid", lambda: inputs.lognormal_signed(2048, 38), 10, 2.0,
     dict(alphabet=1, alphabet_size=300)),
]


def _alpha(o):
    if o.get("alphabet"):
        return ("uniform" if o["alphabet"] == 1 else "quantile", o["alphabet_size"])
    return None


@pytest.mark.parametrize("case", OPT_BUDGET_CASES, ids=[c[0] for c in OPT_BUDGET_CASES])
def test_optimal_budget_search_parity(case):
    """Budget mode on the optimal DP: the lowest-vNMSE supported point with
    H(Xhat) <= b (queries aimed at b, certified by the chord)."""
    name, mk, s, b, o = case
    x = mk()
    _say("optimal budget", name, x.size, s, b)
    r = pipeline.solve(x, s, b, exact_s=bool(o.get("exact_s", 0)), dp="optimal",
                       alphabet=_alpha(o))
    opts = ecasq.ecasq_default_options(dp_objective=1, optimal_scan=1, **o)
    g = ecasq.ecasq_solve(_dev(x), s, b, options=opts)
    _compare(g, r)
    if r.status == 0:
        assert g[2]["entropy"] <= b


@pytest.mark.parametrize("dp", ["approx", "optimal"])
@pytest.mark.parametrize("case", OPT_BUDGET_CASES, ids=[c[0] for c in OPT_BUDGET_CASES])
def test_timeshare_parity(case, dp):
    name, mk, s, b, o = case
    x = mk()
    _say("timeshare", dp, name, x.size, s, b)
    r = pipeline.solve_timeshare(x, s, b, exact_s=bool(o.get("exact_s", 0)), dp=dp,
                                 alphabet=_alpha(o))
    extra = dict(dp_objective=1, optimal_scan=1) if dp == "optimal" else {}
    opts = ecasq.ecasq_default_options(**extra, **o)
    gm, gp, alpha = ecasq.ecasq_solve_timeshare(_dev(x), s, b, options=opts)
    assert alpha == r["alpha"]
    _compare(gm, r["minus"])
    _compare(gp, r["plus"])
    if alpha > 0.0:
        key = "entropy" if dp == "optimal" else "entropy_surrogate"
        mix = alpha * gp[2][key] + (1.0 - alpha) * gm[2][key]
        assert abs(mix - b) <= 1e-12 * b
        assert gm[2]["vnmse"] >= alpha * gp[2]["vnmse"] + (1 - alpha) * gm[2]["vnmse"]


@pytest.mark.parametrize("alpha,seed", [(0.0, 3), (0.3, 4), (0.77, 2 ** 40 + 5), (1.0, 6)])
def test_quantize_timeshare_bit_exact(alpha, seed):
    x = inputs.lognormal_signed(50000, 40)
    lo, hi = float(x.min()), float(x.max())
    cm = np.array([lo, -1.0, 0.5, 2.0, hi])
    cp = np.array([lo, -3.0, -0.2, 0.1, 1.0, 6.0, hi])
    _say("quantize timeshare", alpha, seed)
    sym, part, ent, hist = ecasq.ecasq_quantize_timeshare(_dev(x), torch.from_numpy(cm),
                                                          torch.from_numpy(cp), alpha, seed)
    osym, opart, ohist, oent = pipeline.quantize_timeshare(x, cm, cp, alpha, seed)
    np.testing.assert_array_equal(part.cpu().numpy(), opart)
    np.testing.assert_array_equal(sym.cpu().numpy(), osym)
    np.testing.assert_array_equal(hist.cpu().numpy(), ohist)
    assert _close(float(ent), oent, 1e-12)
    if alpha == 0.0:
        s0, e0, _ = ecasq.ecasq_quantize(_dev(x), torch.from_numpy(cm), seed)
        assert np.array_equal(s0.cpu().numpy(), sym.cpu().numpy()) and float(e0) == float(ent)


def test_timeshare_full_size_weights():
    """The 2^18 weight-like workload at b = 2 bits: the time-share of the
    search's final pair has H(I,B) = b and a vNMSE no larger than the
    unrefined budget solution; the time-shared rounding puts a share alpha of
    the entries on the second codebook."""
    x = inputs.make("weights_256k", seed=0)
    xd = _dev(x)
    b = 2.0
    _say("timeshare full size")
    gm, gp, alpha = ecasq.ecasq_solve_timeshare(xd, 32, b)
    im, ip = gm[2], gp[2]
    _say("  alpha", alpha, "t", im["t"], ip["t"], "H", im["entropy_surrogate"],
         ip["entropy_surrogate"])
    assert 0.0 <= alpha < 1.0
    if alpha > 0.0:
        mix_h = alpha * ip["entropy_surrogate"] + (1 - alpha) * im["entropy_surrogate"]
        assert abs(mix_h - b) <= 1e-12 * b
        assert im["entropy_surrogate"] <= b < ip["entropy_surrogate"]
    g1 = ecasq.ecasq_solve(xd, 32, b, options=ecasq.ecasq_default_options(refine_rounds=0))
    np.testing.assert_array_equal(g1[1].cpu().numpy(), gm[1].cpu().numpy())
    mix_v = alpha * ip["vnmse"] + (1 - alpha) * im["vnmse"]
    assert mix_v <= im["vnmse"] * (1 + 1e-12)
    sym, part, ent, hist = ecasq.ecasq_quantize_timeshare(xd, gm[0], gp[0], alpha, 11)
    n = x.size
    share = float(part.sum()) / n
    assert abs(share - alpha) <= 5 * math.sqrt(max(alpha * (1 - alpha), 1e-12) / n) + 1e-12
    assert int(hist.sum()) == n


REFINED_CASES = OPT_BUDGET_CASES + [
    ("weights_2k_b2", lambda: inputs.make("weights_256k", seed=11, d=2048), 16, 2.0, {}),
    ("student_2k_b1.5", lambda: inputs.make("student_t_1m", seed=11, d=2048), 16, 1.5, {}),
    ("lognormal_2k_b2.5_exh", lambda: inputs.make("lognormal_16k", seed=11, d=2048), 32, 2.5,
     dict(refine_exhaustive=1)),
]


@pytest.mark.parametrize("case", REFINED_CASES, ids=[c[0] for c in REFINED_CASES])
def test_refinement_aware_search_parity(case):
    """Budget search on the refined codebooks' true H(Xhat) (dp_objective 2):
    every point is dp_APX's traceback refined at its multiplier; the answer is
    the feasible point of lowest vNMSE."""
    name, mk, s, b, o = case
    x = mk()
    _say("refined search", name, x.size, s, b)
    r = pipeline.solve(x, s, b, exact_s=bool(o.get("exact_s", 0)), dp="refined",
                       recovery="backpointers", width=1, alphabet=_alpha(o),
                       exhaustive=bool(o.get("refine_exhaustive", 0)))
    opts = ecasq.ecasq_default_options(dp_objective=2, **o)
    g = ecasq.ecasq_solve(_dev(x), s, b, options=opts)
    _compare(g, r)
    if r.status == 0:
        assert g[2]["entropy"] <= b


def test_refinement_aware_budget_sweep():
    x = inputs.student_t(3000, 44)
    budgets = (1.0, 2.0, 3.0)
    _say("refined budget sweep")
    rs = pipeline.solve_budgets(x, 16, budgets, refine_rounds=5, recovery="backpointers",
                                width=1, dp="refined")
    gs = ecasq.ecasq_solve_budgets(_dev(x), 16, budgets,
                                   options=ecasq.ecasq_default_options(dp_objective=2))
    for g, r in zip(gs, rs):
        _compare(g, r)
