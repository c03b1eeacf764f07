"""GPU parity at the full sizes of the evaluation workloads, through the C ABI.

lognormal_16k (d = 16384, s = 32, budgets 1.5, 2.5, 3.5): every search point,
the codebook before and after refinement, the multipliers and the metrics
against the oracle's own end-to-end solves, stored by
tests/golden/make_lognormal_16k.py (the oracle takes about three minutes per
budget at this size).

weights_256k (d = 2^18, s = 32, b = 2, five refinement rounds) and
student_t_1m (d = 2^20, s = 64, budgets 1, 2, 3, 4 sharing their solves), where
one oracle DP solve would take hours, are verified step by step from what the
library records (ecasq_inspect_*):
  search      the oracle's search, run on the GPU's points in place of its own
              solves, asks for exactly the multipliers the GPU solved, in order,
              and ends on the same pair, multiplier and pass count;
  DP          the final solve is re-run with every layer dumped; the oracle
              recomputes from the GPU's previous layer each chain column's
              value and lowest argmin (the traceback must follow them) and a
              sample of other columns' values, bit for bit;
  refinement  the oracle's refinement of the GPU's unrefined codebook at the
              GPU's multiplier equals the GPU's refined codebook, rounds too;
  metrics     MSE, vNMSE, H(Xhat), H(I,B), objective, rate from the oracle's
              sums over the returned codebook, to 1e-9;
  rounding    the final stochastic rounding (Philox seed 0) symbol for symbol.
"""
import math
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import pipeline
from paper_2608_18147_amd import ecasq, inputs
from tests.conftest import ROOT

pytestmark = pytest.mark.gpu

REL = 1e-9
METRICS = ("mse", "vnmse", "entropy", "entropy_surrogate", "objective", "rate_total")


def _say(*a):
    # straight to the terminal: a long case keeps printing while it runs
    sys.__stdout__.write("[case] " + " ".join(str(v) for v in a) + "\n")
    sys.__stdout__.flush()


def _dev(x):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda")


def _close(a, b, rel=REL):
    return abs(a - b) <= rel * max(abs(a), abs(b))


def _golden16k():
    out = {}
    with open(os.path.join(ROOT, "tests", "golden", "lognormal_16k_solutions.txt")) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if line:
                k, v = (a.strip() for a in line.split("=", 1))
                out[k] = v
    return out


def _hexes(s):
    return np.array([float.fromhex(a) for a in s.split()])


@pytest.fixture
def inspect_log():
    ecasq.ecasq_inspect_enable(True)
    yield
    ecasq.ecasq_inspect_enable(False)


# ---------------------------------------------------------------- 16k, stored


@pytest.mark.parametrize("b", [1.5, 2.5, 3.5])
def test_lognormal_16k_equals_stored_oracle_solves(b, inspect_log):
    """d = 16384 end to end (histogram, search, traceback, refinement,
    metrics) against the oracle's stored solves, with R = 5 and R = 0."""
    g = _golden16k()
    x = inputs.make("lognormal_16k", 0)
    xd = _dev(x)
    tag = f"b{b}"
    _say("lognormal_16k", tag)
    cb, rk, info = ecasq.ecasq_solve(xd, 32, b)
    traj = ecasq.ecasq_inspect_points()
    res = ecasq.ecasq_inspect_results()
    want = _hexes(g[f"{tag}.traj"]).reshape(-1, 4)
    np.testing.assert_array_equal(traj, want)
    assert info["p"] == int(g["p"]) and info["status"] == int(g[f"{tag}.status"])
    assert info["dp_solves"] == int(g[f"{tag}.solves"])
    assert info["search_passes"] == int(g[f"{tag}.passes"])
    assert info["lambda"] == float.fromhex(g[f"{tag}.lambda"])
    assert len(res) == 1 and res[0]["lam_B"] == float.fromhex(g[f"{tag}.lambda_B"])
    r0 = [int(a) for a in g[f"{tag}.R0.rank"].split()]
    r5 = [int(a) for a in g[f"{tag}.R5.rank"].split()]
    assert list(res[0]["pre"]) == r0 and list(res[0]["post"]) == r5
    assert list(rk.cpu().numpy()[: info["t"]]) == r5
    assert info["refine_rounds_run"] == int(g[f"{tag}.R5.rounds"])
    for k in METRICS:
        assert _close(info[k], float.fromhex(g[f"{tag}.R5.{k}"])), k
    cb0, rk0, info0 = ecasq.ecasq_solve(xd, 32, b, options=ecasq.ecasq_default_options(
        refine_rounds=0))
    assert list(rk0.cpu().numpy()[: info0["t"]]) == r0 and info0["refine_rounds_run"] == 0
    for k in METRICS:
        assert _close(info0[k], float.fromhex(g[f"{tag}.R0.{k}"])), k


# ---------------------------------------------------- 2^18 and 2^20, stepwise


def _check_search(H, s, b, traj, info, res, cache=None):
    """Replay the oracle's search on the GPU's points."""
    sr = pipeline.search(H, s, b, width=1, cache=cache, replay=traj)
    assert sr["solves"] == len(traj) == info["dp_solves"]
    assert sr["passes"] == info["search_passes"]
    assert sr["lam"] == res["lam_B"] and sr["lam_final"] == info["lambda"]
    assert sr["t"] == len(res["pre"]) and sr["status"] == info["status"]
    return sr


def _check_dp(xd, H, s, lam, chain, rng, nsample):
    """The solve at lam with every layer dumped: the traceback's chain follows
    the lowest argmins the oracle recomputes from the GPU's previous layers,
    and sampled columns' values are the oracle's, bit for bit."""
    F, _, _, _, out = ecasq.ecasq_dp_trace(xd, s, lam, schedule=1, argmins=False)
    F = F.cpu().numpy()
    p = H.p
    lamp = lam * H.s2tot
    t = len(chain)
    imax = min(s, p)
    assert int(out[3]) == t and chain[0] == 0 and chain[-1] == p - 1
    assert F[t][p - 1] == out[0]
    zeros = np.zeros(p)
    for i in range(t, 2, -1):
        j = int(chain[i - 1])
        Fo, Ko, _, _ = pipeline.dp_columns(H, i, lamp, F[i - 1], zeros, zeros, cols=[j])
        assert Fo[0] == F[i][j], (i, j)
        assert Ko[0] == chain[i - 2], (i, j, Ko[0], chain[i - 2])
    Fo, _, _, _ = pipeline.dp_columns(H, 2, lamp, cols=[int(chain[1])])
    assert Fo[0] == F[2][int(chain[1])]
    # final layer choice (eq. apx_final): the lowest i with the least F_i[p-1]
    last = [F[i][p - 1] for i in range(2, imax + 1)]
    assert 2 + int(np.argmin(last)) == t
    for i in range(3, imax + 1):
        cols = np.unique(np.concatenate([rng.integers(i - 1, p, nsample), [p - 1]]))
        Fo, _, _, _ = pipeline.dp_columns(H, i, lamp, F[i - 1], zeros, zeros, cols=cols)
        np.testing.assert_array_equal(Fo, F[i][cols], err_msg=f"layer {i}")


def _check_refine_and_metrics(H, b, info, res, rounds=5):
    u, n, _ = pipeline.refine(H, res["pre"], info["lambda"] * H.s2tot, b, True, rounds)
    np.testing.assert_array_equal(u, res["post"])
    assert n == info["refine_rounds_run"]
    m = pipeline.chain_metrics(H, res["post"], info["lambda"])
    for k in METRICS:
        assert _close(info[k], m[k]), (k, info[k], m[k])


def _check_rounding(x, xd, cb, t):
    sym, ent, hist = ecasq.ecasq_quantize(xd, cb[:t], 0)
    s_o, h_o, e_o = pipeline.quantize(x, cb[:t].cpu().numpy(), 0)
    np.testing.assert_array_equal(sym.cpu().numpy(), s_o)
    np.testing.assert_array_equal(hist.cpu().numpy(), h_o)
    assert abs(float(ent) - e_o) <= 1e-12


def test_weights_256k_solve_step_by_step(inspect_log):
    """2^18 weight-like vector, s = 32, b = 2, R = 5: the bench's workload."""
    x = inputs.make("weights_256k", 0)
    xd = _dev(x)
    _say("weights_256k solve")
    cb, rk, info = ecasq.ecasq_solve(xd, 32, 2.0)
    traj = ecasq.ecasq_inspect_points()
    res = ecasq.ecasq_inspect_results()
    assert len(res) == 1 and info["status"] == 0
    res = res[0]
    np.testing.assert_array_equal(rk.cpu().numpy()[: info["t"]], res["post"])
    _say("oracle prepare", x.size)
    H = pipeline.prepare(x)
    assert info["p"] == H.p
    _check_search(H, 32, 2.0, traj, info, res)
    _say("dump and check the final solve's layers")
    _check_dp(xd, H, 32, res["lam_B"], res["pre"], np.random.default_rng(40), 24)
    _say("refinement, metrics, rounding")
    _check_refine_and_metrics(H, 2.0, info, res)
    _check_rounding(x, xd, cb, info["t"])


@pytest.mark.timeout(900)
def test_student_t_1m_budget_sweep_step_by_step(inspect_log, capfd):
    """2^20 Student-t vector, s = 64, budgets 1, 2, 3, 4 in one call sharing
    their solves (each search starts from the earlier ones' points), R = 5,
    then the final rounding of every budget's codebook.  Runs for minutes:
    its progress lines go to the terminal as it runs."""
    with capfd.disabled():
        _student_t_1m_sweep()


def _student_t_1m_sweep():
    x = inputs.make("student_t_1m", 0)
    xd = _dev(x)
    budgets = (1.0, 2.0, 3.0, 4.0)
    _say("student_t_1m budget sweep (about 40 solves; one line each)")
    ecasq.ecasq_timing_enable(True, verbose=True)
    try:
        out = ecasq.ecasq_solve_budgets(xd, 64, budgets)
    finally:
        ecasq.ecasq_timing_enable(False)
    traj = ecasq.ecasq_inspect_points()
    res = ecasq.ecasq_inspect_results()
    assert len(res) == len(budgets)
    assert len(traj) == sum(o[2]["dp_solves"] for o in out)
    _say("oracle prepare", x.size)
    H = pipeline.prepare(x)
    cache = pipeline.LambdaCache()
    rng = np.random.default_rng(41)
    at = 0
    for k, b in enumerate(budgets):
        cb, rk, info = out[k]
        n = info["dp_solves"]
        _say("budget", b, "solves", n, "t", info["t"])
        assert info["status"] == 0 and info["p"] == H.p
        np.testing.assert_array_equal(rk.cpu().numpy()[: info["t"]], res[k]["post"])
        _check_search(H, 64, b, traj[at: at + n], info, res[k], cache=cache)
        at += n
        _check_dp(xd, H, 64, res[k]["lam_B"], res[k]["pre"], rng, 3)
        _check_refine_and_metrics(H, b, info, res[k])
        _check_rounding(x, xd, cb, info["t"])
