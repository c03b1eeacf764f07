"""GPU parity of the optimal lambda-ECASQ DP (Sec. 4) against the CPU oracle,
through the C ABI (ecasq_solve_optimal, ecasq_opt_trace).

The scan over every predecessor evaluates the oracle's operations in the same
order, so its layers, argmins, codebook and DP value must agree bit for bit.
The monotone-bracket scan (the SMAWK acceleration) reaches the same optimum;
where rounding could let it pick another codebook of equal cost, the test
checks the value to rounding and the codebook's validity instead.
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
    return abs(a - b) <= rel * max(abs(a), abs(b), 1e-300)


def _rounded(d, seed):
    return (np.round(inputs.normal(d, seed) * 6.0) / 6.0).astype(np.float32)


CASES = [
    # name, input, s, lambda, options (exact_s, alphabet)
    ("normal_300", lambda: inputs.normal(300, 3), 8, 0.05, {}),
    ("lognormal_700", lambda: inputs.lognormal_signed(700, 4), 12, 0.02, {}),
    ("dups_p50", lambda: _rounded(5000, 5), 16, 0.1, {}),
    ("s_ge_p", lambda: inputs.normal(40, 6), 64, 0.01, {}),
    ("lambda0_asq", lambda: inputs.normal(400, 7), 10, 0.0, {}),
    ("lambda_large", lambda: inputs.normal(400, 8), 10, 50.0, {}),
    ("exact_s", lambda: inputs.lognormal_signed(500, 9), 9, 0.1, dict(exact_s=1)),
    ("s2", lambda: inputs.normal(300, 10), 2, 0.1, {}),
    ("uniform_grid_400", lambda: inputs.lognormal_signed(2048, 11), 12, 0.05,
     dict(alphabet=1, alphabet_size=400)),
    ("quantile_grid_300", lambda: inputs.student_t(2048, 12), 10, 0.05,
     dict(alphabet=2, alphabet_size=300)),
]


def _oracle(x, s, lam, o):
    alpha = None
    if o.get("alphabet"):
        alpha = ("uniform" if o["alphabet"] == 1 else "quantile", o["alphabet_size"])
    return pipeline.solve_optimal(x, s, lam, exact_s=bool(o.get("exact_s", 0)), alphabet=alpha)


def _compare(g, r):
    cb, rk, info = g
    assert info["t"] == r.t and info["p"] == r.p
    np.testing.assert_array_equal(rk.cpu().numpy(), r.rank)
    np.testing.assert_array_equal(cb.cpu().numpy(), r.codebook)
    for k in ("mse", "vnmse", "entropy", "entropy_surrogate", "objective", "rate_total"):
        assert _close(info[k], getattr(r, k)), (k, info[k], getattr(r, k))
    assert info["dp_solves"] == 1 and info["refine_rounds_run"] == 0
    assert info["cells"] == r.cells
    assert info["status"] == 0


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_optimal_full_scan_bit_exact(case):
    name, mk, s, lam, o = case
    x = mk()
    _say("optimal full", name, x.size, s, lam, o)
    r = _oracle(x, s, lam, o)
    opts = ecasq.ecasq_default_options(optimal_scan=1, **o)
    _compare(ecasq.ecasq_solve_optimal(_dev(x), s, lam, options=opts), r)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_optimal_monotone_brackets(case):
    """The bracketed scan reaches the oracle's optimum: the same codebook, or
    (where rounding reorders two near-equal candidates) one whose objective
    equals the optimum to rounding."""
    name, mk, s, lam, o = case
    x = mk()
    _say("optimal monotone", name, x.size, s, lam, o)
    r = _oracle(x, s, lam, o)
    opts = ecasq.ecasq_default_options(**o)
    cb, rk, info = ecasq.ecasq_solve_optimal(_dev(x), s, lam, options=opts)
    if np.array_equal(rk.cpu().numpy(), r.rank):
        _compare((cb, rk, info), r)
    else:
        _say("  different codebook of equal cost", name)
        assert abs(info["objective"] - r.objective) <= 1e-12 * max(1.0, r.objective)
        u = rk.cpu().numpy()
        assert u[0] == 0 and u[-1] == r.p - 1 and np.all(np.diff(u) > 0) and len(u) <= s


@pytest.mark.parametrize("name,mk,s,lam", [
    ("lognormal_300", lambda: inputs.lognormal_signed(300, 21), 7, 0.03),
    ("normal_520", lambda: inputs.normal(520, 22), 6, 0.2),   # j tiles of 256, ragged
])
def test_optimal_layers_bit_exact(name, mk, s, lam):
    """Every layer's values dp(i, l, j) and argmins of the full scan equal the
    oracle's at every valid (l, j); the DP value too; the monotone scan gives
    the same layers up to rounding-level differences."""
    x = mk()
    H = pipeline.prepare(x)
    p = H.p
    _say("optimal layers", name, p, s, lam)
    lamp = lam * H.s2tot
    ro = pipeline.opt_dp(H, s, lamp, dump=True)
    opts = ecasq.ecasq_default_options(optimal_scan=1)
    F, K, chain, J, cells = ecasq.ecasq_opt_trace(_dev(x), s, lam, p, options=opts)
    F = F.cpu().numpy()
    K = K.cpu().numpy()
    imax = min(s, p)
    for i in range(2, imax + 1):
        ls = [0] if i == 2 else list(range(i - 2, p - 1))
        for l in ls:
            js = np.arange(l + 1, p)
            np.testing.assert_array_equal(F[i, js, l], ro["F"][i, l, js], err_msg=f"F {i} {l}")
            if i >= 3:
                np.testing.assert_array_equal(K[i, l, js], ro["K"][i, l, js],
                                              err_msg=f"K {i} {l}")
    assert J == ro["J"] and chain == list(ro["chain"]) and cells == ro["cells"]
    opts = ecasq.ecasq_default_options(optimal_scan=0)
    Fm, Km, chm, Jm, _ = ecasq.ecasq_opt_trace(_dev(x), s, lam, p, options=opts)
    assert abs(Jm - J) <= 1e-12 * abs(J)
    same = sum(int(np.array_equal(Km.cpu().numpy()[i, l, l + 1:], K[i, l, l + 1:]))
               for i in range(3, imax + 1) for l in range(i - 2, p - 1))
    total = sum(1 for i in range(3, imax + 1) for l in range(i - 2, p - 1))
    _say("  monotone rows identical", same, "of", total)
    assert same >= total - 3


def test_optimal_degenerate_inputs_and_errors():
    xc = np.full(300, -1.5, dtype=np.float32)
    cb, rk, info = ecasq.ecasq_solve_optimal(_dev(xc), 8, 0.1)
    assert info["t"] == 1 and cb.cpu().numpy().tolist() == [-1.5] and info["mse"] == 0.0
    x2 = np.array([0.5, 2.0, 0.5, 2.0, 2.0], dtype=np.float32)
    cb, rk, info = ecasq.ecasq_solve_optimal(_dev(x2), 8, 0.1)
    r = pipeline.solve_optimal(x2, 8, 0.1)
    _compare((cb, rk, info), r)
    xb = torch.from_numpy(inputs.normal(3000, 13)).to(torch.bfloat16)
    _say("optimal bf16")
    cb, rk, info = ecasq.ecasq_solve_optimal(xb.to("cuda"), 16, 0.1,
                                             options=ecasq.ecasq_default_options(optimal_scan=1))
    _compare((cb, rk, info), pipeline.solve_optimal(xb.to(torch.float32).numpy(), 16, 0.1))
    x = inputs.normal(100, 14)
    for bad in (dict(s=1, lam=0.1), dict(s=8, lam=-1.0), dict(s=8, lam=float("nan"))):
        with pytest.raises(ecasq.EcasqError):
            ecasq.ecasq_solve_optimal(_dev(x), bad["s"], bad["lam"])
    with pytest.raises(ecasq.EcasqError):
        ecasq.ecasq_solve_optimal(_dev(x), 8, 0.1,
                                  options=ecasq.ecasq_default_options(optimal_scan=2))


def test_optimal_full_size_bf16_weights():
    """The 2^18-entry weight-like vector in bf16 (p about 4000 permissible
    values), s = 64, lambda = 0.1 (the paper's runtime setting): the
    bracketed and full scans reach the same optimum; the optimum is at least
    as good as the approximate DP's codebook on the true objective, and no
    better than the approximate DP's surrogate optimum minus lambda (from
    H(Xhat) <= H(I,B) <= H(Xhat) + 1)."""
    x = inputs.make("weights_256k", seed=0)
    xb = torch.from_numpy(x).to(torch.bfloat16).to("cuda")
    s, lam = 64, 0.1
    _say("optimal full size bf16", xb.numel())
    gm = ecasq.ecasq_solve_optimal(xb, s, lam)
    gf = ecasq.ecasq_solve_optimal(xb, s, lam, options=ecasq.ecasq_default_options(optimal_scan=1))
    im, iff = gm[2], gf[2]
    _say("  p", im["p"], "t", im["t"], iff["t"], "objective", im["objective"], iff["objective"])
    assert abs(im["objective"] - iff["objective"]) <= 1e-12 * iff["objective"]
    assert im["p"] > 3000
    ga = ecasq.ecasq_solve_lagrangian(xb, s, lam,
                                      options=ecasq.ecasq_default_options(refine_rounds=0))
    ia = ga[2]
    assert iff["objective"] <= ia["objective"] * (1 + 1e-12)
    j_sur = ia["vnmse"] + lam * ia["entropy_surrogate"]
    assert j_sur <= iff["objective"] + lam + 1e-12
