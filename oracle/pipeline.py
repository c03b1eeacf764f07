"""Oracle pipeline: histogram, exact prefix sums, search, recovery, refinement,
final stochastic rounding.

TEST INFRASTRUCTURE ONLY.  Plain Python/numpy for the O(d) steps, the C oracle
(native.py) for the O(s p^2) dynamic programs.

Paper references (arXiv 2608.18147):
  weighted histogram of the sorted input       Sec. 2 (sorting, duplicates)
  prefix sums N, S, S2 and closed forms        App. D
  budget search on lambda                      Sec. 3 and Sec. 5 (lambda tuning)
  Hirschberg recovery                          Sec. 5 / Sec. 4.2
  three-colour refinement                      Sec. 6
  SQ rounding                                  Sec. 2
"""
import math
from dataclasses import dataclass, field

import numpy as np

from . import native
from .philox import philox4x32_10

F32_LSB_EXP = 149  # every float32 is an integer multiple of 2^-149


def histogram(x):
    """Sorted distinct values and their counts.  -0 is folded into +0.

    x: any float array whose values are exact in float32 (f32/f16/bf16)."""
    xf = np.asarray(x).astype(np.float64).ravel()
    if not np.all(np.isfinite(xf)):
        raise ValueError("non-finite input")
    xf = xf + 0.0
    v, c = np.unique(xf, return_counts=True)
    return v, c.astype(np.int64)


def exact_prefix(v, c):
    """Inclusive prefix sums N, S = sum c v, S2 = sum c v^2, each the correctly
    rounded fp64 value of the exact sum (App. D prefix quantities).

    Exactness: every value is K * 2^-149 with integer K, so the sums are exact
    Python integers; int -> float conversion rounds to nearest even and the
    power-of-two rescale is exact."""
    p = len(v)
    N = np.empty(p)
    S = np.empty(p)
    S2 = np.empty(p)
    scale = 1 << F32_LSB_EXP
    acc_n = acc_s = acc_s2 = 0
    for k in range(p):
        num, den = float(v[k]).as_integer_ratio()
        K = num * (scale // den)
        ck = int(c[k])
        acc_n += ck
        acc_s += ck * K
        acc_s2 += ck * K * K
        N[k] = float(acc_n)
        S[k] = math.ldexp(float(acc_s), -F32_LSB_EXP)
        S2[k] = math.ldexp(float(acc_s2), -2 * F32_LSB_EXP)
    return N, S, S2


@dataclass
class Hist:
    v: np.ndarray
    c: np.ndarray
    N: np.ndarray
    S: np.ndarray
    S2: np.ndarray
    d: int

    @property
    def p(self):
        return len(self.v)

    @property
    def s2tot(self):
        return float(self.S2[-1])

    def args(self):
        return (native.dptr(self.v), native.dptr(self.N), native.dptr(self.S),
                native.dptr(self.S2), self.p, self.d)


def uniform_alphabet(v, m):
    """m permissible values evenly spaced over [min X, max X] (App. D with
    P != X; App. F.7 'uniform min-max grid'): p_0 = min X, p_{m-1} = max X,
    p_k = min X + k * ((max X - min X) / (m - 1)) in between, each operation
    rounded to nearest; values that round onto their predecessor are dropped."""
    lo, hi = float(v[0]), float(v[-1])
    if len(v) == 1:
        return np.array([lo])
    step = (hi - lo) / float(m - 1)
    P = [lo]
    for k in range(1, m - 1):
        q = lo + float(k) * step
        if q > P[-1] and q < hi:
            P.append(q)
    P.append(hi)
    return np.array(P)


def quantile_alphabet(v, c, m):
    """m permissible values at the ranks floor(k (d - 1) / (m - 1)) of the
    sorted input (a quantile grid drawn from X, App. F.7), repeats dropped; the
    first and last are min X and max X."""
    d = int(np.sum(c))
    cum = np.cumsum(c)
    P = []
    for k in range(m):
        r = (k * (d - 1)) // (m - 1) if m > 1 else 0
        i = int(np.searchsorted(cum, r, side="right"))  # first i with cum[i] > r
        if not P or v[i] > P[-1]:
            P.append(float(v[i]))
    return np.array(P)


def on_alphabet(v, c, N, S, S2, P):
    """Prefix quantities of X at the permissible values: N(p), S(p), S2(p) are
    the count, sum and sum of squares of the entries <= p (App. D), taken from
    the exact prefix sums at the last input value <= p."""
    idx = np.searchsorted(v, P, side="right") - 1
    Nn = np.empty(len(P)); Sn = np.empty(len(P)); S2n = np.empty(len(P))
    cn = np.empty(len(P), dtype=np.int64)
    prev = 0
    for k, i in enumerate(idx):
        Nn[k], Sn[k], S2n[k] = N[i], S[i], S2[i]
        cn[k] = int(N[i]) - prev
        prev = int(N[i])
    return cn, Nn, Sn, S2n


def prepare(x, alphabet=None):
    """Histogram with exact prefix sums over the permissible values: the
    distinct input values (P = X), or a grid ('uniform', m) / ('quantile', m)."""
    v, c = histogram(x)
    N, S, S2 = exact_prefix(v, c)
    d = int(np.asarray(x).size)
    if alphabet is not None:
        kind, m = alphabet
        P = uniform_alphabet(v, m) if kind == "uniform" else quantile_alphabet(v, c, m)
        c, N, S, S2 = on_alphabet(v, c, N, S, S2, P)
        v = P
    return Hist(np.ascontiguousarray(v), c, N, S, S2, d)


def interval(H, a, b):
    """(C, U, D, P) of (v_a, v_b] in the canonical arithmetic."""
    out = np.zeros(4)
    native.lib().orc_interval(*H.args(), a, b, native.dptr(out))
    return tuple(out)


def dp_forward(H, s, lamp, exact_s=False, backpointers=False, dump=False):
    """One approximate-DP solve at lambda' (MSE units).  Returns dict."""
    L = native.lib()
    out = np.zeros(5)
    bp = np.zeros((s + 1) * H.p, dtype=np.int32) if backpointers else None
    fd = np.full((s + 1) * H.p, np.inf) if dump else None
    lastF = np.full(s + 1, np.inf)
    L.orc_dp_forward(*H.args(), s, int(exact_s), lamp, native.dptr(out),
                     native.iptr(bp) if bp is not None else None,
                     native.dptr(fd) if fd is not None else None, native.dptr(lastF))
    r = dict(J=out[0], mse=out[1], phi=out[2], t=int(out[3]), cells=int(out[4]), lastF=lastF)
    if bp is not None:
        r["bp"] = bp.reshape(s + 1, H.p)
        chain = np.zeros(r["t"], dtype=np.int32)
        L.orc_traceback(native.iptr(bp), H.p, r["t"], native.iptr(chain))
        r["chain_bp"] = chain
    if fd is not None:
        r["F"] = fd.reshape(s + 1, H.p)
    return r


def dp_columns(H, layer, lamp, Fprev=None, Mprev=None, Pprev=None, cols=()):
    """Columns `cols` of DP layer `layer` recomputed from the previous layer
    (eq. apx_base for layer 2, eq. apx_rec otherwise): (F, k*, M, Ph) arrays."""
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    n = len(cols)
    F = np.zeros(n)
    K = np.zeros(n, dtype=np.int32)
    M = np.zeros(n)
    Ph = np.zeros(n)
    if layer == 2:
        Fprev = Mprev = Pprev = np.zeros(1)
    args = [np.ascontiguousarray(a, dtype=np.float64) for a in (Fprev, Mprev, Pprev)]
    native.lib().orc_dp_columns(*H.args(), layer, lamp, *(native.dptr(a) for a in args), n,
                                cols.ctypes.data_as(native.ctypes.POINTER(native.ctypes.c_int64)),
                                native.dptr(F), native.iptr(K), native.dptr(M), native.dptr(Ph))
    return F, K, M, Ph


def hirschberg(H, t, lamp):
    chain = np.zeros(t, dtype=np.int32)
    import ctypes
    cells = ctypes.c_int64(0)
    native.lib().orc_hirschberg(*H.args(), t, lamp, native.iptr(chain), ctypes.byref(cells))
    return chain, int(cells.value)


def chain_metrics(H, chain, lam):
    out = np.zeros(6)
    chain = np.ascontiguousarray(chain, dtype=np.int32)
    native.lib().orc_chain_metrics(*H.args(), len(chain), native.iptr(chain), lam,
                                   native.dptr(out))
    return dict(mse=out[0], vnmse=out[1], entropy=out[2], entropy_surrogate=out[3],
                objective=out[4], rate_total=out[5])


def refine(H, chain, lamp, b=math.inf, budget=False, rounds=5, exhaustive=False):
    import ctypes
    u = np.ascontiguousarray(chain, dtype=np.int32).copy()
    moves = ctypes.c_int32(0)
    n = native.lib().orc_refine(*H.args(), len(u), native.iptr(u), lamp, b, int(budget), rounds,
                                int(exhaustive), ctypes.byref(moves))
    return u, int(n), int(moves.value)


def refine_local(H, chain, r, m, lamp):
    """Local objective of mover r placed at unique index m (Sec. 6)."""
    u = np.ascontiguousarray(chain, dtype=np.int32)
    return native.lib().orc_refine_local(*H.args(), len(u), native.iptr(u), r, m, lamp)


def refine_search(H, chain, r, lamp, exhaustive=False):
    """The position mover r's search finds (before the strict-improvement test)."""
    u = np.ascontiguousarray(chain, dtype=np.int32)
    return int(native.lib().orc_refine_search(*H.args(), len(u), native.iptr(u), r, lamp,
                                              int(exhaustive)))


def refine_substep(H, chain, colour, lamp, exhaustive=False):
    """One colour substep without the budget guard: (new chain, movers moved)."""
    u = np.ascontiguousarray(chain, dtype=np.int32)
    nu = np.zeros_like(u)
    n = native.lib().orc_refine_substep(*H.args(), len(u), native.iptr(u), colour, lamp,
                                        int(exhaustive), native.iptr(nu))
    return nu, int(n)


class ReplayMismatch(AssertionError):
    """The search's queries differ from a recorded trajectory."""


class LambdaCache:
    """Points (lambda, H(I,B), vNMSE, t) solved on one input, shared by the
    searches for several budgets."""

    def __init__(self, cap=4096):
        self.pts = np.zeros(4 * cap)
        self.n = np.zeros(1, dtype=np.int32)
        self.cap = cap


def search(H, s, b, exact_s=False, max_passes=32, width=8, cache=None, aim=True, dp="approx",
           refine_rounds=5, exhaustive=False, replay=None):
    """Budget search on lambda in passes of `width` (8 or 1) multipliers; with
    a LambdaCache, points solved by earlier searches are reused.  aim: width-1
    queries aimed at H = b before the certifying chord query (the batched row
    solver runs the plain chord search: aim=False).  dp: 'approx' searches the
    approximate DP's (H(I,B), vNMSE) points, 'optimal' the optimal DP's
    (H(Xhat), vNMSE) points (width 1), 'refined' the points (H(Xhat), vNMSE)
    of the approximate DP's codebooks after refinement at their multiplier
    (width 1; the answer is the feasible point of lowest vNMSE found).  Also
    returns A, the infeasible point the final chord starts from (lamA etc.
    NaN when there is none).

    replay: a recorded trajectory (rows lambda, H, vNMSE, t) whose points
    stand in for the solves, in order; raises ReplayMismatch when the search
    asks for a multiplier other than the next recorded one, or for more
    solves than were recorded."""
    out = np.zeros(13)
    cap = 1024
    traj = np.zeros(4 * cap)
    if cache is not None:
        cptr, nptr, ccap = native.dptr(cache.pts), native.iptr(cache.n), cache.cap
    else:
        cptr, nptr, ccap = None, None, 0
    kind = {"approx": 0, "optimal": 1, "refined": 2}[dp]
    rp, nrp = None, 0
    if replay is not None:
        rep = np.ascontiguousarray(np.asarray(replay, dtype=np.float64).reshape(-1, 4))
        rp, nrp = native.dptr(rep), len(rep)
    rc = native.lib().orc_search(*H.args(), s, b, int(exact_s), max_passes, width, int(aim),
                                 kind, refine_rounds, int(exhaustive), cptr, nptr, ccap,
                                 native.dptr(traj), cap, rp, nrp, native.dptr(out))
    if rc == -2:
        raise ReplayMismatch(f"query {int(out[4])} differs from the recorded trajectory")
    if rc != 0:
        raise ValueError("search width must be 1 or 8")
    n = int(out[4])
    return dict(lam=out[0], H=out[1], M=out[2], t=int(out[3]), solves=n, cells=int(out[5]),
                status=int(out[6]), lam_final=out[7], passes=int(out[8]),
                traj=traj[: 4 * min(n, cap)].reshape(-1, 4), lamA=out[9], HA=out[10],
                MA=out[11], tA=-1 if math.isnan(out[12]) else int(out[12]))


@dataclass
class Result:
    codebook: np.ndarray
    rank: np.ndarray
    t: int
    p: int
    lam: float
    mse: float
    vnmse: float
    entropy: float
    entropy_surrogate: float
    objective: float
    rate_total: float
    dp_solves: int
    refine_rounds: int
    cells: int
    status: int
    traj: np.ndarray = field(default=None)
    passes: int = 0
    dp_value: float = None   # the optimal DP's own value (lambda' units)


def _finish(H, chain, lam, solves, rounds, cells, status, traj=None):
    m = chain_metrics(H, chain, lam)
    return Result(codebook=H.v[chain].copy(), rank=np.asarray(chain, dtype=np.int32), t=len(chain),
                  p=H.p, lam=lam, mse=m["mse"], vnmse=m["vnmse"], entropy=m["entropy"],
                  entropy_surrogate=m["entropy_surrogate"], objective=m["objective"],
                  rate_total=m["rate_total"], dp_solves=solves, refine_rounds=rounds,
                  cells=cells, status=status, traj=traj)


def _recover(H, t, lam, recovery="hirschberg", s=None, exact_s=False, dp="approx",
             refine_rounds=5, exhaustive=False):
    """Codebook (unique indices) with t values at lambda (vNMSE units): by
    Hirschberg (Sec. 5), or by a traceback through the argmins of a solve at
    the same multiplier ('backpointers'); the optimal DP's own traceback for
    dp='optimal'."""
    if H.p == 1:
        return np.zeros(1, dtype=np.int32), 0
    if t == 2 or not math.isfinite(lam):
        return np.array([0, H.p - 1], dtype=np.int32), 0
    if dp == "optimal":
        r = opt_dp(H, s, lam * H.s2tot, exact_s)
        assert r["t"] == t
        return r["chain"], 0
    if dp == "refined":
        r = dp_forward(H, s, lam * H.s2tot, exact_s, backpointers=True)
        assert r["t"] == t
        chain = r["chain_bp"]
        if refine_rounds > 0 and len(chain) >= 3:
            chain, _, _ = refine(H, chain, lam * H.s2tot, math.inf, False, refine_rounds,
                                 exhaustive)
        return chain, 0
    if recovery == "backpointers":
        r = dp_forward(H, s, lam * H.s2tot, exact_s, backpointers=True)
        assert r["t"] == t
        return r["chain_bp"], 0
    return hirschberg(H, t, lam * H.s2tot)


def solve(x, s, b, refine_rounds=5, exhaustive=False, exact_s=False, max_passes=32,
          recovery="hirschberg", width=8, aim=True, alphabet=None, dp="approx"):
    """Budget mode: the lowest-MSE supported solution with H(I,B) <= b
    (recovered at the multiplier it was found at), then refinement at the
    final chord slope with the budget guard on H(Xhat).  dp='optimal': the
    lowest-MSE supported solution of the optimal DP with H(Xhat) <= b (width
    1, no refinement)."""
    H = prepare(x, alphabet)
    rr = refine_rounds
    if dp != "approx":
        width, refine_rounds = 1, 0
    sr = search(H, s, b, exact_s, max_passes, width, aim=aim, dp=dp, refine_rounds=rr,
                exhaustive=exhaustive)
    chain, hcells = _recover(H, sr["t"], sr["lam"], recovery, s, exact_s, dp, rr, exhaustive)
    lam = sr["lam_final"]
    rounds = 0
    if refine_rounds > 0 and math.isfinite(lam) and len(chain) >= 3:
        chain, rounds, _ = refine(H, chain, lam * H.s2tot, b, True, refine_rounds, exhaustive)
    r = _finish(H, chain, lam, sr["solves"], rounds, sr["cells"] + hcells, sr["status"],
                sr["traj"])
    r.passes = sr["passes"]
    return r


def solve_budgets(x, s, budgets, refine_rounds=5, exhaustive=False, exact_s=False,
                  max_passes=32, recovery="hirschberg", width=8, aim=True, alphabet=None,
                  dp="approx"):
    """Budget mode for several budgets on one input, in the given order, the
    searches sharing one LambdaCache.  Per budget as solve(); dp_solves and
    cells count the solves that budget's search ran."""
    H = prepare(x, alphabet)
    rr = refine_rounds
    if dp != "approx":
        width, refine_rounds = 1, 0
    cache = LambdaCache()
    res = []
    for b in budgets:
        sr = search(H, s, b, exact_s, max_passes, width, cache, aim, dp, rr, exhaustive)
        chain, hcells = _recover(H, sr["t"], sr["lam"], recovery, s, exact_s, dp, rr, exhaustive)
        lam = sr["lam_final"]
        rounds = 0
        if refine_rounds > 0 and math.isfinite(lam) and len(chain) >= 3:
            chain, rounds, _ = refine(H, chain, lam * H.s2tot, b, True, refine_rounds, exhaustive)
        r = _finish(H, chain, lam, sr["solves"], rounds, sr["cells"] + hcells, sr["status"],
                    sr["traj"])
        r.passes = sr["passes"]
        res.append(r)
    return res


def solve_lagrangian(x, s, lam, refine_rounds=0, exhaustive=False, exact_s=False,
                     recovery="hirschberg", alphabet=None):
    """Fixed-multiplier mode: min vNMSE + lambda H(I,B), then refinement on
    vNMSE + lambda H(Xhat) without a budget guard."""
    H = prepare(x, alphabet)
    if H.p == 1:
        return _finish(H, np.zeros(1, dtype=np.int32), lam, 0, 0, 0, 0)
    r = dp_forward(H, s, lam * H.s2tot, exact_s)
    chain, hcells = _recover(H, r["t"], lam, recovery, s, exact_s)
    rounds = 0
    if refine_rounds > 0 and len(chain) >= 3:
        chain, rounds, _ = refine(H, chain, lam * H.s2tot, math.inf, False, refine_rounds,
                                  exhaustive)
    return _finish(H, chain, lam, 1, rounds, r["cells"] + hcells, 0)


def opt_dp(H, s, lamp, exact_s=False, dump=False):
    """Optimal lambda-ECASQ over states (i, l, j) (Sec. 4), every admissible
    predecessor scanned.  Returns dict(J = MSE + lambda' H(Xhat) of the optimum,
    t, chain, cells[, K, F per layer])."""
    L = native.lib()
    out = np.zeros(3)
    chain = np.zeros(max(s, 1), dtype=np.int32)
    imax = min(s, H.p)
    K = np.zeros((imax + 1) * H.p * H.p, dtype=np.int32) if dump else None
    F = np.zeros((imax + 1) * H.p * H.p) if dump else None
    rc = L.orc_opt_dp(*H.args(), s, int(exact_s), lamp, native.iptr(chain), native.dptr(out),
                      native.iptr(K) if dump else None, native.dptr(F) if dump else None)
    assert rc == 0
    t = int(out[1])
    r = dict(J=out[0], t=t, chain=chain[:t].copy(), cells=int(out[2]))
    if dump:
        r["K"] = K.reshape(imax + 1, H.p, H.p)
        r["F"] = F.reshape(imax + 1, H.p, H.p)
    return r


def solve_optimal(x, s, lam, exact_s=False, alphabet=None):
    """Optimal lambda-ECASQ at a fixed multiplier (vNMSE units): the codebook
    minimising vNMSE + lambda H(Xhat) with at most s values (exactly s with
    exact_s) drawn from the permissible values (Sec. 4; App. D)."""
    H = prepare(x, alphabet)
    r = opt_dp(H, s, lam * H.s2tot, exact_s)
    res = _finish(H, r["chain"], lam, 1, 0, r["cells"], 0)
    res.dp_value = r["J"]
    return res


def solve_timeshare(x, s, b, exact_s=False, max_passes=32, recovery="backpointers", width=1,
                    aim=True, alphabet=None, dp="approx"):
    """Two-way time-sharing (Sec. 7, App. E): the search's final pair, B (the
    best supported point with H <= b, 'minus') and A (the supported point the
    final chord starts from, H > b, 'plus'), and the share alpha of entries
    quantized with A such that alpha H_A + (1 - alpha) H_B = b, H being the
    search's entropy (H(I,B) for the approximate DP, H(Xhat) for the optimal
    DP).  Without such a pair (lambda = 0 feasible, an infeasible budget,
    p <= 2) alpha = 0 and both quantizers are B.  No refinement.
    Returns dict(minus, plus (Results), alpha, H_mix, M_mix, status, solves,
    cells)."""
    H = prepare(x, alphabet)
    if dp == "optimal":
        width = 1
    sr = search(H, s, b, exact_s, max_passes, width, aim=aim, dp=dp)
    cm, c1 = _recover(H, sr["t"], sr["lam"], recovery, s, exact_s, dp)
    alpha = 0.0
    cp, c2 = cm, 0
    lam_p = sr["lam"]
    if sr["status"] == 0 and sr["tA"] > 0 and H.p > 2:
        alpha = (b - sr["H"]) / (sr["HA"] - sr["H"])
        cp, c2 = _recover(H, sr["tA"], sr["lamA"], recovery, s, exact_s, dp)
        lam_p = sr["lamA"]
    cells = sr["cells"] + c1 + c2
    minus = _finish(H, cm, sr["lam"], sr["solves"], 0, cells, sr["status"])
    plus = _finish(H, cp, lam_p, sr["solves"], 0, cells, sr["status"])
    minus.passes = plus.passes = sr["passes"]
    HA = sr["HA"] if alpha > 0.0 else sr["H"]
    MA = sr["MA"] if alpha > 0.0 else sr["M"]
    return dict(minus=minus, plus=plus, alpha=alpha, H_mix=alpha * HA + (1.0 - alpha) * sr["H"],
                M_mix=alpha * MA + (1.0 - alpha) * sr["M"], status=sr["status"],
                solves=sr["solves"], cells=cells, HA=HA, HB=sr["H"], MA=MA, MB=sr["M"])


def uniforms(n, seed, stream=0):
    """u_i in [0,1) for i < n: one Philox4x32-10 call per pair of entries.
    Entries 2j and 2j+1 share the counter (j_lo, j_hi, stream, 0) with key
    (seed_lo, seed_hi); entry 2j takes 53 bits of words 0 and 1, entry 2j+1
    of words 2 and 3 (bits = (w_hi << 32 | w_lo) >> 11, u = bits 2^-53).
    Stream 0 drives the rounding, stream 1 the time-sharing partition.  (Sec.
    2 asks for an independent uniform per entry and fixes no generator; the
    four words of one call are independent outputs of it.)"""
    m = (n + 1) // 2
    j = np.arange(m, dtype=np.uint64)
    c0 = (j & np.uint64(0xFFFFFFFF)).astype(np.uint64)
    c1 = (j >> np.uint64(32)).astype(np.uint64)
    z = np.zeros(m, dtype=np.uint64)
    c2 = np.full(m, stream, dtype=np.uint64)
    k0 = np.full(m, seed & 0xFFFFFFFF, dtype=np.uint64)
    k1 = np.full(m, (seed >> 32) & 0xFFFFFFFF, dtype=np.uint64)
    w0, w1, w2, w3 = philox4x32_10(c0, c1, c2, z, k0, k1)
    bits = np.empty(2 * m, dtype=np.uint64)
    bits[0::2] = ((w1 << np.uint64(32)) | w0) >> np.uint64(11)
    bits[1::2] = ((w3 << np.uint64(32)) | w2) >> np.uint64(11)
    return bits[:n].astype(np.float64) * 2.0 ** -53


def quantize(x, codebook, seed):
    """Unbiased SQ of every entry in its original order (Sec. 2): bracket
    q_r < x <= q_{r+1} (x <= q_0 maps to r = 0), round up iff u < (x-q_r)/(q_{r+1}-q_r).
    Returns (symbols uint8, histogram int64, plug-in entropy of the symbols)."""
    xf = np.asarray(x).astype(np.float64).ravel() + 0.0
    q = np.asarray(codebook, dtype=np.float64)
    t = len(q)
    n = len(xf)
    if t == 1:
        sym = np.zeros(n, dtype=np.uint8)
    else:
        r = np.clip(np.searchsorted(q, xf, side="left") - 1, 0, t - 2)
        pu = (xf - q[r]) / (q[r + 1] - q[r])
        u = uniforms(n, seed)
        sym = (r + (u < pu)).astype(np.uint8)
    hist = np.bincount(sym, minlength=t).astype(np.int64)
    ent = 0.0
    for nq in hist:
        if nq > 0:
            y = nq / n
            ent -= y * math.log2(y)
    return sym, hist, ent


def _plugin_entropy(sym, t):
    n = len(sym)
    hist = np.bincount(sym, minlength=t).astype(np.int64)
    ent = 0.0
    for nq in hist:
        if nq > 0:
            y = nq / n
            ent -= y * math.log2(y)
    return hist, ent


def quantize_timeshare(x, cb_minus, cb_plus, alpha, seed):
    """Time-shared final rounding (Sec. 7): entry i uses cb_plus iff its
    partition uniform (Philox stream 1) is below alpha, else cb_minus, and is
    then rounded as quantize() rounds it (stream 0), its symbol indexing its
    own codebook.  The two parts are entropy-coded separately: the entropy is
    (n_minus H_minus + n_plus H_plus) / d with each part's plug-in entropy.
    Returns (symbols, part (1 = plus), hist (minus counts then plus counts),
    entropy)."""
    xf = np.asarray(x).astype(np.float64).ravel() + 0.0
    n = len(xf)
    part = (uniforms(n, seed, 1) < alpha).astype(np.uint8)
    sym = np.zeros(n, dtype=np.uint8)
    u = uniforms(n, seed, 0)
    ent = 0.0
    hists = []
    for which, q in ((0, cb_minus), (1, cb_plus)):
        q = np.asarray(q, dtype=np.float64)
        t = len(q)
        sel = part == which
        if t == 1:
            sy = np.zeros(int(sel.sum()), dtype=np.uint8)
        else:
            xs = xf[sel]
            r = np.clip(np.searchsorted(q, xs, side="left") - 1, 0, t - 2)
            pu = (xs - q[r]) / (q[r + 1] - q[r])
            sy = (r + (u[sel] < pu)).astype(np.uint8)
        sym[sel] = sy
        hist, e = _plugin_entropy(sy, t) if len(sy) else (np.zeros(t, dtype=np.int64), 0.0)
        hists.append(hist)
        ent += len(sy) * e
    return sym, part, np.concatenate(hists), ent / n
