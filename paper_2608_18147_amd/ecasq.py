"""Python binding of libecasq (include/ecasq.h): argument marshalling only.

Every step of the computation runs in the library's HIP kernels; PyTorch
provides device memory and the current stream.  The functions carry the C
names.  If libecasq.so is missing or cannot be loaded, the first call raises:
there is no fallback.
"""
import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libecasq.so")

ECASQ_OK = 0
ECASQ_EINVAL = -1
ECASQ_ENONFINITE = -2
ECASQ_EINFEASIBLE = -3
ECASQ_ENOMEM = -4
ECASQ_EHIP = -5
ECASQ_EWORKSPACE = -6

_DTYPES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}


class ecasq_options(ctypes.Structure):
    _fields_ = [
        ("refine_rounds", ctypes.c_int32),
        ("refine_exhaustive", ctypes.c_int32),
        ("exact_s", ctypes.c_int32),
        ("max_search_passes", ctypes.c_int32),
        ("recovery", ctypes.c_int32),
        ("search_width", ctypes.c_int32),
        ("dp_schedule", ctypes.c_int32),
        ("alphabet", ctypes.c_int32),
        ("alphabet_size", ctypes.c_int32),
        ("optimal_scan", ctypes.c_int32),
        ("dp_objective", ctypes.c_int32),
    ]


class ecasq_info(ctypes.Structure):
    _fields_ = [
        ("t", ctypes.c_int32),
        ("p", ctypes.c_int32),
        ("lambda_", ctypes.c_double),
        ("mse", ctypes.c_double),
        ("vnmse", ctypes.c_double),
        ("entropy", ctypes.c_double),
        ("entropy_surrogate", ctypes.c_double),
        ("objective", ctypes.c_double),
        ("rate_total", ctypes.c_double),
        ("dp_solves", ctypes.c_int32),
        ("refine_rounds_run", ctypes.c_int32),
        ("cells", ctypes.c_int64),
        ("status", ctypes.c_int32),
        ("search_passes", ctypes.c_int32),
    ]

    def as_dict(self):
        d = {k: getattr(self, k) for k, _ in self._fields_}
        d["lambda"] = d.pop("lambda_")
        return d


class EcasqError(RuntimeError):
    def __init__(self, status):
        self.status = status
        super().__init__(f"ecasq status {status}: {ecasq_status_string(status)}")


_lib = None
EXPORTS = (
    "ecasq_default_options", "ecasq_solve", "ecasq_solve_ex", "ecasq_solve_lagrangian",
    "ecasq_quantize", "ecasq_solve_batched", "ecasq_workspace_size", "ecasq_status_string",
    "ecasq_histogram", "ecasq_dp_trace", "ecasq_timing_enable", "ecasq_timing_read",
    "ecasq_solve_budgets", "ecasq_solve_optimal", "ecasq_opt_trace",
    "ecasq_solve_timeshare", "ecasq_quantize_timeshare", "ecasq_encode_bound", "ecasq_encode",
    "ecasq_decode", "ecasq_quantize_noalloc", "ecasq_inspect_enable", "ecasq_inspect_points",
    "ecasq_inspect_results",
)


def lib():
    """Load libecasq.so (built in place by build.py); raises if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with python -m "
                           "paper_2608_18147_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
    P = ctypes.POINTER
    L.ecasq_default_options.argtypes = [P(ecasq_options)]
    L.ecasq_default_options.restype = None
    L.ecasq_solve.argtypes = [vp, i32, i64, i32, dbl, vp, vp, vp, P(ecasq_info)]
    L.ecasq_solve_ex.argtypes = [vp, i32, i64, i32, dbl, P(ecasq_options), vp, vp, vp,
                                 P(ecasq_info), vp, ctypes.c_size_t]
    L.ecasq_solve_lagrangian.argtypes = [vp, i32, i64, i32, dbl, P(ecasq_options), vp, vp, vp,
                                         P(ecasq_info)]
    L.ecasq_solve_budgets.argtypes = [vp, i32, i64, i32, i32, P(dbl), P(ecasq_options), vp, vp,
                                      vp, P(ecasq_info)]
    L.ecasq_quantize.argtypes = [vp, i32, i64, vp, i32, ctypes.c_uint64, vp, vp, vp, vp]
    L.ecasq_quantize_noalloc.argtypes = [vp, i32, i64, vp, i32, ctypes.c_uint64, vp, vp, vp, vp]
    L.ecasq_solve_optimal.argtypes = [vp, i32, i64, i32, dbl, P(ecasq_options), vp, vp, vp,
                                      P(ecasq_info)]
    L.ecasq_opt_trace.argtypes = [vp, i32, i64, i32, dbl, P(ecasq_options), vp, i64, vp, vp,
                                  P(i32), P(dbl)]
    L.ecasq_solve_timeshare.argtypes = [vp, i32, i64, i32, dbl, P(ecasq_options), vp, vp, vp,
                                        P(dbl), P(ecasq_info)]
    L.ecasq_quantize_timeshare.argtypes = [vp, i32, i64, vp, i32, vp, i32, dbl,
                                           ctypes.c_uint64, vp, vp, vp, vp, vp]
    L.ecasq_encode_bound.argtypes = [i64, i32]
    L.ecasq_encode_bound.restype = ctypes.c_size_t
    L.ecasq_encode.argtypes = [vp, i64, i32, vp, vp, ctypes.c_size_t, P(i64)]
    L.ecasq_decode.argtypes = [vp, i64, i64, i32, vp, vp]
    L.ecasq_solve_batched.argtypes = [vp, i32, i64, i64, i32, dbl, P(ecasq_options), vp, vp,
                                      vp, vp]
    L.ecasq_workspace_size.argtypes = [i64, i32, i32]
    L.ecasq_workspace_size.restype = ctypes.c_size_t
    L.ecasq_status_string.argtypes = [i32]
    L.ecasq_status_string.restype = ctypes.c_char_p
    L.ecasq_histogram.argtypes = [vp, i32, i64, vp, vp, vp, vp, vp, P(i64)]
    L.ecasq_dp_trace.argtypes = [vp, i32, i64, i32, i32, P(dbl), i32, vp, vp, vp, vp, vp,
                                 P(dbl)]
    L.ecasq_inspect_enable.argtypes = [i32]
    L.ecasq_inspect_enable.restype = None
    L.ecasq_inspect_points.argtypes = [vp, i32]
    L.ecasq_inspect_points.restype = i32
    L.ecasq_inspect_results.argtypes = [vp, vp, i32]
    L.ecasq_inspect_results.restype = i32
    L.ecasq_timing_enable.argtypes = [i32]
    L.ecasq_timing_enable.restype = None
    L.ecasq_timing_read.argtypes = [i32, P(dbl), P(i64), P(i64), i32]
    L.ecasq_timing_read.restype = None
    for name in ("ecasq_solve", "ecasq_solve_ex", "ecasq_solve_lagrangian", "ecasq_quantize",
                 "ecasq_solve_batched", "ecasq_histogram", "ecasq_dp_trace",
                 "ecasq_solve_budgets", "ecasq_solve_optimal", "ecasq_opt_trace",
                 "ecasq_solve_timeshare", "ecasq_quantize_timeshare", "ecasq_encode",
                 "ecasq_decode", "ecasq_quantize_noalloc"):
        getattr(L, name).restype = i32
    _lib = L
    return L


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check_x(x):
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise TypeError("x must be a CUDA (HIP) tensor")
    if x.dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {x.dtype}")
    return x.contiguous().reshape(-1)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _raise(st, allow=(ECASQ_OK,)):
    if st not in allow:
        raise EcasqError(st)


def ecasq_default_options(**overrides):
    o = ecasq_options()
    lib().ecasq_default_options(ctypes.byref(o))
    for k, v in overrides.items():
        setattr(o, k, int(v))
    return o


def ecasq_status_string(status):
    return lib().ecasq_status_string(int(status)).decode()


def ecasq_workspace_size(d, s, flags=0):
    return int(lib().ecasq_workspace_size(int(d), int(s), int(flags)))


def ecasq_solve(x, s, bits_per_entry, options=None, stream=None, workspace=None):
    """Budget mode.  Returns (codebook fp64 [t], rank int32 [t], info dict)."""
    x = _check_x(x)
    cb = torch.empty(int(s), dtype=torch.float64, device=x.device)
    rk = torch.empty(int(s), dtype=torch.int32, device=x.device)
    info = ecasq_info()
    if options is None and workspace is None:
        st = lib().ecasq_solve(_ptr(x), _DTYPES[x.dtype], x.numel(), int(s),
                               float(bits_per_entry), _stream(stream), _ptr(cb), _ptr(rk),
                               ctypes.byref(info))
    else:
        o = options if options is not None else ecasq_default_options()
        ws = _ptr(workspace)
        nb = workspace.numel() * workspace.element_size() if workspace is not None else 0
        st = lib().ecasq_solve_ex(_ptr(x), _DTYPES[x.dtype], x.numel(), int(s),
                                  float(bits_per_entry), ctypes.byref(o), _stream(stream),
                                  _ptr(cb), _ptr(rk), ctypes.byref(info), ws, nb)
    _raise(st, (ECASQ_OK, ECASQ_EINFEASIBLE))
    t = info.t
    return cb[:t], rk[:t], info.as_dict()


ecasq_solve_ex = ecasq_solve


def ecasq_solve_budgets(x, s, budgets, options=None, stream=None):
    """Several budgets on one input with shared DP solves.  Returns a list of
    (codebook fp64 [t], rank int32 [t], info dict), one per budget."""
    x = _check_x(x)
    nb = len(budgets)
    cb = torch.empty((nb, int(s)), dtype=torch.float64, device=x.device)
    rk = torch.empty((nb, int(s)), dtype=torch.int32, device=x.device)
    infos = (ecasq_info * nb)()
    o = options if options is not None else ecasq_default_options()
    bs = (ctypes.c_double * nb)(*[float(b) for b in budgets])
    st = lib().ecasq_solve_budgets(_ptr(x), _DTYPES[x.dtype], x.numel(), int(s), nb, bs,
                                   ctypes.byref(o), _stream(stream), _ptr(cb), _ptr(rk), infos)
    _raise(st, (ECASQ_OK, ECASQ_EINFEASIBLE))
    return [(cb[k, :infos[k].t], rk[k, :infos[k].t], infos[k].as_dict()) for k in range(nb)]


def ecasq_solve_lagrangian(x, s, lam, options=None, stream=None):
    """Fixed multiplier (vNMSE units).  Returns (codebook, rank, info dict)."""
    x = _check_x(x)
    cb = torch.empty(int(s), dtype=torch.float64, device=x.device)
    rk = torch.empty(int(s), dtype=torch.int32, device=x.device)
    info = ecasq_info()
    o = options if options is not None else ecasq_default_options()
    st = lib().ecasq_solve_lagrangian(_ptr(x), _DTYPES[x.dtype], x.numel(), int(s), float(lam),
                                      ctypes.byref(o), _stream(stream), _ptr(cb), _ptr(rk),
                                      ctypes.byref(info))
    _raise(st)
    t = info.t
    return cb[:t], rk[:t], info.as_dict()


def ecasq_solve_optimal(x, s, lam, options=None, stream=None):
    """Optimal lambda-ECASQ (Sec. 4) at lam (vNMSE units).  Returns (codebook,
    rank, info dict)."""
    x = _check_x(x)
    cb = torch.empty(int(s), dtype=torch.float64, device=x.device)
    rk = torch.empty(int(s), dtype=torch.int32, device=x.device)
    info = ecasq_info()
    o = options if options is not None else ecasq_default_options()
    st = lib().ecasq_solve_optimal(_ptr(x), _DTYPES[x.dtype], x.numel(), int(s), float(lam),
                                   ctypes.byref(o), _stream(stream), _ptr(cb), _ptr(rk),
                                   ctypes.byref(info))
    _raise(st)
    t = info.t
    return cb[:t], rk[:t], info.as_dict()


def ecasq_opt_trace(x, s, lam, p, options=None, stream=None):
    """Every layer of the optimal DP for an input with p permissible values.
    Returns (F [imax+1, p, p] with F[i, j, l] = dp(i, l, j), K [imax+1, p, p]
    with K[i, l, j] the minimising k, chain list, DP value, cells); entries
    outside a layer's valid (l, j) are unspecified."""
    x = _check_x(x)
    imax = min(int(s), int(p))
    cap = (imax + 1) * p * p
    F = torch.empty(cap, dtype=torch.float64, device=x.device)
    K = torch.empty(cap, dtype=torch.int32, device=x.device)
    chain = (ctypes.c_int32 * int(s))()
    out = (ctypes.c_double * 4)()
    o = options if options is not None else ecasq_default_options()
    st = lib().ecasq_opt_trace(_ptr(x), _DTYPES[x.dtype], x.numel(), int(s), float(lam),
                               ctypes.byref(o), _stream(stream), cap, _ptr(F), _ptr(K), chain,
                               out)
    _raise(st)
    if int(out[2]) != p:
        raise ValueError(f"input has {int(out[2])} permissible values, not {p}")
    t = int(out[1])
    return (F.view(imax + 1, p, p), K.view(imax + 1, p, p), list(chain[:t]), out[0],
            int(out[3]))


def ecasq_solve_timeshare(x, s, bits_per_entry, options=None, stream=None):
    """Two-way time-sharing (Sec. 7).  Returns (minus, plus, alpha): minus
    and plus are (codebook, rank, info dict) of B (H <= b) and A (H > b);
    alpha is the share of entries quantized with plus."""
    x = _check_x(x)
    cb = torch.empty((2, int(s)), dtype=torch.float64, device=x.device)
    rk = torch.empty((2, int(s)), dtype=torch.int32, device=x.device)
    infos = (ecasq_info * 2)()
    alpha = ctypes.c_double(0.0)
    o = options if options is not None else ecasq_default_options()
    st = lib().ecasq_solve_timeshare(_ptr(x), _DTYPES[x.dtype], x.numel(), int(s),
                                     float(bits_per_entry), ctypes.byref(o), _stream(stream),
                                     _ptr(cb), _ptr(rk), ctypes.byref(alpha), infos)
    _raise(st, (ECASQ_OK, ECASQ_EINFEASIBLE))
    out = [(cb[k, :infos[k].t], rk[k, :infos[k].t], infos[k].as_dict()) for k in range(2)]
    return out[0], out[1], alpha.value


def ecasq_quantize_timeshare(x, codebook0, codebook1, alpha, seed, stream=None):
    """Returns (symbols uint8 [d], part uint8 [d] (1 = codebook1), entropy
    (0-d fp64 tensor), hist int64 [t0 + t1])."""
    x = _check_x(x)
    c0 = codebook0.to(device=x.device, dtype=torch.float64).contiguous()
    c1 = codebook1.to(device=x.device, dtype=torch.float64).contiguous()
    t0, t1 = c0.numel(), c1.numel()
    sym = torch.empty(x.numel(), dtype=torch.uint8, device=x.device)
    part = torch.empty(x.numel(), dtype=torch.uint8, device=x.device)
    ent = torch.empty((), dtype=torch.float64, device=x.device)
    hist = torch.empty(t0 + t1, dtype=torch.int64, device=x.device)
    st = lib().ecasq_quantize_timeshare(_ptr(x), _DTYPES[x.dtype], x.numel(), _ptr(c0), t0,
                                        _ptr(c1), t1, float(alpha),
                                        ctypes.c_uint64(int(seed) & (2 ** 64 - 1)),
                                        _stream(stream), _ptr(sym), _ptr(part), _ptr(ent),
                                        _ptr(hist))
    _raise(st)
    return sym, part, ent, hist


def ecasq_encode(symbols, t, stream=None):
    """rANS-code uint8 symbols (device) over t values.  Returns the stream as
    a uint8 device tensor."""
    if not isinstance(symbols, torch.Tensor) or not symbols.is_cuda or symbols.dtype != torch.uint8:
        raise TypeError("symbols must be a uint8 CUDA (HIP) tensor")
    sym = symbols.contiguous()
    d = sym.numel()
    cap = lib().ecasq_encode_bound(d, int(t))
    if cap == 0:
        raise ValueError("d or t out of range")
    out = torch.empty(cap, dtype=torch.uint8, device=sym.device)
    n = ctypes.c_int64(0)
    st = lib().ecasq_encode(_ptr(sym), d, int(t), _stream(stream), _ptr(out), cap,
                            ctypes.byref(n))
    _raise(st)
    return out[: n.value]


def ecasq_decode(data, d, t, stream=None):
    """Decode a stream of ecasq_encode back to d uint8 symbols (device)."""
    data = data.contiguous()
    sym = torch.empty(int(d), dtype=torch.uint8, device=data.device)
    st = lib().ecasq_decode(_ptr(data), data.numel(), int(d), int(t), _stream(stream), _ptr(sym))
    _raise(st)
    return sym


def ecasq_quantize(x, codebook, seed, stream=None):
    """Returns (symbols uint8 [d], empirical entropy (0-d fp64 tensor), hist int64 [t])."""
    x = _check_x(x)
    cb = codebook.to(device=x.device, dtype=torch.float64).contiguous()
    t = cb.numel()
    sym = torch.empty(x.numel(), dtype=torch.uint8, device=x.device)
    ent = torch.empty((), dtype=torch.float64, device=x.device)
    hist = torch.empty(t, dtype=torch.int64, device=x.device)
    st = lib().ecasq_quantize(_ptr(x), _DTYPES[x.dtype], x.numel(), _ptr(cb), t,
                              ctypes.c_uint64(int(seed) & (2 ** 64 - 1)), _stream(stream),
                              _ptr(sym), _ptr(ent), _ptr(hist))
    _raise(st)
    return sym, ent, hist


def ecasq_quantize_noalloc(x, codebook, seed, symbols, entropy, hist=None, stream=None):
    """ecasq_quantize into caller-provided outputs, with no allocation inside
    the library: symbols uint8 [d], entropy 0-d fp64, hist int64 [t] or None
    (all on x's device).  codebook must be a contiguous fp64 tensor there."""
    x = _check_x(x)
    if (codebook.dtype != torch.float64 or not codebook.is_contiguous()
            or codebook.device != x.device):
        raise TypeError("codebook must be a contiguous fp64 tensor on x's device")
    t = codebook.numel()
    st = lib().ecasq_quantize_noalloc(_ptr(x), _DTYPES[x.dtype], x.numel(), _ptr(codebook), t,
                                      ctypes.c_uint64(int(seed) & (2 ** 64 - 1)),
                                      _stream(stream), _ptr(symbols), _ptr(entropy),
                                      _ptr(hist) if hist is not None else None)
    _raise(st)
    return symbols, entropy, hist


def ecasq_solve_batched(x, s, bits_per_entry, options=None, stream=None):
    """x: [n, d] rows.  Returns (codebooks fp64 [n, s], t int32 [n], infos uint8 view)."""
    if x.dim() != 2:
        raise ValueError("x must be [n, d]")
    n, d = x.shape
    xc = _check_x(x)
    cbs = torch.zeros((n, int(s)), dtype=torch.float64, device=x.device)
    tt = torch.zeros(n, dtype=torch.int32, device=x.device)
    infos = torch.zeros((n, ctypes.sizeof(ecasq_info)), dtype=torch.uint8, device=x.device)
    o = options if options is not None else ecasq_default_options()
    st = lib().ecasq_solve_batched(_ptr(xc), _DTYPES[x.dtype], n, d, int(s),
                                   float(bits_per_entry), ctypes.byref(o), _stream(stream),
                                   _ptr(cbs), _ptr(tt), _ptr(infos))
    _raise(st, (ECASQ_OK, ECASQ_EINFEASIBLE))
    return cbs, tt, infos


def infos_to_dicts(infos):
    """Decode the device info array of ecasq_solve_batched."""
    raw = infos.cpu().numpy().tobytes()
    sz = ctypes.sizeof(ecasq_info)
    return [ecasq_info.from_buffer_copy(raw[i * sz:(i + 1) * sz]).as_dict()
            for i in range(len(raw) // sz)]


def ecasq_histogram(x, stream=None):
    """Sorted distinct values and exact prefix sums: (v, N, S, S2) fp64 [p]."""
    x = _check_x(x)
    d = x.numel()
    bufs = [torch.empty(d, dtype=torch.float64, device=x.device) for _ in range(4)]
    p = ctypes.c_int64(0)
    st = lib().ecasq_histogram(_ptr(x), _DTYPES[x.dtype], d, _stream(stream),
                               *[_ptr(b) for b in bufs], ctypes.byref(p))
    _raise(st)
    return tuple(b[: p.value] for b in bufs)


def ecasq_dp_trace(x, s, lam, stream=None, accumulators=False, schedule=0, argmins=True):
    """All layers of forward solves at one multiplier (lam a number) or at the
    8 multipliers of a search pass (lam a sequence of 8).  Returns F
    [nlam, s+1, d] fp64 (NaN where unset), kstar [nlam, s+1, d] int32 (-1
    where unset), the accumulators M and Ph like F (None unless asked for),
    and per multiplier (J, MSE, H(I,B), i*, cells).  With a scalar lam the
    leading nlam axis is dropped."""
    x = _check_x(x)
    d = x.numel()
    scalar = not hasattr(lam, "__len__")
    lams = [float(lam)] if scalar else [float(v) for v in lam]
    n = len(lams)
    shape = (n, int(s) + 1, d)
    F = torch.full(shape, float("nan"), dtype=torch.float64, device=x.device)
    K = torch.full(shape, -1, dtype=torch.int32, device=x.device) if argmins else None
    M = torch.full(shape, float("nan"), dtype=torch.float64, device=x.device) if accumulators else None
    Ph = torch.full(shape, float("nan"), dtype=torch.float64, device=x.device) if accumulators else None
    la = (ctypes.c_double * n)(*lams)
    out = (ctypes.c_double * (5 * n))()
    st = lib().ecasq_dp_trace(_ptr(x), _DTYPES[x.dtype], d, int(s), n, la, int(schedule),
                              _stream(stream), _ptr(F), _ptr(K), _ptr(M), _ptr(Ph), out)
    _raise(st)
    res = [tuple(out[5 * m:5 * m + 5]) for m in range(n)]
    if scalar:
        return (F[0], K[0] if K is not None else None, M[0] if M is not None else None,
                Ph[0] if Ph is not None else None, res[0])
    return F, K, M, Ph, res


def ecasq_inspect_enable(on=True):
    lib().ecasq_inspect_enable(1 if on else 0)


def ecasq_inspect_points():
    """The recorded search points as a float64 array [n, 4]: lambda, H, vNMSE,
    t (clears them)."""
    n = lib().ecasq_inspect_points(None, 0)
    out = np.zeros((max(n, 1), 4))
    lib().ecasq_inspect_points(out.ctypes.data_as(ctypes.c_void_p), n)
    return out[:n]


def ecasq_inspect_results():
    """The recorded budget results (clears them): dicts with lam_B (the
    multiplier the codebook was found at), lam_final (the refinement's), pre
    and post (value indices before and after refinement)."""
    n = lib().ecasq_inspect_results(None, None, 0)
    lams = np.zeros(2 * max(n, 1))
    ch = np.zeros(514 * max(n, 1), dtype=np.int32)
    lib().ecasq_inspect_results(lams.ctypes.data_as(ctypes.c_void_p),
                                ch.ctypes.data_as(ctypes.c_void_p), n)
    out = []
    for k in range(n):
        row = ch[514 * k: 514 * (k + 1)]
        out.append(dict(lam_B=float(lams[2 * k]), lam_final=float(lams[2 * k + 1]),
                        pre=row[1: 1 + row[0]].copy(), post=row[258: 258 + row[257]].copy()))
    return out


def ecasq_timing_enable(on=True, verbose=False):
    lib().ecasq_timing_enable((2 if verbose else 1) if on else 0)


TIMING_SINGLE = 0  # one multiplier per DP layer launch
TIMING_PASS = 1    # the 8 multipliers of a search pass per launch
TIMING_SWEEP = 2   # one whole solve of DP schedule 1
TIMING_OPT = 3     # one layer of the optimal DP
TIMING_BATCHED = 4  # one launch of ecasq_solve_batched


def ecasq_timing_read(variant=TIMING_PASS, reset=False):
    """(milliseconds, launches, cells) of the timed DP layer kernel launches of
    one variant; cells are (column, predecessor) pairs, each evaluated for
    every multiplier of its launch."""
    ms = ctypes.c_double(0)
    n = ctypes.c_int64(0)
    c = ctypes.c_int64(0)
    lib().ecasq_timing_read(int(variant), ctypes.byref(ms), ctypes.byref(n), ctypes.byref(c),
                            1 if reset else 0)
    return ms.value, n.value, c.value
