"""Build and load the C oracle (ecasq_oracle.c) through ctypes.

TEST INFRASTRUCTURE ONLY: only tests/, __graft_entry__ and bench.py's
cpu_baseline leg may use it.
"""
import ctypes
import os
import subprocess

import numpy as np

from . import log2_table

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ecasq_oracle.c")
_SO = os.path.join(_HERE, "libecasq_oracle.so")

CFLAGS = ["-O2", "-std=c11", "-mfma", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
          "-shared", "-Wall", "-Wextra"]

_lib = None


def build():
    """Compile the oracle library in place (always recompiles)."""
    tmp = _SO + ".tmp"
    subprocess.run(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
    os.replace(tmp, _SO)
    return _SO


def _stale():
    return (not os.path.exists(_SO)) or os.path.getmtime(_SO) < os.path.getmtime(_SRC)


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if _stale():
        build()
    L = ctypes.CDLL(_SO)
    dp = ctypes.POINTER(ctypes.c_double)
    ip = ctypes.POINTER(ctypes.c_int32)
    i64p = ctypes.POINTER(ctypes.c_int64)
    i64 = ctypes.c_int64
    i32 = ctypes.c_int32
    d = ctypes.c_double
    L.orc_set_log2_table.argtypes = [dp, dp]
    L.orc_log2c.argtypes = [d]
    L.orc_log2c.restype = d
    L.orc_h.argtypes = [d]
    L.orc_h.restype = d
    hist = [dp, dp, dp, dp, i64, i64]
    L.orc_dp_forward.argtypes = hist + [i32, i32, d, dp, ip, dp, dp]
    L.orc_traceback.argtypes = [ip, i64, i32, ip]
    L.orc_hirschberg.argtypes = hist + [i32, d, ip, i64p]
    L.orc_chain_metrics.argtypes = hist + [i32, ip, d, dp]
    L.orc_opt_dp.argtypes = hist + [i32, i32, d, ip, dp, ip, dp]
    L.orc_refine.argtypes = hist + [i32, ip, d, d, i32, i32, i32, ip]
    L.orc_refine_local.argtypes = hist + [i32, ip, i32, i64, d]
    L.orc_refine_local.restype = d
    L.orc_refine_search.argtypes = hist + [i32, ip, i32, d, i32]
    L.orc_refine_search.restype = i64
    L.orc_refine_substep.argtypes = hist + [i32, ip, i32, d, i32, ip]
    L.orc_refine_substep.restype = i32
    L.orc_search.argtypes = hist + [i32, d, i32, i32, i32, i32, i32, i32, i32, dp, ip, i32, dp,
                                    i32, dp, i32, dp]
    L.orc_exp2c.argtypes = [d]
    L.orc_exp2c.restype = d
    L.orc_aim_query.argtypes = [d, d, d, d, d]
    L.orc_aim_query.restype = d
    L.orc_set_exp2_table.argtypes = [dp, dp]
    L.orc_interval.argtypes = hist + [i64, i64, dp]
    L.orc_dp_columns.argtypes = hist + [i32, d, dp, dp, dp, i64, i64p, dp, ip, dp, dp]
    L.orc_dp_columns.restype = None
    invc, lc = log2_table.build_table()
    a = np.asarray(invc, dtype=np.float64)
    b = np.asarray(lc, dtype=np.float64)
    L.orc_set_log2_table(a.ctypes.data_as(dp), b.ctypes.data_as(dp))
    et, ec = log2_table.build_exp2_table()
    ea = np.asarray(et, dtype=np.float64)
    eb = np.asarray(ec, dtype=np.float64)
    L.orc_set_exp2_table(ea.ctypes.data_as(dp), eb.ctypes.data_as(dp))
    L._tables = (a, b, ea, eb)
    _lib = L
    return L


def dptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def iptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
