"""Host-side checks of the C-ABI library that need no GPU: it loads, exports
every symbol include/ecasq.h declares, and its pure host functions behave."""
import ctypes
import os
import re

import pytest

from paper_2608_18147_amd import ecasq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "ecasq.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ecasq_[a-z_]+)\s*\(", src)))


def test_library_loads_and_exports_every_declared_symbol():
    L = ecasq.lib()
    names = _declared()
    assert "ecasq_solve" in names and "ecasq_quantize" in names
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(ecasq.EXPORTS)


def test_status_strings_and_defaults():
    assert ecasq.ecasq_status_string(0) == "ok"
    assert "NaN" in ecasq.ecasq_status_string(-2)
    o = ecasq.ecasq_default_options()
    assert (o.refine_rounds, o.refine_exhaustive, o.exact_s, o.max_search_passes, o.recovery,
            o.search_width, o.dp_schedule, o.alphabet, o.alphabet_size) == \
        (5, 0, 0, 32, 0, 1, 1, 0, 0)


def test_workspace_size_is_linear_in_d():
    a = ecasq.ecasq_workspace_size(1 << 16, 32)
    b = ecasq.ecasq_workspace_size(1 << 18, 32)
    assert 3.5 < b / a < 4.5
    assert ecasq.ecasq_workspace_size(0, 32) == 0
    assert ecasq.ecasq_workspace_size(1024, 1) == 0
    # stored argmins add (s+1) * d int32
    extra = ecasq.ecasq_workspace_size(1 << 16, 32, 1) - a
    assert extra >= 33 * (1 << 16) * 4


def test_argument_errors_before_any_device_work():
    """Argument errors come back synchronously (no GPU is touched)."""
    L = ecasq.lib()
    info = ecasq.ecasq_info()
    fake = ctypes.c_void_p(0x1000)
    # null x, d < 1, s < 2, NaN budget
    assert L.ecasq_solve(None, 0, 10, 4, 2.0, None, fake, None, ctypes.byref(info)) == -1
    assert L.ecasq_solve(fake, 0, 0, 4, 2.0, None, fake, None, ctypes.byref(info)) == -1
    assert L.ecasq_solve(fake, 0, 10, 1, 2.0, None, fake, None, ctypes.byref(info)) == -1
    assert L.ecasq_solve(fake, 0, 10, 4, float("nan"), None, fake, None,
                         ctypes.byref(info)) == -1
    assert L.ecasq_solve(fake, 0, 10, 4, -1.0, None, fake, None, ctypes.byref(info)) == -1
    assert L.ecasq_solve(fake, 7, 10, 4, 2.0, None, fake, None, ctypes.byref(info)) == -1
    assert L.ecasq_quantize(fake, 0, 10, None, 3, 0, None, fake, fake, None) == -1
    assert L.ecasq_quantize(fake, 0, 10, fake, 0, 0, None, fake, fake, None) == -1
    assert L.ecasq_solve_lagrangian(fake, 0, 10, 4, -0.5, None, None, fake, None, None) == -1
