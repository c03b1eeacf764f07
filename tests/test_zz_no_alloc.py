"""The allocation-free rounding entry point (ecasq_quantize_noalloc) against
ecasq_quantize through the C ABI: symbols, counts and entropy bit for bit, on
two calls in a row, the second with a smaller input and codebook (so counts
left in the shared device array by the first call would show)."""
import numpy as np
import pytest
import torch

from paper_2608_18147_amd import ecasq, inputs

pytestmark = pytest.mark.gpu


def _codebook(x, t):
    xs = np.sort(x.astype(np.float64))
    idx = np.unique(np.linspace(0, len(xs) - 1, t).round().astype(np.int64))
    return torch.from_numpy(np.unique(xs[idx])).to("cuda")


def _check(x, t, seed):
    xd = torch.from_numpy(x).to("cuda")
    cb = _codebook(x, t)
    s_ref, e_ref, h_ref = ecasq.ecasq_quantize(xd, cb, seed)
    sym = torch.empty(x.size, dtype=torch.uint8, device="cuda")
    ent = torch.empty((), dtype=torch.float64, device="cuda")
    hist = torch.empty(cb.numel(), dtype=torch.int64, device="cuda")
    ecasq.ecasq_quantize_noalloc(xd, cb, seed, sym, ent, hist)
    torch.cuda.synchronize()
    assert torch.equal(sym, s_ref)
    assert torch.equal(hist, h_ref)
    assert float(ent) == float(e_ref)
    assert int(hist.sum()) == x.size


def test_noalloc_quantize_matches_quantize_twice():
    _check(inputs.student_t(1 << 20, 3), 200, 11)
    _check(inputs.normal(3000, 4), 5, 12)


def test_noalloc_quantize_without_hist_and_limits():
    x = inputs.normal(4097, 5)
    xd = torch.from_numpy(x).to("cuda")
    cb = _codebook(x, 17)
    s_ref, e_ref, _ = ecasq.ecasq_quantize(xd, cb, 3)
    sym = torch.empty(x.size, dtype=torch.uint8, device="cuda")
    ent = torch.empty((), dtype=torch.float64, device="cuda")
    ecasq.ecasq_quantize_noalloc(xd, cb, 3, sym, ent, None)
    torch.cuda.synchronize()
    assert torch.equal(sym, s_ref) and float(ent) == float(e_ref)
    big = torch.linspace(-1, 1, 257, dtype=torch.float64, device="cuda")
    with pytest.raises(ecasq.EcasqError):
        ecasq.ecasq_quantize_noalloc(xd, big, 3, sym, ent, None)
