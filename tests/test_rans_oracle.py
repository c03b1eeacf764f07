"""Pins of the rANS entropy coder in the oracle (Duda, arXiv:1311.2540): the
stream decodes back to the symbols, each segment's length is within the
coder's state size of the model's ideal code length, and the quantized
frequencies track the symbol counts."""
import math

import numpy as np

from oracle import pipeline, rans


def _streams():
    rng = np.random.default_rng(50)
    yield "uniform_t17", rng.integers(0, 17, size=9000), 17
    p = np.array([0.9, 0.05, 0.03, 0.02])
    yield "skewed_t4", rng.choice(4, size=12001, p=p), 4
    yield "one_symbol_present_t8", np.full(5000, 3), 8
    yield "t1", np.zeros(4100, dtype=np.int64), 1
    yield "t256", rng.integers(0, 256, size=20000), 256
    yield "short", np.array([1, 0, 1]), 2
    yield "single", np.array([0]), 2
    x = rng.standard_normal(30000).astype(np.float32)
    q = np.array([float(x.min()), -1.0, -0.3, 0.2, 0.9, float(x.max())])
    yield "rounded_symbols", pipeline.quantize(x, q, 5)[0], len(q)


def test_rans_round_trip_and_length():
    for name, sym, t in _streams():
        sym = [int(s) for s in sym]
        data = rans.encode(sym, t)
        assert rans.decode(data, len(sym), t) == sym, name
        hist = [sym.count(q) for q in range(t)]
        f = rans.quantize_freqs(hist)
        c = [sum(f[:q]) for q in range(t)]
        for a in range(0, len(sym), rans.SEG):
            seg = sym[a:a + rans.SEG]
            nbytes = len(rans.encode_segment(seg, f, c))
            ideal = rans.ideal_bits(seg, f)
            # the final state (32 bits) and the initial state bound the excess
            assert ideal - 32 <= 8 * nbytes <= ideal + 40, (name, a, nbytes, ideal)
        nseg = (len(sym) + rans.SEG - 1) // rans.SEG
        assert len(data) == 2 * t + 4 * nseg + sum(
            len(rans.encode_segment(sym[a:a + rans.SEG], f, c))
            for a in range(0, len(sym), rans.SEG))


def test_rans_frequencies():
    rng = np.random.default_rng(51)
    for t in (1, 2, 5, 64, 256):
        for _ in range(20):
            n = rng.integers(0, 1000, size=t)
            n[rng.random(t) < 0.3] = 0
            if n.sum() == 0:
                n[0] = 1
            f = rans.quantize_freqs(list(n))
            assert sum(f) == rans.M and min(f) >= 1 and max(f) <= rans.M
            d = n.sum()
            for q in range(t):
                # every frequency stays within t units of its exact share
                assert abs(f[q] - n[q] * rans.M / d) <= t + 1


def test_rans_rate_approaches_entropy():
    """On a long stream the coded payload is within 0.5% (plus the per-segment
    states) of the plug-in entropy of the symbols."""
    rng = np.random.default_rng(52)
    p = np.array([0.5, 0.25, 0.125, 0.0625, 0.0625])
    sym = rng.choice(5, size=200000, p=p)
    data = rans.encode(sym, 5)
    hist = np.bincount(sym, minlength=5)
    H = -sum((n / len(sym)) * math.log2(n / len(sym)) for n in hist if n)
    nseg = (len(sym) + rans.SEG - 1) // rans.SEG
    payload_bits = 8 * (len(data) - 2 * 5 - 4 * nseg)
    assert payload_bits <= len(sym) * H * 1.005 + 40 * nseg
    assert payload_bits >= len(sym) * H - 32 * nseg
