"""Entropy coding of the final symbols with range asymmetric numeral systems
(rANS; J. Duda, "Asymmetric numeral systems: entropy coding combining speed of
Huffman coding with compression rate of arithmetic coding", arXiv:1311.2540).

TEST INFRASTRUCTURE ONLY: only tests/, __graft_entry__ and bench.py's
cpu_baseline leg may use the oracle.

It realises the rate the paper charges (App. F.1): the payload at about
H(Xhat) bits per entry plus a 16-bit descriptor per codebook value (here the
symbol's quantized frequency).  Plain Python loops, written from the
definition:

  frequencies  f_q = max(1, floor(n_q M / d)), M = 2^16, then the sum is made
               M: a surplus is added to the largest f (lowest q among ties); a
               deficit is taken one unit at a time from the largest f > 1
               (lowest q among ties); cumulative c_q = f_0 + ... + f_{q-1}.
  state        x in [L, 256 L), L = 2^23, bytes out.
  encode       symbols of a segment in reverse order; for symbol q: while
               x >= 2^15 f_q emit the low byte of x and shift x right by 8;
               then x = floor(x / f_q) 2^16 + (x mod f_q) + c_q.  At the end
               emit x's four bytes, low first.  The segment's stream is the
               emitted bytes in reverse order (so it starts with x, big-endian).
  decode       x = the first four bytes (big-endian); per symbol: slot =
               x mod 2^16, q = the symbol with c_q <= slot < c_q + f_q,
               x = f_q floor(x / 2^16) + slot - c_q, then while x < L:
               x = 256 x + next byte.  A stream decodes back to x = L.
  format       t little-endian u16 (f_q - 1), then one little-endian u32 per
               segment of 4096 symbols (the end of its bytes, counted from the
               start of the payload), then the segments' bytes.
"""
import math

M_BITS = 16
M = 1 << M_BITS
L = 1 << 23
SEG = 4096


def quantize_freqs(hist):
    """Counts n_q (q < t) -> frequencies f_q >= 1 summing to M."""
    t = len(hist)
    d = int(sum(int(n) for n in hist))
    f = [max(1, (int(n) * M) // d) if d > 0 else 1 for n in hist]
    diff = M - sum(f)
    if diff > 0:
        j = max(range(t), key=lambda q: (f[q], -q))
        f[j] += diff
    while diff < 0:
        j = max((q for q in range(t) if f[q] > 1), key=lambda q: (f[q], -q))
        f[j] -= 1
        diff += 1
    return f


def _cum(f):
    c, acc = [], 0
    for v in f:
        c.append(acc)
        acc += v
    return c


def encode_segment(symbols, f, c):
    x = L
    out = []
    for q in reversed(symbols):
        fq = f[q]
        x_max = (1 << 15) * fq
        while x >= x_max:
            out.append(x & 0xFF)
            x >>= 8
        x = ((x // fq) << M_BITS) + (x % fq) + c[q]
    for k in range(4):
        out.append((x >> (8 * k)) & 0xFF)
    return bytes(reversed(out))


def decode_segment(data, n, f, c):
    x = (data[0] << 24) | (data[1] << 16) | (data[2] << 8) | data[3]
    pos = 4
    out = []
    for _ in range(n):
        slot = x & (M - 1)
        q = 0
        while c[q] + f[q] <= slot:
            q += 1
        x = f[q] * (x >> M_BITS) + slot - c[q]
        while x < L:
            x = (x << 8) | data[pos]
            pos += 1
        out.append(q)
    assert x == L and pos == len(data), "corrupt segment"
    return out


def encode(symbols, t):
    """symbols (values < t) -> the coded stream (bytes)."""
    symbols = [int(s) for s in symbols]
    d = len(symbols)
    hist = [0] * t
    for s in symbols:
        hist[s] += 1
    f = quantize_freqs(hist)
    c = _cum(f)
    segs = [encode_segment(symbols[a:a + SEG], f, c) for a in range(0, d, SEG)]
    head = b"".join((v - 1).to_bytes(2, "little") for v in f)
    ends, acc = [], 0
    for sg in segs:
        acc += len(sg)
        ends.append(acc.to_bytes(4, "little"))
    return head + b"".join(ends) + b"".join(segs)


def decode(data, d, t):
    """The coded stream of d symbols over t values -> the symbols."""
    f = [int.from_bytes(data[2 * q:2 * q + 2], "little") + 1 for q in range(t)]
    c = _cum(f)
    nseg = (d + SEG - 1) // SEG
    base = 2 * t
    ends = [int.from_bytes(data[base + 4 * k:base + 4 * k + 4], "little") for k in range(nseg)]
    pay = base + 4 * nseg
    out, start = [], 0
    for k in range(nseg):
        n = min(SEG, d - k * SEG)
        out.extend(decode_segment(data[pay + start:pay + ends[k]], n, f, c))
        start = ends[k]
    return out


def ideal_bits(symbols, f):
    """The model's ideal code length: sum of -log2(f_q / M)."""
    return sum(-math.log2(f[int(s)] / M) for s in symbols)
