"""Oracle-side table for the canonical base-2 logarithm.

TEST INFRASTRUCTURE ONLY: nothing in the product path may import this module.

The paper's entropy terms h(y) = -y log2 y (Sec. 4, definition of h; Sec. 5,
the Phi terms of the surrogate entropy) need a base-2 logarithm evaluated in
fp64.  The paper does not fix how it is computed.  For bit-exact parity the
oracle and the GPU evaluate the same fixed operation sequence (a table-driven
reduction in the style of Tang 1990).  This module builds the oracle's own copy
of the 1024-entry table with mpmath; the GPU library builds its copy with an
independent integer-arithmetic generator.  Every entry is a correctly rounded
double, so both copies must agree bit for bit.

Entry i covers the inputs whose reduced mantissa bits (y's high word minus the
offset word OFF_HI) have i in bits 10..19:
    c_i   = the double whose high word is OFF_HI + (2i+1)*2^9, low word 0
            (OFF_HI is chosen so that the entry holding 1.0 has c = 1.0
            exactly: there r = z - 1 is exact and log2 keeps full relative
            accuracy next to 1)
    invc_i = RN(1 / c_i)                      (an IEEE division)
    lc_i   = RN(log2(1 / invc_i))             (correctly rounded via mpmath)
"""
import struct

import mpmath

OFF_HI = 0x3FE6A200  # high word of a double near 1/sqrt(2); centres an entry on 1.0
TABLE_BITS = 10
TABLE_SIZE = 1 << TABLE_BITS


def _double_from_words(hi, lo=0):
    return struct.unpack("<d", struct.pack("<Q", (hi << 32) | lo))[0]


def _round_checked(x):
    """Round an mpf to the nearest double, refusing near-ties."""
    d = float(x)  # mpmath rounds to nearest
    # reject if x lies within 2^-40 ulp of a rounding midpoint
    import math
    ulp = math.ulp(d)
    frac = (x - mpmath.mpf(d)) / ulp
    if abs(abs(frac) - 0.5) < mpmath.mpf(2) ** -40:
        raise ArithmeticError("ambiguous rounding in log2 table")
    return d


def build_table():
    """Return (invc, lc): two lists of TABLE_SIZE doubles."""
    mpmath.mp.prec = 256
    invc, lc = [], []
    i_one = ((0x3FF00000 - OFF_HI) >> (20 - TABLE_BITS)) & (TABLE_SIZE - 1)
    for i in range(TABLE_SIZE):
        c = _double_from_words(OFF_HI + ((2 * i + 1) << (20 - TABLE_BITS - 1)))
        assert (c == 1.0) == (i == i_one)
        ic = 1.0 / c
        invc.append(ic)
        lc.append(_round_checked(-mpmath.log(mpmath.mpf(ic), 2)))
    return invc, lc


# --------------------------------------------------------------------------
# Canonical base-2 exponential (used by the budget search's aimed query).
#
# exp2c(y) splits y = k/64 + r with k = RN(64 y) and |r| <= 1/128, and forms
# 2^(k/64) = 2^floor(k/64) * T[k mod 64] with T[i] = RN(2^(i/64)) and
# 2^r - 1 = r (C1 + C2 r + ... + C5 r^4) with C_k = RN(ln(2)^k / k!) (Tang
# 1989, table-driven exp).  Both tables here come from mpmath; the GPU library
# derives its copy with exact integer arithmetic.

EXP2_TABLE_SIZE = 64


def build_exp2_table():
    """Return (T, C): T[i] = RN(2^(i/64)) for i < 64 and C = [C1..C5]."""
    mpmath.mp.prec = 256
    T = [_round_checked(mpmath.power(2, mpmath.mpf(i) / EXP2_TABLE_SIZE))
         for i in range(EXP2_TABLE_SIZE)]
    ln2 = mpmath.log(2)
    C = [_round_checked(ln2 ** k / mpmath.factorial(k)) for k in range(1, 6)]
    return T, C
