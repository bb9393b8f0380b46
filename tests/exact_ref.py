"""Exact-rational reference for pinning the oracle (tests only).

Independent of ``oracle/``: the format's values are enumerated from the
definition of the bit codes (IEEE-754-style layout: bias, subnormals, the
all-ones exponent reserved), and rounding picks the nearest enumerated value
by bisection over exact ``Fraction`` values.  Ties go to the neighbour that is
an even multiple of the gap between the two neighbours (round-half-to-even on
the significand).  A magnitude that rounds past the largest finite value
(to the next power of two, which is what an unbounded exponent would give)
becomes INF.

Only used for formats of at most 16 bits, where full enumeration is cheap.
"""
from __future__ import annotations

import bisect
import math
from fractions import Fraction
from functools import lru_cache


def default_bias(e: int) -> int:
    return (1 << (e - 1)) - 1


@lru_cache(maxsize=None)
def values(e: int, m: int, bias: int) -> tuple:
    """All non-negative finite values, indexed by their code (ascending)."""
    out = []
    for ef in range(0, (1 << e) - 1):          # all-ones exponent is INF/NaN
        for mant in range(1 << m):
            if ef == 0:                         # subnormal: 0.mant * 2^(1-bias)
                v = Fraction(mant, 1 << m) * Fraction(2) ** (1 - bias)
            else:                               # normal: 1.mant * 2^(ef-bias)
                v = (1 + Fraction(mant, 1 << m)) * Fraction(2) ** (ef - bias)
            out.append(v)
    return tuple(out)


def emax(e: int, m: int, bias: int) -> int:
    return (1 << e) - 2 - bias


def round_exact(y, e: int, m: int, bias: int | None = None):
    """Round the exact value y (Fraction/float/int) to the format.

    Returns a Fraction, or a float +-inf / nan."""
    if bias is None:
        bias = default_bias(e)
    if isinstance(y, float):
        if math.isnan(y) or math.isinf(y):
            return y
        neg = math.copysign(1.0, y) < 0
        y = Fraction(y)
    else:
        y = Fraction(y)
        neg = y < 0
    a = abs(y)
    ext = list(values(e, m, bias)) + [Fraction(2) ** (emax(e, m, bias) + 1)]
    i = bisect.bisect_right(ext, a) - 1
    if i == len(ext) - 1:
        r = ext[-1]                             # at or past the next power of two
    elif a == ext[i]:
        r = ext[i]
    else:
        lo, hi = ext[i], ext[i + 1]
        dlo, dhi = a - lo, hi - a
        if dlo < dhi:
            r = lo
        elif dhi < dlo:
            r = hi
        else:
            gap = hi - lo
            r = lo if (lo / gap).numerator % 2 == 0 else hi
    if r == ext[-1]:
        return -math.inf if neg else math.inf
    return -r if neg else r


def to_float(v) -> float:
    """Fraction or float -> float, keeping the sign of zero for floats only."""
    return float(v)


def sum_exact(qs, e: int, m: int, bias: int | None = None):
    """Sequential sum with the accumulator rounded after every add."""
    s = None
    for q in qs:
        if s is None:
            s = q
            continue
        if isinstance(s, float) or isinstance(q, float):
            s = round_exact(float(s) + float(q), e, m, bias)   # INF/NaN arithmetic
        else:
            t = s + q
            s = round_exact(t, e, m, bias) if t != 0 else Fraction(0)
    return s


def ceil_log2_exact(t: Fraction) -> int:
    """Smallest integer c with 2^c >= t (t > 0)."""
    c = t.numerator.bit_length() - t.denominator.bit_length()
    while Fraction(2) ** c < t:
        c += 1
    while Fraction(2) ** (c - 1) >= t:
        c -= 1
    return c


def chain_exact(xs, e, m, bias=None, kahan=False):
    """A chain of adds with every intermediate rounded: plain or Kahan."""
    s = xs[0]
    c = Fraction(0)
    for x in xs[1:]:
        if kahan:
            y = round_exact(x - c, e, m, bias)
            t = round_exact(s + y, e, m, bias)
            c = round_exact(round_exact(t - s, e, m, bias) - y, e, m, bias)
            s = t
        else:
            s = round_exact(s + x, e, m, bias)
    return s


def hierarchical_exact(qs, k, seg, e, m, bias=None, kahan=False):
    """Groups of k consecutive workers summed at their master, then the
    masters' ring starting at master `seg`."""
    W = len(qs)
    ng = W // k
    sums = [chain_exact(qs[g * k:(g + 1) * k], e, m, bias, kahan) for g in range(ng)]
    order = [sums[(seg + i) % ng] for i in range(ng)]
    return chain_exact(order, e, m, bias, kahan)
