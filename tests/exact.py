"""Exact-rational reference rules used to pin the fp64 oracle.

Nothing here calls the oracle or the GPU library: rounding is done by
searching the enumerated fp16 grid (decoded by numpy) and by brute force
over candidate codes, in Python Fractions.
"""
import bisect
from fractions import Fraction

import numpy as np

F16_MAX = Fraction(65504)


def _grid():
    bits = np.arange(0x0000, 0x7C00, dtype=np.uint16)  # +0 .. largest finite
    vals = bits.view(np.float16).astype(np.float64)
    fr = [Fraction(float(v)) for v in vals]
    # IEEE overflow: the next value past 65504 on the binade's grid is 2^16,
    # whose significand is even; rounding to it means overflow (+inf).
    fr.append(Fraction(65536))
    b = [int(x) for x in bits] + [0x7C00]
    return fr, b


_GRID_VALS, _GRID_BITS = _grid()


def f16_round_exact(q):
    """fp16 bit pattern nearest to the rational q, ties to even significand,
    overflow to inf, signed zero kept for q == 0 only via the sign of q."""
    q = Fraction(q)
    sign = 0x8000 if q < 0 else 0
    a = abs(q)
    if a >= _GRID_VALS[-1]:
        return sign | 0x7C00
    i = bisect.bisect_left(_GRID_VALS, a)
    if _GRID_VALS[i] == a:
        return sign | _GRID_BITS[i]
    lo, hi = i - 1, i
    dlo = a - _GRID_VALS[lo]
    dhi = _GRID_VALS[hi] - a
    if dlo < dhi:
        pick = lo
    elif dhi < dlo:
        pick = hi
    else:
        pick = lo if (_GRID_BITS[lo] & 1) == 0 else hi
    return sign | _GRID_BITS[pick]


def f16_value(bits):
    return Fraction(float(np.array([bits], dtype=np.uint16).view(np.float16)[0]))


def nearest_code(w, s, Q):
    """argmin over integer c in [-Q, Q] of |w - c*s|, ties to the even c;
    0 when s == 0 (brute force over every candidate)."""
    w = Fraction(w)
    s = Fraction(s)
    if s == 0:
        return 0
    best = None
    for c in range(-Q, Q + 1):
        d = abs(w - c * s)
        if best is None or d < best[0] or (d == best[0] and c % 2 == 0):
            best = (d, c)
    return best[1]


def block_scale_bits(block, Q):
    """fp16 scale of a block by the exact rule: nearest fp16 to absmax/Q."""
    a = max(abs(Fraction(float(v))) for v in block)
    return f16_round_exact(a / Q)


def dot_exact(xs, cs, s_bits_per_block, block=32):
    """sum_b s_b * sum_{k in b} x_k c_k in exact rationals."""
    total = Fraction(0)
    for b, sb in enumerate(s_bits_per_block):
        part = sum(Fraction(float(xs[k])) * int(cs[k]) for k in range(b * block, (b + 1) * block))
        total += f16_value(sb) * part
    return total
