"""Exact rational arithmetic of the runtime quantizer for tiny inputs (test infrastructure).

Inputs are dyadic rationals (any finite float is one), so the unnormalized
Hadamard transform u = H_b x is an exact rational vector.  Eq. (5) applied to
z = u / sqrt(b) gives z / delta = u * q / (r * max|u|): the sqrt(b) cancels, so
the codes are exact rationals rounded half-to-even, with no floating point at
all.  delta = r * max|u| / (q * sqrt(b)) is returned as the exact rational
r * max|u| / q together with b, so a caller can compare it with a float.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence, Tuple


def hadamard_apply(x: Sequence[Fraction], b: int) -> List[Fraction]:
    """u = (I (x) H_b) x with H_b[i][j] = (-1)^popcount(i & j), by the matrix definition."""
    K = len(x)
    assert K % b == 0
    out: List[Fraction] = []
    for k0 in range(0, K, b):
        for i in range(b):
            s = Fraction(0)
            for j in range(b):
                sign = -1 if bin(i & j).count("1") % 2 else 1
                s += sign * x[k0 + j]
            out.append(s)
    return out


def round_half_even(v: Fraction) -> int:
    fl = v.numerator // v.denominator
    rem = v - fl
    if rem > Fraction(1, 2):
        return fl + 1
    if rem < Fraction(1, 2):
        return fl
    return fl if fl % 2 == 0 else fl + 1


def quantize_token(x: Sequence[float], b: int, bits: int, r: Fraction = Fraction(1),
                   chan_mult: Sequence[float] = None) -> Tuple[List[int], Fraction, List[Fraction]]:
    """Exact eq. (5) for one token.

    Returns (codes, r*A/q, ratios) where A = max|H x| (unnormalized), so that the
    paper's delta equals (r*A/q) / sqrt(b), and ratios[c] = z_c / delta exactly.
    """
    xs = [Fraction(float(v)) for v in x]
    if chan_mult is not None:
        xs = [a * Fraction(float(m)) for a, m in zip(xs, chan_mult)]
    u = hadamard_apply(xs, b)
    q = 2 ** (bits - 1) - 1
    A = max((abs(v) for v in u), default=Fraction(0))
    if A == 0:
        return [0] * len(u), Fraction(0), [Fraction(0)] * len(u)
    ratios = [v * q / (r * A) for v in u]
    codes = [max(-q, min(q, round_half_even(t))) for t in ratios]
    return codes, r * A / q, ratios
