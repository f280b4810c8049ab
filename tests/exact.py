"""Exact rational arithmetic used to pin the oracle (tests only).

Independent of the oracle: these helpers know nothing of its rounding rules,
they compute exact values with Python's Fraction and round them to fp32 by the
IEEE definition (nearest, ties to even).
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np


def frac(v) -> Fraction:
    return Fraction(float(v))


def rn32(q: Fraction) -> np.float32:
    """The fp32 value nearest to q (ties to even), subnormals included."""
    if q == 0:
        return np.float32(0.0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    # e = floor(log2 a)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    elif Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp_exp = max(e, -126) - 23
    ulp = Fraction(2) ** ulp_exp
    m = a / ulp
    lo = m.numerator // m.denominator
    rem = m - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    val = Fraction(lo) * ulp
    return np.float32(sign * float(val))


def ulp32(x: float) -> float:
    x = abs(float(np.float32(x)))
    return float(np.spacing(np.float32(x)))


def exact_l1_fixed(v) -> int:
    """sum floor(|v_i| * 2^80) with Python integers."""
    total = 0
    for x in np.asarray(v, dtype=np.float32).tolist():
        f = abs(Fraction(x)) * (2 ** 80)
        total += f.numerator // f.denominator
    return total
