"""Exact rational models used to pin the oracle (test helper).

Rounding of an exact rational to an IEEE binary format with p significant
bits, round-to-nearest-even, written from the format's definition; fmaf as
"exact a*b + c, rounded once to binary32".  Python's Fraction arithmetic is
exact, so these are independent of both the C oracle and the HIP path.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

INF = float("inf")


def _floor_log2(a: Fraction) -> int:
    """floor(log2 a) for a > 0, exactly."""
    e = a.numerator.bit_length() - a.denominator.bit_length()
    # 2^e <= a < 2^(e+2) holds for this estimate; correct it by comparison.
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    return e


def round_binary(q: Fraction, p: int, emin: int, emax: int) -> Fraction | float:
    """Round exact q to the nearest number with p significant bits, minimum
    normal exponent emin and maximum exponent emax; ties to even; values that
    round beyond the largest finite number become +-inf."""
    if q == 0:
        return Fraction(0)
    s = -1 if q < 0 else 1
    a = -q if q < 0 else q
    e = max(_floor_log2(a), emin)
    ulp = Fraction(2) ** (e - p + 1)
    n = a / ulp
    fl = math.floor(n)
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    r = fl * ulp
    max_finite = (Fraction(2) - Fraction(2) ** (1 - p)) * Fraction(2) ** emax
    if r > max_finite:
        return s * INF
    return s * r


def round_f32(q: Fraction):
    return round_binary(q, 24, -126, 127)


def round_f16(q: Fraction):
    return round_binary(q, 11, -14, 15)


def fmaf(a, b, c):
    """binary32 fused multiply-add: exact a*b + c, one rounding."""
    r = round_f32(Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c)))
    return np.float32(float(r))


def f32(x) -> Fraction:
    return Fraction(float(np.float32(x)))
