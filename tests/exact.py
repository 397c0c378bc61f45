"""Exact-arithmetic helpers for pinning the oracle (tests only).

Rounding a rational to the nearest fp32 value (ties to even) lets a test
replay a chain of fused multiply-adds with one rounding per step, independent
of both the oracle's C code and the hardware."""

from fractions import Fraction

import numpy as np

_F32_MAX = Fraction((2 ** 24 - 1) * 2 ** 104)


def round_f32(q: Fraction) -> np.float32:
    """Nearest binary32 value to q, ties to even (gradual underflow kept)."""
    if q == 0:
        return np.float32(0.0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    quantum = Fraction(2) ** (e - 23)
    k = a / quantum
    n = k.numerator // k.denominator
    rem = k - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = n * quantum
    if r > _F32_MAX:
        # at or beyond the rounding boundary to infinity
        return np.float32(sign * np.inf)
    return np.float32(sign * float(r))


def fr(x) -> Fraction:
    return Fraction(float(x))


def fma_f32(a, b, c) -> np.float32:
    """fp32 fused multiply-add with a single rounding."""
    return round_f32(fr(a) * fr(b) + fr(c))
