"""Exact-arithmetic helpers for the oracle pins (rational numbers, no floats)."""
from fractions import Fraction

import numpy as np


def fraction_of(x) -> Fraction:
    return Fraction(float(x))


def round_half_even(x: Fraction) -> int:
    fl = x.numerator // x.denominator
    rem = x - fl
    if rem > Fraction(1, 2):
        return fl + 1
    if rem < Fraction(1, 2):
        return fl
    return fl if fl % 2 == 0 else fl + 1


def fp32_round(x: Fraction) -> np.float32:
    """Correctly rounded (nearest-even) binary32 value of an exact rational."""
    if x == 0:
        return np.float32(0.0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)                       # subnormal quantum 2^-149
    quantum = Fraction(2) ** (e - 23)
    m = round_half_even(a / quantum)
    val = float(m) * float(quantum)        # exact in double: m < 2^25
    return np.float32(sign * val)
