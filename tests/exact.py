"""Exact-rational helpers for the oracle's pins (test infrastructure).

rn32(Fraction) is round-to-nearest-even to binary32 with gradual underflow
and overflow to infinity, written from the IEEE 754 definition with Python
integers; it is itself pinned against numpy's float64 -> float32 conversion.
"""
from fractions import Fraction

import numpy as np


def ilog2(q: Fraction) -> int:
    q = abs(q)
    e = q.numerator.bit_length() - q.denominator.bit_length()
    if Fraction(2) ** e > q:
        e -= 1
    return e


def rn_binary(q: Fraction, p: int, emin: int) -> Fraction:
    """Round q to p significant bits, RNE, with quantum >= 2^(emin - p + 1)."""
    if q == 0:
        return Fraction(0)
    s = -1 if q < 0 else 1
    a = abs(q)
    quantum = max(ilog2(a) - p + 1, emin - p + 1)
    u = a / Fraction(2) ** quantum
    n = u.numerator // u.denominator
    rem = u - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return s * n * Fraction(2) ** quantum


def rn32(q: Fraction) -> np.float32:
    r = rn_binary(q, 24, -126)
    if abs(r) >= Fraction(2) ** 128:
        return np.float32(np.inf if r > 0 else -np.inf)
    if r == 0:
        return np.float32(-0.0 if q < 0 else 0.0)  # underflow keeps the sign
    return np.float32(float(r))


def f(x) -> Fraction:
    return Fraction(float(x))


def bf(h) -> Fraction:
    return Fraction(float((np.uint32(int(h)) << np.uint32(16)).view(np.float32)))
