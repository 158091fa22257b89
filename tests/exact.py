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


def rnbf(q: Fraction) -> Fraction:
    """RNE of q to bfloat16 (8 significant bits, binary32's exponent range,
    gradual underflow) as an exact rational; None for an overflow."""
    r = rn_binary(q, 8, -126)
    return None if abs(r) >= Fraction(2) ** 128 else r


def f(x) -> Fraction:
    return Fraction(float(x))


def bf(h) -> Fraction:
    return Fraction(float((np.uint32(int(h)) << np.uint32(16)).view(np.float32)))


def rn32_sqrt(q: Fraction) -> np.float32:
    """RN32 of the exact square root of q >= 0: a binary32 candidate from the
    float64 root, then moved while a neighbour is nearer, each comparison made
    exactly on squares (an exact square root is never halfway between two
    binary32 values, so no tie can occur)."""
    import math
    assert q >= 0
    if q == 0:
        return np.float32(0.0)
    c = np.float32(math.sqrt(float(q)))
    while True:
        up = np.nextafter(c, np.float32(np.inf))
        dn = np.nextafter(c, np.float32(0))
        if ((f(c) + f(up)) / 2) ** 2 < q:
            c = up
        elif ((f(c) + f(dn)) / 2) ** 2 > q:
            c = dn
        else:
            return c
