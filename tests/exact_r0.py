"""Exact-rational model of rule R0, written independently of the C oracle.

Each function computes the exact real result with ``fractions.Fraction`` and
rounds it once: 24 significant bits, ties to even, unbounded exponent; a
rounded magnitude below 2^-126 becomes zero of the result's sign (IEEE-754
tininess after rounding, then flush); inputs below 2^-126 read as zero of the
same sign.  Used only to pin the oracle's primitives.
"""
import math
from fractions import Fraction as F

import numpy as np

TWO = F(2)
MIN_NORMAL = TWO ** -126


def sign_of(x: float) -> int:
    return -1 if math.copysign(1.0, x) < 0 else 1


def daz(x: float) -> float:
    if x != 0.0 and abs(x) < 2.0 ** -126:
        return math.copysign(0.0, x)
    return x


def _floor_log2(m: F) -> int:
    e = m.numerator.bit_length() - m.denominator.bit_length()
    while TWO ** e > m:
        e -= 1
    while TWO ** (e + 1) <= m:
        e += 1
    return e


def round24(m: F) -> F:
    """Round m > 0 to 24 significant bits, ties to even, unbounded exponent."""
    q = _floor_log2(m) - 23
    scaled = m / TWO ** q
    fl = scaled.numerator // scaled.denominator
    rem = scaled - fl
    if rem > F(1, 2) or (rem == F(1, 2) and fl % 2 == 1):
        fl += 1
    return fl * TWO ** q


def r0(x: F, zero_sign: int = 1) -> np.float32:
    if x == 0:
        return np.float32(math.copysign(0.0, zero_sign))
    s = -1 if x < 0 else 1
    r = round24(abs(x))
    if r < MIN_NORMAL:
        return np.float32(math.copysign(0.0, s))
    if r >= TWO ** 128:
        return np.float32(s * math.inf)
    return np.float32(s * float(r))


def add(a, b):
    a, b = daz(float(a)), daz(float(b))
    x = F(a) + F(b)
    zs = -1 if (x == 0 and sign_of(a) < 0 and sign_of(b) < 0) else 1
    return r0(x, zs)


def mul(a, b):
    a, b = daz(float(a)), daz(float(b))
    return r0(F(a) * F(b), sign_of(a) * sign_of(b))


def fma(a, b, c):
    a, b, c = daz(float(a)), daz(float(b)), daz(float(c))
    p = F(a) * F(b)
    x = p + F(c)
    zs = 1
    if x == 0 and p == 0 and c == 0 and sign_of(a) * sign_of(b) < 0 and sign_of(c) < 0:
        zs = -1
    return r0(x, zs)


def div(a, b):
    a, b = daz(float(a)), daz(float(b))
    return r0(F(a) / F(b), sign_of(a) * sign_of(b))


def sqrt_is_correctly_rounded(x: float, r: float) -> bool:
    """r == RN(sqrt(x)) checked with exact brackets (no square-root routine involved)."""
    x = daz(float(x))
    if x == 0:
        return r == 0 and sign_of(r) == sign_of(x)
    R = F(float(r))
    e = _floor_log2(R)
    ulp_up = TWO ** (e - 23)
    ulp_down = ulp_up / 2 if R == TWO ** e else ulp_up
    lo, hi = R - ulp_down / 2, R + ulp_up / 2
    X = F(x)
    if lo * lo < X < hi * hi:
        return True
    # exact ties cannot occur for square roots of binary32 values; a boundary hit means not RN
    return False


def bf16(x) -> np.float32:
    """RNE to 8 significant bits of a binary32 value (after DAZ), as a float32 value."""
    x = daz(float(x))
    if x == 0:
        return np.float32(x)
    s = -1 if x < 0 else 1
    m = abs(F(x))
    q = _floor_log2(m) - 7
    scaled = m / TWO ** q
    fl = scaled.numerator // scaled.denominator
    rem = scaled - fl
    if rem > F(1, 2) or (rem == F(1, 2) and fl % 2 == 1):
        fl += 1
    v = fl * TWO ** q
    if v >= TWO ** 128:
        return np.float32(s * math.inf)
    return np.float32(s * float(v))
