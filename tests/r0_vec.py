"""Vectorised model of rule R0 (numpy), written independently of the C oracle.

Each operation computes its result in binary64 and rounds it once more to binary32.  For +, -, x and / of
binary32 operands this double rounding is innocuous (53 >= 2*24 + 2), so the binary64 value decides the
binary32 result exactly; the flush of R0 (a result whose 24-bit rounding with unbounded exponent is below
2^-126 becomes zero of its sign) is applied on the binary64 value: the rounding with unbounded exponent is
below 2^-126 exactly when the value is below 2^-126 (1 - 2^-25) in magnitude, and no quotient or product of
binary32 values lies within 2^-49 (relative) of that boundary without equalling it.  Inputs below 2^-126
read as zero of their sign.  `test_oracle_r4_spec.py` checks this model against the exact-rational model
(`exact_r0`) before using it.
"""
import numpy as np

MIN_NORMAL = np.float32(2.0 ** -126)
TINY_BOUND = 2.0 ** -126 * (1.0 - 2.0 ** -25)


def f32(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32)


def daz(x):
    x = np.asarray(x, np.float32)
    return np.where((x != 0) & (np.abs(x) < MIN_NORMAL), np.copysign(np.float32(0.0), x), x).astype(np.float32)


def _round(v64):
    with np.errstate(over="ignore", invalid="ignore"):
        r = v64.astype(np.float32)
    tiny = np.abs(v64) < TINY_BOUND
    return np.where(tiny, np.copysign(np.float32(0.0), v64).astype(np.float32), r).astype(np.float32)


def add(a, b):
    a, b = daz(a).astype(np.float64), daz(b).astype(np.float64)
    with np.errstate(invalid="ignore"):
        return _round(a + b)


def sub(a, b):
    return add(a, -np.asarray(b, np.float32))


def mul(a, b):
    a, b = daz(a).astype(np.float64), daz(b).astype(np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        return _round(a * b)


def div(a, b):
    a, b = daz(a).astype(np.float64), daz(b).astype(np.float64)
    with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
        return _round(a / b)


def bf16_bits(x):
    """RNE of a binary32 value (after DAZ) to bf16, as uint16 bit patterns."""
    u = daz(x).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)
