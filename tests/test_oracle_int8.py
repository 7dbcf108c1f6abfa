"""Pins for the oracle's int8 quantised linear (R13): the 1/sqrt(127) constant from exact arithmetic,
closed forms of the LSQ step re-pin, round-half-even and clamping of the quantiser against an exact
rational model, and the integer GEMM against exact integer matrix products."""
from decimal import Decimal, getcontext
from fractions import Fraction as F

import numpy as np
import pytest

import exact_r0 as R
import oracle

RNG = np.random.default_rng(13)


def bits(x):
    return np.atleast_1d(np.asarray(x, np.float32)).view(np.uint32)


def f32(u):
    return np.array([u], np.uint32).view(np.float32)[0]


def nearest_f32(v: Decimal) -> np.float32:
    f = np.float32(float(v))
    u = int(bits(f)[0])
    cands = [f32(u - 1), f32(u), f32(u + 1)]
    return min(cands, key=lambda c: abs(Decimal(float(c)) - v))


def test_inv_sqrt_qmax_constant():
    # the step re-pin multiplies by RN32(1/sqrt(127)); a row of ones of length 64 gives step 2 * that constant
    getcontext().prec = 60
    c = nearest_f32(Decimal(1) / Decimal(127).sqrt())
    s = oracle.quant_scales(np.full((1, 64), 0x3F80, np.uint16))  # bf16 1.0
    assert bits(s)[0] == bits(np.float32(2) * c)[0]


@pytest.mark.parametrize("val,k", [(0x3F00, 96), (0x4040, 100), (0x3DCC, 2048), (0xBF80, 3)])
def test_quant_scale_constant_rows_closed_form(val, k):
    # |w| = v constant: R1 sum is the exact multiple k*v (small integers times a power-of-two-rich value), so
    # s = RN(RN(2 RN(k v * RN(1/k))) * c) evaluated in exact arithmetic
    v = abs(float(np.array([val << 16], np.uint32).view(np.float32)[0]))
    c = float(f32(0x3DB5BB09))
    total = np.float32(v * k)
    assert float(total) == v * k
    inv_k = np.float32(1.0 / k)
    mean = R.mul(total, inv_k)
    want = R.mul(R.mul(np.float32(2.0), mean), np.float32(c))
    got = oracle.quant_scales(np.full((2, k), val, np.uint16))
    assert np.all(bits(got) == bits(want))


def test_quant_scale_sign_and_power_of_two_invariance():
    w = RNG.integers(0x3000, 0x4200, (5, 300)).astype(np.uint16)  # positive bf16 patterns
    s = oracle.quant_scales(w)
    assert np.array_equal(bits(oracle.quant_scales(w | 0x8000)), bits(s))          # sign of w is ignored
    assert np.array_equal(bits(oracle.quant_scales(w + (3 << 7))), bits(s * np.float32(8)))  # exponent + 3


def test_quantize_ties_clamp_and_specials():
    x = np.array([[0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 126.5, 127.5, -127.5, -128.5, 1e30, -1e30, np.inf, -np.inf,
                   np.nan, -0.0]], np.float32)
    q = oracle.quantize(x, 1.0, per_row=False)
    assert q.tolist() == [[0, 2, 2, 0, -2, -2, 126, 127, -128, -128, 127, -128, 127, -128, 0, 0]]
    # a step that is not > 0 (zero, negative, NaN, subnormal that flushes) quantises to 0
    for s in (0.0, -1.0, np.nan, 1e-40):
        assert np.all(oracle.quantize(x, s, per_row=False) == 0)
    # bf16 input: a subnormal bf16 reads as zero; exact multiples of the step reproduce the integer
    xb = np.array([[0x0001, 0x8005, 0x4040, 0xC0A0]], np.uint16)  # subnormals, 3.0, -5.0
    assert oracle.quantize(xb, 1.0, per_row=False).tolist() == [[0, 0, 3, -5]]


def test_quantize_matches_exact_rational_model():
    x = (RNG.standard_normal((40, 50)) * 3).astype(np.float32)
    s = np.abs(RNG.standard_normal(40)).astype(np.float32) * np.float32(0.05) + np.float32(0.001)
    q = oracle.quantize(x, s, per_row=True)
    for r in range(40):
        for k in range(50):
            t = R.div(x[r, k], s[r])  # RN(x / s)
            fr = F(float(t))
            n = fr.numerator // fr.denominator
            rem = fr - n
            if rem > F(1, 2) or (rem == F(1, 2) and n % 2 == 1):
                n += 1
            assert q[r, k] == max(-128, min(127, n)), (r, k)


@pytest.mark.parametrize("m,n,k", [(7, 9, 33), (16, 5, 256), (3, 4, 1)])
def test_gemm_i8_exact_integer_product(m, n, k):
    a = RNG.integers(-128, 128, (m, k)).astype(np.int8)
    b = RNG.integers(-128, 128, (n, k)).astype(np.int8)
    sb = (np.abs(RNG.standard_normal(n)) * 0.01).astype(np.float32)
    acc, y = oracle.gemm_i8(a, b, np.float32(0.037), sb)
    want = a.astype(np.int64) @ b.astype(np.int64).T
    assert np.array_equal(acc.astype(np.int64), want)
    for i in range(m):
        for j in range(n):
            wy = R.mul(R.mul(np.float32(float(want[i, j])) if abs(want[i, j]) < 2 ** 24 else
                             np.float32(R.r0(F(int(want[i, j])))), np.float32(0.037)), sb[j])
            assert bits(y[i, j]) == bits(wy), (i, j)


def test_gemm_i8_extreme_range():
    # the largest |acc| the bound on k allows: k = 65536 terms of (-128)(-128) = 2^30
    k = 65536
    a = np.full((1, k), -128, np.int8)
    acc, y = oracle.gemm_i8(a, a, np.float32(1.0), np.ones(1, np.float32))
    assert acc[0, 0] == 2 ** 30 and y[0, 0] == np.float32(2.0 ** 30)
