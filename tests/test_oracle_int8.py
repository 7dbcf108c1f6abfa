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


def sylvester(n):
    h = np.array([[1]], np.int64)
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h


def test_fwht_matches_the_hadamard_matrix_on_integers():
    # integer inputs keep every butterfly exact, so the transform must equal H_256 v / 16 exactly
    H = sylvester(256)
    v = RNG.integers(-1000, 1001, (3, 256)).astype(np.float32)
    want = (v.astype(np.float64) @ H.T) / 16.0
    got = oracle.fwht256(v)
    assert np.array_equal(got.astype(np.float64), want)
    assert np.array_equal(oracle.fwht256(got), v)  # the scaled transform is an involution in the exact regime


def rot(x):
    return oracle.fwht256(x)


def one_hot_blocks(rows, L, rng, sign=True):
    # 127 at one position per block of 256 (random sign): rotating such a row gives values +-127/16
    v = np.zeros((rows, L), np.float32)
    for r in range(rows):
        for b in range(L // 256):
            v[r, b * 256 + rng.integers(0, 256)] = 127.0 * (rng.choice([-1, 1]) if sign else 1)
    return v


def test_qlinear_bwd_exact_regime_dx():
    # dy and W^ built so that both rotated operands are integers in [-127, 127] with 127 present: every step
    # is 1, quantisation is exact, and dx must be the exact product rounded once
    rng = np.random.default_rng(5)
    T, N, K = 256, 512, 48
    U = rng.integers(-127, 128, (T, N)).astype(np.float32)
    U[0, 0] = 127
    dy = rot(U)                                   # rot(dy) = U exactly
    V = one_hot_blocks(K, N, rng)                 # rows k of W^ transposed, rotated
    wt = rot(V)                                   # W^T: values +-127/16
    qw = np.rint(wt.T * 16).astype(np.int8)       # W^ = qw / 16 exactly
    sw = np.full(N, 1 / 16, np.float32)
    qx = np.zeros((T, K), np.int8)
    dx, _ = oracle.qlinear_bwd(dy, qx, 1.0, qw, sw, want_dw=False)
    exact = U.astype(np.int64) @ V.astype(np.int64).T
    assert np.array_equal(bits(dx), bits(exact.astype(np.float32)))


def test_qlinear_bwd_exact_regime_dw():
    rng = np.random.default_rng(6)
    T, N, K = 512, 64, 40
    G = rng.integers(-127, 128, (N, T)).astype(np.float32)
    G[0, 0] = -127
    dy = rot(G).T.copy()                          # rot along T of dy^T rows = G
    V2 = one_hot_blocks(K, T, rng)
    xt = rot(V2)                                  # X^ transposed: +-127/16
    qx = np.rint(xt.T * 16).astype(np.int8)       # X^ = qx / 16 exactly
    qw = np.zeros((N, K), np.int8)
    _, dw = oracle.qlinear_bwd(dy, qx, 1 / 16, qw, np.ones(N, np.float32), want_dx=False)
    exact = G.astype(np.int64) @ V2.astype(np.int64).T
    assert np.array_equal(bits(dw), bits(exact.astype(np.float32)))


def test_qlinear_bwd_error_against_float64():
    # general inputs: the int8 gradients approximate the float64 products of the dequantised operands
    rng = np.random.default_rng(7)
    T, N, K = 512, 512, 64
    dy = (rng.standard_normal((T, N)) * 1e-3).astype(np.float32)
    dy[3, 7] = 0.05  # an outlier, which the rotation spreads
    qx = rng.integers(-128, 128, (T, K)).astype(np.int8)
    qw = rng.integers(-128, 128, (N, K)).astype(np.int8)
    sx, sw = np.float32(0.02), (np.abs(rng.standard_normal(N)) * 0.001 + 1e-4).astype(np.float32)
    dx, dw = oracle.qlinear_bwd(dy, qx, sx, qw, sw)
    W = sw[:, None].astype(np.float64) * qw
    X = float(sx) * qx.astype(np.float64)
    for got, want in ((dx, dy.astype(np.float64) @ W), (dw, dy.astype(np.float64).T @ X)):
        rel = np.linalg.norm(got - want) / np.linalg.norm(want)
        assert rel < 0.05, rel
