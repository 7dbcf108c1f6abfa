"""Pins for the oracle GEMM (R2): closed forms, invariants, the R1 order along K, error bound."""
import math
from fractions import Fraction as F

import numpy as np
import pytest

import canon_formulations as CF
import oracle
import paper_2609_17380_amd.inputs as I

RNG = np.random.default_rng(7)


def to_bf16(x):
    u = np.asarray(x, np.float32).view(np.uint32)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def widen(u):
    return (u.astype(np.uint32) << 16).view(np.float32)


def bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


@pytest.mark.parametrize("m,n,k", [(128, 128, 256), (37, 45, 70), (1, 1, 1), (5, 3, 1000), (64, 33, 0)])
def test_integer_inputs_give_exact_product(m, n, k):
    a = RNG.integers(-8, 9, (m, k))
    b = RNG.integers(-8, 9, (k, n))
    c = oracle.gemm(to_bf16(a.astype(np.float32)), to_bf16(b.astype(np.float32)))
    assert np.array_equal(c.astype(np.int64), a @ b)
    if k == 0:
        assert np.all(bits(c) == 0)  # empty sums are +0


def test_layouts_and_transpose_identity():
    a = I.normal_bf16((40, 300), 0, 1)
    b = I.normal_bf16((300, 24), 0, 2)
    c = oracle.gemm(a, b)
    assert np.array_equal(bits(c), bits(oracle.gemm(np.ascontiguousarray(a.T), b, trans_a=True)))
    assert np.array_equal(bits(c), bits(oracle.gemm(a, np.ascontiguousarray(b.T), trans_b=True)))
    assert np.array_equal(bits(c), bits(oracle.gemm(np.ascontiguousarray(a.T), np.ascontiguousarray(b.T), True, True)))
    # C^T = B^T A^T bit for bit (the K order is the same logical index)
    assert np.array_equal(bits(c.T), bits(oracle.gemm(np.ascontiguousarray(b.T), np.ascontiguousarray(a.T))))


def test_sign_and_power_of_two_scaling():
    a = I.normal_bf16((20, 200), 1, 1)
    b = I.normal_bf16((200, 30), 1, 2)
    c = oracle.gemm(a, b)
    assert np.array_equal(bits(-c), bits(oracle.gemm(a ^ np.uint16(0x8000), b)))
    a4 = to_bf16(widen(a) * np.float32(4.0))
    assert np.array_equal(bits(c * np.float32(4.0)), bits(oracle.gemm(a4, b)))


def test_each_element_is_the_canonical_dot_product():
    a = I.normal_bf16((8, 1572 * 32 - 9), 2, 1)
    b = I.normal_bf16((1572 * 32 - 9, 5), 2, 2)
    c = oracle.gemm(a, b)
    for i in range(8):
        for j in range(5):
            prods = widen(a[i]) * widen(b[:, j])  # exact in float32
            assert bits(c[i, j]) == bits(CF.canonical_sum(list(prods)))


def test_cfg1_error_bound_and_negative_control():
    # 128x256 . 256x128, bf16 N(0,1) with seed 0: 8 chunks of 32 per output
    a = I.normal_bf16((128, 256), 0, I.TENSOR_IDS["gemm_a"])
    b = I.normal_bf16((256, 128), 0, I.TENSOR_IDS["gemm_b"])
    c = oracle.gemm(a, b)
    af, bf = widen(a).astype(np.float64), widen(b).astype(np.float64)
    exact = af @ bf  # products are exact; the float64 sum of 256 of them is within 2^-40 relative
    u = 2.0 ** -24
    g = (31 + 3) * u / (1 - (31 + 3) * u)
    assert np.all(np.abs(c - exact) <= g * (np.abs(af) @ np.abs(bf)) + 1e-30)
    # a flat left-to-right chain over all 256 terms gives different bits for some outputs
    differ = 0
    for i in range(0, 128, 16):
        for j in range(0, 128, 16):
            s = np.float32(0)
            for kk in range(256):
                s = np.float32(s + np.float32(af[i, kk] * bf[kk, j]))
            differ += bits(s) != bits(c[i, j])
    assert differ > 0


@pytest.mark.parametrize("kind", ["wide", "tiny", "ties", "cancel"])
def test_adversarial_operands_match_exact_model(kind):
    # every output of a 6x7x70 product (three chunks, a ragged one) against the exact-rational R0 model of the
    # canonical dot product: subnormal products and partials, ties, cancellation and signed zeros
    import adversarial as ADV
    a, b = ADV.gemm_operands(kind, 6, 7, 70)
    c = oracle.gemm(a, b)
    af, bf = widen(a), widen(b)
    for i in range(6):
        for j in range(7):
            want = CF.canonical_dot_r0([float(x) for x in af[i]], [float(y) for y in bf[:, j]])
            assert bits(c[i, j]) == bits(want), (kind, i, j, c[i, j], want)


def test_adversarial_closed_forms():
    import adversarial as ADV
    # cancel: every product meets its negation next in the chain, so every partial and every output is +0
    a, b = ADV.gemm_operands("cancel", 9, 11, 2 * 32 * 3)
    assert np.all(bits(oracle.gemm(a, b)) == 0)
    # huge: same-signed products of at least 2^124 overflow inside the first chunk: +-inf by the column's sign
    a, b = ADV.gemm_operands("huge", 5, 8, 70)
    c = oracle.gemm(a, b)
    sign = np.where(b[0] >> 15, -1.0, 1.0).astype(np.float32)
    assert np.array_equal(bits(c), bits(np.broadcast_to(sign * np.float32(np.inf), c.shape)))
