"""Pins for the oracle's R0 primitives and R4 functions.

R0 (IEEE-754 binary32, round to nearest even, flush of subnormals with the
tininess-after-rounding test) is checked element by element against an exact
rational model on random and adversarial inputs; the R4 constants against their
mathematical definitions; cexp and clog against libm within a stated bound.
"""
import math
import os
import re
from decimal import Decimal, getcontext
from fractions import Fraction as F

import numpy as np
import pytest

import adversarial as ADV
import exact_r0 as X
import oracle

RNG = np.random.default_rng(12345)


def f32_from_bits(u):
    return np.asarray(u, dtype=np.uint32).view(np.float32)


def random_floats(n, exp_lo=0, exp_hi=254):
    return ADV.random_floats(RNG, n, exp_lo, exp_hi)


def bits(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


A, B, C = ADV.triples()


@pytest.mark.parametrize("op", ["add", "sub", "mul", "fma", "div"])
def test_r0_ops_match_exact_rational(op):
    if op == "div":
        keep = np.abs(B) >= np.float32(2.0 ** -126)
        a, b, c = A[keep], B[keep], C[keep]
    else:
        a, b, c = A, B, C
    got = oracle.prim(op, a, b, c)
    want = np.empty_like(got)
    for i in range(a.size):
        if op == "add":
            want[i] = X.add(a[i], b[i])
        elif op == "sub":
            want[i] = X.add(a[i], -b[i])
        elif op == "mul":
            want[i] = X.mul(a[i], b[i])
        elif op == "fma":
            want[i] = X.fma(a[i], b[i], c[i])
        else:
            want[i] = X.div(a[i], b[i])
    finite = np.isfinite(want)
    bad = np.nonzero((bits(got) != bits(want)) & finite)[0]
    assert bad.size == 0, f"{op}: {bad.size} mismatches, first {a[bad[:3]]} {b[bad[:3]]} {got[bad[:3]]} {want[bad[:3]]}"


def test_r0_sqrt_correctly_rounded():
    x = np.abs(np.concatenate([random_floats(4000, 0, 254), random_floats(2000, 120, 135)]))
    r = oracle.prim("sqrt", x)
    for xi, ri in zip(x, r):
        assert X.sqrt_is_correctly_rounded(float(xi), float(ri)), (xi, ri)


def test_bf16_round_to_nearest_even():
    x = np.concatenate([random_floats(5000, 1, 253),
                        f32_from_bits((RNG.integers(0, 1 << 15, 2000, dtype=np.uint32) << 16) | 0x8000),  # ties
                        f32_from_bits(RNG.integers(0, 1 << 23, 200, dtype=np.uint32))])                      # subnormals
    x = x[np.isfinite(x)]
    got = oracle.prim("bf16", x)
    want = np.array([X.bf16(v) for v in x], np.float32)
    assert np.array_equal(bits(got), bits(want))


def _consts_from_source():
    src = open(os.path.join(os.path.dirname(oracle.__file__), "canon_ref.c")).read()
    def grab(name):
        return [int(h[:-1], 16) for h in re.findall(r"0x[0-9A-Fa-f]{8}u", src.split(name, 1)[1].split(";", 1)[0])]
    return {n: grab(n) for n in ("EXP_L2E", "EXP_LN2_HI", "EXP_LN2_LO", "EXP_C[8]", "LOG_SQRT2", "LOG_INV[5]",
                                 "ATTN_SCALE_128")}


def _rn32_bits(fr: F) -> int:
    return int(np.float32(float(X.round24(fr))).view(np.uint32))


def test_r4_constants_are_rn32_of_their_definitions():
    getcontext().prec = 60
    ln2 = F(Decimal(2).ln())
    k = _consts_from_source()
    assert k["EXP_L2E"] == [_rn32_bits(1 / ln2)]
    hi = k["EXP_LN2_HI"][0]
    hi_val = F(float(f32_from_bits(hi)))
    assert abs(hi_val - ln2) < F(1, 2 ** 16) and (hi & 0x1FF) == 0  # <= 15 significant bits: k*hi exact
    assert k["EXP_LN2_LO"] == [_rn32_bits(ln2 - hi_val)]
    assert k["EXP_C[8]"] == [_rn32_bits(F(1, math.factorial(n))) for n in range(8)]
    assert k["LOG_SQRT2"] == [_rn32_bits(F(Decimal(2).sqrt()))]
    assert k["LOG_INV[5]"] == [_rn32_bits(F(1, j)) for j in (3, 5, 7, 9, 11)]
    assert k["ATTN_SCALE_128"] == [_rn32_bits(1 / F(Decimal(128).sqrt()))]


def ulp_err(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.abs(got - ref) / np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)


def test_cexp_special_values_and_accuracy():
    sp = oracle.prim("exp", np.array([0.0, -0.0, 1.0, -1.0], np.float32))
    assert bits(sp)[0] == 0x3F800000 and bits(sp)[1] == 0x3F800000  # cexp(+-0) = 1 exactly
    x = np.concatenate([np.linspace(-86.5, 0, 200001, dtype=np.float32), random_floats(20000, 100, 132)])
    x = x[(x > -86.5) & (x < 88.0)]
    got = oracle.prim("exp", x)
    err = ulp_err(got, np.exp(x.astype(np.float64)))
    assert err.max() <= 3.0, err.max()
    assert oracle.prim("exp", np.array([-100.0, -90.0], np.float32)).tolist() == [0.0, 0.0]
    assert np.isinf(oracle.prim("exp", np.array([89.0], np.float32))[0])
    # monotone (non-decreasing) along a dense increasing grid
    g = np.linspace(-20, 20, 400001, dtype=np.float32)
    assert np.all(np.diff(oracle.prim("exp", g)) >= 0)


def test_clog_accuracy():
    assert oracle.prim("log", np.array([1.0], np.float32))[0] == 0.0
    x = np.concatenate([np.linspace(1, 1e5, 200001, dtype=np.float32), random_floats(20000, 1, 254)])
    x = x[np.isfinite(x) & (x > 0)]
    got = oracle.prim("log", x)
    ref = np.log(x.astype(np.float64))
    nz = np.abs(ref) > 1e-3
    assert ulp_err(got[nz], ref[nz]).max() <= 3.0
    assert np.max(np.abs(got[~nz] - ref[~nz])) < 1e-9


def test_sigmoid_silu_accuracy():
    x = np.linspace(-30, 30, 100001, dtype=np.float32)
    s = oracle.prim("sigmoid", x).astype(np.float64)
    ref = 1 / (1 + np.exp(-x.astype(np.float64)))
    assert np.max(np.abs(s - ref) / ref) < 5e-7
    si = oracle.prim("silu", x).astype(np.float64)
    ref_si = x * ref
    assert np.max(np.abs(si - ref_si) / np.maximum(np.abs(ref_si), 1e-30)) < 1e-6
