"""The canonical functions of R4 (cexp, clog, sigmoid, silu, the SwiGLU forward and backward) evaluated as
their op sequences are written in the CANON-v1 rule text, in an R0 model independent of the oracle, and
compared with the oracle bit for bit.

The sequences are transcribed from the rule text (not from the oracle's source): a transposed Horner step,
a wrong constant, a dropped reduction term or another association gives other bits on some input.  The
vectorised model (`r0_vec`) is itself checked against the exact-rational model (`exact_r0`) on adversarial
operands, and the transcription is evaluated in the exact-rational model too on a few thousand inputs.
"""
import numpy as np
import pytest

import adversarial as ADV
import exact_r0 as X
import oracle
import r0_vec as V

RNG = np.random.default_rng(4242)

# constants as the rule text gives them
L2E, LN2_HI, LN2_LO = 0x3FB8AA3B, 0x3F317200, 0x35BFBE8E
EXP_C = [0x3F800000, 0x3F800000, 0x3F000000, 0x3E2AAAAB, 0x3D2AAAAB, 0x3C088889, 0x3AB60B61, 0x39500D01]
SQRT2 = 0x3FB504F3
INV_ODD = {3: 0x3EAAAAAB, 5: 0x3E4CCCCD, 7: 0x3E124925, 9: 0x3DE38E39, 11: 0x3DBA2E8C}


def c(bits):
    return V.f32(np.uint32(bits))


class ExactOps:
    """The exact-rational model, elementwise over arrays."""

    @staticmethod
    def _map(fn, *args):
        args = np.broadcast_arrays(*[np.asarray(a, np.float32) for a in args])
        out = np.empty(args[0].shape, np.float32)
        for idx in np.ndindex(out.shape):
            out[idx] = fn(*[a[idx] for a in args])
        return out

    add = staticmethod(lambda a, b: ExactOps._map(X.add, a, b))
    sub = staticmethod(lambda a, b: ExactOps._map(lambda x, y: X.add(x, -y), a, b))
    mul = staticmethod(lambda a, b: ExactOps._map(X.mul, a, b))
    div = staticmethod(lambda a, b: ExactOps._map(X.div, a, b))
    daz = staticmethod(lambda a: ExactOps._map(lambda x: np.float32(X.daz(float(x))), a))


def cexp_spec(x, ops):
    x = ops.daz(np.asarray(x, np.float32))
    t = ops.mul(x, c(L2E))
    with np.errstate(invalid="ignore"):
        k = np.rint(t).astype(np.float32)                     # nearest integer, ties to even
    big, small = k > 127, k < -125
    kk = np.where(big | small | ~np.isfinite(k), np.float32(0), k).astype(np.float32)
    r = ops.sub(ops.sub(x, ops.mul(kk, c(LN2_HI))), ops.mul(kk, c(LN2_LO)))
    p = np.full(x.shape, c(EXP_C[7]), np.float32)
    for i in range(6, -1, -1):
        p = ops.add(ops.mul(p, r), c(EXP_C[i]))
    scale = np.ldexp(np.float32(1.0), kk.astype(np.int32)).astype(np.float32)
    out = ops.mul(p, scale)
    out = np.where(big, np.float32(np.inf), out)
    out = np.where(small, np.float32(0.0), out)
    out = np.where(np.isnan(x), np.float32(np.nan), out)
    return out.astype(np.float32)


def clog_spec(x, ops):
    x = ops.daz(np.asarray(x, np.float32))
    special_ninf = x == 0
    special_nan = (x < 0) | np.isnan(x)
    special_inf = np.isposinf(x)
    ok = ~(special_ninf | special_nan | special_inf)
    xs = np.where(ok, x, np.float32(1.0)).astype(np.float32)
    u = xs.view(np.uint32)
    e = ((u >> 23) & 0xFF).astype(np.int64) - 127
    f = ((u & 0x7FFFFF) | 0x3F800000).astype(np.uint32).view(np.float32)
    hi = f > c(SQRT2)
    f = np.where(hi, ops.mul(f, np.float32(0.5)), f).astype(np.float32)
    e = e + hi
    one = np.float32(1.0)
    s = ops.div(ops.sub(f, one), ops.add(f, one))
    z = ops.mul(s, s)
    q = np.full(x.shape, c(INV_ODD[11]), np.float32)
    for j in (9, 7, 5, 3):
        q = ops.add(ops.mul(q, z), c(INV_ODD[j]))
    q = ops.add(ops.mul(q, z), one)
    lf = ops.mul(ops.add(s, s), q)
    E = e.astype(np.float32)
    out = ops.add(ops.mul(E, c(LN2_HI)), ops.add(ops.mul(E, c(LN2_LO)), lf))
    out = np.where(special_ninf, np.float32(-np.inf), out)
    out = np.where(special_nan, np.float32(np.nan), out)
    out = np.where(special_inf, np.float32(np.inf), out)
    return out.astype(np.float32)


def sigmoid_spec(x, ops):
    x = ops.daz(np.asarray(x, np.float32))
    return ops.div(np.float32(1.0), ops.add(np.float32(1.0), cexp_spec(-x, ops)))


def silu_spec(x, ops):
    return ops.mul(x, sigmoid_spec(x, ops))


def same_bits(a, b):
    a, b = np.asarray(a, np.float32), np.asarray(b, np.float32)
    both_nan = np.isnan(a) & np.isnan(b)
    return (a.view(np.uint32) == b.view(np.uint32)) | both_nan


def test_vector_model_matches_exact_model():
    A, B, C = ADV.triples()
    A, B = A[:3000], B[:3000]
    fin = np.isfinite(A) & np.isfinite(B)
    A, B = A[fin], B[fin]
    for name, vf, xf in [("add", V.add, X.add), ("mul", V.mul, X.mul)]:
        got = vf(A, B)
        want = np.array([xf(a, b) for a, b in zip(A, B)], np.float32)
        ok = same_bits(got, want) | ~np.isfinite(want)
        assert ok.all(), (name, A[~ok][:3], B[~ok][:3])
    keep = np.abs(B) >= 2.0 ** -126
    got = V.div(A[keep], B[keep])
    want = np.array([X.div(a, b) for a, b in zip(A[keep], B[keep])], np.float32)
    ok = same_bits(got, want) | ~np.isfinite(want)
    assert ok.all()


def exp_inputs(n):
    bitsr = RNG.integers(0, 1 << 32, n, dtype=np.uint64).astype(np.uint32)
    x = bitsr.view(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) < 110)]
    dense = RNG.uniform(-104.0, 89.0, n).astype(np.float32)
    # neighbourhoods of the points where k changes (t = k + 1/2) and of the range limits
    ks = np.arange(-130, 131, dtype=np.float64)
    mids = ((ks + 0.5) * np.log(2.0)).astype(np.float32)
    near = np.concatenate([mids + np.float32(d) * np.spacing(mids) for d in range(-40, 41)])
    special = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-40, -1e-40, 88.72, 88.73, -87.33, -87.34,
                        -86.64, -86.65], np.float32)
    return np.concatenate([x, dense, near, special]).astype(np.float32)


def log_inputs(n):
    bitsr = RNG.integers(0, 1 << 31, n, dtype=np.uint64).astype(np.uint32)  # every positive binade
    x = bitsr.view(np.float32)
    near1 = (1.0 + RNG.uniform(-0.3, 0.5, n)).astype(np.float32)
    s2 = c(SQRT2)
    around = np.concatenate([[s2 * np.float32(2.0 ** j)] for j in range(-126, 127)]).astype(np.float32)
    around = np.concatenate([np.nextafter(around, np.float32(0)), around, np.nextafter(around, np.float32(np.inf))])
    special = np.array([0.0, -0.0, -1.0, np.inf, -np.inf, np.nan, 1.0, 2.0, 0.5, 1e-40, 50304.0], np.float32)
    return np.concatenate([x, near1, around, special]).astype(np.float32)


def test_cexp_equals_rule_text():
    x = exp_inputs(1 << 21)
    got = oracle.prim("exp", x)
    want = cexp_spec(x, V)
    ok = same_bits(got, want)
    assert ok.all(), (x[~ok][:5], got[~ok][:5], want[~ok][:5])


def test_clog_equals_rule_text():
    x = log_inputs(1 << 21)
    got = oracle.prim("log", x)
    want = clog_spec(x, V)
    ok = same_bits(got, want)
    assert ok.all(), (x[~ok][:5], got[~ok][:5], want[~ok][:5])


def test_sigmoid_silu_equal_rule_text():
    x = np.concatenate([RNG.uniform(-100, 100, 1 << 20), RNG.standard_normal(1 << 18) * 4]).astype(np.float32)
    assert same_bits(oracle.prim("sigmoid", x), sigmoid_spec(x, V)).all()
    assert same_bits(oracle.prim("silu", x), silu_spec(x, V)).all()


def test_swiglu_equals_rule_text():
    n = 1 << 19
    g = (RNG.standard_normal(n) * 3).astype(np.float32)
    u = RNG.standard_normal(n).astype(np.float32)
    da = (RNG.standard_normal(n) * 1e-3).astype(np.float32)
    a, dg, du = oracle.swiglu(g, u, da)
    one = np.float32(1.0)
    sig = sigmoid_spec(g, V)
    assert np.array_equal(a, V.bf16_bits(V.mul(silu_spec(g, V), u)))
    assert np.array_equal(du, V.bf16_bits(V.mul(da, V.mul(g, sig))))
    dsg = V.mul(sig, V.add(one, V.mul(g, V.sub(one, sig))))
    assert np.array_equal(dg, V.bf16_bits(V.mul(V.mul(da, u), dsg)))
    # negative control: the other association of the gate gradient, RN(da RN(u dsg)), differs somewhere
    assert not np.array_equal(dg, V.bf16_bits(V.mul(da, V.mul(u, dsg))))


@pytest.mark.parametrize("fn,spec,gen", [("exp", cexp_spec, exp_inputs), ("log", clog_spec, log_inputs)])
def test_rule_text_in_exact_model(fn, spec, gen):
    x = gen(1 << 12)
    x = RNG.choice(x, 1500, replace=False)
    got = oracle.prim(fn, x)
    assert same_bits(got, spec(x, ExactOps)).all()


def test_transcription_detects_mutations():
    """A dropped low part of ln 2, a one-unit change of the 1/2! or 1/3! coefficient, or a different split of
    the clog tail changes the bits of the transcription on these inputs, so the comparisons above can see
    such mistakes."""
    global LN2_LO
    x = exp_inputs(1 << 16)
    want = oracle.prim("exp", x)
    saved = LN2_LO
    LN2_LO = 0
    try:
        assert not same_bits(want, cexp_spec(x, V)).all()
    finally:
        LN2_LO = saved
    for i in (2, 3):
        saved = EXP_C[i]
        EXP_C[i] = saved + 1
        try:
            assert not same_bits(want, cexp_spec(x, V)).all(), i
        finally:
            EXP_C[i] = saved
    y = log_inputs(1 << 16)
    wlog = oracle.prim("log", y)
    saved = INV_ODD[3]
    INV_ODD[3] = saved + 1
    try:
        assert not same_bits(wlog, clog_spec(y, V)).all()
    finally:
        INV_ODD[3] = saved
