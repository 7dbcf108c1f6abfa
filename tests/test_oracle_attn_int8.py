"""Pins for R17 (int8 P.V per block inside the attention forward) and R18 (dQ accumulated in 64-bit fixed
point), the two attention-kernel variants of the paper's training-details paragraph on int8 computation.

R17: an exact regime (every block's step a power of two, so codes, integer sums, dequantisation and the sum
over blocks are all exact) against exact rational products, with a different step in every block so that a
wrong block size breaks it; invariance under key permutations inside a block, and a negative control across
blocks; causality through whole blocks; a float64 error bound from the quantisation steps.
R18: the fixed-point value of single products against exact rational arithmetic (ties, signs, flushed
inputs, wrap modulo 2^64); the final rounding against the exact-rational R0 model; invariance of whole rows
under any key order (where the R2 GEMM changes bits); exact sums, closed-form wrap-around and vanishing
products; the window never reads masked entries; the float64 error bound.
"""
from fractions import Fraction as Fr

import numpy as np
import pytest

import exact_r0 as R
import oracle

RNG = np.random.default_rng(1717)


def bf16_of(vals) -> np.ndarray:
    """bf16 bit patterns of values that are exactly representable in bf16."""
    f = np.asarray(vals, np.float32)
    u = f.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value not representable in bf16"
    return (u >> 16).astype(np.uint16)


def widen(h) -> np.ndarray:
    return (np.asarray(h, np.uint16).astype(np.uint32) << 16).view(np.float32)


def bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def rand_bf16(shape, std=1.0, rng=RNG):
    x = (rng.standard_normal(shape) * std).astype(np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)  # truncation is fine for inputs


# ---------------------------------------------------------------------------------------------- R17
def exact_regime_inputs(S, hd, rng):
    """P: in tile (qb, kb) the entries are k * 2^-(7+e) with |k| <= 127 and one entry of magnitude
    127 * 2^-(7+e), e drawn per tile; V: in key block kb the entries are m * 2^-(3+f) with one of magnitude
    127 * 2^-(3+f).  Then each step is exactly 2^-(7+e) (resp. 2^-(3+f)): RN(127 * 2^-n * RN(1/127)) rounds
    1 - 2^-28 up to 1."""
    nb = (S + 63) // 64
    P = np.zeros((S, S), np.float64)
    V = np.zeros((S, hd), np.float64)
    ep = rng.integers(0, 6, (nb, nb))
    ev = rng.integers(0, 6, nb)
    for kb in range(nb):
        k0, k1 = 64 * kb, min(64 * kb + 64, S)
        m = rng.integers(-127, 128, (k1 - k0, hd)).astype(np.float64)
        m.flat[rng.integers(0, m.size)] = 127 * rng.choice([-1, 1])
        V[k0:k1] = m * 2.0 ** -(3 + ev[kb])
        for qb in range(nb):
            i0, i1 = 64 * qb, min(64 * qb + 64, S)
            k = rng.integers(-127, 128, (i1 - i0, k1 - k0)).astype(np.float64)
            k.flat[rng.integers(0, k.size)] = 127 * rng.choice([-1, 1])
            P[i0:i1, k0:k1] = k * 2.0 ** -(7 + ep[qb, kb])
    return bf16_of(P), bf16_of(V), P, V


@pytest.mark.parametrize("S,hd", [(128, 8), (100, 4), (192, 16), (64, 3)])
def test_pv_i8_exact_regime_equals_exact_product(S, hd):
    P16, V16, P, V = exact_regime_inputs(S, hd, np.random.default_rng(S * 31 + hd))
    O = oracle.attn_pv_i8(P16, V16)
    # every quantity is a multiple of 2^-20 below 2^14 in magnitude: the float64 product is exact
    want = (P @ V).astype(np.float32)
    assert np.array_equal(bits(O), bits(want))


def test_pv_i8_exact_regime_breaks_with_other_block_sizes():
    """The same inputs quantised with blocks of 32 or 128 keys would use other steps: check that the exact
    regime depends on the 64-block grid (the exact product is not reproduced when the tile exponents are
    shifted by half a block)."""
    S, hd = 192, 8
    P16, V16, P, V = exact_regime_inputs(S, hd, np.random.default_rng(5))
    shift = np.roll(np.arange(S), 32)  # keys moved by half a block, P columns and V rows together
    O = oracle.attn_pv_i8(np.ascontiguousarray(P16[:, shift]), np.ascontiguousarray(V16[shift]))
    want = (P[:, shift] @ V[shift]).astype(np.float32)
    assert not np.array_equal(bits(O), bits(want))


def test_pv_i8_invariant_under_key_permutation_inside_blocks():
    S, hd = 192, 16
    P16 = rand_bf16((S, S), 0.02)
    P16 &= 0x7FFF
    V16 = rand_bf16((S, hd))
    O = oracle.attn_pv_i8(P16, V16)
    perm = np.concatenate([64 * b + RNG.permutation(64) for b in range(3)])
    Op = oracle.attn_pv_i8(np.ascontiguousarray(P16[:, perm]), np.ascontiguousarray(V16[perm]))
    assert np.array_equal(bits(O), bits(Op))
    # negative control: exchanging keys between blocks changes the steps and the bits
    swap = np.arange(S)
    swap[[3, 70, 150]] = swap[[150, 3, 70]]
    Os = oracle.attn_pv_i8(np.ascontiguousarray(P16[:, swap]), np.ascontiguousarray(V16[swap]))
    assert not np.array_equal(bits(O), bits(Os))


def causal_probs(S, rng):
    raw = rng.standard_normal((S, S)).astype(np.float32)
    P = np.empty((S, S), np.uint16)
    oracle.lib().cref_softmax_causal(1, S, raw.ctypes.data, np.float32(0.3), P.ctypes.data)
    return P


def test_pv_i8_causal_blocks():
    """Query block 0 of a causal P sees key block 0 only: values of later keys cannot reach its rows, and a
    row whose P block is all +0 beyond the diagonal gets +0 terms."""
    S, hd = 192, 8
    P16 = causal_probs(S, RNG)
    V16 = rand_bf16((S, hd))
    O = oracle.attn_pv_i8(P16, V16)
    V2 = V16.copy()
    V2[64:] = rand_bf16((S - 64, hd))
    O2 = oracle.attn_pv_i8(P16, V2)
    assert np.array_equal(bits(O[:64]), bits(O2[:64]))
    assert not np.array_equal(bits(O[64:]), bits(O2[64:]))
    # row 0 is p = 1 on key 0 and +0 elsewhere: O[0] is V[0] up to its block's quantisation step
    V = widen(V16).astype(np.float64)
    sv = np.abs(V[:64]).max() / 127
    assert np.all(np.abs(O[0] - V[0]) <= sv / 2 * (1 + 2 ** -20) + np.abs(V[0]) * 2 ** -21)


def test_pv_i8_within_quantisation_bound():
    S, hd = 256, 16
    P16 = causal_probs(S, RNG)
    V16 = rand_bf16((S, hd))
    O = oracle.attn_pv_i8(P16, V16).astype(np.float64)
    P, V = widen(P16).astype(np.float64), widen(V16).astype(np.float64)
    exact = P @ V
    bound = np.zeros_like(exact)
    for kb in range(S // 64):
        ks = slice(64 * kb, 64 * kb + 64)
        sv = np.abs(V[ks]).max() / 127
        for qb in range(S // 64):
            qs = slice(64 * qb, 64 * qb + 64)
            sp = np.abs(P[qs, ks]).max() / 127
            # |p v - p^ v^| <= |p| sv/2 + sp/2 (|v| + sv/2), plus the two dequantisation roundings
            bound[qs] += (np.abs(P[qs, ks]) @ np.full((64, hd), sv / 2)
                          + np.full((64, 64), sp / 2) @ (np.abs(V[ks]) + sv / 2)) * (1 + 2 ** -22)
    bound += np.abs(exact) * 2 ** -20 + 1e-30
    assert np.all(np.abs(O - exact) <= bound)
    # and the quantisation error is the error of an int8 product: about 1% of the row scale, not 0
    assert np.abs(O - exact).max() > 0


# ---------------------------------------------------------------------------------------------- R18
def fx_exact(a16, b16, F):
    """the definition in exact rational arithmetic: nearest integer (ties to even) to a*b*2^F, mod 2^64"""
    a = R.daz(float(widen(a16)))
    b = R.daz(float(widen(b16)))
    x = Fr(a) * Fr(b) * Fr(2) ** F
    return round(x) % (1 << 64)  # Fraction.__round__ rounds half to even


def test_fx_product_against_exact_arithmetic():
    F = 40
    pats = list(rand_bf16((400,), 1.0)) + list(rand_bf16((200,), 1e-6)) + list(rand_bf16((200,), 1e5))
    pats += [0x0001, 0x8001, 0x007F, 0x0080, 0x8080, 0x3F80, 0xBF80, 0x0000, 0x8000, 0x7F7F, 0xFF7F]
    pats = np.array(pats, np.uint16)
    rng = np.random.default_rng(3)
    for _ in range(3000):
        a, b = int(rng.choice(pats)), int(rng.choice(pats))
        f = int(rng.choice([1, 13, 40, 62]))
        assert oracle.fx_product(a, b, f) == fx_exact(a, b, f), (hex(a), hex(b), f)


@pytest.mark.parametrize("F", [10, 40, 62])
def test_fx_product_ties_round_to_even(F):
    # 1.5 * 2^-F -> 2; 2.5 * 2^-F -> 2; 0.5 * 2^-F -> 0; -1.5 * 2^-F -> -2 (mod 2^64)
    def pat(v):
        return int(bf16_of([v])[0])
    for prod, want in [(1.5, 2), (2.5, 2), (0.5, 0), (-1.5, -2), (3.5, 4)]:
        a, b = pat(prod), pat(2.0 ** -F)
        assert oracle.fx_product(a, b, F) == want % (1 << 64)


def test_fx_to_f32_against_exact_r0():
    rng = np.random.default_rng(4)
    cases = [int(v) for v in rng.integers(-(1 << 63), (1 << 63) - 1, 500, dtype=np.int64)]
    cases += [int(v) for v in rng.integers(-(1 << 30), 1 << 30, 300)]
    cases += [1, -1, (1 << 24) + 1, (1 << 25) + 3, -(1 << 63), (1 << 63) - 1, 3 << 40, 0]
    for s in cases:
        for F in (1, 20, 40, 62):
            got = oracle.fx_to_f32(s, F)
            want = R.r0(Fr(s) / Fr(2) ** F) if s != 0 else np.float32(0.0)
            assert bits(got) == bits(want), (s, F)
    # flush: 2^-126 survives at F = 62 only as 2^64 ulps; a sum of 1 at F = 62 is 2^-62, a normal number
    assert oracle.fx_to_f32(1, 62) == np.float32(2.0 ** -62)


def brute_dq(dS16, K16, F, window=0):
    S, hd = K16.shape
    out = np.empty((S, hd), np.float32)
    for i in range(S):
        j0 = max(0, i - window + 1) if window else 0
        for c in range(hd):
            tot = sum(fx_exact(int(dS16[i, j]), int(K16[j, c]), F) for j in range(j0, i + 1)) % (1 << 64)
            s = tot - (1 << 64) if tot >= 1 << 63 else tot
            out[i, c] = R.r0(Fr(s) / Fr(2) ** F) if s else np.float32(0.0)
    return out


@pytest.mark.parametrize("S,hd,F,window", [(12, 3, 40, 0), (9, 2, 20, 4), (16, 2, 62, 0)])
def test_dq_fixed_brute_force(S, hd, F, window):
    dS16 = rand_bf16((S, S), 1e-3)
    K16 = rand_bf16((S, hd), 1.0)
    got = oracle.attn_dq_fixed(dS16, K16, F, window)
    assert np.array_equal(bits(got), bits(brute_dq(dS16, K16, F, window)))


def test_dq_fixed_row_is_invariant_under_key_order():
    """The last query sees every key: any order of the keys gives the same fixed-point row, while the R2
    GEMM's chained fp32 order changes bits."""
    S, hd = 256, 16
    dS16 = rand_bf16((S, S), 1e-2)
    K16 = rand_bf16((S, hd), 1.0)
    last = oracle.attn_dq_fixed(dS16, K16, 40)[S - 1]
    changed = False
    for seed in range(3):
        perm = np.random.default_rng(seed).permutation(S)
        dSp = dS16.copy()
        dSp[S - 1] = dS16[S - 1, perm]
        got = oracle.attn_dq_fixed(dSp, np.ascontiguousarray(K16[perm]), 40)[S - 1]
        assert np.array_equal(bits(got), bits(last))
        g0 = oracle.gemm(dS16[S - 1:], K16)
        g1 = oracle.gemm(np.ascontiguousarray(dSp[S - 1:]), np.ascontiguousarray(K16[perm]))
        changed |= not np.array_equal(bits(g0), bits(g1))
    assert changed


def test_dq_fixed_exact_sums():
    # dS = a * 2^-10, K = b * 2^-2 with small integers: every product and sum is exact at F = 40
    S, hd = 96, 8
    a = RNG.integers(-100, 101, (S, S)).astype(np.float64)
    b = RNG.integers(-100, 101, (S, hd)).astype(np.float64)
    dS, K = a * 2.0 ** -10, b * 2.0 ** -2
    got = oracle.attn_dq_fixed(bf16_of(dS), bf16_of(K), 40)
    want = (np.tril(dS) @ K).astype(np.float32)  # exact in float64, then rounded once
    assert np.array_equal(bits(got), bits(want))


def test_dq_fixed_wraps_modulo_2_64_and_small_products_vanish():
    # at F = 62 a product of 2 is 2^63, which wraps to -2^63: one such term reads -2, two of them 0
    S = 3
    dS = np.zeros((S, S), np.float32)
    dS[1, :2] = 1.0
    dS[2, :1] = 1.0
    K = np.full((S, 1), 2.0, np.float32)
    got = oracle.attn_dq_fixed(bf16_of(dS), bf16_of(K), 62)[:, 0]
    assert got[2] == np.float32(-2.0) and got[1] == 0.0 and got[0] == 0.0
    # products below half a unit of 2^-F vanish; exactly half rounds to the even 0
    dS = np.zeros((2, 2), np.float32)
    dS[1, 0] = 2.0 ** -41
    dS[1, 1] = 2.0 ** -42
    got = oracle.attn_dq_fixed(bf16_of(dS), bf16_of(np.ones((2, 1), np.float32)), 40)
    assert got[1, 0] == 0.0


def test_dq_fixed_window_reads_no_masked_entry():
    S, hd, W = 64, 4, 9
    dS16 = rand_bf16((S, S), 1e-2)
    K16 = rand_bf16((S, hd))
    i, j = np.indices((S, S))
    seen = (j <= i) & (j > i - W)
    clean = np.where(seen, dS16, 0).astype(np.uint16)
    garbage = np.where(seen, dS16, rand_bf16((S, S), 1e3)).astype(np.uint16)
    a = oracle.attn_dq_fixed(clean, K16, 40, W)
    assert np.array_equal(bits(a), bits(oracle.attn_dq_fixed(garbage, K16, 40, W)))
    # and with every entry outside the window zero, the windowed result is the causal one
    assert np.array_equal(bits(a), bits(oracle.attn_dq_fixed(clean, K16, 40, 0)))


def test_dq_fixed_within_float64_bound():
    S, hd, F = 128, 16, 40
    dS16 = rand_bf16((S, S), 1e-3)
    K16 = rand_bf16((S, hd))
    got = oracle.attn_dq_fixed(dS16, K16, F).astype(np.float64)
    exact = np.tril(widen(dS16).astype(np.float64)) @ widen(K16).astype(np.float64)
    n = np.arange(1, S + 1)[:, None]
    assert np.all(np.abs(got - exact) <= n * 2.0 ** -(F + 1) + np.abs(exact) * 2 ** -24 * 1.0001)


# ---------------------------------------------------------------------------------------------- in the block
import paper_2609_17380_amd.inputs as I  # noqa: E402


def block_case(pv, dq, Hkv=0, qk=0, win=0, S=80):
    d, H, F, B = 64, 2, 96, 2
    hd = d // H
    cfg = oracle.ModelCfg(1, d, H, hd, F, 97, S, B, np.float32(1e-5), Hkv, qk, 0, win, 0, np.float32(0), pv, dq)
    kvw = (Hkv or H) * hd
    shapes = [(d,), (d + 2 * kvw, d), (d, d), (d,), (2 * F, d), (d, F)]
    w = [I.normal_bf16(s, 3, 900 + i, std=0.1, mean=1.0) if len(s) == 1 else I.normal_bf16(s, 3, 900 + i, std=0.08)
         for i, s in enumerate(shapes)]
    x = I.bf16_bits_to_f32(I.normal_bf16((B * S, d), 1, I.TENSOR_IDS["x_in"]))
    dy = I.bf16_bits_to_f32(I.normal_bf16((B * S, d), 1, I.TENSOR_IDS["dy_in"]))
    cos, sin = I.rope_tables(S, hd)
    return oracle.block_fwd_bwd(cfg, B, x, dy, w, cos, sin), d, kvw


def relerr(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.mark.parametrize("Hkv,qk,win", [(0, 0, 0), (1, 1, 20)])
def test_block_fixed_point_dq_changes_only_the_query_path(Hkv, qk, win):
    """R18 replaces only the dQ contraction: the forward and every gradient that does not flow through dQ
    (W_o, the MLP, the key and value rows of W_qkv) are bit-identical to the plain block; the rest stays
    within the fixed-point resolution of it, and a coarse grid (F = 12) visibly loses small products."""
    (y0, dx0, dw0), d, kvw = block_case(0, 0, Hkv, qk, win)
    (y1, dx1, dw1), _, _ = block_case(0, 40, Hkv, qk, win)
    assert np.array_equal(bits(y0), bits(y1))
    for i in (2, 3, 4, 5):
        assert np.array_equal(bits(dw0[i]), bits(dw1[i]))
    assert np.array_equal(bits(dw0[1][d:]), bits(dw1[1][d:]))
    # dQ is rounded to bf16 before the weight gradient: at F = 40 the fixed-point and the chained fp32 dQ
    # almost always round alike
    assert relerr(dw1[1][:d], dw0[1][:d]) < 1e-5
    assert relerr(dx1, dx0) < 1e-5
    # a coarse grid loses the small products: F = 12 is far from the fp32 contraction
    (_, _, dw2), _, _ = block_case(0, 12, Hkv, qk, win)
    assert relerr(dw2[1][:d], dw0[1][:d]) > 1e-3


@pytest.mark.parametrize("Hkv,qk,win", [(0, 0, 0), (1, 1, 20)])
def test_block_int8_pv_is_a_quantised_forward(Hkv, qk, win):
    """R17 changes O (an int8 product per block) and hence everything after it; the block stays within the
    int8 quantisation error of the plain block, and the backward is the unquantised one (straight-through):
    the MLP weight gradients move only through the changed activations."""
    (y0, dx0, dw0), d, _ = block_case(0, 0, Hkv, qk, win)
    (y1, dx1, dw1), _, _ = block_case(1, 0, Hkv, qk, win)
    assert not np.array_equal(bits(y0), bits(y1))
    assert relerr(y1, y0) < 2e-2
    assert relerr(dx1, dx0) < 5e-2
    for i in range(6):
        assert relerr(dw1[i], dw0[i]) < 1e-1, i
