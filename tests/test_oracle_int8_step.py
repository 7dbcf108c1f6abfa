"""Pins for R19, the int8 projections inside the block and the step (the paper's W8A8 quantisation-aware
training): the LSQ gradient of an activation step against exact rational arithmetic (ties to even, the clamp
bounds, flushed and non-positive steps) and closed forms; blocks and full steps with int8 projections against
a float64 autograd model of LSQ fake quantisation with straight-through gradients (``torch_model_ref.qlinear``,
independent of the oracle); the step's declared order (activation steps after each layer's weights, no
weight decay) through AdamW of the reduced gradient."""
import math
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

import exact_r0 as R0
import oracle
import paper_2609_17380_amd.inputs as I
import torch_model_ref as R

NAMES = ["attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down", "sx_qkv", "sx_o", "sx_gate_up", "sx_down"]


def bits(x):
    return np.atleast_1d(np.asarray(x, np.float32)).view(np.uint32)


def bf16_of(vals):
    u = np.asarray(vals, np.float32).view(np.uint32)
    assert np.all((u & 0xFFFF) == 0)
    return (u >> 16).astype(np.uint16)


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def gamma(K):
    return np.float32(1.0 / math.sqrt(127.0 * K))


def exact_lsq(x16, s, dx):
    """the definition with exact rationals: delta from the correctly rounded quotient, then one rounding of
    each product, the R1 sum is exact here (the test keeps every partial sum exactly representable)"""
    tot = Fr(0)
    for xv, g in zip(x16.ravel(), dx.ravel()):
        x = float((np.uint32(xv) << 16).view(np.float32))
        v = float(R0.div(np.float32(x), np.float32(s)))
        if v < -128:
            dl = -128.0
        elif v > 127:
            dl = 127.0
        else:
            dl = float(round(Fr(v))) - v  # Fraction rounds half to even
        tot += Fr(float(R0.mul(np.float32(g), np.float32(dl))))
    return R0.mul(np.float32(float(tot)), gamma(x16.shape[1]))


def test_lsq_grad_zero_on_the_grid():
    """Activations on the integer grid of the step have delta = 0 (round(v) - v = 0): the gradient is +0."""
    rng = np.random.default_rng(0)
    s = np.float32(0.125)
    x = bf16_of(rng.integers(-128, 128, (16, 48)).astype(np.float32) * s)
    dx = rng.standard_normal((16, 48)).astype(np.float32)
    g = oracle.lsq_step_grad(x, s, dx)
    assert bits(g)[0] == 0


@pytest.mark.parametrize("T,K", [(8, 40), (3, 96), (32, 64)])
def test_lsq_grad_exact_regime(T, K):
    """s = 2^-3 and x = m 2^-5 (v = m / 4: ties at every odd half) with some x beyond the clamp bounds, small
    integer upstream gradients: every delta and product is exact and every partial sum representable, so the
    result is the exact sum times RN32(1/sqrt(127 K)), rounded once."""
    rng = np.random.default_rng(T * K)
    s = np.float32(0.125)
    m = rng.integers(-255, 256, (T, K))  # 8-bit integers: x = m / 32 is a bf16 value
    m[0, :4] = [2000, -2000, 508, -516]  # v = 500, -500 (clamped), 127 (in range), -129 (below -128)
    x = bf16_of(m.astype(np.float32) / 32)
    dx = rng.integers(-9, 10, (T, K)).astype(np.float32)
    got = oracle.lsq_step_grad(x, s, dx)
    assert bits(got)[0] == bits(exact_lsq(x, s, dx))[0]


def test_lsq_grad_ties_round_to_even():
    """v = 2.5 rounds to 2 (delta -0.5), v = 3.5 to 4 (delta +0.5): with dx = 1 the two cancel exactly, while
    rounding half away from zero would leave +1 and truncation -1 (times the gradient scale)."""
    s = np.float32(1.0)
    x = bf16_of(np.array([[2.5, 3.5]], np.float32))
    dx = np.ones((1, 2), np.float32)
    assert bits(oracle.lsq_step_grad(x, s, dx))[0] == 0
    x = bf16_of(np.array([[2.5, 2.5]], np.float32))  # two ties to even: delta -0.5 each
    want = R0.mul(np.float32(-1.0), gamma(2))
    assert bits(oracle.lsq_step_grad(x, s, dx))[0] == bits(want)[0]


def test_lsq_grad_bounds_and_degenerate_steps():
    s = np.float32(0.5)
    x = bf16_of(np.array([[100.0, -100.0, 63.5, -64.5]], np.float32))  # v = 200, -200, 127, -129
    dx = np.array([[1.0, 1.0, 4.0, 2.0]], np.float32)
    # deltas 127, -128, 0, -128 (v < -128 takes the lower bound)
    want = R0.mul(np.float32(127 - 128 + 0 - 256), gamma(4))
    assert bits(oracle.lsq_step_grad(x, s, dx))[0] == bits(want)[0]
    for bad in (0.0, -0.5, 2.0 ** -130):  # a step that is not > 0 once flushed has no gradient
        assert bits(oracle.lsq_step_grad(x, np.float32(bad), dx))[0] == 0


def block_case(cfg, B, seed=3):
    d, F = cfg.d_model, cfg.d_ffn
    H, hd = cfg.n_heads, cfg.head_dim
    kvw = (cfg.n_kv_heads or H) * hd
    shapes = [(d,), (d + 2 * kvw, d), (d, d), (d,), (2 * F, d), (d, F)]
    w = [I.normal_bf16(s, seed, 900 + i, std=0.1, mean=1.0) if len(s) == 1 else
         I.normal_bf16(s, seed, 900 + i, std=0.05) for i, s in enumerate(shapes)]
    w += [np.array([I.bf16_pattern(v)], np.uint16) for v in I.ACT_STEPS.values()]
    T = B * cfg.seq
    x = I.bf16_bits_to_f32(I.normal_bf16((T, d), seed, I.TENSOR_IDS["x_in"]))
    dy = I.bf16_bits_to_f32(I.normal_bf16((T, d), seed, I.TENSOR_IDS["dy_in"]))
    return w, x, dy


@pytest.mark.parametrize("Hkv,qk,win", [(0, 0, 0), (1, 1, 40)])
def test_block_int8_projections_match_float64_qat(Hkv, qk, win):
    """The int8 block against the float64 LSQ fake-quantisation model: the forward to float rounding (both
    quantise the same bf16 operands with the same steps), the gradients within the error of R14's rotated
    int8 backward (a few per cent), the activation steps' gradients within 30% (sums of products of both
    signs)."""
    d, H, F, S, B = 256, 2, 256, 128, 2
    hd = d // H
    cfg = oracle.ModelCfg(1, d, H, hd, F, 97, S, B, np.float32(1e-5), Hkv, qk, 0, win, 0, np.float32(0), 0, 0, 1)
    w, x, dy = block_case(cfg, B)
    cos, sin = I.rope_tables(S, hd)
    y, dx, dw = oracle.block_fwd_bwd(cfg, B, x, dy, w, cos, sin)
    xt = torch.tensor(x, dtype=R.DT, requires_grad=True)
    wt = {n: R.bf16_tensor(t, requires_grad=True) for n, t in zip(NAMES, w)}
    scale = float(np.float32(1 / math.sqrt(hd)))
    yt = R.block(xt, wt, B, S, H, hd, F, float(np.float32(1e-5)), torch.tensor(cos, dtype=R.DT),
                 torch.tensor(sin, dtype=R.DT), scale, Hkv=Hkv or None, qk_norm=bool(qk), window=win, int8=True)
    yt.backward(torch.tensor(dy, dtype=R.DT))
    assert rel(y, yt.detach().numpy()) < 1e-5
    assert rel(dx, xt.grad.numpy()) < 5e-2
    for n, g in zip(NAMES[:6], dw[:6]):
        assert rel(g, wt[n].grad.numpy()) < 1e-1, n
    for n, g in zip(NAMES[6:], dw[6:]):
        assert rel(g, wt[n].grad.numpy()) < 0.3, n
    # the plain block differs: the int8 projections are really in use
    cfg0 = oracle.ModelCfg(1, d, H, hd, F, 97, S, B, np.float32(1e-5), Hkv, qk, 0, win, 0, np.float32(0), 0, 0, 0)
    y0, _, _ = oracle.block_fwd_bwd(cfg0, B, x, dy, w[:6], cos, sin)
    assert rel(y0, y) > 1e-4


def test_step_int8_projections_match_float64_and_declared_order():
    L, d, H, F, V, S, mb = 2, 256, 2, 256, 97, 128, 2
    hd = d // H
    cfg = oracle.ModelCfg(L, d, H, hd, F, V, S, mb, np.float32(1e-5), 1, 1, 1, 48, 2, np.float32(1e-4), 0, 0, 1)
    plan = oracle.Plan(1, 2, 1)
    R_ = 2
    params = I.model_params(L, d, F, V, seed=9, std=0.05, kv_dim=hd, embed_norm=True, int8_linear=True)
    windows = I.uniform_int((R_ * mb, S + 1), 9, I.TENSOR_IDS["windows"], V)
    cos, sin = I.rope_tables(S, hd)
    k = oracle.AdamWConsts(*I.adamw_constants())
    p_or = [p.copy() for p in params]
    m = [np.zeros(p.shape, np.float32) for p in params]
    v = [np.zeros(p.shape, np.float32) for p in params]
    loss, grads = oracle.step(cfg, plan, p_or, m, v, windows, cos, sin, k, want_grads=True)
    pt = [R.bf16_tensor(p, requires_grad=True) for p in params]
    tcfg = dict(d=d, H=H, hd=hd, F=F, L=L, eps=float(np.float32(1e-5)), Hkv=1, qk_norm=True, embed_norm=True,
                swa_window=48, swa_full_every=2, z_loss=float(np.float32(1e-4)), int8_linear=True)
    scale = float(np.float32(1 / math.sqrt(hd)))
    tot = 0
    for r in range(R_):
        tok = torch.tensor(windows[[r + R_ * s for s in range(mb)]], dtype=torch.long)
        tot = tot + R.model_loss(pt, tok, tcfg, torch.tensor(cos, dtype=R.DT), torch.tensor(sin, dtype=R.DT),
                                 scale) / R_
    tot.backward()
    # a code that rounds the other way in fp32 and in float64 (RN32(x/s) at a rounding boundary) moves the loss
    assert abs(float(loss) - float(tot.detach())) < 5e-4 * abs(float(tot.detach()))
    names = [n for n, _, _, _ in I.model_param_shapes(L, d, F, V, hd, True, True)]
    for n, g, p in zip(names, grads, pt):
        if ".sx_" not in n:
            assert rel(g, p.grad.numpy()) < 1e-1, n
    # an activation step's gradient is a sum of 10^4-10^5 terms of both signs: the few per cent error of the
    # rotated int8 backward in each term leaves an absolute error, checked against the size of these
    # gradients across the model (a wrong sign, bound or gradient scale is off by far more)
    sx = [(g[0], float(p.grad.numpy()[0])) for n, g, p in zip(names, grads, pt) if ".sx_" in n]
    rms = math.sqrt(sum(r * r for _, r in sx) / len(sx))
    for got, ref in sx:
        assert abs(float(got) - ref) < 0.5 * rms, (got, ref, rms)
    # post-step parameters are AdamW of the reduced gradient, activation steps without weight decay
    p2 = [p.copy() for p in params]
    m2 = [np.zeros(p.shape, np.float32) for p in params]
    v2 = [np.zeros(p.shape, np.float32) for p in params]
    decay = [t[3] for t in I.model_param_shapes(L, d, F, V, hd, True, True)]
    assert sum(decay) == 4 * L + 1 and len(decay) == 3 + 10 * L + 1
    oracle.adamw(p2, m2, v2, grads, decay, k)
    for a, b in zip(p_or, p2):
        assert np.array_equal(a, b)
    assert any(not np.array_equal(a, b) for a, b in zip(p_or[8:12], params[8:12]))  # steps moved
