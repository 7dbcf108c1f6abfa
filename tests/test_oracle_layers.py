"""Pins for RMSNorm (R3), causal softmax (R5), cross-entropy (R6) and AdamW (R9) in the oracle."""
import math

import numpy as np
import pytest
import torch

import exact_r0 as X
import oracle
import paper_2609_17380_amd.inputs as I

RNG = np.random.default_rng(99)


def to_bf16(x):
    u = np.asarray(x, np.float32).view(np.uint32)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def widen(u):
    return (u.astype(np.uint32) << 16).view(np.float32)


def bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def test_rmsnorm_constant_rows_closed_form():
    # rows of +-2^e with eps = 0: mean square = 2^2e, rstd = 2^-e exactly, y = sign * g exactly
    cols = 96
    e = RNG.integers(-20, 20, 16)
    x = (np.exp2(e)[:, None] * RNG.choice([-1, 1], (16, 1)) * np.ones((16, cols))).astype(np.float32)
    g = to_bf16(RNG.standard_normal(cols).astype(np.float32))
    y, rstd = oracle.rownorm_fwd(x, g, 0.0)
    assert np.array_equal(rstd, np.exp2(-e).astype(np.float32))
    assert np.array_equal(widen(y), (np.sign(x) * widen(g)[None, :]).astype(np.float32))


def test_rmsnorm_matches_float64_autograd():
    rows, cols, eps = 64, 2048 + 96, 1e-5
    x = (RNG.standard_normal((rows, cols)) * 3).astype(np.float32)
    g = to_bf16((1 + 0.1 * RNG.standard_normal(cols)).astype(np.float32))
    dy = RNG.standard_normal((rows, cols)).astype(np.float32)
    y, rstd = oracle.rownorm_fwd(x, g, np.float32(eps))
    dx, dg = oracle.rownorm_bwd(x, g, rstd, dy)
    xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    gt = torch.tensor(widen(g), dtype=torch.float64, requires_grad=True)
    r = torch.rsqrt((xt * xt).mean(dim=1, keepdim=True) + float(np.float32(eps)))
    yt = xt * r * gt
    yt.backward(torch.tensor(dy, dtype=torch.float64))
    assert rel(rstd, r.detach().numpy()[:, 0]) < 1e-6
    assert np.max(np.abs(widen(y) - yt.detach().numpy()) / (np.abs(yt.detach().numpy()) + 1e-6)) < 2 ** -7
    assert rel(dx, xt.grad.numpy()) < 1e-5
    assert rel(dg, gt.grad.numpy()) < 1e-5


def test_softmax_uniform_rows_are_exact_powers_of_two():
    s = 64
    raw = np.full((1, s, s), 0.75, np.float32)
    p = widen(oracle.softmax_causal(raw, 1.0))[0]
    for i in range(s):
        n = i + 1
        if n & (n - 1) == 0:
            assert np.all(p[i, :n] == np.float32(1.0 / n))
        assert np.all(bits(p[i, n:]) == 0)  # masked keys are +0


def test_softmax_matches_float64():
    s = 200
    raw = RNG.standard_normal((3, s, s)).astype(np.float32) * 4
    c = np.float32(1 / math.sqrt(128))
    p = widen(oracle.softmax_causal(raw, c))
    sc = raw.astype(np.float64) * float(c)
    mask = np.tril(np.ones((s, s), bool))
    sc = np.where(mask, sc, -np.inf)
    ref = np.exp(sc - sc.max(-1, keepdims=True))
    ref /= ref.sum(-1, keepdims=True)
    assert np.max(np.abs(p - ref)) < 2 ** -8
    assert np.max(np.abs(p.astype(np.float64).sum(-1) - 1)) < 0.02


def test_xent_uniform_logits_closed_form():
    V, T = 50304, 4
    logits = np.zeros((T, V), np.uint16)
    tgt = np.array([0, 7, 50303, 1234], np.int32)
    dl, rl, ml = oracle.xent(logits, tgt, np.float32(1 / T))
    clog_v = oracle.prim("log", np.array([V], np.float32))[0]
    assert np.all(bits(rl) == bits(clog_v)) and abs(float(clog_v) - math.log(V)) < 2e-6
    # S = V exactly (sums of ones), p = RN32(1/V); off-target d = bf16(p/4); target d = bf16(RN(RN(p - 1)/4))
    p = X.div(1.0, float(V))
    off = X.bf16(X.mul(p, 0.25))
    on = X.bf16(X.mul(X.add(p, -1.0), 0.25))
    d = widen(dl)
    want = np.full((T, V), off, np.float32)
    want[np.arange(T), tgt] = on
    assert np.array_equal(bits(d), bits(want))


def test_xent_matches_float64():
    T, V = 16, 50304
    logits = I.normal_bf16((T, V), 0, I.TENSOR_IDS["logits"], std=2.0)
    tgt = I.uniform_int((T,), 0, I.TENSOR_IDS["targets"], V)
    invT = np.float32(1 / T)
    dl, rl, ml = oracle.xent(logits, tgt, invT)
    lt = torch.tensor(widen(logits), dtype=torch.float64, requires_grad=True)
    loss = torch.nn.functional.cross_entropy(lt, torch.tensor(tgt, dtype=torch.long), reduction="none")
    loss.mean().backward()
    assert np.max(np.abs(rl - loss.detach().numpy())) < 1e-5
    assert abs(float(ml) - float(loss.mean())) < 1e-5
    ref = lt.grad.numpy()
    assert np.max(np.abs(widen(dl) - ref) / (np.abs(ref) + 1e-12)) < 2 ** -7


def adamw_consts(lr=3e-4, b1=0.9, b2=0.95, eps=1e-8, wd=0.1, t=1):
    return oracle.AdamWConsts(lr, b1, 1 - b1, b2, 1 - b2, 1 / (1 - b1 ** t), 1 / (1 - b2 ** t), eps, 1 - lr * wd)


def test_adamw_first_step_closed_form_and_decay_mask():
    n = 10000
    p0 = I.normal_bf16((n,), 0, I.TENSOR_IDS["adam_p"], std=0.02)
    g = (I.normal_f32((n,), 0, I.TENSOR_IDS["adam_g"]) * 1e-3).astype(np.float32)
    k = adamw_consts()
    outs = []
    for decay in (1, 0):
        p = p0.copy(); m = np.zeros(n, np.float32); v = np.zeros(n, np.float32)
        oracle.adamw([p], [m], [v], [g], [decay], k)
        outs.append(p)
        # t = 1, m = v = 0: the update is lr * g / (|g| + eps) ~ lr * sign(g)
        ref = widen(p0).astype(np.float64) * (1 - 3e-4 * 0.1 if decay else 1.0) - 3e-4 * g / (np.abs(g) + 1e-8)
        assert np.max(np.abs(widen(p) - ref) / np.maximum(np.abs(ref), 1e-4)) < 2 ** -7
        assert np.array_equal(m, (np.float32(0.1) * g).astype(np.float32))
    assert np.any(outs[0] != outs[1])
