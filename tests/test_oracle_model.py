"""Pins for the oracle's decoder block and full step against a float64 autograd model.

The float64 model (``torch_model_ref``) shares nothing with the oracle; agreement is to a tolerance set by
fp32-versus-fp64 accumulation and the bf16 rounding points (a wrong sign, index, operand or dropped term
shows up as an O(1) relative error).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_17380_amd.inputs as I
import torch_model_ref as R

NAMES = ["attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down"]


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def small_cfg(L=1, d=64, H=2, F=96, V=97, S=48, mb=2):
    return oracle.ModelCfg(L, d, H, d // H, F, V, S, mb, np.float32(1e-5))


def block_weights(d, F, seed, std):
    shapes = [(d,), (3 * d, d), (d, d), (d,), (2 * F, d), (d, F)]
    w = []
    for i, s in enumerate(shapes):
        if len(s) == 1:
            w.append(I.normal_bf16(s, seed, 900 + i, std=0.1, mean=1.0))
        else:
            w.append(I.normal_bf16(s, seed, 900 + i, std=std))
    return w


def test_block_fwd_bwd_matches_float64_autograd():
    cfg = small_cfg(d=64, H=2, F=96, S=48)
    B, S, d, F, H = 2, cfg.seq, cfg.d_model, cfg.d_ffn, cfg.n_heads
    hd = d // H
    x16 = I.normal_bf16((B * S, d), 0, I.TENSOR_IDS["x_in"])
    dy16 = I.normal_bf16((B * S, d), 0, I.TENSOR_IDS["dy_in"])
    x, dy = I.bf16_bits_to_f32(x16), I.bf16_bits_to_f32(dy16)
    w = block_weights(d, F, 0, 0.08)
    cos, sin = I.rope_tables(S, hd)
    y, dx, dw = oracle.block_fwd_bwd(cfg, B, x, dy, w, cos, sin)

    xt = torch.tensor(x, dtype=R.DT, requires_grad=True)
    wt = {n: R.bf16_tensor(t, requires_grad=True) for n, t in zip(NAMES, w)}
    scale = float(np.float32(1 / math.sqrt(hd)))
    yt = R.block(xt, wt, B, S, H, hd, F, float(np.float32(1e-5)), torch.tensor(cos, dtype=R.DT),
                 torch.tensor(sin, dtype=R.DT), scale)
    yt.backward(torch.tensor(dy, dtype=R.DT))
    assert rel(y, yt.detach().numpy()) < 1e-4
    assert rel(dx, xt.grad.numpy()) < 5e-3
    for n, g in zip(NAMES, dw):
        assert rel(g, wt[n].grad.numpy()) < 5e-3, n


def test_step_matches_float64_autograd_and_plan():
    cfg = small_cfg(L=2, d=64, H=2, F=96, V=97, S=40, mb=2)
    plan = oracle.Plan(1, 2, 2)
    R_ = plan.dp_shard * plan.dp_replicate
    M = R_ * plan.accum * cfg.micro_seqs
    params = I.model_params(cfg.n_layers, cfg.d_model, cfg.d_ffn, cfg.vocab, seed=0, std=0.05)
    windows = I.uniform_int((M, cfg.seq + 1), 0, I.TENSOR_IDS["windows"], cfg.vocab)
    cos, sin = I.rope_tables(cfg.seq, cfg.head_dim)
    k = oracle.AdamWConsts(*I.adamw_constants())
    p_or = [p.copy() for p in params]
    m = [np.zeros(p.shape, np.float32) for p in params]
    v = [np.zeros(p.shape, np.float32) for p in params]
    loss, grads = oracle.step(cfg, plan, p_or, m, v, windows, cos, sin, k, want_grads=True)

    # float64 reference: mean over all microbatches of the mean token loss (the plan's exact meaning)
    pt = [R.bf16_tensor(p, requires_grad=True) for p in params]
    tcfg = dict(d=cfg.d_model, H=cfg.n_heads, hd=cfg.head_dim, F=cfg.d_ffn, L=cfg.n_layers,
                eps=float(np.float32(1e-5)))
    scale = float(np.float32(1 / math.sqrt(cfg.head_dim)))
    tot = 0
    for r in range(R_):
        rows = [r + R_ * s for s in range(cfg.micro_seqs)]
        tok = torch.tensor(windows[rows], dtype=torch.long)
        tot = tot + R.model_loss(pt, tok, tcfg, torch.tensor(cos, dtype=R.DT), torch.tensor(sin, dtype=R.DT),
                                 scale) / R_
    tot.backward()
    assert abs(float(loss) - float(tot)) < 1e-5 * abs(float(tot))
    assert abs(float(loss) - math.log(cfg.vocab)) < 0.5
    for i, (g, p) in enumerate(zip(grads, pt)):
        assert rel(g, p.grad.numpy()) < 5e-3, i
    # post-step parameters are AdamW of the reduced gradient
    p2 = [p.copy() for p in params]
    m2 = [np.zeros(p.shape, np.float32) for p in params]
    v2 = [np.zeros(p.shape, np.float32) for p in params]
    decay = [t[3] for t in I.model_param_shapes(cfg.n_layers, cfg.d_model, cfg.d_ffn, cfg.vocab)]
    oracle.adamw(p2, m2, v2, grads, decay, k)
    for a, b in zip(p_or, p2):
        assert np.array_equal(a, b)
    # a second run gives identical bits
    p3 = [p.copy() for p in params]
    m3 = [np.zeros(p.shape, np.float32) for p in params]
    v3 = [np.zeros(p.shape, np.float32) for p in params]
    loss3, _ = oracle.step(cfg, plan, p3, m3, v3, windows, cos, sin, k)
    assert np.float32(loss3).view(np.uint32) == np.float32(loss).view(np.uint32)
    assert all(np.array_equal(a, b) for a, b in zip(p_or, p3))
