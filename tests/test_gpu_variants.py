"""The paper's model variants (R16) on the device against the oracle, bit for bit: the sliding-window softmax,
the cross-entropy with z-loss, the fp32-output RMSNorm of the embedding norm, decoder blocks with grouped
key/value heads, gain-free QK-norm and windows, and full steps with every variant on."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import (DEV, assert_bits, dev_bf16, dev_f32, dev_i32, host_f32, host_u16,
                      poisoned_workspace)

pytestmark = pytest.mark.gpu

NAMES = ["attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down"]


# (1, 4200, 600) and (1, 4104, 10): windows that start past whole staging segments of 2048 keys
@pytest.mark.parametrize("bh,s,win", [(3, 200, 16), (2, 64, 1), (4, 2048, 512), (2, 70, 33), (1, 2304, 512),
                                      (1, 2304, 2000), (2, 96, 96), (1, 4200, 600), (1, 4104, 10),
                                      # windows up to 512 keep the row's band in registers; a partial last chunk
                                      (2, 1000, 100), (1, 4096, 257), (1, 4096, 512),
                                      # longer windows on rows held in registers (2049 .. 4096 keys)
                                      (1, 4096, 1000), (1, 3000, 2999)])
def test_softmax_window(bh, s, win):
    print(f"softmax window {bh}x{s}x{s} w={win}", flush=True)
    raw = I.normal_f32((bh, s, s), 1, I.TENSOR_IDS["scores"]) * np.float32(8)
    c = np.float32(1 / math.sqrt(128))
    want = oracle.softmax_causal(raw, c, window=win)
    p = torch.empty((bh, s, s), dtype=torch.bfloat16, device=DEV)
    C.softmax_xent(C.SOFTMAX_CAUSAL, bh * s, s, dev_f32(raw), p, scale=float(c), window=win)
    torch.cuda.synchronize()
    assert_bits(host_u16(p), want, "probs")


@pytest.mark.parametrize("rows,vocab", [(7, 1000), (16, 50304), (3, 33), (2, 51208), (4, 128256)])
@pytest.mark.parametrize("z", [1e-4, 0.05])
def test_xent_z_loss(rows, vocab, z):
    print(f"xent z={z} {rows}x{vocab}", flush=True)
    logits = I.normal_bf16((rows, vocab), 2, I.TENSOR_IDS["logits"], std=2.0)
    tgt = I.uniform_int((rows,), 2, I.TENSOR_IDS["targets"], vocab)
    invT = np.float32(1.0 / rows)
    zf = np.float32(z)
    dl_o, rl_o, ml_o = oracle.xent(logits, tgt, invT, z_loss=zf)
    dl = torch.empty((rows, vocab), dtype=torch.bfloat16, device=DEV)
    rl = torch.empty(rows, dtype=torch.float32, device=DEV)
    ml = torch.empty(1, dtype=torch.float32, device=DEV)
    C.softmax_xent(C.XENT, rows, vocab, dev_bf16(logits), dl, targets=dev_i32(tgt), inv_tokens=float(invT),
                   row_loss=rl, mean_loss=ml, z_loss=float(zf))
    torch.cuda.synchronize()
    assert_bits(host_u16(dl), dl_o, "dlogits")
    assert_bits(host_f32(rl), rl_o, "row_loss")
    assert_bits(host_f32(ml), np.array([ml_o], np.float32), "mean_loss")


@pytest.mark.parametrize("rows,cols", [(5, 96), (64, 2048), (33, 2048 + 96), (7, 1001)])
def test_rownorm_fwd_f32(rows, cols):
    print(f"rownorm f32 {rows}x{cols}", flush=True)
    x = (I.normal_f32((rows, cols), 3, 3) * 2).astype(np.float32)
    g = I.normal_bf16((cols,), 3, 200, std=0.1, mean=1.0)
    eps = np.float32(1e-5)
    y_o, r_o = oracle.rownorm_fwd_f32(x, g, eps)
    y = torch.empty((rows, cols), dtype=torch.float32, device=DEV)
    r = torch.empty(rows, dtype=torch.float32, device=DEV)
    C.rownorm(C.FWD_F32, rows, cols, dev_f32(x), dev_bf16(g), eps, y=y, rstd=r)
    torch.cuda.synchronize()
    assert_bits(host_f32(y), y_o, "y")
    assert_bits(host_f32(r), r_o, "rstd")


def cfgs(L, d, H, F, V, S, mb, Hkv=0, qk=0, en=0, win=0, every=0, z=0.0):
    hd = d // H
    args = (L, d, H, hd, F, V, S, mb, np.float32(1e-5), Hkv, qk, en, win, every, np.float32(z))
    return oracle.ModelCfg(*args), C.ModelCfg(*args)


# S a multiple of 128 takes the grouped dK/dV GEMMs with per-head skip ranges; other S the full contraction
@pytest.mark.parametrize("d,H,Hkv,qk,win,F,S,batch", [(256, 4, 2, 0, 0, 384, 96, 2), (256, 4, 1, 1, 0, 320, 130, 1),
                                                     (256, 4, 4, 1, 40, 384, 96, 2), (256, 2, 1, 1, 33, 256, 130, 1),
                                                     (512, 4, 2, 1, 64, 384, 160, 1), (256, 4, 2, 1, 17, 384, 96, 2),
                                                     (256, 4, 2, 1, 0, 384, 256, 1), (256, 4, 1, 0, 100, 256, 384, 1),
                                                     (512, 8, 2, 1, 64, 384, 256, 2), (256, 4, 1, 1, 1, 256, 128, 1),
                                                     (256, 4, 2, 0, 300, 256, 256, 1),
                                                     # more score tiles than resident workgroups (1024 and 2048)
                                                     (256, 2, 2, 0, 0, 256, 1024, 4), (512, 16, 4, 1, 200, 512, 1024, 1),
                                                     (256, 2, 1, 1, 300, 256, 1000, 4),
                                                     # windows far shorter than the sequence: P and dS stay
                                                     # unwritten beyond the products' reach (poisoned workspace)
                                                     (256, 2, 2, 1, 50, 256, 512, 1), (256, 4, 1, 0, 64, 256, 640, 1),
                                                     # head dim 48: a ragged second chunk in every per-row reduction
                                                     (192, 4, 4, 0, 0, 256, 96, 2),
                                                     # head dim 544: 17 chunks per attention row dot (the wide path)
                                                     (544, 1, 1, 0, 0, 256, 64, 1)])
def test_block_variants_bit_exact(d, H, Hkv, qk, win, F, S, batch):
    print(f"block d={d} H={H} Hkv={Hkv} qk={qk} win={win} F={F} S={S} B={batch}", flush=True)
    hd = d // H
    cfg_o, cfg_c = cfgs(1, d, H, F, 100, S, batch, Hkv=Hkv, qk=qk, win=win)
    T = batch * S
    x = I.bf16_bits_to_f32(I.normal_bf16((T, d), 4, I.TENSOR_IDS["x_in"]))
    dy = I.bf16_bits_to_f32(I.normal_bf16((T, d), 4, I.TENSOR_IDS["dy_in"]))
    kvw = Hkv * hd
    shapes = [(d,), (d + 2 * kvw, d), (d, d), (d,), (2 * F, d), (d, F)]
    w = [I.normal_bf16(s, 4, I.TENSOR_IDS[n], std=(0.1 if len(s) == 1 else 0.05), mean=(1.0 if len(s) == 1 else 0.0))
         for s, n in zip(shapes, NAMES)]
    cos, sin = I.rope_tables(S, hd)
    y_o, dx_o, dw_o = oracle.block_fwd_bwd(cfg_o, batch, x, dy, w, cos, sin)
    ws = poisoned_workspace(C.block_workspace_bytes(cfg_c, batch))
    y = torch.empty((T, d), dtype=torch.float32, device=DEV)
    dx = torch.empty_like(y)
    dw = [torch.empty(s, dtype=torch.float32, device=DEV) for s in shapes]
    C.block_fwd_bwd(cfg_c, batch, dev_f32(x), dev_f32(dy), [dev_bf16(t) for t in w], dev_f32(cos), dev_f32(sin), y,
                    dx, dw, ws)
    torch.cuda.synchronize()
    assert_bits(host_f32(y), y_o, "y")
    assert_bits(host_f32(dx), dx_o, "dx")
    for n, g, go in zip(NAMES, dw, dw_o):
        assert_bits(host_f32(g), go, "d" + n)


def run_step(L, d, H, F, V, S, mb, plan, variant, seed=0, clip=None):
    hd = d // H
    cfg_o, cfg_c = cfgs(L, d, H, F, V, S, mb, **variant)
    Hkv = variant.get("Hkv", 0) or H
    en = bool(variant.get("en", 0))
    params = I.model_params(L, d, F, V, seed=seed, std=0.02, kv_dim=Hkv * hd, embed_norm=en)
    R = plan[1] * plan[2]
    windows = I.uniform_int((R * plan[0] * mb, S + 1), seed, I.TENSOR_IDS["windows"], V)
    cos, sin = I.rope_tables(S, hd)
    k = I.adamw_constants()
    po = [p.copy() for p in params]
    mo = [np.zeros(p.shape, np.float32) for p in params]
    vo = [np.zeros(p.shape, np.float32) for p in params]
    res = oracle.step(cfg_o, oracle.Plan(*plan), po, mo, vo, windows, cos, sin, oracle.AdamWConsts(*k),
                      want_grads=True, clip=oracle.ClipCfg(*clip) if clip else None)
    pg = [dev_bf16(p) for p in params]
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    gg = [torch.empty(p.shape, dtype=torch.float32, device=DEV) for p in params]
    cplan = C.DPPlan(*plan)
    ws = poisoned_workspace(C.step_workspace_bytes(cfg_c, cplan))
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    norm = torch.zeros(1, dtype=torch.float32, device=DEV)
    state = torch.zeros(1, dtype=torch.int32, device=DEV)
    cc = C.make_clip(*clip, norm, state) if clip else None
    C.step(cfg_c, cplan, pg, mg, vg, dev_i32(windows), dev_f32(cos), dev_f32(sin), C.AdamWConsts(*k), ws, loss,
           grads_out=gg, clip=cc)
    torch.cuda.synchronize()
    return res, (po, mo, vo), (host_f32(loss), [host_f32(g) for g in gg], [host_u16(p) for p in pg],
                               [host_f32(m) for m in mg], [host_f32(v) for v in vg], host_f32(norm))


@pytest.mark.parametrize("variant,plan", [
    (dict(Hkv=2, qk=1, en=1, win=24, every=2, z=1e-4), (1, 2, 1)),
    (dict(Hkv=1, qk=1, en=1, win=40, every=0, z=0.05), (2, 1, 1)),
    (dict(Hkv=2), (1, 1, 2)),
    (dict(win=17, every=3, z=1e-4), (1, 2, 1)),
    (dict(en=1), (1, 1, 1)),
    (dict(Hkv=2, qk=1, en=1, win=48, every=2, z=1e-4, S=128), (1, 2, 1)),
])
def test_step_variants_bit_exact(variant, plan):
    print(f"step variant {variant} plan {plan}", flush=True)
    clip = (1.0, 5.0, 5) if variant.get("qk") else None
    variant = dict(variant)
    S = variant.pop("S", 64)
    res, (po, mo, vo), (lg, gg, pg, mg, vg, ng) = run_step(3, 256, 4, 256, 300, S, 2, plan, variant, clip=clip)
    loss_o, g_o = res[0], res[1]
    assert_bits(lg, np.array([loss_o], np.float32), "loss")
    if clip:
        assert_bits(ng, np.array([res[2]["norm"]], np.float32), "pre-clip norm")
    for i in range(len(po)):
        assert_bits(gg[i], g_o[i], f"grad {i}")
        assert_bits(pg[i], po[i], f"param {i}")
        assert_bits(mg[i], mo[i], f"m {i}")
        assert_bits(vg[i], vo[i], f"v {i}")
