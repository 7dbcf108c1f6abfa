"""The int8 attention kernels on the device against the oracle, bit for bit: P.V in int8 per block (R17) and
dQ accumulated in 64-bit fixed point (R18), as standalone entry points (ragged sequences, grouped heads,
windows, masked entries holding garbage that must not be read, the exact path for huge products, sampled
rows at the paper's 4096-token shape) and inside decoder blocks and full steps."""
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


def seen_mask(S, window):
    i, j = np.indices((S, S))
    m = j <= i
    if window:
        m &= j > i - window
    return m


def probs(B, H, S, window, seed):
    """causal (windowed) softmax rows from the oracle, with garbage bf16 in the masked entries"""
    raw = I.normal_f32((B * H, S, S), seed, I.TENSOR_IDS["scores"]) * np.float32(4)
    P = oracle.softmax_causal(raw, np.float32(1 / math.sqrt(128)), window=window).reshape(B, H, S, S)
    junk = I.normal_bf16((B, H, S, S), seed, 77, std=3.0)
    return np.where(seen_mask(S, window), P, junk).astype(np.uint16)


def pv_case(B, H, Hkv, S, hd, window, seed=0):
    P = probs(B, H, S, window, seed)
    V = I.normal_bf16((B, Hkv, S, hd), seed, I.TENSOR_IDS["x_in"])
    G = H // Hkv
    want = np.empty((B, S, H, hd), np.float32)
    seen = seen_mask(S, window)
    for b in range(B):
        for h in range(H):
            Ph = np.where(seen, P[b, h], 0).astype(np.uint16)
            want[b, :, h, :] = oracle.attn_pv_i8(Ph, V[b, h // G])
    return P, V, want


def run_pv(B, H, Hkv, S, hd, window, P, V):
    ws = torch.empty(C.attn_pv_i8_workspace_bytes(B, Hkv, S, hd), dtype=torch.uint8, device=DEV)
    of = torch.empty((B, S, H * hd), dtype=torch.float32, device=DEV)
    ob = torch.empty((B, S, H * hd), dtype=torch.bfloat16, device=DEV)
    C.attn_pv_i8(B, H, Hkv, S, hd, window, dev_bf16(P), dev_bf16(V), ws, o_f32=of, o_bf16=ob)
    torch.cuda.synchronize()
    return host_f32(of), host_u16(ob)


@pytest.mark.parametrize("B,H,Hkv,S,hd,window", [(2, 2, 2, 64, 32, 0), (1, 4, 2, 100, 32, 0), (2, 2, 1, 192, 128, 0),
                                                  (1, 2, 2, 200, 64, 40), (1, 4, 1, 130, 128, 7),
                                                  (1, 2, 2, 320, 96, 0), (1, 1, 1, 33, 256, 0)])
def test_pv_i8_standalone(B, H, Hkv, S, hd, window):
    print(f"pv_i8 B={B} H={H} Hkv={Hkv} S={S} hd={hd} window={window}", flush=True)
    P, V, want = pv_case(B, H, Hkv, S, hd, window)
    of, ob = run_pv(B, H, Hkv, S, hd, window, P, V)
    assert_bits(of, want.reshape(B, S, H * hd), "O fp32")
    wb = (want.reshape(-1).view(np.uint32) + 0x7FFF + ((want.reshape(-1).view(np.uint32) >> 16) & 1)) >> 16
    assert_bits(ob.reshape(-1), wb.astype(np.uint16), "O bf16")


def test_pv_i8_long_sequence_sampled():
    """The paper's 4096-token rows (64 key blocks: two chains of 32 blocks folded) for one head, and a
    windowed head; every row checked."""
    for window in (0, 512):
        print(f"pv_i8 S=4096 window={window}", flush=True)
        P, V, want = pv_case(1, 1, 1, 4096, 128, window, seed=3)
        of, _ = run_pv(1, 1, 1, 4096, 128, window, P, V)
        assert_bits(of, want.reshape(1, 4096, 128), "O fp32")


def dq_case(B, H, Hkv, S, hd, window, F, seed=0, std=1e-3, kstd=1.0):
    dS = I.normal_bf16((B, H, S, S), seed, 78, std=std)
    junk = I.normal_bf16((B, H, S, S), seed, 79, std=1e4)
    dS = np.where(seen_mask(S, window), dS, junk).astype(np.uint16)
    K = I.normal_bf16((B, Hkv, S, hd), seed, 80, std=kstd)
    G = H // Hkv
    want = np.empty((B, S, H, hd), np.float32)
    for b in range(B):
        for h in range(H):
            want[b, :, h, :] = oracle.attn_dq_fixed(dS[b, h], K[b, h // G], F, window)
    return dS, K, want


def run_dq(B, H, Hkv, S, hd, window, F, dS, K):
    dQ = torch.empty((B, S, H * hd), dtype=torch.float32, device=DEV)
    C.attn_dq_fixed(B, H, Hkv, S, hd, window, F, dev_bf16(dS), dev_bf16(K), dQ)
    torch.cuda.synchronize()
    return host_f32(dQ)


@pytest.mark.parametrize("B,H,Hkv,S,hd,window,F", [(2, 2, 2, 64, 16, 0, 40), (1, 4, 2, 100, 64, 0, 40),
                                                    (1, 2, 1, 200, 128, 33, 40), (2, 2, 2, 96, 32, 0, 12),
                                                    (1, 2, 2, 70, 128, 0, 62), (1, 1, 1, 129, 64, 1, 24)])
def test_dq_fixed_standalone(B, H, Hkv, S, hd, window, F):
    print(f"dq_fixed B={B} H={H} Hkv={Hkv} S={S} hd={hd} window={window} F={F}", flush=True)
    dS, K, want = dq_case(B, H, Hkv, S, hd, window, F)
    assert_bits(run_dq(B, H, Hkv, S, hd, window, F, dS, K), want.reshape(B, S, H * hd), "dQ")


@pytest.mark.parametrize("F,std", [(40, 2.0 ** 14), (62, 1.0), (50, 64.0)])
def test_dq_fixed_exact_path_and_wraparound(F, std):
    """Products of 2^51 and more (times 2^F) take the exact path; sums past 2^63 wrap modulo 2^64."""
    print(f"dq_fixed large products F={F} std={std}", flush=True)
    dS, K, want = dq_case(1, 2, 1, 96, 32, 0, F, seed=5, std=std, kstd=std)
    assert_bits(run_dq(1, 2, 1, 96, 32, 0, F, dS, K), want.reshape(1, 96, 64), "dQ")


@pytest.mark.parametrize("S,window", [(2048, 0), (4096, 512)])
def test_dq_fixed_long_sequence(S, window):
    print(f"dq_fixed S={S} hd=128 window={window} (one head)", flush=True)
    dS, K, want = dq_case(1, 1, 1, S, 128, window, 40, seed=7)
    assert_bits(run_dq(1, 1, 1, S, 128, window, 40, dS, K), want.reshape(1, S, 128), "dQ")


def cfgs(L, d, H, F, V, S, mb, Hkv=0, qk=0, en=0, win=0, every=0, z=0.0, pv=0, dq=0):
    hd = d // H
    args = (L, d, H, hd, F, V, S, mb, np.float32(1e-5), Hkv, qk, en, win, every, np.float32(z), pv, dq)
    return oracle.ModelCfg(*args), C.ModelCfg(*args)


@pytest.mark.parametrize("d,H,Hkv,qk,win,F,S,batch,pv,dq", [
    (64, 2, 0, 0, 0, 96, 96, 2, 1, 0), (64, 2, 0, 0, 0, 96, 96, 2, 0, 40), (64, 2, 1, 1, 20, 96, 130, 1, 1, 40),
    (256, 2, 1, 1, 0, 256, 192, 1, 1, 40), (256, 4, 2, 1, 40, 384, 128, 2, 1, 40), (128, 2, 2, 0, 0, 128, 64, 1, 1, 12),
    (256, 4, 1, 1, 64, 256, 512, 1, 1, 40)])
def test_block_int8_attention_bit_exact(d, H, Hkv, qk, win, F, S, batch, pv, dq):
    print(f"block pv={pv} dq={dq} d={d} H={H} Hkv={Hkv} qk={qk} win={win} S={S} B={batch}", flush=True)
    hd = d // H
    cfg_o, cfg_c = cfgs(1, d, H, F, 100, S, batch, Hkv=Hkv, qk=qk, win=win, pv=pv, dq=dq)
    T = batch * S
    x = I.bf16_bits_to_f32(I.normal_bf16((T, d), 4, I.TENSOR_IDS["x_in"]))
    dy = I.bf16_bits_to_f32(I.normal_bf16((T, d), 4, I.TENSOR_IDS["dy_in"]))
    kvw = (Hkv or H) * hd
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


def test_step_paper_attention_bit_exact():
    """A full step with every variant of the paper's architecture and both int8-path attention kernels."""
    L, d, H, F, V, S, mb, plan = 3, 256, 2, 256, 300, 128, 2, (1, 2, 1)
    variant = dict(Hkv=1, qk=1, en=1, win=48, every=2, z=1e-4, pv=1, dq=40)
    print(f"step {variant} plan {plan}", flush=True)
    hd = d // H
    cfg_o, cfg_c = cfgs(L, d, H, F, V, S, mb, **variant)
    params = I.model_params(L, d, F, V, seed=0, std=0.02, kv_dim=hd, embed_norm=True)
    R = plan[1] * plan[2]
    windows = I.uniform_int((R * plan[0] * mb, S + 1), 0, I.TENSOR_IDS["windows"], V)
    cos, sin = I.rope_tables(S, hd)
    k = I.adamw_constants()
    po = [p.copy() for p in params]
    mo = [np.zeros(p.shape, np.float32) for p in params]
    vo = [np.zeros(p.shape, np.float32) for p in params]
    loss_o, g_o, info = oracle.step(cfg_o, oracle.Plan(*plan), po, mo, vo, windows, cos, sin, oracle.AdamWConsts(*k),
                                    want_grads=True, clip=oracle.ClipCfg(1.0, 5.0, 5))
    pg = [dev_bf16(p) for p in params]
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    gg = [torch.empty(p.shape, dtype=torch.float32, device=DEV) for p in params]
    cplan = C.DPPlan(*plan)
    ws = poisoned_workspace(C.step_workspace_bytes(cfg_c, cplan))
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    norm = torch.zeros(1, dtype=torch.float32, device=DEV)
    state = torch.zeros(1, dtype=torch.int32, device=DEV)
    C.step(cfg_c, cplan, pg, mg, vg, dev_i32(windows), dev_f32(cos), dev_f32(sin), C.AdamWConsts(*k), ws, loss,
           grads_out=gg, clip=C.make_clip(1.0, 5.0, 5, norm, state))
    torch.cuda.synchronize()
    assert_bits(host_f32(loss), np.array([loss_o], np.float32), "loss")
    assert_bits(host_f32(norm), np.array([info["norm"]], np.float32), "pre-clip norm")
    for i in range(len(po)):
        assert_bits(host_f32(gg[i]), g_o[i], f"grad {i}")
        assert_bits(host_u16(pg[i]), po[i], f"param {i}")
        assert_bits(host_f32(mg[i]), mo[i], f"m {i}")
        assert_bits(host_f32(vg[i]), vo[i], f"v {i}")


def test_int8_attention_rejects_unsupported_shapes():
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    P = torch.empty(64 * 64, dtype=torch.bfloat16, device=DEV)
    for hd in (48, 16):  # not a multiple of 32
        with pytest.raises(C.CanonError):
            C.attn_pv_i8(1, 1, 1, 64, hd, 0, P, P, ws, o_f32=torch.empty(64 * hd, device=DEV))
    with pytest.raises(C.CanonError):  # head_dim outside {16, 32, 64, 128}
        C.attn_dq_fixed(1, 1, 1, 64, 96, 0, 40, P, P, torch.empty(64 * 96, device=DEV))
    with pytest.raises(C.CanonError):  # frac_bits outside [1, 62]
        C.attn_dq_fixed(1, 1, 1, 64, 64, 0, 63, P, P, torch.empty(64 * 64, device=DEV))
    _, cfg_c = cfgs(1, 64, 4, 96, 100, 64, 1, pv=1)  # head_dim 16
    with pytest.raises(C.CanonError):
        C.block_fwd_bwd(cfg_c, 1, *([torch.empty(1, device=DEV)] * 2), [P] * 6, *([torch.empty(1, device=DEV)] * 4),
                        [torch.empty(1, device=DEV)] * 6, ws)
