"""canon_block_fwd_bwd and canon_step against the oracle, bit for bit, at configurations the oracle runs in
seconds (several GEMM tiles, ragged sequence tails, head size 128 as in the 1B shape)."""
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


def block_case(d, H, F, S, batch, std):
    hd = d // H
    cfg_o = oracle.ModelCfg(1, d, H, hd, F, 100, S, batch, np.float32(1e-5))
    cfg_c = C.ModelCfg(1, d, H, hd, F, 100, S, batch, np.float32(1e-5))
    T = batch * S
    x = I.bf16_bits_to_f32(I.normal_bf16((T, d), 0, I.TENSOR_IDS["x_in"]))
    dy = I.bf16_bits_to_f32(I.normal_bf16((T, d), 0, I.TENSOR_IDS["dy_in"]))
    shapes = [(d,), (3 * d, d), (d, d), (d,), (2 * F, d), (d, F)]
    w = [I.normal_bf16(s, 0, I.TENSOR_IDS[n], std=(0.1 if len(s) == 1 else std), mean=(1.0 if len(s) == 1 else 0.0))
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


@pytest.mark.parametrize("d,H,F,S,batch,std", [(256, 2, 384, 96, 2, 0.05), (128, 1, 256, 64, 1, 0.08),
                                              (256, 2, 320, 130, 1, 0.02)])
def test_block_bit_exact(d, H, F, S, batch, std):
    print(f"block d={d} H={H} F={F} S={S} B={batch}", flush=True)
    block_case(d, H, F, S, batch, std)


def run_step(L, d, H, F, V, S, mb, plan, seed=0, grads=True, windows=None):
    hd = d // H
    params = I.model_params(L, d, F, V, seed=seed, std=0.02)
    R = plan[1] * plan[2]
    if windows is None:
        windows = I.uniform_int((R * plan[0] * mb, S + 1), seed, I.TENSOR_IDS["windows"], V)
    cos, sin = I.rope_tables(S, hd)
    k = I.adamw_constants()
    po = [p.copy() for p in params]
    mo = [np.zeros(p.shape, np.float32) for p in params]
    vo = [np.zeros(p.shape, np.float32) for p in params]
    loss_o, g_o = oracle.step(oracle.ModelCfg(L, d, H, hd, F, V, S, mb, np.float32(1e-5)), oracle.Plan(*plan), po, mo,
                              vo, windows, cos, sin, oracle.AdamWConsts(*k), want_grads=grads)
    cfg = C.ModelCfg(L, d, H, hd, F, V, S, mb, np.float32(1e-5))
    cplan = C.DPPlan(*plan)
    pg = [dev_bf16(p) for p in params]
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    gg = [torch.empty(p.shape, dtype=torch.float32, device=DEV) for p in params] if grads else None
    ws = poisoned_workspace(C.step_workspace_bytes(cfg, cplan))
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    C.step(cfg, cplan, pg, mg, vg, dev_i32(windows), dev_f32(cos), dev_f32(sin), C.AdamWConsts(*k), ws, loss,
           grads_out=gg)
    torch.cuda.synchronize()
    return (loss_o, g_o, po, mo, vo), (host_f32(loss), [host_f32(g) for g in gg] if grads else None,
                                       [host_u16(p) for p in pg], [host_f32(m) for m in mg], [host_f32(v) for v in vg])


@pytest.mark.parametrize("plan", [(1, 2, 2), (2, 2, 1), (1, 1, 3)])
def test_step_bit_exact(plan):
    print(f"step plan={plan}", flush=True)
    (lo, go, po, mo, vo), (lg, gg, pg, mg, vg) = run_step(2, 256, 2, 256, 300, 64, 2, plan)
    assert_bits(lg, np.array([lo], np.float32), "loss")
    for i in range(len(po)):
        assert_bits(gg[i], go[i], f"grad {i}")
        assert_bits(pg[i], po[i], f"param {i}")
        assert_bits(mg[i], mo[i], f"m {i}")
        assert_bits(vg[i], vo[i], f"v {i}")


def test_step_with_heavily_repeated_tokens():
    """Token draws skewed like text: one token takes ~60% of each 2048-token microbatch (more than 1024
    occurrences: the embedding backward's chunk chain runs over 39 chunks and the fold over them), others
    ~10% and ~2% (several chunks), the rest uniform."""
    L, d, H, F, V, S, mb, plan = 1, 128, 1, 128, 300, 2048, 1, (1, 2, 1)
    rng = np.random.default_rng(17)
    n = plan[1] * mb
    win = rng.integers(0, V, size=(n, S + 1)).astype(np.int32)
    u = rng.random((n, S + 1))
    win[u < 0.60] = 7
    win[(u >= 0.60) & (u < 0.70)] = 11
    win[(u >= 0.70) & (u < 0.72)] = 13
    counts = [(win[i, :S] == 7).sum() for i in range(n)]
    print(f"step skewed tokens: token 7 occurs {counts} times per microbatch", flush=True)
    assert min(counts) > 1024
    (lo, go, po, mo, vo), (lg, gg, pg, mg, vg) = run_step(L, d, H, F, V, S, mb, plan, windows=win)
    assert_bits(lg, np.array([lo], np.float32), "loss")
    assert_bits(gg[0], go[0], "embedding gradient")
    for i in range(len(po)):
        assert_bits(gg[i], go[i], f"grad {i}")
        assert_bits(pg[i], po[i], f"param {i}")


def test_step_rejects_bad_tokens_without_update():
    L, d, H, F, V, S, mb = 1, 128, 1, 128, 50, 32, 1
    cfg = C.ModelCfg(L, d, H, d // H, F, V, S, mb, np.float32(1e-5))
    cplan = C.DPPlan(1, 1, 1)
    params = I.model_params(L, d, F, V, seed=0)
    windows = I.uniform_int((1, S + 1), 0, 50, V)
    windows[0, 5] = V + 3  # out of range
    cos, sin = I.rope_tables(S, d // H)
    pg = [dev_bf16(p) for p in params]
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    ws = poisoned_workspace(C.step_workspace_bytes(cfg, cplan))
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    C.step(cfg, cplan, pg, mg, vg, dev_i32(windows), dev_f32(cos), dev_f32(sin), C.AdamWConsts(*I.adamw_constants()),
           ws, loss)
    torch.cuda.synchronize()
    assert np.isnan(host_f32(loss)[0])
    for a, b in zip(pg, params):
        assert np.array_equal(host_u16(a), b)


@pytest.mark.parametrize("plan", [(1, 2, 2), (2, 1, 3)])
def test_step_state_digest_matches_oracle_state(plan):
    """The per-step audit hash computed inside canon_step equals H1 of the oracle's own step outputs (windows,
    parameters, m, v, reduced gradient), written by the oracle's hash code, and canon_state_hash of the
    device outputs; a second run of the same step gives the same digest."""
    from oracle import state_hash as H
    L, d, H_, F, V, S, mb = 2, 128, 1, 128, 200, 64, 1
    hd = d // H_
    params = I.model_params(L, d, F, V, seed=3, std=0.02)
    R = plan[1] * plan[2]
    windows = I.uniform_int((R * plan[0] * mb, S + 1), 3, I.TENSOR_IDS["windows"], V)
    cos, sin = I.rope_tables(S, hd)
    k = I.adamw_constants()
    po = [p.copy() for p in params]
    mo = [np.zeros(p.shape, np.float32) for p in params]
    vo = [np.zeros(p.shape, np.float32) for p in params]
    _, g_o = oracle.step(oracle.ModelCfg(L, d, H_, hd, F, V, S, mb, np.float32(1e-5)), oracle.Plan(*plan), po, mo, vo,
                         windows, cos, sin, oracle.AdamWConsts(*k), want_grads=True)
    want = H.state_digest([windows.astype(np.int32).tobytes()] + [p.astype(np.uint16).tobytes() for p in po] +
                          [m.tobytes() for m in mo] + [v.tobytes() for v in vo] + [g.tobytes() for g in g_o])
    cfg = C.ModelCfg(L, d, H_, hd, F, V, S, mb, np.float32(1e-5))
    cplan = C.DPPlan(*plan)
    ws = poisoned_workspace(C.step_workspace_bytes(cfg, cplan))
    digests = []
    for run in range(2):
        pg = [dev_bf16(p) for p in params]
        mg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
        vg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
        gg = [torch.empty(p.shape, dtype=torch.float32, device=DEV) for p in params]
        win = dev_i32(windows)
        loss = torch.zeros(1, dtype=torch.float32, device=DEV)
        dig = torch.zeros(32, dtype=torch.uint8, device=DEV)
        C.step(cfg, cplan, pg, mg, vg, win, dev_f32(cos), dev_f32(sin), C.AdamWConsts(*k), ws, loss, grads_out=gg,
               state_digest=dig)
        torch.cuda.synchronize()
        digests.append(bytes(dig.cpu().numpy()))
        state = [win] + pg + mg + vg + gg
        hws = torch.empty(C.state_hash_workspace_bytes(state), dtype=torch.uint8, device=DEV)
        d2 = torch.zeros(32, dtype=torch.uint8, device=DEV)
        C.state_hash(state, d2, hws)
        torch.cuda.synchronize()
        assert bytes(d2.cpu().numpy()) == digests[-1]
    print(f"step digest {digests[0].hex()[:16]}.. oracle {want.hex()[:16]}..", flush=True)
    assert digests[0] == want and digests[1] == want
