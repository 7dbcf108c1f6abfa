"""The HIP path at the workloads' own shapes against the oracle's digests.

* One decoder block forward and backward at d_model 2048, 16 heads of 128, FFN 8192, seq 2048, batch 1.
* A full-width training step: 2 layers, d_model 2048, FFN 8192, vocab 50304, seq 2048, plan (1, 2, 1), with
  the global-norm clip: loss, pre-clip norm, every reduced gradient, and the post-AdamW parameters and moments.
* The int8 quantised linear's backward at the gate/up projection (T 8192, N 16384, K 2048): dx and dW.

The expected values are SHA-256 digests of every output tensor, written by
``tests/golden/make_full_shape_golden.py`` from the CPU oracle on the same seeded inputs (``full_shape_cases``).
"""
import json
import os

import numpy as np
import pytest
import torch

import full_shape_cases as FC
import paper_2609_17380_amd.canon as C
from gpu_util import DEV, dev_bf16, dev_f32, dev_i32, host_f32, host_u16, poisoned_workspace

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(case):
    with open(os.path.join(GOLDEN, f"full_shape_{case}.json")) as f:
        return json.load(f)


def check(golden, got: dict):
    bad = []
    for e in golden["tensors"]:
        a = got[e["name"]]
        assert list(a.shape) == e["shape"], e["name"]
        if FC.digest(a) != e["sha256"]:
            bad.append(f"{e['name']}: head bits gpu {FC.head_bits(a)} oracle {e['head_bits']}")
    assert not bad, f"{len(bad)} of {len(golden['tensors'])} tensors differ from the oracle:\n" + "\n".join(bad[:12])


def test_block_d2048_seq2048_matches_oracle():
    g = load("block")
    c = FC.BLOCK
    assert g["config"]["d"] == c["d"] and g["config"]["S"] == c["S"] and g["config"]["F"] == c["F"]
    print(f"block d={c['d']} H={c['H']} F={c['F']} S={c['S']} batch={c['batch']}", flush=True)
    x, dy, w, cos, sin = FC.block_inputs(c)
    cfg = C.ModelCfg(1, c["d"], c["H"], c["hd"], c["F"], 100, c["S"], c["batch"], np.float32(c["eps"]))
    T = c["batch"] * c["S"]
    ws = poisoned_workspace(C.block_workspace_bytes(cfg, c["batch"]))
    y = torch.empty((T, c["d"]), dtype=torch.float32, device=DEV)
    dx = torch.empty_like(y)
    dw = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in w]
    C.block_fwd_bwd(cfg, c["batch"], dev_f32(x), dev_f32(dy), [dev_bf16(t) for t in w], dev_f32(cos), dev_f32(sin),
                    y, dx, dw, ws)
    torch.cuda.synchronize()
    got = {"y": host_f32(y), "dx": host_f32(dx)}
    for n, t in zip(FC.BLOCK_NAMES, dw):
        got["d" + n] = host_f32(t)
    check(g, got)


def test_step_full_width_matches_oracle():
    g = load("step")
    c = FC.STEP
    assert g["config"]["V"] == c["V"] and g["config"]["L"] == c["L"] and tuple(g["config"]["plan"]) == c["plan"]
    print(f"step L={c['L']} d={c['d']} F={c['F']} V={c['V']} S={c['S']} mb={c['mb']} plan={c['plan']}", flush=True)
    params, windows, cos, sin, k = FC.step_inputs(c)
    cfg = C.ModelCfg(c["L"], c["d"], c["H"], c["hd"], c["F"], c["V"], c["S"], c["mb"], np.float32(c["eps"]))
    plan = C.DPPlan(*c["plan"])
    pg = [dev_bf16(p) for p in params]
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    gg = [torch.empty(p.shape, dtype=torch.float32, device=DEV) for p in params]
    ws = poisoned_workspace(C.step_workspace_bytes(cfg, plan))
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    norm = torch.zeros(1, dtype=torch.float32, device=DEV)
    state = torch.zeros(1, dtype=torch.int32, device=DEV)
    C.step(cfg, plan, pg, mg, vg, dev_i32(windows), dev_f32(cos), dev_f32(sin), C.AdamWConsts(*k), ws, loss,
           grads_out=gg, clip=C.make_clip(*c["clip"], norm, state))
    torch.cuda.synchronize()
    assert int(state.cpu()[0]) == g["skip_state"]
    names = [n for n, *_ in FC.I.model_param_shapes(c["L"], c["d"], c["F"], c["V"])]
    got = {"loss": host_f32(loss), "norm": host_f32(norm)}
    for n, t in zip(names, gg):
        got["grad." + n] = host_f32(t)
    for n, t in zip(names, pg):
        got["param." + n] = host_u16(t)
    for n, t in zip(names, mg):
        got["m." + n] = host_f32(t)
    for n, t in zip(names, vg):
        got["v." + n] = host_f32(t)
    print(f"loss gpu {float(got['loss'][0]):.6f} oracle {g['loss']:.6f}", flush=True)
    check(g, got)


def test_qlinear_bwd_gate_up_shape_matches_oracle():
    g = load("qlinear")
    c = FC.QLIN
    assert (g["config"]["T"], g["config"]["N"], g["config"]["K"]) == (c["T"], c["N"], c["K"])
    print(f"qlinear_bwd T={c['T']} N={c['N']} K={c['K']}", flush=True)
    dy, qx, sx, qw, sw = FC.qlin_inputs(c)
    T, N, K = c["T"], c["N"], c["K"]
    ws = torch.empty(C.qlinear_bwd_workspace_bytes(T, N, K), dtype=torch.uint8, device=DEV)
    dx = torch.empty((T, K), dtype=torch.float32, device=DEV)
    dw = torch.empty((N, K), dtype=torch.float32, device=DEV)
    C.qlinear_bwd(T, N, K, dev_f32(dy), torch.from_numpy(qx).to(DEV), dev_f32(sx), torch.from_numpy(qw).to(DEV),
                  dev_f32(sw), dx, dw, ws)
    torch.cuda.synchronize()
    check(g, {"dx": host_f32(dx), "dw": host_f32(dw)})
