"""canon_rownorm, canon_softmax_xent, canon_grad_accum and canon_adamw against the oracle, bit for bit."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import DEV, assert_bits, dev_bf16, dev_f32, dev_i32, host_f32, host_u16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rows,cols", [(5, 96), (64, 2048), (33, 2048 + 96), (8192, 2048), (7, 1001),
                                       (1541, 64)])
def test_rownorm_fwd_bwd(rows, cols):
    print(f"rownorm {rows}x{cols}", flush=True)
    x = (I.normal_f32((rows, cols), 0, 3) * 2).astype(np.float32)
    g = I.normal_bf16((cols,), 0, 200, std=0.1, mean=1.0)
    dy = I.normal_f32((rows, cols), 0, 4)
    eps = np.float32(1e-5)
    y_o, r_o = oracle.rownorm_fwd(x, g, eps)
    dx_o, dg_o = oracle.rownorm_bwd(x, g, r_o, dy)
    dx_, dg_, ddy = dev_f32(x), dev_bf16(g), dev_f32(dy)
    y = torch.empty((rows, cols), dtype=torch.bfloat16, device=DEV)
    r = torch.empty(rows, dtype=torch.float32, device=DEV)
    C.rownorm(C.FWD, rows, cols, dx_, dg_, eps, y=y, rstd=r)
    dx = torch.empty((rows, cols), dtype=torch.float32, device=DEV)
    dgn = torch.empty(cols, dtype=torch.float32, device=DEV)
    C.rownorm(C.BWD, rows, cols, dx_, dg_, eps, rstd=r, dy=ddy, dx=dx, dgain=dgn)
    torch.cuda.synchronize()
    assert_bits(host_u16(y), y_o, "y")
    assert_bits(host_f32(r), r_o, "rstd")
    assert_bits(host_f32(dx), dx_o, "dx")
    assert_bits(host_f32(dgn), dg_o, "dgain")


# rows of 2049 .. 4096 keys are held in registers and chained in two halves: 2052 (a lone last chunk), 3000 (a
# ragged last chunk), 4096 (128 full chunks); 4100 takes the staged kernel (two staging segments and a third)
@pytest.mark.parametrize("bh,s", [(3, 200), (2, 64), (4, 2048), (2, 70), (1, 33), (1, 2304), (1, 2052), (2, 3000),
                                  (1, 4096), (1, 4100)])
def test_softmax_causal(bh, s):
    print(f"softmax {bh}x{s}x{s}", flush=True)
    raw = I.normal_f32((bh, s, s), 0, I.TENSOR_IDS["scores"]) * np.float32(8)
    c = np.float32(1 / math.sqrt(128))
    want = oracle.softmax_causal(raw, c)
    p = torch.empty((bh, s, s), dtype=torch.bfloat16, device=DEV)
    C.softmax_xent(C.SOFTMAX_CAUSAL, bh * s, s, dev_f32(raw), p, scale=float(c))
    torch.cuda.synchronize()
    assert_bits(host_u16(p), want, "probs")


@pytest.mark.parametrize("rows,vocab", [(7, 1000), (16, 50304), (3, 33), (4, 1004), (2, 51208)])
def test_xent(rows, vocab):
    print(f"xent {rows}x{vocab}", flush=True)
    logits = I.normal_bf16((rows, vocab), 0, I.TENSOR_IDS["logits"], std=2.0)
    tgt = I.uniform_int((rows,), 0, I.TENSOR_IDS["targets"], vocab)
    invT = np.float32(1.0 / rows)
    dl_o, rl_o, ml_o = oracle.xent(logits, tgt, invT)
    dl = torch.empty((rows, vocab), dtype=torch.bfloat16, device=DEV)
    rl = torch.empty(rows, dtype=torch.float32, device=DEV)
    ml = torch.empty(1, dtype=torch.float32, device=DEV)
    C.softmax_xent(C.XENT, rows, vocab, dev_bf16(logits), dl, targets=dev_i32(tgt), inv_tokens=float(invT),
                   row_loss=rl, mean_loss=ml)
    torch.cuda.synchronize()
    assert_bits(host_u16(dl), dl_o, "dlogits")
    assert_bits(host_f32(rl), rl_o, "row_loss")
    assert_bits(host_f32(ml), np.array([ml_o], np.float32), "mean_loss")


def test_xent_full_size_sampled_rows():
    rows, vocab = 8192, 50304
    print("xent full 8192x50304", flush=True)
    logits = I.normal_bf16((rows, vocab), 0, I.TENSOR_IDS["logits"], std=2.0)
    tgt = I.uniform_int((rows,), 0, I.TENSOR_IDS["targets"], vocab)
    invT = np.float32(1.0 / rows)
    dl = torch.empty((rows, vocab), dtype=torch.bfloat16, device=DEV)
    rl = torch.empty(rows, dtype=torch.float32, device=DEV)
    ml = torch.empty(1, dtype=torch.float32, device=DEV)
    C.softmax_xent(C.XENT, rows, vocab, dev_bf16(logits), dl, targets=dev_i32(tgt), inv_tokens=float(invT),
                   row_loss=rl, mean_loss=ml)
    torch.cuda.synchronize()
    rl_h = host_f32(rl)
    sample = np.array([0, 1, 4097, rows - 1] + list(np.random.default_rng(2).integers(0, rows, 12)))
    dl_o, rl_o, _ = oracle.xent(logits[sample], tgt[sample], invT)
    assert_bits(host_u16(dl)[sample], dl_o, "dlogits rows")
    assert_bits(rl_h[sample], rl_o, "row_loss rows")
    # all row losses and their canonical mean, from the oracle (no logit gradients, to keep it fast)
    _, rl_all, ml_all = oracle.xent(logits, tgt, invT, want_dlogits=False)
    assert_bits(rl_h, rl_all, "row_loss all")
    assert_bits(host_f32(ml), np.array([ml_all], np.float32), "mean_loss")


@pytest.mark.parametrize("plan", [(1, 8, 1), (1, 1, 8), (2, 4, 1), (1, 2, 3), (3, 2, 3), (1, 1, 7), (1, 16, 1),
                                  (2, 2, 4), (1, 32, 2), (1, 1, 1)])
@pytest.mark.parametrize("n,offset", [(100003, 0), (4099, 1), (3, 0), (1, 0)])
def test_grad_accum(plan, n, offset):
    # up to 16 buffers with 16-byte aligned pointers take the vector kernel (n % 4 tail included); more
    # buffers, or a pointer off 16-byte alignment (offset 1), take the one-element-per-thread kernel
    accum, shard, rep = plan
    print(f"grad_accum plan {plan} n={n} offset={offset}", flush=True)
    grads = [I.normal_f32((n,), 0, I.TENSOR_IDS["grads"] + i, std=1e-3) for i in range(accum * shard * rep)]
    want = oracle.grad_accum(grads, accum, shard, rep)
    out = torch.empty(n + offset, dtype=torch.float32, device=DEV)[offset:]
    dg = []
    for g in grads:
        t = torch.empty(n + offset, dtype=torch.float32, device=DEV)
        t[offset:] = dev_f32(g)
        dg.append(t[offset:])
    C.grad_accum(C.DPPlan(accum, shard, rep), n, dg, out)
    torch.cuda.synchronize()
    assert_bits(host_f32(out), want, f"plan {plan}")


@pytest.mark.parametrize("offset", [0, 1])
def test_adamw(offset):
    # offset 1 puts every pointer off 16-byte alignment
    sizes = [1000, 37, 4096]
    k = I.adamw_constants()
    ps = [I.normal_bf16((s,), 1, 40 + i, std=0.02) for i, s in enumerate(sizes)]
    gs = [I.normal_f32((s,), 1, 50 + i, std=1e-3) for i, s in enumerate(sizes)]
    ms = [I.normal_f32((s,), 1, 60 + i, std=1e-4) for i, s in enumerate(sizes)]
    vs = [np.abs(I.normal_f32((s,), 1, 70 + i, std=1e-6)) for i, s in enumerate(sizes)]
    mask = [1, 0, 1]
    po, mo, vo = [p.copy() for p in ps], [m.copy() for m in ms], [v.copy() for v in vs]
    oracle.adamw(po, mo, vo, gs, mask, oracle.AdamWConsts(*k))
    def shifted(t):
        if not offset:
            return t
        u = torch.empty(t.numel() + offset, dtype=t.dtype, device=DEV)
        u[offset:] = t
        return u[offset:]

    pg, mg, vg = [shifted(dev_bf16(p)) for p in ps], [shifted(dev_f32(m)) for m in ms], [shifted(dev_f32(v)) for v in vs]
    C.adamw(pg, mg, vg, [shifted(dev_f32(g)) for g in gs], mask, C.AdamWConsts(*k))
    torch.cuda.synchronize()
    for i in range(3):
        assert_bits(host_u16(pg[i]), po[i], f"p{i}")
        assert_bits(host_f32(mg[i]), mo[i], f"m{i}")
        assert_bits(host_f32(vg[i]), vo[i], f"v{i}")
