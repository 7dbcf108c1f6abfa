"""Benchmark: one canonical-order training-step replay of the 1B-shaped decoder on one MI355X.

Workload (the configuration the metric is quoted on): 16 layers, d_model 2048, 16 heads of 128, SwiGLU FFN
8192, vocab 50304, sequence 2048, global batch 32 sequences run as 8 emulated data-parallel ranks of 4
sequences (Algorithm 1 with dp_shard 8), then AdamW.  Inputs are seeded and synthetic (uniform random tokens,
N(0, 0.02) weights) and resident in HBM before timing starts.

Printed JSON line:
  value        whole-step throughput in algorithmic TFLOP/s (GEMM + causal attention FLOPs / step time)
  ms_per_step  the step-replay time
  roofline     the dominant kernel (the canonical GEMM) on the fp32 matrix-core peak it runs on
  cpu_baseline the CPU oracle timed on a bounded row sample of the same GEMM workload
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA = 157.3   # TFLOP/s, MI355X dense fp32 matrix
PEAK_BF16_MFMA = 2500.0  # TFLOP/s, MI355X dense bf16 matrix
PEAK_HBM = 8000.0        # GB/s
PEAK_INT8_MFMA = 5000.0  # TOP/s, MI355X dense int8 matrix
PEAK_VALU_OPS = 78.6     # T lane-operations/s: 256 CUs x 4 SIMDs x 32 lanes x 2.4 GHz (the fp32 vector rate, 157.3
                         # TFLOP/s counting an FMA as 2; counters show kernels issuing above a 16-lane rate)
SHA_BLOCK_VALU = 1698    # VALU instructions of one SHA-256 compression in hash_leaves_kernel's block loop (gfx950 ISA)

L, D, H, HD, F, V, S, MB = 16, 2048, 16, 128, 8192, 50304, 2048, 4
PLAN = (1, 8, 1)
METRIC = "canonical-order GEMM TFLOP/s (% of bf16 peak), bit-exact; 1B step replay secs"


def attn_pairs(S, window):
    """(query, key) pairs a head computes over in one sequence: causal, or the sliding window."""
    if not window or window >= S:
        return S * (S + 1) // 2
    return window * (window + 1) // 2 + (S - window) * window


def step_flops_open1b(L, d, H, Hkv, hd, F, V, S, mb, window, full_every, ranks=1):
    """Algorithmic FLOP of one step of the paper's own architecture (grouped heads, hybrid windows): every
    forward and backward GEMM, attention over visible (query, key) pairs only."""
    T = mb * S
    N = d + 2 * Hkv * hd
    fwd_layer = 2 * T * (d * N + d * d + d * 2 * F + F * d)
    total = 0
    for l in range(L):
        full = (full_every and (l + 1) % full_every == 0) or l == L - 1
        pairs = attn_pairs(S, 0 if full else window)
        total += 3 * fwd_layer + mb * H * pairs * 12 * hd  # QK^T, PV forward; dP, dQ, dK, dV backward
    return ranks * (total + 3 * 2 * T * d * V)


def step_flops(L=L, d=D, H=H, hd=HD, F=F, V=V, S=S, mb=MB, ranks=8):
    """Algorithmic FLOPs of one step: every GEMM of forward and backward (2 per multiply-add), attention
    counted over the unmasked (causal) entries only."""
    T = mb * S
    fwd_layer = 2 * T * (d * 3 * d + d * d + d * 2 * F + F * d)
    causal = mb * H * (S * (S + 1) // 2) * hd * 2  # one causal S x S x hd product
    attn_fwd, attn_bwd = 2 * causal, 4 * causal
    head = 2 * T * d * V
    per_mb = L * (3 * fwd_layer + attn_fwd + attn_bwd) + 3 * head
    return per_mb * ranks


def gemm_traffic_from_profile():
    """HBM bytes per launch of the dominant GEMM from the committed counter summary, or None when the GEMM
    source has changed since the counters were taken."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", "gemm_8192x16384x2048_launch_and_traffic.md")
    src = os.path.join(ROOT, "paper_2609_17380_amd", "csrc", "gemm.hip")
    if not os.path.exists(prof):
        return None
    fields = dict(l.split(":", 1) for l in open(prof) if l.startswith(("traffic_bytes_per_launch:", "gemm_source_sha256:")))
    if fields.get("gemm_source_sha256", "").strip() != hashlib.sha256(open(src, "rb").read()).hexdigest():
        return None
    return int(fields["traffic_bytes_per_launch"])


# GEMM shapes of the 1B decoder over one microbatch of 8192 tokens: (name, m, n, k, A stored [k, m], B stored [n, k])
GEMM_SWEEP = [("qkv", 8192, 6144, 2048, 0, 1), ("out", 8192, 2048, 2048, 0, 1), ("gate_up", 8192, 16384, 2048, 0, 1),
              ("down", 8192, 2048, 8192, 0, 1), ("head", 8192, 50304, 2048, 0, 1),
              ("wgrad_qkv", 6144, 2048, 8192, 1, 0), ("wgrad_out", 2048, 2048, 8192, 1, 0),
              ("wgrad_gate_up", 16384, 2048, 8192, 1, 0), ("wgrad_down", 2048, 8192, 8192, 1, 0),
              ("wgrad_head", 50304, 2048, 8192, 1, 0),
              ("dgrad_qkv", 8192, 2048, 6144, 0, 0), ("dgrad_gate_up", 8192, 2048, 16384, 0, 0),
              ("dgrad_down", 8192, 8192, 2048, 0, 0), ("dgrad_head", 8192, 2048, 50304, 0, 0)]


def _timed(torch, stream, fn, reps, warm=1):
    for _ in range(warm):
        fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def _hbm(ms, nbytes):
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "ms": round(ms, 4), "bytes": int(nbytes), "achieved": round(gbs, 1), "unit": "GB/s",
            "peak": PEAK_HBM, "frac": round(gbs / PEAK_HBM, 4)}


KERNEL_GROUPS = ("gemm", "int8", "rows", "embed", "plan", "block", "attn_i8", "open1b")


def kernel_table(C, I, torch, np, stream, dev, groups=KERNEL_GROUPS):
    """Each entry point at the shapes of the single-kernel workloads: the GEMM sweep over the 1B shapes, RMSNorm
    over a microbatch, causal softmax at 16 heads x 2048 x 2048, cross-entropy 8192 x 50304, the ordered sum of 8
    gradient buffers of 1.2e9 fp32, AdamW over 1.2e9 parameters, the global gradient norm (and clip) over the
    1B gradient, and one decoder block forward + backward.
    Inputs are seeded N(0, sigma) draws made on the device (the values do not change the work); bytes are the
    algorithmic minimum each kernel must move."""
    g = torch.Generator(device=dev)
    g.manual_seed(0)

    def randn(shape, std=1.0, dtype=torch.float32):
        return (torch.randn(shape, generator=g, device=dev, dtype=torch.float32) * std).to(dtype)

    class Entries(dict):  # each entry is printed when it is measured (a long table shows its progress)
        def __setitem__(self, k_, v_):
            super().__setitem__(k_, v_)
            frac = f"{100 * v_['frac']:.1f}%" if v_.get("frac") is not None else "no single roofline"
            print(f"bench:   {k_}: {v_['ms']} ms, {v_['achieved']} {v_['unit']} ({frac})", file=sys.stderr, flush=True)

        def update(self, other):
            for k_, v_ in other.items():
                self[k_] = v_

    out = Entries()
    print("bench: kernel table", file=sys.stderr, flush=True)

    def want(group):
        return group in groups

    if want("gemm"):
        for si, (name, m, n, k, ta, tb) in enumerate(GEMM_SWEEP):
            a = randn((k, m) if ta else (m, k), dtype=torch.bfloat16)
            b = randn((n, k) if tb else (k, n), dtype=torch.bfloat16)
            c = torch.empty((m, n), dtype=torch.float32, device=dev)
            lda, ldb = a.shape[1], b.shape[1]
            # warm launches (ten before the first shape of the sweep, which otherwise carries the clock ramp after
            # the step replays and the state hash)
            ms = _timed(torch, stream, lambda: C.gemm(m, n, k, a, lda, b, ldb, c, n, ta, tb, stream=stream), 5,
                        warm=10 if si == 0 else 2)
            tf = 2.0 * m * n * k / (ms * 1e-3) / 1e12
            out[f"gemm_{name}_{m}x{n}x{k}"] = {"bound": "mfma", "ms": round(ms, 4), "achieved": round(tf, 2),
                                               "unit": "TFLOP/s", "peak": PEAK_FP32_MFMA,
                                               "frac": round(tf / PEAK_FP32_MFMA, 4),
                                               "pct_bf16_peak": round(100 * tf / PEAK_BF16_MFMA, 3)}
            del a, b, c

    if want("int8"):
        # the int8 quantised linear (the paper's W8A8 path): exact int8 GEMM with dequantisation at the
        # projection shapes of the 1B decoder, and the quantisers
        for name, m, n, k in [("qkv", 8192, 6144, 2048), ("gate_up", 8192, 16384, 2048), ("down", 8192, 2048, 8192),
                              ("out", 8192, 2048, 2048)]:
            qa = torch.randint(-128, 128, (m, k), generator=g, device=dev, dtype=torch.int8)
            qb = torch.randint(-128, 128, (n, k), generator=g, device=dev, dtype=torch.int8)
            sa = torch.full((1,), 0.01, device=dev)
            sb = torch.full((n,), 0.001, device=dev)
            yq = torch.empty((m, n), dtype=torch.float32, device=dev)
            ms = _timed(torch, stream, lambda: C.gemm_i8(m, n, k, qa, k, qb, k, y=yq, sa=sa, sb=sb, stream=stream), 5)
            tops = 2.0 * m * n * k / (ms * 1e-3) / 1e12
            out[f"gemm_i8_{name}_{m}x{n}x{k}"] = {"bound": "mfma", "ms": round(ms, 4), "achieved": round(tops, 1),
                                                  "unit": "TOP/s", "peak": PEAK_INT8_MFMA,
                                                  "frac": round(tops / PEAK_INT8_MFMA, 4)}
            del qa, qb, yq
        # int8 backward of the gate/up projection: rotated straight-through dx and dW (2 GEMMs of 2*T*N*K each)
        Tq, Nq, Kq = 8192, 16384, 2048
        dyq = randn((Tq, Nq), 1e-3)
        qxq = torch.randint(-128, 128, (Tq, Kq), generator=g, device=dev, dtype=torch.int8)
        qwq = torch.randint(-128, 128, (Nq, Kq), generator=g, device=dev, dtype=torch.int8)
        sxq = torch.full((1,), 0.02, device=dev)
        swq = torch.full((Nq,), 0.001, device=dev)
        dxq = torch.empty((Tq, Kq), device=dev)
        dwq = torch.empty((Nq, Kq), device=dev)
        wsq = torch.empty(C.qlinear_bwd_workspace_bytes(Tq, Nq, Kq), dtype=torch.uint8, device=dev)
        ms = _timed(torch, stream, lambda: C.qlinear_bwd(Tq, Nq, Kq, dyq, qxq, sxq, qwq, swq, dxq, dwq, wsq,
                                                        stream=stream), 3)
        tops = 2 * 2.0 * Tq * Nq * Kq / (ms * 1e-3) / 1e12
        out[f"qlinear_bwd_gate_up_{Tq}x{Nq}x{Kq}"] = {"bound": "mfma", "ms": round(ms, 4), "achieved": round(tops, 1),
                                                     "unit": "TOP/s", "peak": PEAK_INT8_MFMA,
                                                     "frac": round(tops / PEAK_INT8_MFMA, 4)}
        del dyq, qxq, qwq, dxq, dwq, wsq
        wq = randn((16384, 2048), 0.02, torch.bfloat16)
        swq = torch.empty(16384, dtype=torch.float32, device=dev)
        ms = _timed(torch, stream, lambda: C.quant_scales(16384, 2048, wq, swq, stream=stream), 10)
        out["quant_scales_16384x2048"] = _hbm(ms, 16384 * 2048 * 2 + 16384 * 4)
        qq = torch.empty((16384, 2048), dtype=torch.int8, device=dev)
        ms = _timed(torch, stream, lambda: C.quantize(16384, 2048, wq, swq, True, qq, stream=stream), 10)
        out["quantize_16384x2048_bf16"] = _hbm(ms, 16384 * 2048 * 3 + 16384 * 4)
        del wq, swq, qq

    if want("rows"):
        T, d = MB * S, D
        x = randn((T, d))
        gain = torch.full((d,), 0x3F80, dtype=torch.int16, device=dev)
        y = torch.empty((T, d), dtype=torch.int16, device=dev)
        rstd = torch.empty(T, dtype=torch.float32, device=dev)
        ms = _timed(torch, stream, lambda: C.rownorm(C.FWD, T, d, x, gain, 1e-5, y=y, rstd=rstd, stream=stream), 20)
        out[f"rownorm_fwd_{T}x{d}"] = _hbm(ms, T * d * (4 + 2) + T * 4 + d * 2)
        dy, dx = randn((T, d)), torch.empty((T, d), dtype=torch.float32, device=dev)
        dgain = torch.empty(d, dtype=torch.float32, device=dev)
        ms = _timed(torch, stream, lambda: C.rownorm(C.BWD, T, d, x, gain, 1e-5, rstd=rstd, dy=dy, dx=dx, dgain=dgain,
                                                    stream=stream), 20)
        out[f"rownorm_bwd_{T}x{d}"] = _hbm(ms, T * d * 12 + T * 4 + d * 6)
        del x, y, rstd, dy, dx, dgain

        bh = 16
        raw = randn((bh, S, S))
        probs = torch.empty((bh, S, S), dtype=torch.int16, device=dev)
        scale = float(np.float32(1 / np.sqrt(128)))
        ms = _timed(torch, stream, lambda: C.softmax_xent(C.SOFTMAX_CAUSAL, bh * S, S, raw, probs, scale=scale,
                                                         stream=stream), 10)
        out[f"softmax_causal_{bh}x{S}x{S}"] = _hbm(ms, bh * (S * (S + 1) // 2) * 4 + bh * S * S * 2)
        del raw, probs

        logits = randn((T, V), std=2.0, dtype=torch.bfloat16)
        tgt = torch.randint(0, V, (T,), generator=g, device=dev, dtype=torch.int32)
        dl = torch.empty((T, V), dtype=torch.bfloat16, device=dev)
        rl = torch.empty(T, dtype=torch.float32, device=dev)
        ml = torch.empty(1, dtype=torch.float32, device=dev)
        ms = _timed(torch, stream, lambda: C.softmax_xent(C.XENT, T, V, logits, dl, targets=tgt, inv_tokens=1.0 / T,
                                                         row_loss=rl, mean_loss=ml, stream=stream), 10)
        out[f"xent_{T}x{V}"] = _hbm(ms, T * V * 4 + T * 8)
        del logits, tgt, dl, rl, ml

    if want("embed"):
        # R11 embedding backward of one 1B microbatch (8192 tokens, d 2048, vocabulary 50304): bound by writing
        # the +0 rows of dE and reading dx once
        Te, Ve = MB * S, V
        tok = torch.randint(0, Ve, (Te,), generator=g, device=dev, dtype=torch.int32)
        dxe = randn((Te, D), 1e-3)
        dE = torch.empty((Ve, D), dtype=torch.float32, device=dev)
        wse = torch.empty(C.embed_bwd_workspace_bytes(Te, D), dtype=torch.uint8, device=dev)
        ms = _timed(torch, stream, lambda: C.embed_bwd(Te, Ve, D, tok, dxe, dE, wse, stream=stream), 10)
        out[f"embed_bwd_{Te}x{D}_v{Ve}"] = _hbm(ms, Te * D * 4 + Ve * D * 4 + Te * 4)
        del tok, dxe, dE, wse

    if want("plan"):
        n = 1_200_000_000
        grads = [randn((n,), std=1e-3) for _ in range(8)]
        gsum = torch.empty(n, dtype=torch.float32, device=dev)
        ms = _timed(torch, stream, lambda: C.grad_accum(C.DPPlan(1, 8, 1), n, grads, gsum, stream=stream), 3)
        out["grad_accum_8x1.2e9"] = _hbm(ms, 9 * n * 4)
        del grads
        torch.cuda.empty_cache()
        p = randn((n,), std=0.02, dtype=torch.bfloat16)
        m1 = torch.zeros(n, dtype=torch.float32, device=dev)
        v1 = torch.zeros(n, dtype=torch.float32, device=dev)
        consts = C.AdamWConsts(*I.adamw_constants())
        ms = _timed(torch, stream, lambda: C.adamw([p], [m1], [v1], [gsum], [1], consts, stream=stream), 3)
        out["adamw_1.2e9"] = _hbm(ms, n * 24)
        del p, m1, v1
        # R15 over the whole 1B gradient in one flat buffer (the step's launch): the norm alone (clip not
        # engaged: 4 bytes read per element), then norm + in-place clip (engaged: 12 bytes per element)
        P = sum(int(np.prod(sh)) for _, sh, _, _ in I.model_param_shapes(L, D, F, V))
        gflat = randn((P,), std=1e-3)
        nrm = torch.empty(1, dtype=torch.float32, device=dev)
        cws = torch.empty(C.clip_grad_norm_workspace_bytes([gflat]), dtype=torch.uint8, device=dev)
        off = C.make_clip(float(np.float32(1e30)), float("inf"), 0, nrm)
        ms = _timed(torch, stream, lambda: C.clip_grad_norm([gflat], off, cws, stream=stream), 5)
        out[f"global_norm_{P}"] = _hbm(ms, 4 * P)
        on = C.make_clip(1e-30, float("inf"), 0, nrm)  # coef < 1 every call: the clip pass runs each time
        ms = _timed(torch, stream, lambda: C.clip_grad_norm([gflat], on, cws, stream=stream), 3)
        out[f"global_norm_and_clip_{P}"] = _hbm(ms, 12 * P)
        del gflat, gsum, cws
        torch.cuda.empty_cache()

    if want("block"):
        cfg = C.ModelCfg(1, D, H, HD, F, V, S, 1, np.float32(1e-5))
        xb, dyb = randn((S, D)), randn((S, D)).to(torch.bfloat16).float()
        w = [torch.full((D,), 0x3F80, dtype=torch.int16, device=dev), randn((3 * D, D), 0.02, torch.bfloat16),
             randn((D, D), 0.02, torch.bfloat16), torch.full((D,), 0x3F80, dtype=torch.int16, device=dev),
             randn((2 * F, D), 0.02, torch.bfloat16), randn((D, F), 0.02, torch.bfloat16)]
        dw = [torch.empty(t.shape, dtype=torch.float32, device=dev) for t in w]
        cos, sin = I.rope_tables(S, HD)
        cos, sin = torch.from_numpy(cos).to(dev), torch.from_numpy(sin).to(dev)
        yb, dxb = torch.empty_like(xb), torch.empty_like(xb)
        wsb = torch.empty(C.block_workspace_bytes(cfg, 1), dtype=torch.uint8, device=dev)
        ms = _timed(torch, stream, lambda: C.block_fwd_bwd(cfg, 1, xb, dyb, w, cos, sin, yb, dxb, dw, wsb,
                                                          stream=stream), 3)
        fl = step_flops(L=1, mb=1, ranks=1) - 3 * 2 * S * D * V  # one block, no head
        out[f"block_fwd_bwd_seq{S}"] = {"bound": "mfma", "ms": round(ms, 3), "achieved": round(fl / (ms * 1e-3) / 1e12, 2),
                                        "unit": "TFLOP/s", "peak": PEAK_FP32_MFMA,
                                        "frac": round(fl / (ms * 1e-3) / 1e12 / PEAK_FP32_MFMA, 4)}
        del xb, dyb, w, dw, yb, dxb, wsb
        torch.cuda.empty_cache()
    if want("attn_i8"):
        out.update(int8_attention(C, torch, stream, dev, randn))
    if want("open1b"):
        out.update(open1b_step(C, I, torch, np, stream, dev))
        out.update(open1b_step(C, I, torch, np, stream, dev, int8_attn=True))
        out.update(open1b_step(C, I, torch, np, stream, dev, int8_attn=True, int8_linear=True))
    return dict(out)


def int8_attention(C, torch, stream, dev, randn):
    """The int8 path's attention kernels at the paper's shape (4 sequences x 16 heads (4 key/value heads) x 4096
    tokens, head_dim 128), full causal and 512-token window: P.V in int8 per block (bound by reading P once:
    2 bytes per visible entry, plus V and O) and dQ in 64-bit fixed point (bound by the VALU: one binary64 fma
    and one 64-bit integer add per product, each issuing at half the 32-lane rate, so 4 lane-operations)."""
    o = O1B
    B, Hh, Hkv, Ss, hd = o["mb"], o["H"], o["Hkv"], o["S"], o["hd"]
    out = {}
    P = randn((B, Hh, Ss, Ss), 1e-3, torch.bfloat16).abs()
    Vt = randn((B, Hkv, Ss, hd), 1.0, torch.bfloat16)
    ob = torch.empty((B, Ss, Hh * hd), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(C.attn_pv_i8_workspace_bytes(B, Hkv, Ss, hd), dtype=torch.uint8, device=dev)
    dQ = torch.empty((B, Ss, Hh * hd), dtype=torch.float32, device=dev)
    for window in (0, o["window"]):
        pairs = attn_pairs(Ss, window)
        ms = _timed(torch, stream, lambda: C.attn_pv_i8(B, Hh, Hkv, Ss, hd, window, P, Vt, ws, o_bf16=ob,
                                                       stream=stream), 3)
        nbytes = 2 * B * Hh * pairs + 2 * B * Hkv * Ss * hd + 2 * B * Ss * Hh * hd
        e = _hbm(ms, nbytes)
        e["int8_tops"] = round(2.0 * B * Hh * pairs * hd / (ms * 1e-3) / 1e12, 1)
        out[f"attn_pv_i8_{B}x{Hh}x{Ss}x{hd}_w{window}"] = e
        ms = _timed(torch, stream, lambda: C.attn_dq_fixed(B, Hh, Hkv, Ss, hd, window, 40, P, Vt, dQ,
                                                          stream=stream), 3)
        prods = B * Hh * pairs * hd
        ops = 4.0 * prods / (ms * 1e-3) / 1e12
        out[f"attn_dq_fixed_{B}x{Hh}x{Ss}x{hd}_w{window}"] = {
            "bound": "alu", "ms": round(ms, 4), "achieved": round(ops, 2), "unit": "T lane-op/s",
            "peak": PEAK_VALU_OPS, "frac": round(ops / PEAK_VALU_OPS, 4),
            "products_per_s": round(prods / (ms * 1e-3), 1)}
    del P, Vt, ob, ws, dQ
    torch.cuda.empty_cache()
    return out


# The paper's own 1B architecture (its hyperparameter table): 24 layers, d 2048, 16 query / 4 key-value heads
# of 128, FFN 5632, vocab 128256, sequence 4096, sliding window 512 with every 5th and the last layer full,
# gain-free QK-norm, embedding norm, z-loss 1e-4; 4 sequences per microbatch.
O1B = dict(L=24, d=2048, H=16, Hkv=4, hd=128, F=5632, V=128256, S=4096, mb=4, window=512, full_every=5)


def open1b_step(C, I, torch, np, stream, dev, int8_attn=False, int8_linear=False):
    """One step of the paper's architecture with every variant on (one rank, one microbatch of 4 x 4096 tokens,
    the clip at 1.0), timed after one warmup step.  int8_attn: also the int8 path's attention kernels (P.V in
    int8 per block, dQ in 64-bit fixed point with 40 fractional bits); int8_linear: the four projections of
    every block in int8 with learned activation steps (the paper's production configuration with both)."""
    o = O1B
    tag = ("all_variants" + ("_int8_attention" if int8_attn and not int8_linear else "")
           + ("_int8_production" if int8_linear else ""))
    print(f"bench: open-1B step ({tag})", file=sys.stderr, flush=True)
    cfg = C.ModelCfg(o["L"], o["d"], o["H"], o["hd"], o["F"], o["V"], o["S"], o["mb"], np.float32(1e-5), o["Hkv"],
                     1, 1, o["window"], o["full_every"], np.float32(1e-4), int(int8_attn), 40 if int8_attn else 0,
                     int(int8_linear))
    plan = C.DPPlan(1, 1, 1)
    params = I.model_params(o["L"], o["d"], o["F"], o["V"], seed=0, std=0.02, kv_dim=o["Hkv"] * o["hd"],
                            embed_norm=True, int8_linear=int8_linear)
    pg = [torch.from_numpy(p.view(np.int16)).to(dev) for p in params]
    del params
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=dev) for p in pg]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=dev) for p in pg]
    windows = torch.from_numpy(I.uniform_int((o["mb"], o["S"] + 1), 0, I.TENSOR_IDS["windows"], o["V"])).to(dev)
    cos, sin = I.rope_tables(o["S"], o["hd"])
    cos, sin = torch.from_numpy(cos).to(dev), torch.from_numpy(sin).to(dev)
    consts = C.AdamWConsts(*I.adamw_constants())
    ws = torch.empty(C.step_workspace_bytes(cfg, plan), dtype=torch.uint8, device=dev)
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    gnorm = torch.zeros(1, dtype=torch.float32, device=dev)
    clip = C.make_clip(1.0, float("inf"), 0, gnorm)
    ms = _timed(torch, stream, lambda: C.step(cfg, plan, pg, mg, vg, windows, cos, sin, consts, ws, loss,
                                              stream=stream, clip=clip), 1)
    fl = step_flops_open1b(o["L"], o["d"], o["H"], o["Hkv"], o["hd"], o["F"], o["V"], o["S"], o["mb"], o["window"],
                           o["full_every"])
    tf = fl / (ms * 1e-3) / 1e12
    res = {"bound": "mfma", "ms": round(ms, 2), "achieved": round(tf, 2), "unit": "TFLOP/s", "peak": PEAK_FP32_MFMA,
           "frac": round(tf / PEAK_FP32_MFMA, 4), "flops": fl, "tokens_per_s": round(o["mb"] * o["S"] / (ms * 1e-3), 1),
           "loss": float(loss.item()), "grad_norm_preclip": float(gnorm.item())}
    del ws, pg, mg, vg
    torch.cuda.empty_cache()
    if int8_linear:  # int8 projections next to fp32 canonical attention and head: no single roofline
        res.update({"bound": "mixed", "peak": None, "frac": None,
                    "note": "algorithmic rate; the int8 projection GEMMs count 2 operations per multiply-add"})
    return {"step_open1b_4x4096_" + tag: res}


def oracle_single_thread(oracle, I, np):
    """The oracle on one host thread: the 128x256x128 canonical GEMM (seed 0), 16 rows of the 8192 x 50304
    cross-entropy and a 2^22-element chunk of the ordered sum of 8 gradient buffers (plus AdamW on it)."""
    res = {}
    oracle.set_threads(1)
    try:
        a = I.normal_bf16((128, 256), 0, I.TENSOR_IDS["gemm_a"])
        b = I.normal_bf16((256, 128), 0, I.TENSOR_IDS["gemm_b"])
        t0 = time.time()
        for _ in range(5):
            oracle.gemm(a, b)
        sec = (time.time() - t0) / 5
        res["gemm_128x256x128_ms"] = round(sec * 1e3, 3)
        res["gemm_128x256x128_gflops"] = round(2 * 128 * 256 * 128 / sec / 1e9, 3)
        rows = 16
        logits = I.normal_bf16((rows, V), 0, I.TENSOR_IDS["logits"], std=2.0)
        tgt = I.uniform_int((rows,), 0, I.TENSOR_IDS["targets"], V).reshape(-1)
        t0 = time.time()
        oracle.xent(logits, tgt, 1.0 / 8192)
        sec = time.time() - t0
        res["xent_16x50304_ms"] = round(sec * 1e3, 2)
        res["xent_gb_per_s"] = round(rows * V * 4 / sec / 1e9, 4)
        n = 1 << 22
        grads = [I.normal_f32((n,), 0, I.TENSOR_IDS["grads"] + r, std=1e-3) for r in range(8)]
        t0 = time.time()
        gsum = oracle.grad_accum(grads, 1, 8, 1)
        sec = time.time() - t0
        res["grad_accum_8x4194304_ms"] = round(sec * 1e3, 1)
        res["grad_accum_gb_per_s"] = round(9 * n * 4 / sec / 1e9, 3)
        p = I.normal_bf16((n,), 0, I.TENSOR_IDS["adam_p"], std=0.02)
        m, v = np.zeros(n, np.float32), np.zeros(n, np.float32)
        t0 = time.time()
        oracle.adamw([p], [m], [v], [gsum], [1], oracle.AdamWConsts(*I.adamw_constants()))
        sec = time.time() - t0
        res["adamw_4194304_ms"] = round(sec * 1e3, 1)
        res["adamw_gb_per_s"] = round(24 * n / sec / 1e9, 3)
    finally:
        oracle.set_threads(os.cpu_count() or 1)
    print(f"bench: oracle on one thread: {res}", file=sys.stderr, flush=True)
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--hash-steps", type=int, default=1,
                    help="steps timed again with the per-step audit hash inside canon_step (0: skip)")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gemm-reps", type=int, default=10)
    ap.add_argument("--no-kernel-table", action="store_true")
    ap.add_argument("--kernels", default=",".join(KERNEL_GROUPS),
                    help="comma-separated groups of the kernel table: " + ",".join(KERNEL_GROUPS))
    ap.add_argument("--no-step", action="store_true",
                    help="time only the kernel table (no step replays, no dominant-GEMM launches); prints its JSON")
    ap.add_argument("--open1b-only", action="store_true",
                    help="time only the paper-architecture step (all variants; without and with the int8 "
                         "attention kernels; the int8 production configuration) and print its entries")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build measures one GPU only (data-parallel ranks are emulated on one device by "
              "Algorithm 1); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_17380_amd.canon as C
    import paper_2609_17380_amd.inputs as I

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    groups = tuple(x for x in args.kernels.split(",") if x)
    if args.no_step:
        print(json.dumps({"kernels": kernel_table(C, I, torch, np, stream, dev, groups)}), flush=True)
        return
    if args.open1b_only:
        res = open1b_step(C, I, torch, np, stream, dev)
        res.update(open1b_step(C, I, torch, np, stream, dev, int8_attn=True))
        res.update(open1b_step(C, I, torch, np, stream, dev, int8_attn=True, int8_linear=True))
        print(json.dumps(res), flush=True)
        return
    print("bench: generating inputs", file=sys.stderr, flush=True)
    t0 = time.time()
    params = I.model_params(L, D, F, V, seed=0, std=0.02)
    pg = [torch.from_numpy(p.view(np.int16)).to(dev) for p in params]
    del params
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=dev) for p in pg]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=dev) for p in pg]
    R = PLAN[1] * PLAN[2]
    windows = torch.from_numpy(I.uniform_int((R * PLAN[0] * MB, S + 1), 0, I.TENSOR_IDS["windows"], V)).to(dev)
    cos, sin = I.rope_tables(S, HD)
    cos, sin = torch.from_numpy(cos).to(dev), torch.from_numpy(sin).to(dev)
    cfg = C.ModelCfg(L, D, H, HD, F, V, S, MB, np.float32(1e-5))
    plan = C.DPPlan(*PLAN)
    consts = C.AdamWConsts(*I.adamw_constants())
    ws = torch.empty(C.step_workspace_bytes(cfg, plan), dtype=torch.uint8, device=dev)
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    # the paper's clip to a global norm of 1.0 (R15) runs in every step; the spike rule is off here, since a
    # skipped update would leave work out of the timed step
    gnorm = torch.zeros(1, dtype=torch.float32, device=dev)
    clip = C.make_clip(1.0, float("inf"), 0, gnorm)
    torch.cuda.synchronize()
    print(f"bench: inputs ready in {time.time() - t0:.1f}s; workspace {ws.numel() / 1e9:.1f} GB",
          file=sys.stderr, flush=True)

    # every replay restores the initial state first (parameters copied back, moments zeroed: 12.8 GB of
    # stores, ~3 ms, inside the timed region), so each timed step recomputes the same step t = 1 and its
    # output state must hash to the same digest as the first
    p0 = [t.clone() for t in pg]
    state = pg + mg + vg
    hws = torch.empty(C.state_hash_workspace_bytes(state), dtype=torch.uint8, device=dev)
    hdig = torch.empty(32, dtype=torch.uint8, device=dev)

    def restore():
        for t, t0 in zip(pg, p0):
            t.copy_(t0)
        for t in mg + vg:
            t.zero_()

    def one_step():
        restore()
        C.step(cfg, plan, pg, mg, vg, windows, cos, sin, consts, ws, loss, stream=stream, clip=clip)

    def state_digest():
        C.state_hash(state, hdig, hws, stream=stream)
        torch.cuda.synchronize()
        return bytes(hdig.cpu().numpy().tobytes()).hex()

    first_loss = first_digest = None
    for i in range(max(args.warmup, 1)):
        one_step()
        torch.cuda.synchronize()
        if first_digest is None:
            first_loss, first_digest = float(loss.item()), state_digest()
        print(f"bench: warmup step {i} loss {loss.item():.5f} pre-clip grad norm {gnorm.item():.5f}",
              file=sys.stderr, flush=True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for i in range(args.steps):
        one_step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    last_digest = state_digest()
    print(f"bench: {args.steps} steps, {ms / 1000:.3f} s/step, loss {loss.item():.5f}; state digest "
          f"{last_digest[:16]}.. (first step {first_digest[:16]}..)", file=sys.stderr, flush=True)
    flops = step_flops()
    value = flops / (ms * 1e-3) / 1e12

    # the paper's hash-on / hash-off comparison: the same step with the per-step audit hash (H1 of the
    # windows, parameters, m, v and reduced gradient, 17.9 GB) computed inside canon_step
    audit = None
    if args.hash_steps > 0:
        sdig = torch.zeros(32, dtype=torch.uint8, device=dev)

        def one_step_hashed():
            restore()
            C.step(cfg, plan, pg, mg, vg, windows, cos, sin, consts, ws, loss, stream=stream, clip=clip,
                   state_digest=sdig)
        one_step_hashed()
        torch.cuda.synchronize()
        ev0.record(stream)
        for i in range(args.hash_steps):
            one_step_hashed()
        ev1.record(stream)
        torch.cuda.synchronize()
        ms_h = ev0.elapsed_time(ev1) / args.hash_steps
        audit = {"steps": args.hash_steps, "ms_per_step_hash_on": round(ms_h, 2), "ms_per_step_hash_off": round(ms, 2),
                 "overhead_pct": round(100 * (ms_h - ms) / ms, 3),
                 "step_state_digest": bytes(sdig.cpu().numpy().tobytes()).hex(),
                 "params_m_v_digest_unchanged": state_digest() == first_digest}
        print(f"bench: hash on {ms_h / 1000:.3f} s/step ({audit['overhead_pct']:.2f}% over hash off); step digest "
              f"{audit['step_state_digest'][:16]}..", file=sys.stderr, flush=True)

    # dominant kernel: the canonical GEMM at the fused gate/up shape (8192 x 16384 x 2048), timed per launch
    gm, gn, gk = MB * S, 2 * F, D
    a = torch.from_numpy(I.normal_bf16((gm, gk), 0, I.TENSOR_IDS["gemm_a"]).view(np.int16)).to(dev)
    b = torch.from_numpy(I.normal_bf16((gn, gk), 0, I.TENSOR_IDS["gemm_b"]).view(np.int16)).to(dev)
    c = torch.empty((gm, gn), dtype=torch.float32, device=dev)
    C.gemm(gm, gn, gk, a, gk, b, gk, c, gn, 0, 1, stream=stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.gemm_reps):
        C.gemm(gm, gn, gk, a, gk, b, gk, c, gn, 0, 1, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    gemm_ms = e0.elapsed_time(e1) / args.gemm_reps
    gemm_flop = 2.0 * gm * gn * gk
    gemm_tf = gemm_flop / (gemm_ms * 1e-3) / 1e12
    # the same shape through an unconstrained library GEMM (hipBLASLt via torch), for the cost of the order
    ab, bb = a.view(torch.bfloat16), b.view(torch.bfloat16)
    torch.matmul(ab, bb.t())
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.gemm_reps):
        torch.matmul(ab, bb.t())
    e1.record(stream)
    torch.cuda.synchronize()
    blas_ms = e0.elapsed_time(e1) / args.gemm_reps
    blas_tf = gemm_flop / (blas_ms * 1e-3) / 1e12
    traffic = gemm_traffic_from_profile()
    roofline = {"bound": "mfma", "achieved": round(gemm_tf, 2), "peak": PEAK_FP32_MFMA, "unit": "TFLOP/s",
                "frac": round(gemm_tf / PEAK_FP32_MFMA, 4), "traffic": traffic,
                "kernel": f"gemm_mfma_kernel {gm}x{gn}x{gk} (fp32 rank-1 MFMA chains)",
                "avg_launch_ms": round(gemm_ms, 4), "pct_bf16_peak": round(100 * gemm_tf / PEAK_BF16_MFMA, 3)}

    del ws, p0, hws
    torch.cuda.empty_cache()
    kernels = {} if args.no_kernel_table else kernel_table(C, I, torch, np, stream, dev, groups)
    if not args.no_kernel_table:
        # the canonical state hash of the post-step state (parameters, both moments): 1,279,854,592 x 10 bytes
        hws = torch.empty(C.state_hash_workspace_bytes(state), dtype=torch.uint8, device=dev)
        hd = torch.empty(32, dtype=torch.uint8, device=dev)
        hms = _timed(torch, stream, lambda: C.state_hash(state, hd, hws, stream=stream), 3)
        hbytes = sum(t.numel() * t.element_size() for t in state)
        # SHA-256 is bound by integer VALU issue, not by HBM: the leaf blocks' compressions at
        # SHA_BLOCK_VALU instructions each (the tree and digest nodes, < 0.1% more, are not counted)
        tops = hbytes / 64 * SHA_BLOCK_VALU / (hms * 1e-3) / 1e12
        kernels["state_hash_params_m_v"] = {
            "bound": "alu", "ms": round(hms, 4), "bytes": int(hbytes),
            "gb_per_s": round(hbytes / (hms * 1e-3) / 1e9, 1), "achieved": round(tops, 2), "unit": "T lane-op/s",
            "peak": PEAK_VALU_OPS, "frac": round(tops / PEAK_VALU_OPS, 4)}
        print(f"bench:   state_hash_params_m_v: {hms:.3f} ms, {kernels['state_hash_params_m_v']['gb_per_s']} GB/s, "
              f"{tops:.2f} T VALU op/s", file=sys.stderr, flush=True)
        del hws

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        ah = a.cpu().numpy().view(np.uint16)
        bh = b.cpu().numpy().view(np.uint16)
        rows, spent = 4, 0.0
        while True:  # grow the row sample until it takes about 10 s
            t1 = time.time()
            oracle.gemm(ah[:rows], bh, trans_b=True)
            spent = time.time() - t1
            if spent > 10.0 or rows >= gm:
                break
            rows = min(gm, int(rows * max(2.0, min(8.0, 12.0 / max(spent, 1e-3)))))
        cpu_tf = 2.0 * rows * gn * gk / spent / 1e12
        cpu = {"value": cpu_tf, "unit": "TFLOP/s", "cores": oracle.num_threads(), "kind": "oracle",
               "sample": f"rows 0..{rows - 1} of the canonical {gm}x{gn}x{gk} gate/up GEMM ({spent:.1f} s)"}
        print(f"bench: oracle {cpu_tf * 1e3:.3f} GFLOP/s on {oracle.num_threads()} threads", file=sys.stderr,
              flush=True)
        cpu["single_thread"] = oracle_single_thread(oracle, I, np)

    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 2), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16 operands, f32 canonical accumulation", "data": "synthetic",
        "config": {"workload": "1B-shaped canonical step replay (16 layers, d 2048, 16x128 heads, FFN 8192, "
                               "vocab 50304, seq 2048; 8 ranks x 4 sequences by Algorithm 1; AdamW)",
                   "global_batch": R * PLAN[0] * MB, "seq_len": S, "parallelism": "dp8 emulated on 1 GPU",
                   "plan": {"accum": PLAN[0], "dp_shard": PLAN[1], "dp_replicate": PLAN[2]},
                   "clip": {"max_norm": 1.0, "spike_rule": "off (a skipped update would drop work)"}},
        "step_replay_seconds": round(ms / 1000, 3), "step_flops": flops, "tokens_per_s": round(
            R * PLAN[0] * MB * S / (ms * 1e-3), 1),
        "gemm_tflops": round(gemm_tf, 2), "gemm_pct_bf16_peak": round(100 * gemm_tf / PEAK_BF16_MFMA, 3),
        "gemm_unconstrained_library_tflops": round(blas_tf, 2),
        "roofline": roofline, "cpu_baseline": cpu, "loss": float(loss.item()), "loss_first_step": first_loss,
        "grad_norm_preclip": float(gnorm.item()),
        "replay": {"state_digest_first_step": first_digest, "state_digest_after_timed_steps": last_digest,
                   "identical": first_digest == last_digest,
                   "note": "each replay restores the initial parameters and zero moments (inside the timed "
                           "region) and recomputes step t = 1; the digest is the canonical state hash (H1) of "
                           "the post-AdamW parameters and both moments"},
        "audit_hash": audit,
        "kernels": kernels,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
