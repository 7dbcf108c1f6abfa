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

L, D, H, HD, F, V, S, MB = 16, 2048, 16, 128, 8192, 50304, 2048, 4
PLAN = (1, 8, 1)
METRIC = "canonical-order GEMM TFLOP/s (% of bf16 peak), bit-exact; 1B step replay secs"


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gemm-reps", type=int, default=10)
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
    torch.cuda.synchronize()
    print(f"bench: inputs ready in {time.time() - t0:.1f}s; workspace {ws.numel() / 1e9:.1f} GB",
          file=sys.stderr, flush=True)

    def one_step():
        C.step(cfg, plan, pg, mg, vg, windows, cos, sin, consts, ws, loss, stream=stream)

    for i in range(args.warmup):
        one_step()
        torch.cuda.synchronize()
        print(f"bench: warmup step {i} loss {loss.item():.5f}", file=sys.stderr, flush=True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for i in range(args.steps):
        one_step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    print(f"bench: {args.steps} steps, {ms / 1000:.3f} s/step, loss {loss.item():.5f}", file=sys.stderr, flush=True)
    flops = step_flops()
    value = flops / (ms * 1e-3) / 1e12

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

    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 2), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16 operands, f32 canonical accumulation", "data": "synthetic",
        "config": {"workload": "1B-shaped canonical step replay (16 layers, d 2048, 16x128 heads, FFN 8192, "
                               "vocab 50304, seq 2048; 8 ranks x 4 sequences by Algorithm 1; AdamW)",
                   "global_batch": R * PLAN[0] * MB, "seq_len": S, "parallelism": "dp8 emulated on 1 GPU",
                   "plan": {"accum": PLAN[0], "dp_shard": PLAN[1], "dp_replicate": PLAN[2]}},
        "step_replay_seconds": round(ms / 1000, 3), "step_flops": flops, "tokens_per_s": round(
            R * PLAN[0] * MB * S / (ms * 1e-3), 1),
        "gemm_tflops": round(gemm_tf, 2), "gemm_pct_bf16_peak": round(100 * gemm_tf / PEAK_BF16_MFMA, 3),
        "gemm_unconstrained_library_tflops": round(blas_tf, 2),
        "roofline": roofline, "cpu_baseline": cpu, "loss": float(loss.item()),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
