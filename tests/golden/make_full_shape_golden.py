"""Writes the oracle's results of the full-shape parity cases as per-tensor SHA-256 digests.

Runs the CPU oracle only (no GPU code is imported):
``python tests/golden/make_full_shape_golden.py [block|step|qlinear]`` writes ``full_shape_<case>.json`` beside this
script (or into ``--out-dir``).
With CANON_REF_PROGRESS=1 the oracle prints a line after each block and head pass.  The GPU parity test
(`tests/test_gpu_full_shape.py`) regenerates the same seeded inputs, runs the HIP path and compares digests.
The oracle needs about 1 TFLOP for the block and 6 TFLOP for the step (minutes to tens of minutes on a few
cores).
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))             # tests/
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))  # repository root

import numpy as np  # noqa: E402

import full_shape_cases as FC  # noqa: E402
import oracle  # noqa: E402


def entry(name, a):
    return {"name": name, "shape": list(a.shape), "dtype": str(a.dtype), "sha256": FC.digest(a),
            "head_bits": FC.head_bits(a)}


def make_block():
    c = FC.BLOCK
    x, dy, w, cos, sin = FC.block_inputs(c)
    cfg = oracle.ModelCfg(1, c["d"], c["H"], c["hd"], c["F"], 100, c["S"], c["batch"], np.float32(c["eps"]))
    t0 = time.time()
    y, dx, dw = oracle.block_fwd_bwd(cfg, c["batch"], x, dy, w, cos, sin)
    secs = time.time() - t0
    out = [entry("y", y), entry("dx", dx)] + [entry("d" + n, g) for n, g in zip(FC.BLOCK_NAMES, dw)]
    return {"case": "block", "config": c, "oracle_seconds": round(secs, 1), "threads": oracle.num_threads(),
            "tensors": out}


def make_step():
    c = FC.STEP
    params, windows, cos, sin, k = FC.step_inputs(c)
    cfg = oracle.ModelCfg(c["L"], c["d"], c["H"], c["hd"], c["F"], c["V"], c["S"], c["mb"], np.float32(c["eps"]))
    m = [np.zeros(p.shape, np.float32) for p in params]
    v = [np.zeros(p.shape, np.float32) for p in params]
    t0 = time.time()
    loss, grads, info = oracle.step(cfg, oracle.Plan(*c["plan"]), params, m, v, windows, cos, sin,
                                    oracle.AdamWConsts(*k), want_grads=True, clip=oracle.ClipCfg(*c["clip"]))
    secs = time.time() - t0
    names = [n for n, *_ in FC.I.model_param_shapes(c["L"], c["d"], c["F"], c["V"])]
    out = [entry("loss", np.array([loss], np.float32)), entry("norm", np.array([info["norm"]], np.float32))]
    for n, g in zip(names, grads):
        out.append(entry("grad." + n, g))
    for n, p in zip(names, params):
        out.append(entry("param." + n, p))
    for n, a in zip(names, m):
        out.append(entry("m." + n, a))
    for n, a in zip(names, v):
        out.append(entry("v." + n, a))
    return {"case": "step", "config": c, "oracle_seconds": round(secs, 1), "threads": oracle.num_threads(),
            "loss": float(loss), "skip_state": info["skip_state"], "skipped": info["skipped"], "tensors": out}


def make_qlinear():
    c = FC.QLIN
    dy, qx, sx, qw, sw = FC.qlin_inputs(c)
    t0 = time.time()
    dx, dw = oracle.qlinear_bwd(dy, qx, sx[0], qw, sw)
    secs = time.time() - t0
    return {"case": "qlinear", "config": c, "oracle_seconds": round(secs, 1), "threads": oracle.num_threads(),
            "tensors": [entry("dx", dx), entry("dw", dw)]}


def main(which, out_dir=HERE):
    for case, fn in (("block", make_block), ("step", make_step), ("qlinear", make_qlinear)):
        if which in (case, "all"):
            print(f"{case}: running the oracle on {oracle.num_threads()} threads", flush=True)
            res = fn()
            path = os.path.join(out_dir, f"full_shape_{case}.json")
            with open(path, "w") as f:
                json.dump(res, f, indent=1)
            print(f"{case}: {res['oracle_seconds']} s on {res['threads']} threads -> {path}", flush=True)


if __name__ == "__main__":
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("case", nargs="?", default="all", choices=["block", "step", "qlinear", "all"])
    ap.add_argument("--out-dir", default=HERE, help="where the JSON files go (default: beside this script)")
    args = ap.parse_args()
    os.makedirs(args.out_dir, exist_ok=True)
    main(args.case, args.out_dir)
