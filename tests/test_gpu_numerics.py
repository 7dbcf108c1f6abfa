"""Device primitives (R0, R4) against the oracle, bit for bit, on adversarial and dense inputs."""
import numpy as np
import pytest
import torch

import adversarial as ADV
import oracle
import paper_2609_17380_amd.canon as C
from gpu_util import assert_bits, dev_f32, host_f32

pytestmark = pytest.mark.gpu

A, B, CC = ADV.triples(seed=777, n=20000)


def run(op, a, b=None, c=None):
    n = a.size
    da = dev_f32(a)
    db = dev_f32(b if b is not None else a)
    dc = dev_f32(c if c is not None else a)
    out = torch.empty(n, dtype=torch.float32, device=da.device)
    C.devmath(op, n, da, db, dc, out)
    torch.cuda.synchronize()
    return host_f32(out)


@pytest.mark.parametrize("op", ["add", "sub", "mul", "fma"])
def test_r0_ops_match_oracle(op):
    print(f"devmath {op} n={A.size}", flush=True)
    assert_bits(run(op, A, B, CC), oracle.prim(op, A, B, CC), op)


def test_division_matches_oracle():
    keep = np.abs(B) >= np.float32(2.0 ** -126)
    a, b = A[keep], B[keep]
    got, want = run("div", a, b), oracle.prim("div", a, b)
    fin = np.isfinite(want)
    assert_bits(got[fin], want[fin], "div")


def test_sqrt_matches_oracle_sampled_bit_patterns():
    u = np.arange(0, 1 << 32, 251, dtype=np.uint64).astype(np.uint32)
    x = u.view(np.float32)
    x = x[np.isfinite(x) & (x >= 0)]
    assert_bits(run("sqrt", x), oracle.prim("sqrt", x), "sqrt")


@pytest.mark.parametrize("op", ["exp", "log", "sigmoid", "silu", "bf16"])
def test_canonical_functions_match_oracle(op):
    rng = np.random.default_rng(5)
    dense = np.linspace(-100, 100, 400001, dtype=np.float32)
    pos = np.exp(np.linspace(-80, 80, 200001)).astype(np.float32)
    rnd = ADV.random_floats(rng, 200000, 0, 254)
    x = np.concatenate([dense, pos, rnd, A])
    x = x[np.isfinite(x)]
    if op == "log":
        x = np.abs(x)
    got, want = run(op, x), oracle.prim(op, x)
    ok = ~(np.isnan(got) & np.isnan(want))
    assert_bits(got[ok], want[ok], op)
