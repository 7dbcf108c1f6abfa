"""canon_embed_bwd (R11) against the oracle, bit for bit: the 1B microbatch (8192 tokens, vocabulary 50304,
d 2048) with uniform and text-like skewed tokens, the paper architecture's 16384-token microbatch with a token
repeated thousands of times, ragged sizes through every sort stage (one block, several blocks with global
merge steps), odd widths on the scalar path, out-of-range tokens and the empty case."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import DEV, assert_bits, dev_f32, dev_i32, host_f32

pytestmark = pytest.mark.gpu


def skewed(T, V, rng, shares=(0.6, 0.1, 0.02)):
    tok = rng.integers(0, V, T).astype(np.int32)
    u = rng.random(T)
    lo = 0.0
    for i, sh in enumerate(shares):
        tok[(u >= lo) & (u < lo + sh)] = 7 + 4 * i
        lo += sh
    return tok


def run(tok, dx, V):
    T, d = dx.shape
    dE = torch.full((V, d), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.empty(C.embed_bwd_workspace_bytes(T, d), dtype=torch.uint8, device=DEV)
    C.embed_bwd(T, V, d, dev_i32(tok), dev_f32(dx), dE, ws)
    torch.cuda.synchronize()
    return host_f32(dE)


@pytest.mark.parametrize("T,V,d,kind", [(8192, 50304, 2048, "uniform"), (8192, 50304, 2048, "skewed"),
                                        (16384, 50304, 2048, "skewed"), (16384, 1000, 64, "single")])
def test_embed_bwd_workload_shapes(T, V, d, kind):
    print(f"embed_bwd T={T} V={V} d={d} {kind}", flush=True)
    rng = np.random.default_rng(T + d)
    if kind == "uniform":
        tok = I.uniform_int((T,), 0, I.TENSOR_IDS["windows"], V).reshape(-1)
    elif kind == "skewed":
        tok = skewed(T, V, rng)
    else:
        tok = np.full(T, 999, np.int32)  # one token everywhere: 512 chunks folded
    dx = I.normal_f32((T, d), 3, I.TENSOR_IDS["dy_in"], std=1e-3)
    if kind != "uniform":
        print(f"  most repeated token: {np.bincount(tok).max()} occurrences", flush=True)
    assert_bits(run(tok, dx, V), oracle.embed_bwd(tok, dx, V), f"dE T={T}")


@pytest.mark.parametrize("T", [1, 2, 31, 33, 2047, 2048, 2049, 5000, 40000])
@pytest.mark.parametrize("d", [1, 5, 64])
def test_embed_bwd_ragged(T, d):
    print(f"embed_bwd ragged T={T} d={d}", flush=True)
    rng = np.random.default_rng(T * 7 + d)
    V = 97
    tok = skewed(T, V, rng, shares=(0.3, 0.05))
    tok[rng.random(T) < 0.01] = -5     # out of range below
    tok[rng.random(T) < 0.01] = V + 3  # and above
    dx = (rng.standard_normal((T, d)) * 2.0 ** rng.integers(-20, 21, (T, d))).astype(np.float32)
    assert_bits(run(tok, dx, V), oracle.embed_bwd(tok, dx, V), f"dE T={T} d={d}")


def test_embed_bwd_empty():
    dE = torch.full((11, 3), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.empty(max(C.embed_bwd_workspace_bytes(0, 3), 1), dtype=torch.uint8, device=DEV)
    t = torch.zeros(1, dtype=torch.int32, device=DEV)
    x = torch.zeros(3, dtype=torch.float32, device=DEV)
    C.embed_bwd(0, 11, 3, t, x, dE, ws)
    torch.cuda.synchronize()
    assert np.all(host_f32(dE).view(np.uint32) == 0)
