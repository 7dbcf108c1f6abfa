"""canon_lsq_step_grad_noalloc (block sums in the library's own device array) against canon_lsq_step_grad
(block sums in a caller workspace), through the C ABI, bit for bit: two calls in a row, the second smaller,
so a stale block sum from the first call would show; a call beyond the array's limit is rejected."""
import numpy as np
import pytest
import torch

import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import DEV, assert_bits, dev_bf16, dev_f32, host_f32

pytestmark = pytest.mark.gpu


def with_workspace(T, K, x, s, dx):
    g = torch.full((1,), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.empty(C.lsq_step_grad_workspace_bytes(T, K), dtype=torch.uint8, device=DEV)
    C.lsq_step_grad(T, K, x, s, dx, g, ws)
    torch.cuda.synchronize()
    return host_f32(g)


def no_alloc(T, K, x, s, dx):
    g = torch.full((1,), float("nan"), dtype=torch.float32, device=DEV)
    C.lsq_step_grad_noalloc(T, K, x, s, dx, g)
    torch.cuda.synchronize()
    return host_f32(g)


def case(T, K, seed, s):
    x16 = I.normal_bf16((T, K), seed, I.TENSOR_IDS["x_in"], std=0.3)
    dx = I.normal_f32((T, K), seed, I.TENSOR_IDS["dy_in"], std=1e-3)
    return dev_bf16(x16), dev_f32(np.array([s], np.float32)), dev_f32(dx)


def test_no_alloc_matches_workspace_entry_twice_in_a_row():
    # first call: 4096 x 2048 (256 block sums); second: 300 x 777 (8 block sums, the last ragged)
    for T, K, seed in [(4096, 2048, 1), (300, 777, 2)]:
        print(f"lsq noalloc T={T} K={K}", flush=True)
        x, s, dx = case(T, K, seed, 0.05)
        want = with_workspace(T, K, x, s, dx)
        got = no_alloc(T, K, x, s, dx)
        assert np.isfinite(want[0])
        assert_bits(got, want, f"noalloc T={T} K={K}")


def test_no_alloc_empty_and_limit():
    x, s, dx = case(4, 8, 3, 0.05)
    assert_bits(no_alloc(0, 8, x, s, dx), with_workspace(0, 8, x, s, dx), "empty")
    big_t = C.lsq_step_grad_noalloc_max_terms() // 8 + 1
    g = torch.zeros(1, dtype=torch.float32, device=DEV)
    with pytest.raises(C.CanonError) as e:
        C.lsq_step_grad_noalloc(big_t, 8, x, s, dx, g)  # validated on the host, nothing is launched
    assert e.value.status == C.EUNSUPPORTED
