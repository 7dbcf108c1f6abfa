"""The gradient plan fed one microbatch at a time (canon_plan_begin / push / finish), stopped after every
microbatch, persisted (the host record's bytes and the device slots copied to host memory), and resumed in
other device memory: the result must equal the oracle's Algorithm 1 and canon_grad_accum bit for bit,
wherever the plan was stopped (the analogue of restarting from a checkpoint and comparing the repeated
steps' hashes)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import DEV, assert_bits, dev_f32, host_f32

pytestmark = pytest.mark.gpu

PLANS = [(1, 8, 1), (2, 4, 1), (1, 2, 4), (3, 1, 5), (2, 3, 3), (1, 1, 7), (1, 1, 1), (4, 2, 2), (1, 1, 13)]


def spread_grads(count, n, seed):
    """Gradients over many binades, so that another association of the plan's sums shows in the bits."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        g = I.normal_f32((n,), 3, I.TENSOR_IDS["grads"] + i, std=1e-3)
        out.append((g * np.exp2(rng.integers(-10, 11, n))).astype(np.float32))
    return out


def state_at(bytes_, shift):
    """A fresh 256-byte aligned device buffer of bytes_ bytes, placed `shift` slots of 256 bytes into a larger
    allocation so that it never has the address of the buffer it replaces."""
    words = bytes_ // 4
    big = torch.empty(words + 64 * (shift + 1), dtype=torch.float32, device=DEV)
    off = (-big.data_ptr() % 256) // 4 + 64 * shift
    return big, big[off:off + words]


def run_plan(plan, dg, n, stop=None, shift=1, tamper=None):
    """Push every gradient; after `stop` pushes persist and resume in new memory.  Returns the result."""
    p = C.DPPlan(*plan)
    nbytes = C.plan_state_bytes(p, n)
    _, state = state_at(nbytes, 0)
    cur = C.plan_begin(p, n)
    for i, g in enumerate(dg):
        if i == stop:
            torch.cuda.synchronize()
            saved_state = state.cpu().numpy().copy()
            saved_cur = bytes(cur)
            del state, cur
            torch.cuda.synchronize()
            _, state = state_at(nbytes, shift)
            state.copy_(torch.from_numpy(saved_state).to(DEV))
            cur = C.PlanCursor.from_buffer_copy(saved_cur)
            if tamper:
                tamper(cur)
        C.plan_push(cur, g, state)
    assert cur.next == len(dg)
    out = torch.empty(n, dtype=torch.float32, device=DEV)
    C.plan_finish(cur, state, out)
    torch.cuda.synchronize()
    return host_f32(out)


@pytest.mark.parametrize("plan", PLANS)
@pytest.mark.parametrize("n", [10007, 1])
def test_plan_stop_and_resume_everywhere(plan, n):
    accum, shard, rep = plan
    total = accum * shard * rep
    print(f"plan resume {plan} n={n}", flush=True)
    grads = spread_grads(total, n, 17 * total + n)
    want = oracle.grad_accum(grads, accum, shard, rep)
    dg = [dev_f32(g) for g in grads]
    fused = torch.empty(n, dtype=torch.float32, device=DEV)
    C.grad_accum(C.DPPlan(*plan), n, dg, fused)
    torch.cuda.synchronize()
    assert_bits(host_f32(fused), want, f"fused plan {plan}")
    assert_bits(run_plan(plan, dg, n), want, f"streamed plan {plan}")
    for stop in range(total + 1):
        assert_bits(run_plan(plan, dg, n, stop=stop, shift=1 + stop % 3), want, f"plan {plan} resumed at {stop}")


def test_resume_with_swapped_slots_changes_bits():
    """Negative control: a resumed record whose two stack entries point at each other's slots (a record the
    calls accept, since each slot is still used once) gives other bits, so the comparisons above would see
    a resume that lost track of the stack."""
    plan, n = (1, 1, 7), 4096
    grads = spread_grads(7, n, 99)
    want = oracle.grad_accum(grads, *plan)
    dg = [dev_f32(g) for g in grads]

    def swap(cur):
        assert cur.depth == 2  # after 6 replicas: levels 2 and 1
        cur.slot[0], cur.slot[1] = cur.slot[1], cur.slot[0]

    got = run_plan(plan, dg, n, stop=6, tamper=swap)
    assert not np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_plan_rejects_push_past_end_and_early_finish():
    plan = C.DPPlan(1, 2, 1)
    n = 64
    state = state_at(C.plan_state_bytes(plan, n), 0)[1]
    g = torch.zeros(n, dtype=torch.float32, device=DEV)
    out = torch.empty(n, dtype=torch.float32, device=DEV)
    cur = C.plan_begin(plan, n)
    with pytest.raises(C.CanonError):
        C.plan_finish(cur, state, out)
    C.plan_push(cur, g, state)
    C.plan_push(cur, g, state)
    before = bytes(cur)
    with pytest.raises(C.CanonError):
        C.plan_push(cur, g, state)
    assert bytes(cur) == before
    with pytest.raises(C.CanonError):  # state buffer too small
        C.plan_finish(cur, state, out, state_bytes=C.plan_state_bytes(plan, n) - 4)
    C.plan_finish(cur, state, out)
    torch.cuda.synchronize()
    assert np.all(host_f32(out).view(np.uint32) == 0)
    assert ctypes.sizeof(cur) == len(before)
