"""R15 on the device against the oracle, bit for bit: canon_clip_grad_norm (pre-clip norm, spike counter,
in-place clip) over single and several tensors (empty, ragged, misaligned, vector and scalar loads), the
full 1B-model gradient in one flat buffer (the step's launch), and the clip inside canon_step."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import (DEV, assert_bits, dev_bf16, dev_f32, dev_i32, host_f32, host_u16,
                      poisoned_workspace)

pytestmark = pytest.mark.gpu

TID = 700


def wide_f32(n, seed, tid=TID):
    """Normal values spread over exponents 2^-12 .. 2^12, so that grouping changes the rounded sum."""
    x = I.normal_f32((n,), seed, tid)
    e = I.uniform_int((n,), seed, tid + 1, 25).astype(np.int64) - 12
    return (x * np.exp2(e)).astype(np.float32)


def bits(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


def same(a, b):
    """Bit-equal, or both NaN (IEEE 754 leaves a NaN result's sign and payload open)."""
    return bool(bits(a) == bits(b)) or bool(np.isnan(a) and np.isnan(b))


def to_device(hosts, misalign=False):
    """Device copies; with misalign, each tensor sits one float past a 16-byte boundary."""
    out = []
    for h in hosts:
        if misalign:
            buf = torch.empty(h.size + 1, dtype=torch.float32, device=DEV)
            t = buf[1:]
            t.copy_(torch.from_numpy(h))
        else:
            t = dev_f32(h)
        out.append(t)
    return out


def device_clip(grads, max_norm, spike_norm, skip_steps, skip_state=0):
    norm = torch.full((1,), -1.0, dtype=torch.float32, device=DEV)
    state = torch.full((1,), skip_state, dtype=torch.int32, device=DEV)
    skipped = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    ws = torch.empty(max(1, C.clip_grad_norm_workspace_bytes(grads)), dtype=torch.uint8, device=DEV)
    C.clip_grad_norm(grads, C.make_clip(max_norm, spike_norm, skip_steps, norm, state, skipped), ws)
    torch.cuda.synchronize()
    return np.float32(host_f32(norm)[0]), int(state.cpu()[0]), int(skipped.cpu()[0])


def oracle_clip(hosts, max_norm, spike_norm, skip_steps, skip_state=0):
    norm = oracle.global_norm(hosts)
    coef, state, skipped = oracle.clip_decide(norm, oracle.ClipCfg(max_norm, spike_norm, skip_steps), skip_state)
    clipped = [h.copy() for h in hosts]
    oracle.clip_apply(clipped, coef)
    return norm, state, skipped, clipped


def check(hosts, max_norm=1.0, spike_norm=5.0, skip_steps=5, skip_state=0, misalign=False):
    grads = to_device(hosts, misalign)
    n_d, s_d, k_d = device_clip(grads, max_norm, spike_norm, skip_steps, skip_state)
    n_o, s_o, k_o, clipped = oracle_clip(hosts, max_norm, spike_norm, skip_steps, skip_state)
    assert same(n_d, n_o), (n_d, n_o)
    assert (s_d, k_d) == (s_o, k_o)
    for i, (g, c) in enumerate(zip(grads, clipped)):
        assert_bits(host_f32(g), c, f"clipped tensor {i}")
    return n_o


@pytest.mark.parametrize("n", [0, 1, 5, 31, 32, 33, 2047, 2048, 2049, 8191, 32767, 32768, 32769, 100003, 1 << 20,
                               3_000_001, 4_194_304])
def test_single_tensor(n):
    print(f"clip single n={n}", flush=True)
    check([wide_f32(n, n)], max_norm=0.5)


@pytest.mark.parametrize("sizes", [[5, 0, 27, 64], [100, 3, 33, 2049], [4096, 0, 8, 32768, 12], [1, 1, 1], [0, 0],
                                   [32, 32, 32], [33, 31, 2048 * 3 + 1, 7], [4, 8, 32768 * 2 + 4, 0, 1000, 40000]])
@pytest.mark.parametrize("misalign", [False, True])
def test_several_tensors(sizes, misalign):
    print(f"clip sizes={sizes} misalign={misalign}", flush=True)
    hosts = [wide_f32(s, 17 + i, TID + 10 * i) for i, s in enumerate(sizes)]
    check(hosts, max_norm=0.5, misalign=misalign)


def test_no_tensors():
    n_d, s_d, k_d = device_clip([], 1.0, 5.0, 5)
    assert bits(n_d) == 0 and (s_d, k_d) == (0, 0)


def test_no_clip_leaves_gradient_untouched():
    hosts = [wide_f32(s, 3 + s) for s in (1000, 4097)]
    norm = check(hosts, max_norm=float(np.float32(1e30)))
    assert norm < 1e30


def test_large_tensor_count():
    rng = np.random.default_rng(9)
    sizes = [int(s) for s in rng.integers(0, 300, 700)]
    hosts = [wide_f32(s, 100 + i, TID + 2 * i) for i, s in enumerate(sizes)]
    check(hosts, max_norm=0.25)


def test_nonfinite_gradients():
    h = wide_f32(5000, 1)
    h[1234] = np.nan
    n = check([h], max_norm=1.0, spike_norm=5.0, skip_steps=5)
    assert np.isnan(n)
    h[1234] = np.float32(3e30)  # the square overflows
    assert check([h], max_norm=1.0, spike_norm=5.0, skip_steps=5) == np.inf


def test_spike_counter_over_steps():
    base = wide_f32(50_000, 2)
    norm0 = float(oracle.global_norm([base]))
    state_d = state_o = 0
    for step, target in enumerate([1.0, 6.0, 1.0, 1.0, 7.0, 1.0, 1.0, 1.0, 1.0, 1.0, 1.0, 0.5]):
        h = (base * np.float32(target / norm0)).astype(np.float32)
        grads = to_device([h])
        n_d, state_d, k_d = device_clip(grads, 1.0, 5.0, 5, state_d)
        n_o, state_o, k_o, _ = oracle_clip([h], 1.0, 5.0, 5, state_o)
        assert bits(n_d) == bits(n_o) and (state_d, k_d) == (state_o, k_o), step


def test_rejects_invalid_settings():
    g = [dev_f32(np.ones(8, np.float32))]
    ws = torch.empty(C.clip_grad_norm_workspace_bytes(g), dtype=torch.uint8, device=DEV)
    with pytest.raises(C.CanonError):
        C.clip_grad_norm(g, C.make_clip(0.0, 5.0, 0), ws)
    with pytest.raises(C.CanonError):
        C.clip_grad_norm(g, C.make_clip(1.0, 5.0, 5), ws)  # spike rule without a counter
    with pytest.raises(C.CanonError):
        C.clip_grad_norm(g, C.make_clip(1.0, 5.0, 0), ws[:16])


def test_full_1b_gradient_in_one_buffer():
    """The norm over the whole gradient of the 16-layer, d = 2048 model (one flat buffer, as in the step)."""
    shapes = I.model_param_shapes(16, 2048, 8192, 50304)
    P = sum(int(np.prod(s)) for _, s, _, _ in shapes)
    print(f"clip full P={P}: generating", flush=True)
    h = I.normal_f32((P,), 11, TID + 5, std=1e-4)
    print("clip full: device", flush=True)
    g = dev_f32(h)
    n_d, s_d, k_d = device_clip([g], 1.0, 5.0, 5)
    got = host_f32(g)
    del g
    print("clip full: oracle", flush=True)
    n_o, s_o, k_o, clipped = oracle_clip([h], 1.0, 5.0, 5)
    assert bits(n_d) == bits(n_o), (n_d, n_o)
    assert (s_d, k_d) == (s_o, k_o) == (0, 0)
    assert 1.0 < n_o < 5.0  # the clip is engaged, the spike rule is not
    assert_bits(got, clipped[0], "clipped full gradient")


# ---- the clip inside the step ----

def run_step(clip, skip_state=0, L=2, d=256, H=2, F=256, V=300, S=64, mb=2, plan=(1, 2, 1), seed=4):
    hd = d // H
    params = I.model_params(L, d, F, V, seed=seed, std=0.02)
    R = plan[1] * plan[2]
    windows = I.uniform_int((R * plan[0] * mb, S + 1), seed, I.TENSOR_IDS["windows"], V)
    cos, sin = I.rope_tables(S, hd)
    k = I.adamw_constants()
    po = [p.copy() for p in params]
    mo = [np.zeros(p.shape, np.float32) for p in params]
    vo = [np.zeros(p.shape, np.float32) for p in params]
    res = oracle.step(oracle.ModelCfg(L, d, H, hd, F, V, S, mb, np.float32(1e-5)), oracle.Plan(*plan), po, mo, vo,
                      windows, cos, sin, oracle.AdamWConsts(*k), want_grads=True,
                      clip=oracle.ClipCfg(*clip) if clip else None, skip_state=skip_state)
    cfg = C.ModelCfg(L, d, H, hd, F, V, S, mb, np.float32(1e-5))
    cplan = C.DPPlan(*plan)
    pg = [dev_bf16(p) for p in params]
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    gg = [torch.empty(p.shape, dtype=torch.float32, device=DEV) for p in params]
    ws = poisoned_workspace(C.step_workspace_bytes(cfg, cplan))
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    norm = torch.full((1,), -1.0, dtype=torch.float32, device=DEV)
    state = torch.full((1,), skip_state, dtype=torch.int32, device=DEV)
    skipped = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    cc = C.make_clip(*clip, norm, state, skipped) if clip else None
    C.step(cfg, cplan, pg, mg, vg, dev_i32(windows), dev_f32(cos), dev_f32(sin), C.AdamWConsts(*k), ws, loss,
           grads_out=gg, clip=cc)
    torch.cuda.synchronize()
    dev = dict(loss=host_f32(loss), grads=[host_f32(x) for x in gg], p=[host_u16(x) for x in pg],
               m=[host_f32(x) for x in mg], v=[host_f32(x) for x in vg], norm=np.float32(host_f32(norm)[0]),
               state=int(state.cpu()[0]), skipped=int(skipped.cpu()[0]))
    return res, (po, mo, vo), params, dev


@pytest.mark.parametrize("clip,skip_state", [((0.05, 5.0, 5), 0), ((1e9, np.inf, 0), 0), ((1.0, 1e-6, 3), 0),
                                             ((1.0, 1e30, 3), 2), ((0.05, 1e30, 5), 1)])
def test_step_with_clip_bit_exact(clip, skip_state):
    print(f"step clip={clip} state={skip_state}", flush=True)
    (loss_o, g_o, info), (po, mo, vo), params, dev = run_step(clip, skip_state)
    assert_bits(dev["loss"], np.array([loss_o], np.float32), "loss")
    assert bits(dev["norm"]) == bits(info["norm"])
    assert (dev["state"], dev["skipped"]) == (info["skip_state"], info["skipped"])
    for i in range(len(po)):
        assert_bits(dev["grads"][i], g_o[i], f"grad {i}")
        assert_bits(dev["p"][i], po[i], f"param {i}")
        assert_bits(dev["m"][i], mo[i], f"m {i}")
        assert_bits(dev["v"][i], vo[i], f"v {i}")
    if info["skipped"]:
        assert all(np.array_equal(a, b) for a, b in zip(dev["p"], params))


def test_step_clip_off_matches_step_without_clip():
    _, _, _, with_clip = run_step((1e9, np.inf, 0))
    (loss_o, _), (po, _, _), _, _ = run_step(None)
    for a, b in zip(with_clip["p"], po):
        assert np.array_equal(a, b)


def test_step_bad_token_with_clip():
    L, d, H, F, V, S, mb = 1, 128, 1, 128, 50, 32, 1
    cfg = C.ModelCfg(L, d, H, d // H, F, V, S, mb, np.float32(1e-5))
    cplan = C.DPPlan(1, 1, 1)
    params = I.model_params(L, d, F, V, seed=0)
    windows = I.uniform_int((1, S + 1), 0, 50, V)
    windows[0, 7] = -1
    cos, sin = I.rope_tables(S, d // H)
    pg = [dev_bf16(p) for p in params]
    mg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    vg = [torch.zeros(p.shape, dtype=torch.float32, device=DEV) for p in params]
    ws = poisoned_workspace(C.step_workspace_bytes(cfg, cplan))
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    norm = torch.zeros(1, dtype=torch.float32, device=DEV)
    state = torch.full((1,), 2, dtype=torch.int32, device=DEV)
    skipped = torch.zeros(1, dtype=torch.int32, device=DEV)
    C.step(cfg, cplan, pg, mg, vg, dev_i32(windows), dev_f32(cos), dev_f32(sin), C.AdamWConsts(*I.adamw_constants()),
           ws, loss, clip=C.make_clip(1.0, 5.0, 5, norm, state, skipped))
    torch.cuda.synchronize()
    assert np.isnan(host_f32(loss)[0]) and np.isnan(host_f32(norm)[0])
    assert int(state.cpu()[0]) == 2 and int(skipped.cpu()[0]) == 1
    for a, b in zip(pg, params):
        assert np.array_equal(host_u16(a), b)
