"""Pins for R15: the global gradient norm, the clip coefficient and the spike-skip rule.

The norm is checked against exact integer arithmetic, closed forms, an independent formulation of the
canonical order (the zero-padded perfect tree over chunk partials of the flat vector), and PyTorch's own
clip routine where the norm is exact; the spike rule against the activation counts the paper reports.
"""
import math
import os

import numpy as np
import pytest
import torch

import canon_formulations as CF
import oracle
import paper_2609_17380_amd.inputs as I

RNG = np.random.default_rng(1515)
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bits(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


def wide(n):
    return (RNG.standard_normal(n) * np.exp2(RNG.integers(-12, 12, n))).astype(np.float32)


def flat_reference(tensors):
    """Independent formulation: squares of the concatenated vector, chunks of 32 over the flat index,
    perfect zero-padded tree, correctly rounded sqrt (numpy float32 arithmetic)."""
    flat = np.concatenate([t.ravel() for t in tensors]) if tensors else np.zeros(0, np.float32)
    sq = (flat * flat).astype(np.float32)
    return np.sqrt(CF.canonical_sum(list(sq)))


# ---- the norm ----

@pytest.mark.parametrize("sizes", [[0], [1], [31], [32, 1], [5, 0, 27, 64], [100, 3, 33, 2049]])
def test_norm_small_integers_exact(sizes):
    ts = [RNG.integers(-40, 41, s).astype(np.float32) for s in sizes]
    q = sum(int((t.astype(np.int64) ** 2).sum()) for t in ts)
    assert q < 2 ** 24  # every partial sum is an integer below 2^24: exact
    # RN24(RN53(sqrt q)) = RN24(sqrt q) since 53 >= 2*24 + 2
    assert bits(oracle.global_norm(ts)) == bits(np.float32(math.sqrt(q)))


def test_norm_closed_forms():
    assert bits(oracle.global_norm([np.ones(1 << 20, np.float32)])) == bits(1024.0)
    halves = [np.full(s, 0.5, np.float32) for s in (300, 724)]  # 1024 * 0.25 = 256
    assert bits(oracle.global_norm(halves)) == bits(16.0)
    assert bits(oracle.global_norm([np.zeros(77, np.float32)])) == 0
    assert bits(oracle.global_norm([])) == 0
    assert bits(oracle.global_norm([np.array([-3.0, 4.0], np.float32)])) == bits(5.0)


def test_norm_of_negatives_equals_norm_of_magnitudes():
    t = wide(999)
    assert bits(oracle.global_norm([t])) == bits(oracle.global_norm([np.abs(t)]))


@pytest.mark.parametrize("seed", range(6))
def test_norm_chunks_run_across_tensor_boundaries(seed):
    rng = np.random.default_rng(seed)
    sizes = [int(s) for s in rng.integers(0, 90, 7)] + [1000]
    ts = [(rng.standard_normal(s) * np.exp2(rng.integers(-12, 12, s))).astype(np.float32) for s in sizes]
    got = oracle.global_norm(ts)
    assert bits(got) == bits(flat_reference(ts))


def test_flat_and_per_tensor_readings_differ_somewhere():
    """The boundary test above has power: chunking each tensor on its own gives other bits here."""
    differs = 0
    for seed in range(20):
        rng = np.random.default_rng(100 + seed)
        ts = [(rng.standard_normal(s) * np.exp2(rng.integers(-12, 12, s))).astype(np.float32)
              for s in (45, 45, 45, 45)]
        per_tensor = [CF.padded_tree(CF.chunk_partials(list((t * t).astype(np.float32)))) for t in ts]
        alt = np.sqrt(CF.padded_tree(per_tensor))
        differs += int(bits(alt) != bits(oracle.global_norm(ts)))
    assert differs > 0


def test_tensor_order_is_the_declared_order():
    ts = [wide(45), wide(1000), wide(19)]
    rev = ts[::-1]
    assert bits(oracle.global_norm(rev)) == bits(flat_reference(rev))
    assert bits(oracle.global_norm(ts)) == bits(flat_reference(ts))


def test_norm_nonfinite():
    t = np.ones(64, np.float32)
    t[40] = np.nan
    assert np.isnan(oracle.global_norm([t]))
    t[40] = 1e20  # square overflows
    assert oracle.global_norm([t]) == np.inf
    assert oracle.global_norm([np.ones(3, np.float32), np.array([np.inf], np.float32)]) == np.inf


def test_norm_flushes_tiny_squares():
    # (2^-70)^2 = 2^-140 is below the normal range and flushes to +0 under R0
    assert bits(oracle.global_norm([np.full(10, 2.0 ** -70, np.float32)])) == 0
    # (2^-60)^2 = 2^-120 is normal: 4 of them sum to 2^-118, sqrt 2^-59
    assert bits(oracle.global_norm([np.full(4, 2.0 ** -60, np.float32)])) == bits(2.0 ** -59)


# ---- the clip ----

def torch_clip(grads, max_norm):
    ps = [torch.nn.Parameter(torch.zeros(g.shape)) for g in grads]
    for p, g in zip(ps, grads):
        p.grad = torch.from_numpy(g.copy())
    tn = torch.nn.utils.clip_grad_norm_(ps, max_norm, foreach=False)
    return float(tn), [p.grad.numpy() for p in ps]


def pythagorean(scale, reps):
    # each tensor is a multiple of (3, 4) or (5, 12): per-tensor norms 5c and 13c are exact, so is the total
    out = []
    for i in range(reps):
        base = np.array([3, 4] if i % 2 == 0 else [5, 12], np.float32)
        out.append((base * np.float32(scale * (i + 1))).astype(np.float32))
    return out


@pytest.mark.parametrize("case", ["one_tensor", "pythagorean"])
@pytest.mark.parametrize("scale", [0.25, 1.0, 3.0, 40.0])
def test_clip_matches_torch_where_the_norm_is_exact(case, scale):
    # exact sums of squares, and per-tensor norms PyTorch rounds without error (it takes the norm of the
    # per-tensor norms): its total is then the correctly rounded norm too
    if case == "one_tensor":
        ts = [(RNG.integers(-9, 10, 300) * np.float32(scale)).astype(np.float32)]
    else:
        ts = pythagorean(scale, 6)
    norm = oracle.global_norm(ts)
    tn, clipped = torch_clip(ts, 1.0)
    assert bits(norm) == bits(np.float32(tn))
    coef, _, _ = oracle.clip_decide(norm, oracle.ClipCfg(1.0, np.inf, 0))
    ours = [t.copy() for t in ts]
    oracle.clip_apply(ours, coef)
    for a, b in zip(ours, clipped):
        assert np.array_equal(bits(a), bits(b))


def test_clip_coefficient_values():
    k = oracle.ClipCfg(1.0, 5.0, 5)
    one = np.float32(1.0)
    for norm in (2.0, 1.0, 0.75, 1e-3, 7.0):
        coef, _, _ = oracle.clip_decide(np.float32(norm), k, 0)
        want = one / np.float32(np.float32(norm) + np.float32(1e-6))
        assert bits(coef) == bits(want), norm
    # norm 1.0: 1/RN(1 + 1e-6) is below 1, so the clip engages (PyTorch's convention)
    coef, _, _ = oracle.clip_decide(np.float32(1.0), k, 0)
    assert coef < 1
    coef, _, _ = oracle.clip_decide(np.float32(0.0), k, 0)
    assert coef == np.float32(1e6) or coef > 1
    coef, _, _ = oracle.clip_decide(np.float32(np.inf), k, 0)
    assert bits(coef) == 0


def test_clip_apply_only_below_one():
    t = wide(100)
    t[7] = np.float32(2.0 ** -140)  # a subnormal stays as it is when no clip applies (no multiply at all)
    u = t.copy()
    oracle.clip_apply([u], np.float32(1.0))
    assert np.array_equal(bits(u), bits(t))
    oracle.clip_apply([u], np.float32(2.0))
    assert np.array_equal(bits(u), bits(t))
    c = np.float32(0.3)
    oracle.clip_apply([u], c)
    want = (t * c).astype(np.float32)
    want[7] = 0.0  # R0 reads the subnormal input as +0
    assert np.array_equal(bits(u), bits(want))


def test_clipped_gradient_has_norm_at_most_max():
    for seed in range(5):
        rng = np.random.default_rng(seed)
        ts = [(rng.standard_normal(s) * 3).astype(np.float32) for s in (500, 77, 2000)]
        norm = oracle.global_norm(ts)
        coef, _, _ = oracle.clip_decide(norm, oracle.ClipCfg(1.0, np.inf, 0))
        oracle.clip_apply(ts, coef)
        exact = math.sqrt(sum(float((t.astype(np.float64) ** 2).sum()) for t in ts))
        assert exact <= 1.0 + 1e-5


# ---- the spike rule ----

def run_protocol(norms, threshold, skip_steps):
    k = oracle.ClipCfg(1.0, threshold, skip_steps)
    state, skipped = 0, []
    for s, n in enumerate(norms):
        _, state, sk = oracle.clip_decide(np.float32(n), k, state)
        if sk:
            skipped.append(s)
    return skipped, state


def test_spike_protocol_reproduces_the_reported_skip_count():
    with open(os.path.join(GOLDEN, "spike_protocol.txt")) as f:
        rows = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    total, thr, k, want = int(rows[0][0]), float(rows[0][1]), int(rows[0][2]), int(rows[0][3])
    norms = np.full(total, 0.8, np.float32)
    spikes = [(int(r[0]), float(r[1])) for r in rows[1:]]
    for step, n in spikes:
        norms[step] = n
    skipped, state = run_protocol(norms, thr, k)
    assert len(skipped) == want
    assert skipped == [s + i for s, _ in spikes for i in range(k)]
    assert state == 0


def test_spike_threshold_is_strict_and_nan_is_a_spike():
    assert run_protocol([5.0, 1.0], 5.0, 5)[0] == []
    assert run_protocol([np.nextafter(np.float32(5), np.float32(6)), 1.0], 5.0, 5)[0] == [0, 1]
    assert run_protocol([np.nan] + [1.0] * 9, 5.0, 5)[0] == [0, 1, 2, 3, 4]
    assert run_protocol([np.inf] + [1.0] * 9, 5.0, 3)[0] == [0, 1, 2]


def test_spike_inside_the_window_restarts_it():
    norms = [1.0, 9.0, 1.0, 1.0, 9.0] + [1.0] * 10
    assert run_protocol(norms, 5.0, 5)[0] == [1, 2, 3, 4, 5, 6, 7, 8]


def test_spike_rule_off():
    assert run_protocol([9.0, np.nan, 1.0], 5.0, 0)[0] == []


def test_invalid_settings_rejected():
    with pytest.raises(ValueError):
        oracle.clip_decide(np.float32(1), oracle.ClipCfg(0.0, 5.0, 5), 0)
    with pytest.raises(ValueError):
        oracle.clip_decide(np.float32(1), oracle.ClipCfg(1.0, 5.0, -1), 0)


# ---- the step ----

def small_setup():
    cfg = oracle.ModelCfg(1, 64, 2, 32, 96, 97, 40, 2, np.float32(1e-5))
    plan = oracle.Plan(2, 1, 1)
    M = plan.accum * cfg.micro_seqs
    params = I.model_params(cfg.n_layers, cfg.d_model, cfg.d_ffn, cfg.vocab, seed=3, std=0.05)
    windows = I.uniform_int((M, cfg.seq + 1), 3, I.TENSOR_IDS["windows"], cfg.vocab)
    cos, sin = I.rope_tables(cfg.seq, cfg.head_dim)
    return cfg, plan, params, windows, cos, sin


def fresh(params):
    return ([p.copy() for p in params], [np.zeros(p.shape, np.float32) for p in params],
            [np.zeros(p.shape, np.float32) for p in params])


@pytest.mark.parametrize("max_norm", [1e-3, 0.05, 1e9])
def test_step_with_clip_is_norm_then_clip_then_adamw(max_norm):
    cfg, plan, params, windows, cos, sin = small_setup()
    k = oracle.AdamWConsts(*I.adamw_constants())
    p0, m0, v0 = fresh(params)
    loss0, g0 = oracle.step(cfg, plan, p0, m0, v0, windows, cos, sin, k, want_grads=True)
    p1, m1, v1 = fresh(params)
    loss1, g1, info = oracle.step(cfg, plan, p1, m1, v1, windows, cos, sin, k, want_grads=True,
                                  clip=oracle.ClipCfg(max_norm, 5.0, 5))
    assert bits(loss0) == bits(loss1)
    assert all(np.array_equal(bits(a), bits(b)) for a, b in zip(g0, g1))  # grads_out: pre-clip
    assert bits(info["norm"]) == bits(flat_reference(g0))
    assert info["skipped"] == 0 and info["skip_state"] == 0
    coef, _, _ = oracle.clip_decide(info["norm"], oracle.ClipCfg(max_norm, 5.0, 5))
    g = [x.copy() for x in g0]
    oracle.clip_apply(g, coef)
    p2, m2, v2 = fresh(params)
    decay = [t[3] for t in I.model_param_shapes(cfg.n_layers, cfg.d_model, cfg.d_ffn, cfg.vocab)]
    oracle.adamw(p2, m2, v2, g, decay, k)
    for a, b in zip(p1 + m1 + v1, p2 + m2 + v2):
        assert np.array_equal(a, b)
    if max_norm >= 1e9:  # no clip: the same update as the step without R15
        for a, b in zip(p0, p1):
            assert np.array_equal(a, b)
    else:
        assert any(not np.array_equal(a, b) for a, b in zip(p0, p1))


def test_step_spike_skips_the_update_and_counts_down():
    cfg, plan, params, windows, cos, sin = small_setup()
    k = oracle.AdamWConsts(*I.adamw_constants())
    p1, m1, v1 = fresh(params)
    _, _, info = oracle.step(cfg, plan, p1, m1, v1, windows, cos, sin, k,
                             clip=oracle.ClipCfg(1.0, 1e-6, 3))
    assert info["skipped"] == 1 and info["skip_state"] == 2
    assert all(np.array_equal(a, b) for a, b in zip(p1, params))
    assert all(not m.any() for m in m1) and all(not v.any() for v in v1)
    # inside the window a calm step is skipped too; the counter runs out after the third
    calm = oracle.ClipCfg(1.0, 1e30, 3)
    _, _, info = oracle.step(cfg, plan, p1, m1, v1, windows, cos, sin, k, clip=calm, skip_state=2)
    assert info["skipped"] == 1 and info["skip_state"] == 1
    _, _, info = oracle.step(cfg, plan, p1, m1, v1, windows, cos, sin, k, clip=calm, skip_state=1)
    assert info["skipped"] == 1 and info["skip_state"] == 0
    _, _, info = oracle.step(cfg, plan, p1, m1, v1, windows, cos, sin, k, clip=calm, skip_state=0)
    assert info["skipped"] == 0
    assert any(not np.array_equal(a, b) for a, b in zip(p1, params))
