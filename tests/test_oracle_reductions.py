"""Pins for R1 (chunked chains + binary-carry fold), Alg. 2 (TreeFold) and Alg. 1 (gradient plan)."""
import math
import os
from fractions import Fraction as F

import numpy as np
import pytest

import canon_formulations as CF
import oracle

RNG = np.random.default_rng(2024)


def wide(n):
    """float32 terms with a wide dynamic range (so that grouping changes bits), away from subnormals."""
    return (RNG.standard_normal(n) * np.exp2(RNG.integers(-20, 20, n))).astype(np.float32)


def bits(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


@pytest.mark.parametrize("n", [0, 1, 5, 31, 32, 33, 64, 65, 100, 224, 256, 1000, 2049, 6144])
def test_rsum_integer_inputs_are_exact(n):
    t = RNG.integers(-1000, 1000, n).astype(np.float32)
    assert float(oracle.rsum(t)) == float(t.astype(np.int64).sum())


def test_rsum_empty_is_positive_zero():
    assert bits(oracle.rsum(np.zeros(0, np.float32))) == 0


def test_rsum_hand_example_chunk_boundaries():
    # chunk 0 = [2^24, 1 x 31]: each 2^24 + 1 is a tie and rounds back to 2^24 (even); chunk 1 = 32 ones = 32.
    # The fold adds the partials: 2^24 + 32.  A plain left-to-right sum would stay at 2^24.  Chunks of 31
    # give partials 2^24, 31, 2: (2^24 + 31) is a tie that rounds to 2^24 + 32 (even), then + 2 = 2^24 + 34.
    t = np.ones(64, np.float32)
    t[0] = 2.0 ** 24
    assert float(oracle.rsum(t)) == 2.0 ** 24 + 32
    assert float(oracle.rsum(t, chunk=64)) == 2.0 ** 24
    assert float(oracle.rsum(t, chunk=31)) == 2.0 ** 24 + 34


@pytest.mark.parametrize("n", [1, 7, 32, 33, 95, 96, 97, 224, 7 * 32, 11 * 32 + 5, 13 * 32, 192 * 32, 1572 * 32 - 17])
def test_rsum_matches_padded_tree_formulation(n):
    t = wide(n)
    assert bits(oracle.rsum(t)) == bits(CF.canonical_sum(list(t)))


def test_rsum_negative_controls():
    # chunk counts with >= 3 set bits distinguish the two readings of Result; flat order differs too
    diff_reading = diff_flat = 0
    for trial in range(20):
        t = wide(13 * 32)
        parts = CF.chunk_partials(list(t))
        want = oracle.rsum(t)
        diff_reading += bits(want) != bits(CF.largest_block_first(parts))
        flat = np.float32(0)
        for v in t:
            flat = np.float32(flat + v)
        diff_flat += bits(want) != bits(flat)
    assert diff_reading > 0 and diff_flat > 0


def test_rsum_error_bound():
    u = 2.0 ** -24
    for n in (100, 2048, 50304):
        t = RNG.standard_normal(n).astype(np.float32)
        exact = sum(F(float(v)) for v in t)
        nc = math.ceil(n / 32)
        m = 31 + math.ceil(math.log2(nc)) if nc > 1 else 31
        gamma = m * u / (1 - m * u)
        bound = gamma * float(np.abs(t.astype(np.float64)).sum())
        assert abs(float(oracle.rsum(t)) - float(exact)) <= bound


def bf16_vals(n, scale_exp=(-8, 8)):
    v = RNG.standard_normal(n) * np.exp2(RNG.integers(*scale_exp, n))
    u = v.astype(np.float32).view(np.uint32)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return u


def widen(u):
    return (u.astype(np.uint32) << 16).view(np.float32)


@pytest.mark.parametrize("n", [1, 31, 32, 128, 2048, 6144 + 7])
def test_rdot_bf16_is_fma_chain_plus_fold(n):
    a, b = bf16_vals(n), bf16_vals(n)
    prods = widen(a) * widen(b)  # bf16 x bf16 products are exact in float32
    assert bits(oracle.rdot_bf16(a, b)) == bits(CF.canonical_sum(list(prods)))


def test_rdot_f32_is_unfused():
    a, b = wide(1000), wide(1000)
    prods = (a * b).astype(np.float32)  # one rounding per product, then the chain
    assert bits(oracle.rdot_f32(a, b)) == bits(CF.canonical_sum(list(prods)))


def test_treefold_golden_stack_bound():
    path = os.path.join(os.path.dirname(__file__), "golden", "treefold_stack.txt")
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    for n_rep, max_entries in rows:
        _, deepest = oracle.treefold(np.ones((int(n_rep), 4), np.float32))
        assert deepest == int(max_entries)


@pytest.mark.parametrize("n", list(range(1, 41)) + [64, 100, 255, 256, 257])
def test_treefold_equals_padded_tree(n):
    parts = wide(n)
    got, _ = oracle.treefold(parts.reshape(n, 1))
    assert bits(got[0]) == bits(CF.padded_tree(list(parts)))


def _plan_formulation(grads, accum, shard, rep):
    """Alg. 1 restated: per replica, the ascending-shard sum of (accum-weighted) rank gradients; the
    replica partials (times the shard reciprocal) folded by the padded tree; then times 1/dp_replicate.
    Each element independently (vectorized over elements with float32 numpy)."""
    ia, ish, irep = (np.float32(1.0 / x) for x in (accum, shard, rep))
    reps = []
    for rp in range(rep):
        inner = None
        for sh in range(shard):
            r = rp * shard + sh
            g = np.zeros_like(grads[0])
            for k in range(accum):
                g = (g + (grads[r * accum + k] * ia).astype(np.float32)).astype(np.float32)
            inner = g if inner is None else (inner + g).astype(np.float32)
        reps.append((inner * ish).astype(np.float32))
    out = np.array([CF.padded_tree([rp[i] for rp in reps]) for i in range(grads[0].size)], np.float32)
    return (out * irep).astype(np.float32)


PLANS = [(1, 8, 1), (1, 1, 8), (1, 2, 4), (2, 4, 1), (1, 1, 6), (1, 1, 7), (3, 2, 3), (2, 3, 5)]


@pytest.mark.parametrize("plan", PLANS)
def test_grad_plan_matches_alg1_formulation(plan):
    accum, shard, rep = plan
    grads = [wide(257) for _ in range(accum * shard * rep)]
    got = oracle.grad_accum(grads, accum, shard, rep)
    assert np.array_equal(bits(got), bits(_plan_formulation(grads, accum, shard, rep)))


def test_grad_plan_exact_mean_for_power_of_two_plans():
    for accum, shard, rep in [(1, 8, 1), (2, 4, 2), (1, 2, 4), (4, 1, 2)]:
        n = accum * shard * rep
        grads = [RNG.integers(-64, 64, 100).astype(np.float32) for _ in range(n)]
        want = np.sum(np.stack(grads).astype(np.float64), axis=0) / n
        assert np.array_equal(oracle.grad_accum(grads, accum, shard, rep).astype(np.float64), want)


def test_grad_plan_negative_controls():
    # (1) a reciprocal multiply differs from a division for a non-power-of-two divisor (the appendix on averages);
    # (2) swapping mesh order (shard-major instead of replica-major) changes bits.
    x = wide(4096)
    got = oracle.grad_accum([x], 1, 1, 1)
    assert np.array_equal(got, x)
    g3 = oracle.grad_accum([x, np.zeros_like(x), np.zeros_like(x)], 3, 1, 1)
    assert np.array_equal(bits(g3), bits((x * np.float32(1 / 3)).astype(np.float32)))
    assert np.any(bits(g3) != bits((x / np.float32(3)).astype(np.float32)))
    grads = [wide(512) for _ in range(6)]
    a = oracle.grad_accum(grads, 1, 2, 3)
    swapped = [grads[sh * 3 + rp] for rp in range(3) for sh in range(2)]  # re-index as if shard-major
    b = oracle.grad_accum(swapped, 1, 2, 3)
    assert np.any(bits(a) != bits(b))
