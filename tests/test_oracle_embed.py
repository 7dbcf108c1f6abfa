"""Pins for the oracle's embedding backward (R11): dE[v] = R1 sum over the ascending positions t with
tok[t] = v of dx[t].

Tokens repeated 33, 100 and 1500 times exercise the multi-chunk path (chains of 32, then Algorithm 2 over
the chain partials).  Integer-valued gradients make every partial exact, so the result must be the exact sum
(this pins the grouping by token, completeness and the +0 rows).  Gradients spread over many binades make the
order matter: the result must equal an independent formulation of R1 over the ascending positions
(a recursive zero-padded tree, `canon_formulations`) and differ from descending, flat and 31-term orders.
"""
import numpy as np
import pytest

import canon_formulations as CF
import oracle

RNG = np.random.default_rng(2026)


def skewed_tokens(counts: dict, n_single: int, vocab: int, rng) -> np.ndarray:
    toks = []
    for v, c in counts.items():
        toks += [v] * c
    rest = [v for v in range(vocab) if v not in counts]
    toks += list(rng.choice(rest, size=n_single, replace=False))
    toks = np.array(toks, np.int32)
    rng.shuffle(toks)
    return toks


def bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def test_repeated_tokens_integer_gradients_are_exact():
    V, d = 300, 24
    counts = {5: 33, 17: 100, 250: 1500, 99: 32, 100: 64, 101: 65}
    tok = skewed_tokens(counts, 40, V, RNG)
    dx = RNG.integers(-8, 9, size=(tok.size, d)).astype(np.float32)
    dE = oracle.embed_bwd(tok, dx, V)
    want = np.zeros((V, d), np.int64)
    np.add.at(want, tok, dx.astype(np.int64))
    assert np.array_equal(dE.astype(np.int64), want)
    absent = np.setdiff1d(np.arange(V), tok)
    assert np.all(bits(dE[absent]) == 0), "rows that never occur must be +0"


def wide_range_grads(T, d, rng):
    return (rng.standard_normal((T, d)) * 2.0 ** rng.integers(-20, 21, size=(T, d))).astype(np.float32)


def test_order_matches_ascending_positions_and_not_others():
    V, d = 64, 8
    counts = {3: 1500, 7: 100, 11: 33, 12: 1}
    tok = skewed_tokens(counts, 20, V, RNG)
    dx = wide_range_grads(tok.size, d, RNG)
    dE = oracle.embed_bwd(tok, dx, V)
    differs_desc = differs_flat = differs_31 = 0
    for v in counts:
        pos = np.nonzero(tok == v)[0]
        for j in range(d):
            terms = dx[pos, j]
            want = CF.canonical_sum(list(terms))
            assert bits(dE[v, j]) == bits(want), (v, j)
            if counts[v] > 32:
                differs_desc += bits(CF.canonical_sum(list(terms[::-1]))) != bits(want)
                flat = np.float32(0.0)
                for t in terms:
                    flat = np.float32(flat + t)
                differs_flat += bits(flat) != bits(want)
                differs_31 += bits(CF.canonical_sum(list(terms), chunk=31)) != bits(want)
    assert differs_desc > 0 and differs_flat > 0 and differs_31 > 0


def test_single_occurrence_and_signed_zero():
    V, d = 10, 4
    tok = np.array([2, 4, 4], np.int32)
    dx = np.array([[1.5, -0.0, 3.0, -2.0], [-0.0, -0.0, 1.0, 2.0], [-0.0, 0.0, 1.0, -2.0]], np.float32)
    dE = oracle.embed_bwd(tok, dx, V)
    # one term: +0 + t; a -0 term gives +0 (the chain starts at +0)
    assert bits(dE[2]).tolist() == bits(np.array([1.5, 0.0, 3.0, -2.0], np.float32)).tolist()
    assert bits(dE[4]).tolist() == bits(np.array([0.0, 0.0, 2.0, 0.0], np.float32)).tolist()


def test_out_of_range_tokens_contribute_nothing():
    V, d = 16, 3
    tok = np.array([1, -1, 16, 1, 400, 2], np.int32)
    dx = np.arange(18, dtype=np.float32).reshape(6, 3)
    dE = oracle.embed_bwd(tok, dx, V)
    want = np.zeros((V, d), np.float32)
    want[1] = dx[0] + dx[3]
    want[2] = dx[5]
    assert np.array_equal(dE, want)


def test_empty_microbatch_gives_zero_rows():
    dE = oracle.embed_bwd(np.zeros(0, np.int32), np.zeros((0, 5), np.float32), 7)
    assert np.all(bits(dE) == 0)


@pytest.mark.parametrize("count", [32, 33, 64, 65, 96, 97, 1024, 1025, 1500])
def test_chunk_boundaries_hand_derived(count):
    """A token's first occurrence carries 2^24 and the others 1.  Chunk 0 absorbs its 31 ones (each
    2^24 + 1 ties to 2^24), later chunks sum their ones exactly, so 64 occurrences give 2^24 + 32 (a flat
    sum gives 2^24).  Every count must also equal the independent formulation."""
    V, d = 8, 2
    tok = np.full(count, 6, np.int32)
    dx = np.ones((count, d), np.float32)
    dx[0] = 2.0 ** 24
    dE = oracle.embed_bwd(tok, dx, V)
    want = CF.canonical_sum(list(dx[:, 0]))
    assert np.all(bits(dE[6]) == bits(want))
    if count == 64:
        assert dE[6, 0] == 2.0 ** 24 + 32
    if count <= 32:
        assert dE[6, 0] == 2.0 ** 24
