"""Alternative formulations of the canonical order, used only to pin the oracle.

These are written differently from the oracle on purpose: the chunk partials
are folded by a recursive, zero-padded perfect binary tree (an equivalent
description of Alg. 2's binary-carry fold with the leftover blocks combined
smallest first), not by a stack.  Arithmetic is numpy float32 (IEEE round to
nearest even); the inputs used with them stay far from the subnormal range,
where R0 and plain IEEE arithmetic agree.
"""
import numpy as np


def padded_tree(parts):
    parts = [np.float32(p) for p in parts]
    n = len(parts)
    if n == 0:
        return np.float32(0.0)
    size = 1
    while size < n:
        size *= 2

    def rec(lo, sz):
        if sz == 1:
            return parts[lo]
        half = sz // 2
        if lo + half >= n:  # the right half is padding only: x + (+0) = x
            return rec(lo, half)
        return np.float32(rec(lo, half) + rec(lo + half, half))

    return rec(0, size)


def largest_block_first(parts):
    """The other reading of Alg. 2's Result (combine the leftover blocks largest first)."""
    parts = [np.float32(p) for p in parts]
    n = len(parts)
    blocks, lo = [], 0
    for bit in reversed(range(n.bit_length())):
        if n >> bit & 1:
            blocks.append(padded_tree(parts[lo:lo + (1 << bit)]))
            lo += 1 << bit
    acc = blocks[0]
    for b in blocks[1:]:
        acc = np.float32(acc + b)
    return acc


def chunk_partials(terms, chunk=32):
    out = []
    for c0 in range(0, len(terms), chunk):
        s = np.float32(0.0)
        for t in terms[c0:c0 + chunk]:
            s = np.float32(s + np.float32(t))
        out.append(s)
    return out


def canonical_sum(terms, chunk=32):
    return padded_tree(chunk_partials(terms, chunk))


def canonical_dot_r0(a, b, chunk=32):
    """The canonical dot product of two float sequences in exact rational arithmetic with the R0 rounding
    model (DAZ inputs, one round to nearest even per fma, flush of tiny results): fma chains of `chunk` terms
    from +0, then the zero-padded tree with absent padding.  Valid over the whole float range."""
    import exact_r0 as R
    n = len(a)
    parts = []
    for c0 in range(0, n, chunk):
        s = np.float32(0.0)
        for x, y in zip(a[c0:c0 + chunk], b[c0:c0 + chunk]):
            s = R.fma(x, y, s)
        parts.append(s)
    if not parts:
        return np.float32(0.0)
    size = 1
    while size < len(parts):
        size *= 2

    def rec(lo, sz):
        if sz == 1:
            return parts[lo]
        half = sz // 2
        if lo + half >= len(parts):
            return rec(lo, half)
        return R.add(rec(lo, half), rec(lo + half, half))

    return rec(0, size)
