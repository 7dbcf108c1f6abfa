"""Canonical state hash: the oracle (TEST INFRASTRUCTURE; only tests, the smoke check and the benchmark's
CPU-baseline leg may use it).

The paper anchors every training step with a sharded canonical hash of each rank's batches, parameters,
optimizer state and gradient shards, computed on the host, and names moving it onto the device as its next
step (appendix on the state-hash overhead; the discussion of runtime overheads).  It does not fix the
hash function, so this build defines one, H1, built from SHA-256 (FIPS 180-4):

* A tensor of n bytes is cut into nb = ceil(n / 64) blocks of 64 bytes (the last one may be shorter).
* It has W = max(1, ceil(nb / 1024)) leaves.  Leaf l holds the blocks l, l + W, l + 2W, ... in that order
  (interleaved, so that neighbouring leaves read neighbouring memory); its digest is SHA-256 of their bytes.
* The leaf digests are folded pairwise level by level, SHA-256(left || right), an odd last node passing up
  unchanged, down to one root.
* tensor digest = SHA-256(0x02 || index (8 bytes, little endian) || n (8 bytes, little endian) || root).
* state digest = SHA-256(0x03 || tensor digest 0 || tensor digest 1 || ...), tensors in the declared order.

The primitive is Python's hashlib.sha256; everything else is spelled out below.
"""
from __future__ import annotations

import hashlib
import math

BLOCK = 64
BLOCKS_PER_LEAF = 1024


def sha256(b: bytes) -> bytes:
    return hashlib.sha256(b).digest()


def leaf_count(n: int) -> int:
    nb = (n + BLOCK - 1) // BLOCK
    return max(1, (nb + BLOCKS_PER_LEAF - 1) // BLOCKS_PER_LEAF)


def leaf_digests(buf: bytes) -> list:
    n = len(buf)
    nb = (n + BLOCK - 1) // BLOCK
    W = leaf_count(n)
    return [sha256(b"".join(buf[BLOCK * b: BLOCK * b + BLOCK] for b in range(l, nb, W))) for l in range(W)]


def merkle_root(level: list) -> bytes:
    while len(level) > 1:
        nxt = [sha256(level[i] + level[i + 1]) for i in range(0, len(level) - 1, 2)]
        if len(level) % 2:
            nxt.append(level[-1])
        level = nxt
    return level[0]


def tensor_digest(buf: bytes, index: int) -> bytes:
    root = merkle_root(leaf_digests(buf))
    return sha256(b"\x02" + index.to_bytes(8, "little") + len(buf).to_bytes(8, "little") + root)


def state_digest(buffers) -> bytes:
    return sha256(b"\x03" + b"".join(tensor_digest(bytes(b), i) for i, b in enumerate(buffers)))
