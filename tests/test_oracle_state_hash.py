"""Pins for the state-hash oracle: the SHA-256 primitive against the FIPS 180-2 example vectors, and the
H1 structure (leaf interleaving, leaf count boundaries, the pairwise fold with a promoted odd node, the
domain bytes) checked against hand-built digests and against single-byte changes."""
import hashlib

import numpy as np
import pytest

from oracle import state_hash as H


@pytest.mark.parametrize("msg,hexd", [
    (b"abc", "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"),
    (b"", "e3b0c44298fc1c149afbf4c8996fb92427ae41e4649b934ca495991b7852b855"),
    (b"abcdbcdecdefdefgefghfghighijhijkijkljklmklmnlmnomnopnopq",
     "248d6a61d20638b8e5c026930c3e6039a33ce45964ff2167f6ecedd419db06c1"),
])
def test_sha256_fips_vectors(msg, hexd):
    assert H.sha256(msg).hex() == hexd


def test_sha256_million_a():
    assert H.sha256(b"a" * 1_000_000).hex() == "cdc76e5c9914fb9281a1c7e284d73e67f1809a48a497200e046d39ccc7112cd0"


@pytest.mark.parametrize("n,w", [(0, 1), (1, 1), (64 * 1024, 1), (64 * 1024 + 1, 2), (64 * 2048, 2),
                                 (64 * 2048 + 64, 3)])
def test_leaf_count_boundaries(n, w):
    assert H.leaf_count(n) == w


def test_interleaved_leaves_and_fold_by_hand():
    rng = np.random.default_rng(0)
    buf = rng.integers(0, 256, 64 * 3000 + 17, dtype=np.uint8).tobytes()   # 3001 blocks -> 3 leaves
    blocks = [buf[64 * i: 64 * i + 64] for i in range(3001)]
    leaves = [hashlib.sha256(b"".join(blocks[l::3])).digest() for l in range(3)]
    assert H.leaf_digests(buf) == leaves
    root = hashlib.sha256(hashlib.sha256(leaves[0] + leaves[1]).digest() + leaves[2]).digest()  # odd leaf promoted
    assert H.merkle_root(leaves) == root
    want = hashlib.sha256(b"\x02" + (7).to_bytes(8, "little") + len(buf).to_bytes(8, "little") + root).digest()
    assert H.tensor_digest(buf, 7) == want


def test_state_digest_sensitivity():
    rng = np.random.default_rng(1)
    bufs = [rng.integers(0, 256, n, dtype=np.uint8).tobytes() for n in (0, 5, 64 * 1024 + 3, 300000)]
    d = H.state_digest(bufs)
    assert d == hashlib.sha256(b"\x03" + b"".join(H.tensor_digest(b, i) for i, b in enumerate(bufs))).digest()
    for t in range(1, 4):
        for pos in (0, len(bufs[t]) // 2, len(bufs[t]) - 1):
            changed = list(bufs)
            bb = bytearray(changed[t])
            bb[pos] ^= 1
            changed[t] = bytes(bb)
            assert H.state_digest(changed) != d
    assert H.state_digest(bufs[::-1]) != d           # tensor order matters
    assert H.state_digest(bufs[:1] + [b""] + bufs[1:]) != d  # so does an empty tensor
