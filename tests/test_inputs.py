"""Pins for the seeded input generator (Philox4x32-10, Salmon et al., SC'11)."""
import numpy as np

import paper_2609_17380_amd.inputs as I

# Known-answer vectors published with the Random123 reference implementation of Philox4x32-10.
KAT = [
    ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
    ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
    ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
     [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
]


def test_philox_known_answers():
    for ctr, key, want in KAT:
        assert I.philox4x32_10(ctr, key).tolist() == want


def test_stream_is_index_addressable():
    full = I.normal_bf16((1000,), seed=0, tid=7)
    part = I.normal_bf16((300,), seed=0, tid=7, start=401)
    assert np.array_equal(full[401:701], part)
    ints = I.uniform_int((999,), seed=3, tid=6, bound=50304)
    assert np.array_equal(ints[5:50], I.uniform_int((45,), seed=3, tid=6, bound=50304, start=5))


def test_distribution_shapes():
    z = I.normal_f32((1 << 18,), seed=0, tid=1)
    assert abs(float(z.mean())) < 0.01 and abs(float(z.std()) - 1) < 0.01
    w = I.bf16_bits_to_f32(I.normal_bf16((1 << 16,), seed=0, tid=2, std=0.02))
    assert abs(float(w.std()) - 0.02) < 0.001
    t = I.uniform_int((1 << 16,), seed=0, tid=6, bound=50304)
    assert t.min() >= 0 and t.max() < 50304
    # different tensor ids give unrelated streams
    assert not np.array_equal(I.normal_bf16((64,), 0, 1), I.normal_bf16((64,), 0, 2))
