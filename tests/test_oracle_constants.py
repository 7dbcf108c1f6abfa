"""Pins for the constants the oracle evaluates on the host from an integer size.

RN32(1/sqrt(n)) serves as the attention scale (n = head_dim) and as LSQ's gradient scale (n = 127 K, K the
features of the projection input).  The oracle decides it exactly; these tests check it against 60-digit
decimal arithmetic and against an exact integer bracket written here, over every head size up to 4096, every
K up to 2^17 and random sizes up to 2^59.  RN32(1/n) of the averages is checked against exact rationals.
"""
from decimal import Decimal, getcontext
from fractions import Fraction as F

import numpy as np
import pytest

import exact_r0 as X
import oracle


def rn32_decimal(n: int) -> int:
    """Bits of RN32(1/sqrt(n)) from a 60-digit decimal value (the error of 1e-60 relative is far below the
    distance of 1/sqrt(n) to any binary32 rounding boundary, which is at least 2^-52 relative)."""
    getcontext().prec = 60
    v = F(1 / Decimal(n).sqrt())
    return int(np.float32(float(X.round24(v))).view(np.uint32))


def bracket_ok(n: int, y: np.float32) -> bool:
    """y = RN32(1/sqrt(n)) iff 1/sqrt(n) lies strictly between the midpoints to y's neighbours; with
    y = m 2^e (2^23 <= m < 2^24) a midpoint P 2^Q lies above 1/sqrt(n) iff P^2 n 2^(2Q) > 1."""
    mant, e = np.frexp(np.float64(y))
    m = int(mant * 2 ** 24)
    e = int(e) - 24
    assert 2 ** 23 <= m < 2 ** 24

    def above(P, Q):  # P 2^Q > 1/sqrt(n)
        return P * P * n > 2 ** (-2 * Q)

    up = above(2 * m + 1, e - 1)
    lo = (4 * m - 1, e - 2) if m == 2 ** 23 else (2 * m - 1, e - 1)
    return up and not above(*lo)


def test_inv_sqrt_head_sizes_against_decimal():
    for hd in range(1, 4097):
        got = int(oracle.inv_sqrt_int(hd).view(np.uint32))
        assert got == rn32_decimal(hd), hd
    assert int(oracle.inv_sqrt_int(128).view(np.uint32)) == 0x3DB504F3


def test_inv_sqrt_lsq_scales_against_decimal():
    # the projection input widths of the 1B workload and the paper's architecture, and a sweep
    ks = sorted(set([2048, 5632, 8192, 11264, 16384, 128256] + list(range(1, 8193))))
    for k in ks:
        got = int(oracle.inv_sqrt_int(127 * k).view(np.uint32))
        assert got == rn32_decimal(127 * k), k


def test_inv_sqrt_exact_bracket_wide_range():
    rng = np.random.default_rng(7)
    ns = list(range(1, 1 << 12)) + [127 * k for k in range(1, (1 << 17) + 1)]
    ns += [int(x) for x in rng.integers(1, 1 << 59, 20000, dtype=np.int64)]
    ns += [4 ** j for j in range(30)] + [4 ** j - 1 for j in range(1, 30)] + [4 ** j + 1 for j in range(30)]
    for n in ns:
        y = oracle.inv_sqrt_int(n)
        assert bracket_ok(n, y), n


def test_inv_sqrt_powers_of_four_are_exact():
    for j in range(30):
        assert float(oracle.inv_sqrt_int(4 ** j)) == 2.0 ** -j


@pytest.mark.parametrize("n", [0, -1, 1 << 60])
def test_inv_sqrt_out_of_range_is_nan(n):
    assert np.isnan(oracle.inv_sqrt_int(n))


def test_bracket_rejects_neighbours():
    """The bracket test itself: one unit up or down is never accepted."""
    for n in [2, 3, 5, 127 * 2048, 127 * 8192, 1000003]:
        y = oracle.inv_sqrt_int(n)
        assert bracket_ok(n, y)
        assert not bracket_ok(n, np.nextafter(y, np.float32(1)))
        assert not bracket_ok(n, np.nextafter(y, np.float32(0)))
