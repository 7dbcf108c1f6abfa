"""Random and adversarial fp32 operands: ties, cancellation, the 2^-126 band, signed zeros, subnormals."""
import numpy as np


def f32_from_bits(u):
    return np.asarray(u, dtype=np.uint32).view(np.float32)


def random_floats(rng, n, exp_lo=0, exp_hi=254):
    sign = rng.integers(0, 2, n, dtype=np.uint32) << 31
    ex = rng.integers(exp_lo, exp_hi + 1, n, dtype=np.uint32) << 23
    man = rng.integers(0, 1 << 23, n, dtype=np.uint32)
    return f32_from_bits(sign | ex | man)


def triples(seed=12345, n=3000):
    rng = np.random.default_rng(seed)
    a, b, c = [], [], []
    a += list(random_floats(rng, n, 0, 254)); b += list(random_floats(rng, n, 0, 254)); c += list(random_floats(rng, n, 0, 254))
    a += list(random_floats(rng, n, 100, 150)); b += list(random_floats(rng, n, 100, 150)); c += list(random_floats(rng, n, 100, 150))
    base = random_floats(rng, n, 110, 140)
    ulp = np.spacing(np.abs(base)).astype(np.float64)
    tie = (ulp / 2 * (2 * rng.integers(0, 4, n) + 1) * rng.choice([-1, 1], n)).astype(np.float32)
    a += list(base); b += list(tie); c += list(tie)
    T = 2.0 ** -126
    ua = (0.5 + rng.random(n) * 0.5).astype(np.float32)
    ub = ((T / ua.astype(np.float64)) * (1 + (rng.random(n) - 0.5) * 2.0 ** -21)).astype(np.float32)
    ub = np.maximum(ub, np.float32(T)) * rng.choice([-1, 1], n).astype(np.float32)
    a += list(ua); b += list(ub); c += [np.float32(0.0)] * n
    a2 = (1.0 + rng.integers(1, 2 ** 23, n) * 2.0 ** -23).astype(np.float32)
    cc = np.full(n, 2.0 ** -124, np.float32) * rng.choice([-1, 1], n).astype(np.float32)
    b2 = ((-(2.0 ** -124 - T * (1 + (rng.random(n) - 0.5) * 2.0 ** -20) * np.sign(cc)) / a2.astype(np.float64))
          ).astype(np.float32)
    a += list(a2); b += list(b2); c += list(cc)
    a += list(base); b += list((-base * (1 + rng.integers(-3, 4, n) * 2.0 ** -23)).astype(np.float32)); c += list(base)
    for za in (0.0, -0.0, 1.5, -1.5, 2.0 ** -130, -(2.0 ** -130)):
        for zb in (0.0, -0.0, 3.0, -3.0):
            for zc in (0.0, -0.0, -4.5):
                a.append(np.float32(za)); b.append(np.float32(zb)); c.append(np.float32(zc))
    return np.array(a, np.float32), np.array(b, np.float32), np.array(c, np.float32)


def _bf16(sign, exp, man):
    return ((np.asarray(sign, np.uint32) << 15) | (np.asarray(exp, np.uint32) << 7) | np.asarray(man, np.uint32)
            ).astype(np.uint16)


def gemm_operands(kind, m, n, k, seed=7):
    """bf16 bit patterns A [m, k] and B [k, n] (logical layouts) that drive a canonical GEMM chain into its
    corner cases.
      wide:   exponents over 2^-64 .. 2^55, so products run from the subnormal range to 2^111
      tiny:   products and partial sums around 2^-126, with bf16 subnormal operands and signed zeros
      ties:   a 2^24 term opens every chunk, then small integers and halves: many exact round-half-even ties
      cancel: every product is cancelled by its neighbour; zeros of both signs
      huge:   same-signed products of at least 2^124: chains overflow to +-inf (never inf - inf)"""
    rng = np.random.default_rng(seed)
    if kind == "wide":
        a = _bf16(rng.integers(0, 2, (m, k)), rng.integers(127 - 64, 127 + 56, (m, k)), rng.integers(0, 128, (m, k)))
        b = _bf16(rng.integers(0, 2, (k, n)), rng.integers(127 - 64, 127 + 56, (k, n)), rng.integers(0, 128, (k, n)))
    elif kind == "tiny":
        def tiny(shape):
            e = rng.integers(127 - 66, 127 - 59, shape)
            e = np.where(rng.random(shape) < 0.05, 0, e)  # subnormal operands (read as zero)
            mant = rng.integers(0, 128, shape)
            mant = np.where((e == 0) & (mant == 0), 1, mant)
            out = _bf16(rng.integers(0, 2, shape), e, mant)
            return np.where(rng.random(shape) < 0.03, _bf16(rng.integers(0, 2, shape), 0, 0), out)
        a, b = tiny((m, k)), tiny((k, n))
    elif kind == "ties":
        small = np.array([0x3F80, 0xBF80, 0x4040, 0xC040, 0x3F00, 0xBF00, 0x3FC0, 0xBFC0], np.uint16)  # +-1, 3, .5, 1.5
        a = small[rng.integers(0, 8, (m, k))]
        b = small[rng.integers(0, 8, (k, n))]
        a[:, ::32] = 0x4580  # 2^12
        b[::32, :] = 0x4580
    elif kind == "cancel":
        a = _bf16(rng.integers(0, 2, (m, k)), rng.integers(100, 150, (m, k)), rng.integers(0, 128, (m, k)))
        a[:, 1::2] = a[:, 0:(k // 2) * 2:2] ^ np.uint16(0x8000)
        b = _bf16(rng.integers(0, 2, (k, n)), rng.integers(100, 150, (k, n)), rng.integers(0, 128, (k, n)))
        b[1::2, :] = b[0:(k // 2) * 2:2, :]
        z = np.repeat(rng.random((m, (k + 1) // 2)) < 0.1, 2, axis=1)[:, :k]  # zero both terms of a pair
        a = np.where(z, _bf16(rng.integers(0, 2, (m, k)), 0, 0), a)
    elif kind == "huge":
        a = _bf16(0, rng.integers(127 + 62, 127 + 64, (m, k)), rng.integers(0, 128, (m, k)))
        sgn = rng.integers(0, 2, n)
        b = _bf16(np.broadcast_to(sgn, (k, n)), rng.integers(127 + 62, 127 + 64, (k, n)), rng.integers(0, 128, (k, n)))
    else:
        raise ValueError(kind)
    return np.ascontiguousarray(a, np.uint16), np.ascontiguousarray(b, np.uint16)


GEMM_KINDS = ("wide", "tiny", "ties", "cancel", "huge")
