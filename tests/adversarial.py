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
