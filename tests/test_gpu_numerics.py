"""Device primitives (R0, R4) against the oracle, bit for bit, on adversarial and dense inputs."""
import numpy as np
import pytest
import torch

import adversarial as ADV
import oracle
import paper_2609_17380_amd.canon as C
from gpu_util import assert_bits, dev_f32, host_f32

pytestmark = pytest.mark.gpu

A, B, CC = ADV.triples(seed=777, n=20000)


def run(op, a, b=None, c=None):
    n = a.size
    da = dev_f32(a)
    db = dev_f32(b if b is not None else a)
    dc = dev_f32(c if c is not None else a)
    out = torch.empty(n, dtype=torch.float32, device=da.device)
    C.devmath(op, n, da, db, dc, out)
    torch.cuda.synchronize()
    return host_f32(out)


@pytest.mark.parametrize("op", ["add", "sub", "mul", "fma"])
def test_r0_ops_match_oracle(op):
    print(f"devmath {op} n={A.size}", flush=True)
    assert_bits(run(op, A, B, CC), oracle.prim(op, A, B, CC), op)


def test_division_matches_oracle():
    keep = np.abs(B) >= np.float32(2.0 ** -126)
    a, b = A[keep], B[keep]
    got, want = run("div", a, b), oracle.prim("div", a, b)
    fin = np.isfinite(want)
    assert_bits(got[fin], want[fin], "div")


def test_sqrt_matches_oracle_sampled_bit_patterns():
    u = np.arange(0, 1 << 32, 251, dtype=np.uint64).astype(np.uint32)
    x = u.view(np.float32)
    x = x[np.isfinite(x) & (x >= 0)]
    assert_bits(run("sqrt", x), oracle.prim("sqrt", x), "sqrt")


@pytest.mark.parametrize("op", ["exp", "log", "sigmoid", "silu", "bf16"])
def test_canonical_functions_match_oracle(op):
    rng = np.random.default_rng(5)
    dense = np.linspace(-100, 100, 400001, dtype=np.float32)
    pos = np.exp(np.linspace(-80, 80, 200001)).astype(np.float32)
    rnd = ADV.random_floats(rng, 200000, 0, 254)
    x = np.concatenate([dense, pos, rnd, A])
    x = x[np.isfinite(x)]
    if op == "log":
        x = np.abs(x)
    got, want = run(op, x), oracle.prim(op, x)
    ok = ~(np.isnan(got) & np.isnan(want))
    assert_bits(got[ok], want[ok], op)


def _oracle_parallel(op, a, b=None, parts=16):
    """The oracle's scalar primitive over a large array, split over host threads (each element is independent;
    ctypes releases the interpreter lock during the call)."""
    import concurrent.futures as cf
    out = np.empty_like(a)
    edges = np.linspace(0, a.size, parts + 1).astype(np.int64)

    def work(i):
        lo, hi = edges[i], edges[i + 1]
        out[lo:hi] = oracle.prim(op, a[lo:hi], None if b is None else b[lo:hi])

    with cf.ThreadPoolExecutor(max_workers=parts) as ex:
        list(ex.map(work, range(parts)))
    return out


def _same_or_both_nan(got, want):
    g, w = got.view(np.uint32), want.view(np.uint32)
    return (g == w) | (np.isnan(got) & np.isnan(want))


def test_sqrt_exhaustive_all_bit_patterns():
    """CRsqrt over all 2^32 binary32 inputs against the oracle (IEEE sqrt after the input flush), in chunks of
    2^28 generated on both sides from the same bit-pattern ranges."""
    chunk = 1 << 28
    bad = 0
    for c0 in range(-(1 << 31), 1 << 31, chunk):
        print(f"sqrt exhaustive: bit patterns {c0 & 0xFFFFFFFF:#010x} .. +2^28", flush=True)
        x_dev = torch.arange(c0, c0 + chunk, dtype=torch.int32, device="cuda").view(torch.float32)
        out = torch.empty(chunk, dtype=torch.float32, device="cuda")
        C.devmath("sqrt", chunk, x_dev, None, None, out)
        torch.cuda.synchronize()
        got = host_f32(out)
        del out, x_dev
        x = np.arange(c0, c0 + chunk, dtype=np.int64).astype(np.int32).view(np.float32)
        want = _oracle_parallel("sqrt", x)
        ok = _same_or_both_nan(got, want)
        if not ok.all():
            i = np.nonzero(~ok)[0][0]
            raise AssertionError(f"sqrt({x[i]!r} = {x.view(np.uint32)[i]:#x}): gpu {got[i]!r} oracle {want[i]!r}; "
                                 f"{(~ok).sum()} in this chunk")
        bad += int((~ok).sum())
    assert bad == 0


def test_division_billion_pairs():
    """CRdiv on 2^30 operand pairs against the oracle: uniformly random bit patterns (every class: zeros,
    subnormals, normals, infinities, NaNs), and pairs whose quotient lands near the overflow threshold and
    near the 2^-126 flush boundary."""
    rng = np.random.default_rng(123)
    chunk = 1 << 27
    for it in range(8):
        print(f"division: pairs {it * chunk} .. {(it + 1) * chunk}", flush=True)
        if it < 6:
            a = rng.integers(0, 1 << 32, chunk, dtype=np.uint64).astype(np.uint32).view(np.float32)
            b = rng.integers(0, 1 << 32, chunk, dtype=np.uint64).astype(np.uint32).view(np.float32)
        else:
            # quotients near 2^128 (it 6) and near 2^-126 (it 7): a random significand pair, exponents chosen
            # so the quotient's exponent is the target give or take one
            target = 127 if it == 6 else -126
            ea = rng.integers(-100, 101, chunk)
            eb = ea - target + rng.integers(-1, 2, chunk)
            ok = (eb >= -126) & (eb <= 127)
            eb = np.where(ok, eb, 0)
            ea = np.where(ok, ea, target)
            ma = rng.integers(1 << 23, 1 << 24, chunk).astype(np.float64)
            mb = rng.integers(1 << 23, 1 << 24, chunk).astype(np.float64)
            sa = rng.choice([-1.0, 1.0], chunk)
            a = (sa * np.ldexp(ma, (ea - 23).astype(np.int32))).astype(np.float32)
            b = np.ldexp(mb, (eb - 23).astype(np.int32)).astype(np.float32)
        out = torch.empty(chunk, dtype=torch.float32, device="cuda")
        da, db = dev_f32(a), dev_f32(b)
        C.devmath("div", chunk, da, db, None, out)
        torch.cuda.synchronize()
        got = host_f32(out)
        del out, da, db
        want = _oracle_parallel("div", a, b)
        ok = _same_or_both_nan(got, want)
        if not ok.all():
            i = np.nonzero(~ok)[0][0]
            raise AssertionError(f"{a[i]!r} / {b[i]!r}: gpu {got[i]!r} oracle {want[i]!r}; {(~ok).sum()} differ")
