"""canon_gemm against the oracle: bit for bit at small shapes (all layouts, ragged tiles, many chunk
counts) and on sampled outputs at the 1B decoder's full GEMM shapes."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import DEV, assert_bits, dev_bf16, host_f32

pytestmark = pytest.mark.gpu


def gpu_gemm(a, b, ta, tb, m, n, k):
    da, db = dev_bf16(a), dev_bf16(b)
    c = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
    C.gemm(m, n, k, da, a.shape[1] if a.ndim == 2 else 1, db, b.shape[1] if b.ndim == 2 else 1, c, n, ta, tb)
    torch.cuda.synchronize()
    return host_f32(c)


def operands(m, n, k, ta, tb, seed):
    a = I.normal_bf16((k, m) if ta else (m, k), seed, I.TENSOR_IDS["gemm_a"])
    b = I.normal_bf16((n, k) if tb else (k, n), seed, I.TENSOR_IDS["gemm_b"])
    return a, b


def test_cfg1_bit_exact():
    # 128x256 . 256x128, bf16 N(0,1), seed 0: 8 chunks of 32 per output
    print("gemm cfg1 128x256x128", flush=True)
    a, b = operands(128, 128, 256, 0, 0, 0)
    assert_bits(gpu_gemm(a, b, 0, 0, 128, 128, 256), oracle.gemm(a, b), "cfg1")


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
@pytest.mark.parametrize("m,n,k", [(37, 45, 70), (130, 260, 96), (64, 128, 33), (1, 1, 1), (200, 3, 1000),
                                   (65, 129, 7 * 32), (96, 200, 13 * 32 + 5)])
def test_layouts_and_ragged_shapes(m, n, k, ta, tb):
    print(f"gemm {m}x{n}x{k} ta={ta} tb={tb}", flush=True)
    a, b = operands(m, n, k, ta, tb, 3)
    assert_bits(gpu_gemm(a, b, ta, tb, m, n, k), oracle.gemm(a, b, bool(ta), bool(tb)), f"{m}x{n}x{k}")


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
@pytest.mark.parametrize("k", [2048, 6144, 6144 + 32, 8192, 16384, 16384 + 96, 50304, 128256])
def test_deep_folds(k, ta, tb):
    # chunk counts 64, 192, 193, 256, 512, 515, 1572, 4008: every fold depth the steps use (stack depths 7, 9,
    # 11 and 12), in every operand layout
    print(f"gemm fold depth k={k} ta={ta} tb={tb}", flush=True)
    m, n = 70, 130
    a, b = operands(m, n, k, ta, tb, 4)
    assert_bits(gpu_gemm(a, b, ta, tb, m, n, k), oracle.gemm(a, b, bool(ta), bool(tb)), f"k={k}")


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
@pytest.mark.parametrize("k", [64, 96, 2048, 2080, 6144, 8192, 16384 + 32, 50304, 128256])
def test_whole_tiles_every_depth(k, ta, tb):
    # whole 64 x 128 tiles (the unchecked 16-byte load path of every chunk), even and odd chunk counts, every
    # stack depth, every layout
    print(f"gemm whole tiles 128x256x{k} ta={ta} tb={tb}", flush=True)
    m, n = 128, 256
    a, b = operands(m, n, k, ta, tb, 8)
    assert_bits(gpu_gemm(a, b, ta, tb, m, n, k), oracle.gemm(a, b, bool(ta), bool(tb)), f"k={k}")


@pytest.mark.parametrize("ta,tb", [(0, 1), (1, 0)])
@pytest.mark.parametrize("m,n,k,accum", [(130, 260, 192, 3), (128, 256, 2048, 2), (64, 128, 32, 4), (70, 90, 8192, 1)])
def test_accum_plan_epilogue(m, n, k, accum, ta, tb):
    """canon_gemm's ACCUM_PLAN epilogue over `accum` microbatches, C cleared to +0 first, against the oracle's
    plan on the oracle's GEMMs: g_r = R7's ascending sum of RN(grad * RN(1/accum)) (one rank: the plan's
    result is g_r itself)."""
    print(f"gemm accum-plan {m}x{n}x{k} accum={accum} ta={ta} tb={tb}", flush=True)
    c = torch.zeros((m, n), dtype=torch.float32, device=DEV)
    inv = float(np.float32(1.0 / accum))
    grads = []
    for j in range(accum):
        a, b = operands(m, n, k, ta, tb, 20 + j)
        C.gemm(m, n, k, dev_bf16(a), a.shape[1], dev_bf16(b), b.shape[1], c, n, ta, tb, accum_scale=inv)
        grads.append(oracle.gemm(a, b, bool(ta), bool(tb)))
    torch.cuda.synchronize()
    want = oracle.grad_accum([g.reshape(-1) for g in grads], accum, 1, 1).reshape(m, n)
    assert_bits(host_f32(c), want, f"accum {m}x{n}x{k}")


def test_k_zero_and_empty():
    c = torch.full((4, 5), float("nan"), dtype=torch.float32, device=DEV)
    a = torch.zeros(4, 1, dtype=torch.bfloat16, device=DEV)
    C.gemm(4, 5, 0, a, 1, a, 5, c, 5)
    torch.cuda.synchronize()
    assert np.all(host_f32(c).view(np.uint32) == 0)  # empty sums are +0
    C.gemm(0, 5, 3, a, 3, a, 5, c, 5)  # no-op


def test_strided_batched_and_determinism():
    bt, m, n, k = 3, 96, 80, 160
    a = I.normal_bf16((bt, m, k), 5, 1)
    b = I.normal_bf16((bt, k, n), 5, 2)
    da, db = dev_bf16(a), dev_bf16(b)
    c = torch.empty((bt, m, n), dtype=torch.float32, device=DEV)
    C.gemm_strided_batched(m, n, k, da, k, m * k, db, n, k * n, c, n, m * n, bt)
    c2 = torch.empty_like(c)
    C.gemm_strided_batched(m, n, k, da, k, m * k, db, n, k * n, c2, n, m * n, bt)
    torch.cuda.synchronize()
    for z in range(bt):
        assert_bits(host_f32(c[z]), oracle.gemm(a[z], b[z]), f"batch {z}")
    assert torch.equal(c.view(torch.int32), c2.view(torch.int32))


@pytest.mark.parametrize("m,n,k", [(200, 300, 128), (130, 260, 70), (64, 128, 32), (257, 129, 97)])
def test_short_contraction_batches(m, n, k):
    """K <= 128 with both operands k-contiguous takes the persistent short-contraction kernel: more tiles than
    resident workgroups (each walks several tiles, ragged ones among them), every batch matrix bit-exact."""
    tiles = -(-m // 64) * -(-n // 128)
    bt = -(-768 // tiles)  # 768 tiles: more than the 512 resident workgroups of 256 CUs
    print(f"gemm short {bt}x {m}x{n}x{k}", flush=True)
    a = I.normal_bf16((bt, m, k), 6, 1)
    b = I.normal_bf16((bt, n, k), 6, 2)
    c = torch.empty((bt, m, n), dtype=torch.float32, device=DEV)
    C.gemm_strided_batched(m, n, k, dev_bf16(a), k, m * k, dev_bf16(b), k, n * k, c, n, m * n, bt, trans_b=1)
    torch.cuda.synchronize()
    got = host_f32(c)
    for z in range(bt):
        assert_bits(got[z], oracle.gemm(a[z], b[z], False, True), f"batch {z}")


def test_invalid_arguments_are_rejected():
    a = torch.zeros(16, dtype=torch.bfloat16, device=DEV)
    c = torch.zeros(16, dtype=torch.float32, device=DEV)
    with pytest.raises(C.CanonError) as e:
        C.gemm(4, 4, 4, a, 2, a, 4, c, 4)  # lda < k
    assert e.value.status == C.EINVAL
    with pytest.raises(C.CanonError) as e:
        C.gemm(4, 4, 4, None, 4, a, 4, c, 4)
    assert e.value.status == C.EINVAL
    with pytest.raises(C.CanonError) as e:
        C.gemm(4, 4, 4, a, 4, a, 4, c, 4, order=C.Order(1, 16, 0, 1))
    assert e.value.status == C.EUNSUPPORTED


# full 1B shapes (8192-token microbatch): all fourteen forward, weight-gradient and input-gradient GEMMs of the
# sweep, and the head's input gradient at the paper architecture's vocabulary (contraction 128256)
FULL = [
    ("qkv", 8192, 6144, 2048, 0, 1), ("out", 8192, 2048, 2048, 0, 1), ("gate_up", 8192, 16384, 2048, 0, 1),
    ("down", 8192, 2048, 8192, 0, 1), ("head", 8192, 50304, 2048, 0, 1),
    ("wgrad_qkv", 6144, 2048, 8192, 1, 0), ("wgrad_out", 2048, 2048, 8192, 1, 0),
    ("wgrad_gate_up", 16384, 2048, 8192, 1, 0), ("wgrad_down", 2048, 8192, 8192, 1, 0),
    ("wgrad_head", 50304, 2048, 8192, 1, 0),
    ("dgrad_qkv", 8192, 2048, 6144, 0, 0), ("dgrad_gate_up", 8192, 2048, 16384, 0, 0),
    ("dgrad_down", 8192, 8192, 2048, 0, 0), ("dgrad_head", 8192, 2048, 50304, 0, 0),
    ("dgrad_head_v128256", 4096, 2048, 128256, 0, 0),
]


@pytest.mark.parametrize("name,m,n,k,ta,tb", FULL)
def test_full_size_sampled(name, m, n, k, ta, tb):
    print(f"gemm full {name} {m}x{n}x{k}", flush=True)
    a, b = operands(m, n, k, ta, tb, 0)
    c = gpu_gemm(a, b, ta, tb, m, n, k)
    assert np.all(np.isfinite(c))
    rng = np.random.default_rng(1)
    idx = [(int(i), int(j)) for i, j in zip(rng.integers(0, m, 48), rng.integers(0, n, 48))]
    idx += [(0, 0), (m - 1, n - 1), (m - 1, 0), (0, n - 1)]
    got = np.array([c[i, j] for i, j in idx], np.float32)
    want = np.array([oracle.rdot_bf16(a[:, i] if ta else a[i], b[j] if tb else b[:, j]) for i, j in idx], np.float32)
    assert_bits(got, want, name)


@pytest.mark.parametrize("kind", ["wide", "tiny", "ties", "cancel", "huge"])
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
@pytest.mark.parametrize("m,n,k", [(130, 260, 192), (70, 130, 167), (128, 256, 224)])
def test_adversarial_operands(kind, ta, tb, m, n, k):
    # the matrix-core chains against the oracle where rounding decides: subnormal products and partial sums
    # (flush), bf16 subnormal operands (read as zero), round-half-even ties, exact cancellation with signed
    # zeros, overflow to infinity; vector-load tiles and ragged tiles
    import adversarial as ADV
    print(f"gemm adversarial {kind} {m}x{n}x{k} ta={ta} tb={tb}", flush=True)
    a, b = ADV.gemm_operands(kind, m, n, k, seed=11)
    a_st = np.ascontiguousarray(a.T) if ta else a
    b_st = np.ascontiguousarray(b.T) if tb else b
    assert_bits(gpu_gemm(a_st, b_st, ta, tb, m, n, k), oracle.gemm(a_st, b_st, bool(ta), bool(tb)),
                f"{kind} {m}x{n}x{k}")
