"""The int8 quantised linear on the GPU against the oracle: LSQ step re-pin (bit-exact fp32), quantiser
(byte-exact), exact int8 GEMM (bit-exact int32) and its dequantisation (bit-exact fp32), at small
shapes with ragged tiles and at the 1B decoder's shapes on sampled rows."""
import numpy as np
import pytest
import torch

import adversarial as ADV
import oracle
import paper_2609_17380_amd.canon as C
import paper_2609_17380_amd.inputs as I
from gpu_util import DEV, assert_bits, dev_bf16, dev_f32, host_f32

pytestmark = pytest.mark.gpu
RNG = np.random.default_rng(8)


def dev_i8(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int8)).to(DEV)


@pytest.mark.parametrize("rows,cols", [(5, 2048), (130, 97), (3, 1), (64, 8192), (2, 32768), (7, 1000), (9, 36)])
def test_quant_scales(rows, cols):
    print(f"quant_scales {rows}x{cols}", flush=True)
    w = I.normal_bf16((rows, cols), 0, I.TENSOR_IDS["gemm_b"], std=0.02)
    w[0, : min(cols, 7)] = np.array([0x0001, 0x8003, 0x7F7F, 0xFF7F, 0x0000, 0x8000, 0x3F80], np.uint16)[: min(cols, 7)]
    want = oracle.quant_scales(w)
    got = torch.empty(rows, dtype=torch.float32, device=DEV)
    C.quant_scales(rows, cols, dev_bf16(w), got)
    torch.cuda.synchronize()
    assert_bits(host_f32(got), want, "scale")


def special_values(shape):
    x = (RNG.standard_normal(shape) * 3).astype(np.float32)
    flat = x.reshape(-1)
    sp = np.array([0.5, 1.5, -2.5, 127.5, -128.5, 1e30, -1e30, np.inf, -np.inf, np.nan, -0.0, 1e-40],
                  np.float32)
    flat[: sp.size] = sp
    return x


@pytest.mark.parametrize("per_row", [True, False])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cols", [301, 304])  # 304: whole 16-byte vectors per row (the vector kernels)
def test_quantize(per_row, dtype, cols):
    rows = 37
    x = special_values((rows, cols))
    s = (np.abs(RNG.standard_normal(rows)) * 0.1 + 0.01).astype(np.float32)
    s[1], s[2], s[3], s[4] = 0.0, -1.0, np.nan, 1e-40  # steps that quantise to 0
    if not per_row:
        s = s[:1]
    if dtype == "bf16":
        xh = (x.view(np.uint32) >> 16).astype(np.uint16)
        want, xd = oracle.quantize(xh, s, per_row), dev_bf16(xh)
    else:
        want, xd = oracle.quantize(x, s, per_row), dev_f32(x)
    q = torch.empty((rows, cols), dtype=torch.int8, device=DEV)
    C.quantize(rows, cols, xd, dev_f32(s), per_row, q)
    torch.cuda.synchronize()
    got = q.cpu().numpy()
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]


def gemm_case(m, n, k, a_off=0, seed=0, extreme=False):
    rng = np.random.default_rng(seed)
    if extreme:
        a = np.full((m, k), -128, np.int8)
        b = np.full((n, k), -128, np.int8)
        b[1::2] = 127
    else:
        a = rng.integers(-128, 128, (m, k)).astype(np.int8)
        b = rng.integers(-128, 128, (n, k)).astype(np.int8)
    sa = np.float32(0.0173)
    sb = (np.abs(rng.standard_normal(n)) * 0.01).astype(np.float32)
    acc_o, y_o = oracle.gemm_i8(a, b, sa, sb)
    ad = torch.empty(m * k + a_off, dtype=torch.int8, device=DEV)
    ad[a_off:] = dev_i8(a).reshape(-1)
    acc = torch.full((m, n), -1, dtype=torch.int32, device=DEV)
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
    C.gemm_i8(m, n, k, ad[a_off:], k, dev_i8(b), k, acc=acc, y=y, sa=dev_f32(np.array([sa])), sb=dev_f32(sb))
    torch.cuda.synchronize()
    assert np.array_equal(acc.cpu().numpy(), acc_o)
    assert_bits(host_f32(y), y_o, "y")


@pytest.mark.parametrize("m,n,k", [(130, 260, 192), (128, 128, 64), (1, 1, 1), (200, 3, 1000), (64, 300, 48),
                                   (129, 129, 4096), (7, 5, 0),
                                   # whole 256 x 256 tiles (64-byte stages loaded three ahead): 1 .. 5 stages
                                   # (the pipeline's start and end cases), many stages
                                   (256, 256, 64), (256, 256, 128), (512, 768, 192), (256, 512, 256),
                                   (512, 256, 320), (768, 512, 2048)])
def test_gemm_i8(m, n, k):
    print(f"gemm_i8 {m}x{n}x{k}", flush=True)
    gemm_case(m, n, k)


@pytest.mark.parametrize("outputs", ["y", "acc"])
def test_gemm_i8_whole_tiles_one_output(outputs):
    """The whole-tile kernel with only the dequantised output (as the quantised linear asks) or only the
    int32 accumulators; the other buffer stays untouched."""
    m, n, k = 512, 512, 320
    rng = np.random.default_rng(11)
    a = rng.integers(-128, 128, (m, k)).astype(np.int8)
    b = rng.integers(-128, 128, (n, k)).astype(np.int8)
    sa = np.float32(0.021)
    sb = (np.abs(rng.standard_normal(n)) * 0.01).astype(np.float32)
    acc_o, y_o = oracle.gemm_i8(a, b, sa, sb)
    acc = torch.full((m, n), -1, dtype=torch.int32, device=DEV)
    y = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
    if outputs == "y":
        C.gemm_i8(m, n, k, dev_i8(a), k, dev_i8(b), k, y=y, sa=dev_f32(np.array([sa])), sb=dev_f32(sb))
    else:
        C.gemm_i8(m, n, k, dev_i8(a), k, dev_i8(b), k, acc=acc)
    torch.cuda.synchronize()
    if outputs == "y":
        assert_bits(host_f32(y), y_o, "y")
        assert np.all(acc.cpu().numpy() == -1)
    else:
        assert np.array_equal(acc.cpu().numpy(), acc_o)
        assert np.all(np.isnan(host_f32(y)))


def test_gemm_i8_misaligned_and_extreme():
    gemm_case(70, 90, 160, a_off=3)           # operand off 16-byte alignment: byte loads
    gemm_case(64, 64, 65536, extreme=True)    # |acc| up to 2^30
    gemm_case(256, 256, 65536, extreme=True)  # the same through the whole-tile kernel


def test_quantised_linear_1b_shapes_sampled():
    # the gate/up projection of the 1B decoder over one microbatch: scales of the weights, quantised weights
    # and activations, int8 GEMM and dequantisation; sampled activation rows through the oracle
    T, K, N = 8192, 2048, 16384
    w = I.normal_bf16((N, K), 0, I.TENSOR_IDS["gemm_b"], std=0.02)
    x = I.normal_f32((T, K), 0, I.TENSOR_IDS["gemm_a"])
    sx = np.array([0.0625], np.float32)  # per-tensor activation step
    wd, xd, sxd = dev_bf16(w), dev_f32(x), dev_f32(sx)
    sw = torch.empty(N, dtype=torch.float32, device=DEV)
    C.quant_scales(N, K, wd, sw)
    qw = torch.empty((N, K), dtype=torch.int8, device=DEV)
    qx = torch.empty((T, K), dtype=torch.int8, device=DEV)
    C.quantize(N, K, wd, sw, True, qw)
    C.quantize(T, K, xd, sxd, False, qx)
    y = torch.empty((T, N), dtype=torch.float32, device=DEV)
    C.gemm_i8(T, N, K, qx, K, qw, K, y=y, sa=sxd, sb=sw)
    torch.cuda.synchronize()
    sw_o = oracle.quant_scales(w)
    assert_bits(host_f32(sw), sw_o, "weight steps")
    qw_o = oracle.quantize(w, sw_o, True)
    assert np.array_equal(qw.cpu().numpy(), qw_o)
    rows = np.concatenate([np.arange(0, 64), RNG.choice(T, 64, replace=False)])
    qx_o = oracle.quantize(x[rows], sx, False)
    assert np.array_equal(qx.cpu().numpy()[rows], qx_o)
    _, y_o = oracle.gemm_i8(qx_o, qw_o, sx[0], sw_o)
    assert_bits(host_f32(y)[rows], y_o, "y rows")


@pytest.mark.parametrize("m,n,k", [(8000, 8100, 320), (4352, 16200, 96)])
def test_gemm_i8_large_ragged_tiles_sampled(m, n, k):
    """Products large enough for the 256 x 256 tiles, with ragged last tile rows, columns and stages: the
    int32 accumulators and the dequantised outputs of sampled rows (the first and last tile rows among them)
    against the oracle."""
    print(f"gemm_i8 {m}x{n}x{k}", flush=True)
    rng = np.random.default_rng(m + n + k)
    a = rng.integers(-128, 128, (m, k)).astype(np.int8)
    b = rng.integers(-128, 128, (n, k)).astype(np.int8)
    sa = np.array([0.013], np.float32)
    sb = (np.abs(rng.standard_normal(n)) * 0.01 + 1e-3).astype(np.float32)
    acc = torch.empty((m, n), dtype=torch.int32, device=DEV)
    y = torch.empty((m, n), dtype=torch.float32, device=DEV)
    C.gemm_i8(m, n, k, torch.from_numpy(a).to(DEV), k, torch.from_numpy(b).to(DEV), k, acc=acc, y=y,
              sa=dev_f32(sa), sb=dev_f32(sb))
    torch.cuda.synchronize()
    rows = np.concatenate([np.arange(0, 8), np.arange(m - 8, m), rng.choice(m, 48, replace=False)])
    acc_o, y_o = oracle.gemm_i8(a[rows], b, sa[0], sb)
    assert np.array_equal(acc.cpu().numpy()[rows], acc_o)
    assert_bits(host_f32(y)[rows], y_o, "y rows")


def qlinear_bwd_case(T, N, K, seed, want_dx=True, want_dw=True, outlier=True):
    rng = np.random.default_rng(seed)
    dy = (rng.standard_normal((T, N)) * 1e-3).astype(np.float32)
    if outlier:
        dy[1, 3] = 0.08
    dy[0, :4] = np.array([1e-40, -0.0, 0.0, 3e-39], np.float32)  # subnormal and signed-zero inputs
    qx = rng.integers(-128, 128, (T, K)).astype(np.int8)
    qw = rng.integers(-128, 128, (N, K)).astype(np.int8)
    sx = np.array([0.021], np.float32)
    sw = (np.abs(rng.standard_normal(N)) * 0.001 + 1e-4).astype(np.float32)
    dx_o, dw_o = oracle.qlinear_bwd(dy, qx, sx[0], qw, sw, want_dx=want_dx, want_dw=want_dw)
    ws = torch.empty(C.qlinear_bwd_workspace_bytes(T, N, K), dtype=torch.uint8, device=DEV)
    dx = torch.full((T, K), float("nan"), device=DEV) if want_dx else None
    dw = torch.full((N, K), float("nan"), device=DEV) if want_dw else None
    C.qlinear_bwd(T, N, K, dev_f32(dy), dev_i8(qx), dev_f32(sx), dev_i8(qw), dev_f32(sw), dx, dw, ws)
    torch.cuda.synchronize()
    if want_dx:
        assert_bits(host_f32(dx), dx_o, "dx")
    if want_dw:
        assert_bits(host_f32(dw), dw_o, "dw")


@pytest.mark.parametrize("T,N,K", [(256, 256, 64), (512, 768, 72), (256, 512, 1), (768, 256, 130)])
def test_qlinear_bwd(T, N, K):
    print(f"qlinear_bwd {T}x{N}x{K}", flush=True)
    qlinear_bwd_case(T, N, K, seed=T + N + K)


def test_qlinear_bwd_one_output_and_mid_size():
    qlinear_bwd_case(256, 96, 40, seed=1, want_dx=False)   # dW only: N need not be a multiple of 256
    qlinear_bwd_case(80, 512, 40, seed=2, want_dw=False)   # dx only: T need not be a multiple of 256
    qlinear_bwd_case(2048, 2048, 512, seed=3)              # several tiles per operand, full rotation blocks


def test_qlinear_bwd_many_blocks():
    """T N = 2^25 rotation blocks' worth of the upstream gradient: the contiguous-direction rotation runs more
    than one grid-stride round per wavefront, the strided-direction one 4096 tiles."""
    print("qlinear_bwd 4096x8192x256", flush=True)
    qlinear_bwd_case(4096, 8192, 256, seed=4)


@pytest.mark.parametrize("s", [0.1, 0.0173, 1.0 / 3.0, 3e-38, 2.0 ** 126, 2.0 ** 127, 1e38, 7.0])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_quantize_per_tensor_near_every_boundary(s, dtype):
    """One step for the whole tensor takes the reciprocal path: values at, just inside and just outside every
    half-integer multiple of the step (and of the clamp bounds), for steps whose reciprocal is inexact, tiny,
    beyond 2^126 (no reciprocal path) or huge; the result must equal the correctly rounded quotient's."""
    s32 = np.float32(s)
    k = np.arange(-131, 132, dtype=np.float64)
    base = (k + 0.5) * np.float64(s32)
    vals = []
    for b in base:
        f = np.float32(b)
        u = int(np.array([f], np.float32).view(np.uint32)[0])
        for du in (-2, -1, 0, 1, 2):
            vals.append(np.array([u + du], np.uint32).view(np.float32)[0] if f != 0 else np.float32(0))
    vals += [np.float32(v) for v in (np.inf, -np.inf, np.nan, 0.0, -0.0, 1e-40, 3e38, -3e38)]
    x = np.array(vals, np.float32)
    x = np.concatenate([x, RNG.standard_normal(4096).astype(np.float32) * np.float32(50 * s32 if s < 1e37 else 1)])
    n = (x.size // 4) * 4
    x = x[:n].reshape(4, -1)
    rows, cols = x.shape
    if dtype == "bf16":
        xh = (x.view(np.uint32) >> 16).astype(np.uint16)
        want, xd = oracle.quantize(xh, np.array([s32]), False), dev_bf16(xh)
    else:
        want, xd = oracle.quantize(x, np.array([s32]), False), dev_f32(x)
    q = torch.empty((rows, cols), dtype=torch.int8, device=DEV)
    C.quantize(rows, cols, xd, dev_f32(np.array([s32])), False, q)
    torch.cuda.synchronize()
    got = q.cpu().numpy()
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]
