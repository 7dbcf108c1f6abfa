"""CPU oracle of the canonical-order training step (CANON-v1).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(the GPU library and its binding) never imports it, and it never imports the
product path; the only shared code is the seeded input generator.

Thin ctypes binding over ``liboracle.so`` (plain C, ``canon_ref.c``).  Arrays
are numpy; bf16 tensors are uint16 bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "canon_ref.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

CFLAGS = ["-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-march=x86-64-v3",
          "-std=c11", "-D_GNU_SOURCE"]


def build() -> str:
    tmp = _LIB + ".tmp"
    subprocess.run(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
    os.replace(tmp, _LIB)  # a process that has the old library loaded keeps its copy
    return _LIB


class ModelCfg(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("seq", ctypes.c_int32), ("micro_seqs", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("n_kv_heads", ctypes.c_int32), ("qk_norm", ctypes.c_int32), ("embed_norm", ctypes.c_int32),
                ("swa_window", ctypes.c_int32), ("swa_full_every", ctypes.c_int32), ("z_loss", ctypes.c_float),
                ("pv_int8", ctypes.c_int32), ("dq_fixed_bits", ctypes.c_int32), ("int8_linear", ctypes.c_int32)]


class Plan(ctypes.Structure):
    _fields_ = [("accum", ctypes.c_int32), ("dp_shard", ctypes.c_int32), ("dp_replicate", ctypes.c_int32)]


class AdamWConsts(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("lr", "beta1", "one_minus_beta1", "beta2", "one_minus_beta2",
                                              "inv_bc1", "inv_bc2", "eps", "decay_factor")]


class ClipCfg(ctypes.Structure):
    """R15 clip settings: clip threshold, spike threshold, updates skipped per spike (0: no spike rule)."""
    _fields_ = [("max_norm", ctypes.c_float), ("spike_norm", ctypes.c_float), ("skip_steps", ctypes.c_int32)]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            raise RuntimeError(f"{_LIB} is not built; run __graft_entry__.build() first")
        lib = ctypes.CDLL(_LIB)
        f, i32, i64, vp = ctypes.c_float, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        sig = {
            "cref_add": (f, [f, f]), "cref_sub": (f, [f, f]), "cref_mul": (f, [f, f]),
            "cref_fma": (f, [f, f, f]), "cref_div": (f, [f, f]), "cref_sqrt": (f, [f]),
            "cref_exp": (f, [f]), "cref_log": (f, [f]), "cref_sigmoid": (f, [f]), "cref_silu": (f, [f]),
            "cref_bf16": (ctypes.c_uint16, [f]),
            "cref_prim": (ctypes.c_int, [i32, i64, vp, vp, vp, vp]),
            "cref_rsum": (f, [vp, i64, i64, i32]),
            "cref_rdot_bf16": (f, [vp, i64, vp, i64, i64, i32]),
            "cref_rdot_f32": (f, [vp, i64, vp, i64, i64, i32]),
            "cref_treefold": (ctypes.c_int, [vp, i64, i64, vp, vp]),
            "cref_gemm": (ctypes.c_int, [i32, i32, i64, i64, i64, vp, i64, vp, i64, vp, i64]),
            "cref_rownorm_fwd": (ctypes.c_int, [i64, i64, vp, vp, f, vp, vp]),
            "cref_rownorm_bwd": (ctypes.c_int, [i64, i64, vp, vp, vp, vp, vp, vp]),
            "cref_softmax_causal": (ctypes.c_int, [i64, i64, vp, f, vp]),
            "cref_softmax_window": (ctypes.c_int, [i64, i64, vp, f, i64, vp]),
            "cref_xent": (ctypes.c_int, [i64, i64, vp, vp, f, vp, vp, vp]),
            "cref_xent_z": (ctypes.c_int, [i64, i64, vp, vp, f, f, vp, vp, vp]),
            "cref_rownorm_fwd_f32": (ctypes.c_int, [i64, i64, vp, vp, f, vp, vp]),
            "cref_grad_accum": (ctypes.c_int, [vp, i64, vp, vp]),
            "cref_adamw": (ctypes.c_int, [i64, vp, vp, vp, vp, vp, vp, vp]),
            "cref_block_fwd_bwd": (ctypes.c_int, [vp, i32, vp, vp, vp, vp, vp, vp, vp, vp]),
            "cref_step": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
            "cref_global_norm": (f, [i64, vp, vp]),
            "cref_clip_decide": (ctypes.c_int, [f, vp, vp, vp, vp]),
            "cref_clip_apply": (ctypes.c_int, [i64, vp, vp, f]),
            "cref_quant_scales": (ctypes.c_int, [i64, i64, vp, vp]),
            "cref_quantize": (ctypes.c_int, [i64, i64, i32, vp, vp, i32, vp]),
            "cref_gemm_i8": (ctypes.c_int, [i64, i64, i64, vp, i64, vp, i64, vp, vp, i64, f, vp]),
            "cref_fwht256": (ctypes.c_int, [i64, vp]),
            "cref_qlinear_bwd": (ctypes.c_int, [i64, i64, i64, vp, vp, f, vp, vp, vp, vp]),
            "cref_attn_pv_i8": (ctypes.c_int, [i64, i64, vp, vp, vp]),
            "cref_attn_dq_fixed": (ctypes.c_int, [i64, i64, i64, i32, vp, vp, vp]),
            "cref_fx_product": (ctypes.c_uint64, [ctypes.c_uint16, ctypes.c_uint16, i32]),
            "cref_fx_to_f32": (f, [ctypes.c_uint64, i32]),
            "cref_lsq_step_grad": (f, [i64, i64, vp, f, vp]),
            "cref_embed_bwd": (ctypes.c_int, [i64, i64, i64, vp, vp, vp]),
            "cref_inv_sqrt_int": (f, [i64]),
            "cref_swiglu": (ctypes.c_int, [i64, vp, vp, vp, vp, vp, vp]),
            "cref_num_threads": (ctypes.c_int, []),
            "cref_set_threads": (None, [ctypes.c_int]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype, fn.argtypes = res, args
        _lib = lib
    return _lib


def lib():
    return _load()


def _p(a: np.ndarray) -> int:
    assert a.flags.c_contiguous, "oracle arrays must be C-contiguous"
    return a.ctypes.data


def _ptr_array(arrs):
    return (ctypes.c_void_p * len(arrs))(*[_p(a) for a in arrs])


def _check(rc):
    if rc != 0:
        raise ValueError(f"oracle call failed with status {rc}")


PRIM_OPS = {"add": 0, "sub": 1, "mul": 2, "fma": 3, "div": 4, "sqrt": 5, "exp": 6, "log": 7, "sigmoid": 8,
            "silu": 9, "bf16": 10}


def prim(op: str, a, b=None, c=None) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = np.ascontiguousarray(a if b is None else b, dtype=np.float32)
    c = np.ascontiguousarray(a if c is None else c, dtype=np.float32)
    out = np.empty_like(a)
    _check(_load().cref_prim(PRIM_OPS[op], a.size, _p(a), _p(b), _p(c), _p(out)))
    return out


def rsum(t, chunk: int = 32) -> np.float32:
    t = np.ascontiguousarray(t, dtype=np.float32)
    return np.float32(_load().cref_rsum(_p(t), t.size, 1, chunk))


def rdot_bf16(a, b, chunk: int = 32) -> np.float32:
    a = np.ascontiguousarray(a, dtype=np.uint16)
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return np.float32(_load().cref_rdot_bf16(_p(a), 1, _p(b), 1, a.size, chunk))


def rdot_f32(a, b, chunk: int = 32) -> np.float32:
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = np.ascontiguousarray(b, dtype=np.float32)
    return np.float32(_load().cref_rdot_f32(_p(a), 1, _p(b), 1, a.size, chunk))


def treefold(parts: np.ndarray):
    parts = np.ascontiguousarray(parts, dtype=np.float32)
    nparts = parts.shape[0]
    length = int(np.prod(parts.shape[1:])) if parts.ndim > 1 else 1
    out = np.empty(parts.shape[1:] if parts.ndim > 1 else (1,), dtype=np.float32)
    deepest = ctypes.c_int32(0)
    _check(_load().cref_treefold(_p(parts), nparts, length, _p(out), ctypes.addressof(deepest)))
    return out, deepest.value


def gemm(a: np.ndarray, b: np.ndarray, trans_a: bool = False, trans_b: bool = False) -> np.ndarray:
    """C = op(A) op(B); a, b uint16 bf16 bit patterns stored row-major; returns fp32 [m, n]."""
    a = np.ascontiguousarray(a, dtype=np.uint16)
    b = np.ascontiguousarray(b, dtype=np.uint16)
    m, k = (a.shape[1], a.shape[0]) if trans_a else a.shape
    kb, n = (b.shape[1], b.shape[0]) if trans_b else b.shape
    assert k == kb
    c = np.empty((m, n), dtype=np.float32)
    _check(_load().cref_gemm(int(trans_a), int(trans_b), m, n, k, _p(a), a.shape[1], _p(b), b.shape[1], _p(c), n))
    return c


def rownorm_fwd(x: np.ndarray, gain: np.ndarray, eps: float):
    x = np.ascontiguousarray(x, dtype=np.float32)
    gain = np.ascontiguousarray(gain, dtype=np.uint16)
    rows, cols = x.shape
    y = np.empty((rows, cols), dtype=np.uint16)
    rstd = np.empty(rows, dtype=np.float32)
    _check(_load().cref_rownorm_fwd(rows, cols, _p(x), _p(gain), eps, _p(y), _p(rstd)))
    return y, rstd


def rownorm_fwd_f32(x: np.ndarray, gain: np.ndarray, eps: float):
    """R3 forward with an fp32 output (the embedding norm of R16)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    gain = np.ascontiguousarray(gain, dtype=np.uint16)
    rows, cols = x.shape
    y = np.empty((rows, cols), dtype=np.float32)
    rstd = np.empty(rows, dtype=np.float32)
    _check(_load().cref_rownorm_fwd_f32(rows, cols, _p(x), _p(gain), eps, _p(y), _p(rstd)))
    return y, rstd


def rownorm_bwd(x, gain, rstd, dy):
    x = np.ascontiguousarray(x, dtype=np.float32)
    gain = np.ascontiguousarray(gain, dtype=np.uint16)
    rstd = np.ascontiguousarray(rstd, dtype=np.float32)
    dy = np.ascontiguousarray(dy, dtype=np.float32)
    rows, cols = x.shape
    dx = np.empty((rows, cols), dtype=np.float32)
    dgain = np.empty(cols, dtype=np.float32)
    _check(_load().cref_rownorm_bwd(rows, cols, _p(x), _p(gain), _p(rstd), _p(dy), _p(dx), _p(dgain)))
    return dx, dgain


def softmax_causal(raw: np.ndarray, scale: float, window: int = 0) -> np.ndarray:
    """R5; with window > 0 (R16), query i sees keys i - window < j <= i."""
    raw = np.ascontiguousarray(raw, dtype=np.float32)
    batch, s, s2 = raw.shape
    assert s == s2
    p = np.empty((batch, s, s), dtype=np.uint16)
    if window:
        _check(_load().cref_softmax_window(batch, s, _p(raw), scale, window, _p(p)))
    else:
        _check(_load().cref_softmax_causal(batch, s, _p(raw), scale, _p(p)))
    return p


def xent(logits: np.ndarray, targets: np.ndarray, inv_tokens: float, want_dlogits: bool = True,
         z_loss: float = 0.0):
    """R6; with z_loss > 0, R16's z-loss in the same pass."""
    logits = np.ascontiguousarray(logits, dtype=np.uint16)
    targets = np.ascontiguousarray(targets, dtype=np.int32)
    rows, vocab = logits.shape
    dl = np.empty((rows, vocab) if want_dlogits else (1,), dtype=np.uint16)
    rl = np.empty(rows, dtype=np.float32)
    ml = ctypes.c_float(0)
    if z_loss:
        _check(_load().cref_xent_z(rows, vocab, _p(logits), _p(targets), inv_tokens, z_loss,
                                   _p(dl) if want_dlogits else None, _p(rl), ctypes.addressof(ml)))
    else:
        _check(_load().cref_xent(rows, vocab, _p(logits), _p(targets), inv_tokens,
                                 _p(dl) if want_dlogits else None, _p(rl), ctypes.addressof(ml)))
    return (dl if want_dlogits else None), rl, np.float32(ml.value)


def grad_accum(grads, accum: int, dp_shard: int, dp_replicate: int) -> np.ndarray:
    grads = [np.ascontiguousarray(g, dtype=np.float32) for g in grads]
    assert len(grads) == accum * dp_shard * dp_replicate
    n = grads[0].size
    out = np.empty(n, dtype=np.float32)
    plan = Plan(accum, dp_shard, dp_replicate)
    _check(_load().cref_grad_accum(ctypes.addressof(plan), n, _ptr_array(grads), _p(out)))
    return out.reshape(grads[0].shape)


def adamw(params, m, v, grads, decay_mask, consts: AdamWConsts):
    """Updates params (uint16), m, v (float32) in place."""
    sizes = np.array([p.size for p in params], dtype=np.int64)
    mask = np.ascontiguousarray(np.asarray(decay_mask, dtype=np.uint8))
    _check(_load().cref_adamw(len(params), _p(sizes), _ptr_array(params), _ptr_array(m), _ptr_array(v),
                              _ptr_array(grads), _p(mask), ctypes.addressof(consts)))


def block_fwd_bwd(cfg: ModelCfg, batch: int, x, dy, w, rope_cos, rope_sin):
    x = np.ascontiguousarray(x, dtype=np.float32)
    dy = np.ascontiguousarray(dy, dtype=np.float32)
    w = [np.ascontiguousarray(t, dtype=np.uint16) for t in w]
    y = np.empty_like(x)
    dx = np.empty_like(x)
    dw = [np.empty(t.shape, dtype=np.float32) for t in w]
    _check(_load().cref_block_fwd_bwd(ctypes.addressof(cfg), batch, _p(x), _p(dy), _ptr_array(w),
                                      _p(np.ascontiguousarray(rope_cos, dtype=np.float32)),
                                      _p(np.ascontiguousarray(rope_sin, dtype=np.float32)),
                                      _p(y), _p(dx), _ptr_array(dw)))
    return y, dx, dw


def step(cfg: ModelCfg, plan: Plan, params, m, v, windows, rope_cos, rope_sin, consts: AdamWConsts,
         want_grads: bool = False, clip: ClipCfg | None = None, skip_state: int = 0):
    """Runs one step; updates params, m, v in place; returns (loss, grads or None).

    With ``clip`` (R15) it returns (loss, grads, info) where info holds the pre-clip ``norm``, the spike
    counter ``skip_state`` after the step and ``skipped``."""
    loss = ctypes.c_float(0)
    norm = ctypes.c_float(0)
    state = ctypes.c_int32(skip_state)
    skipped = ctypes.c_int32(0)
    grads = [np.empty(p.shape, dtype=np.float32) for p in params] if want_grads else None
    windows = np.ascontiguousarray(windows, dtype=np.int32)
    _check(_load().cref_step(ctypes.addressof(cfg), ctypes.addressof(plan), _ptr_array(params), _ptr_array(m),
                             _ptr_array(v), _p(windows), _p(np.ascontiguousarray(rope_cos, dtype=np.float32)),
                             _p(np.ascontiguousarray(rope_sin, dtype=np.float32)), ctypes.addressof(consts),
                             ctypes.addressof(clip) if clip is not None else None,
                             ctypes.addressof(loss), _ptr_array(grads) if grads is not None else None,
                             ctypes.addressof(norm), ctypes.addressof(state), ctypes.addressof(skipped)))
    if clip is None:
        return np.float32(loss.value), grads
    return np.float32(loss.value), grads, {"norm": np.float32(norm.value), "skip_state": state.value,
                                           "skipped": skipped.value}


def global_norm(grads) -> np.float32:
    """R15 pre-clip global norm of a list of fp32 tensors taken end to end in list order."""
    grads = [np.ascontiguousarray(g, dtype=np.float32) for g in grads]
    sizes = np.array([g.size for g in grads], dtype=np.int64)
    return np.float32(_load().cref_global_norm(len(grads), _p(sizes), _ptr_array(grads)))


def clip_decide(norm, clip: ClipCfg, skip_state: int = 0):
    """R15 decision for one step: returns (coef, skip_state after the step, skipped)."""
    coef = ctypes.c_float(0)
    state = ctypes.c_int32(skip_state)
    skipped = ctypes.c_int32(0)
    _check(_load().cref_clip_decide(float(np.float32(norm)), ctypes.addressof(clip), ctypes.addressof(state),
                                    ctypes.addressof(coef), ctypes.addressof(skipped)))
    return np.float32(coef.value), state.value, skipped.value


def clip_apply(grads, coef) -> None:
    """R15: g <- RN(g * coef) in place (float32 arrays) when coef < 1."""
    sizes = np.array([g.size for g in grads], dtype=np.int64)
    _check(_load().cref_clip_apply(len(grads), _p(sizes), _ptr_array(grads), float(np.float32(coef))))


def quant_scales(w: np.ndarray) -> np.ndarray:
    """R13 per-row LSQ step of a bf16 [rows, cols] matrix (uint16 bit patterns)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    out = np.empty(w.shape[0], dtype=np.float32)
    _check(_load().cref_quant_scales(w.shape[0], w.shape[1], _p(w), _p(out)))
    return out


def quantize(x: np.ndarray, scale, per_row: bool) -> np.ndarray:
    """R13 quantisation of an fp32 (float32 array) or bf16 (uint16 array) [rows, cols] tensor to int8."""
    x = np.ascontiguousarray(x)
    dtype = 0 if x.dtype == np.float32 else 1
    assert x.dtype in (np.float32, np.uint16)
    s = np.ascontiguousarray(np.atleast_1d(np.asarray(scale, dtype=np.float32)))
    q = np.empty(x.shape, dtype=np.int8)
    _check(_load().cref_quantize(x.shape[0], x.shape[1], dtype, _p(x), _p(s), int(per_row), _p(q)))
    return q


def gemm_i8(a: np.ndarray, b: np.ndarray, sa: float, sb: np.ndarray):
    """R13 int8 GEMM: a [m, k], b [n, k] int8 -> (exact int32 acc [m, n], dequantised fp32 y [m, n])."""
    a = np.ascontiguousarray(a, dtype=np.int8)
    b = np.ascontiguousarray(b, dtype=np.int8)
    m, k = a.shape
    n = b.shape[0]
    sb = np.ascontiguousarray(sb, dtype=np.float32)
    acc = np.empty((m, n), dtype=np.int32)
    y = np.empty((m, n), dtype=np.float32)
    _check(_load().cref_gemm_i8(m, n, k, _p(a), k, _p(b), k, _p(acc), _p(y), n, np.float32(sa), _p(sb)))
    return acc, y


def fwht256(v: np.ndarray) -> np.ndarray:
    """R14 block Walsh-Hadamard rotation (blocks of 256 along the flattened array), returned as a copy."""
    out = np.array(v, dtype=np.float32, copy=True, order="C")
    _check(_load().cref_fwht256(out.size, _p(out)))
    return out


def qlinear_bwd(dy: np.ndarray, qx: np.ndarray, sx: float, qw: np.ndarray, sw: np.ndarray, want_dx=True,
                want_dw=True):
    """R14 int8 backward: (dx [T, K], dw [N, K]) from dy [T, N] and the forward's codes and steps."""
    dy = np.ascontiguousarray(dy, dtype=np.float32)
    qx = np.ascontiguousarray(qx, dtype=np.int8)
    qw = np.ascontiguousarray(qw, dtype=np.int8)
    sw = np.ascontiguousarray(sw, dtype=np.float32)
    T, N = dy.shape
    K = qx.shape[1]
    dx = np.empty((T, K), np.float32) if want_dx else None
    dw = np.empty((N, K), np.float32) if want_dw else None
    _check(_load().cref_qlinear_bwd(T, N, K, _p(dy), _p(qx), np.float32(sx), _p(qw), _p(sw),
                                    _p(dx) if dx is not None else None, _p(dw) if dw is not None else None))
    return dx, dw


def attn_pv_i8(P: np.ndarray, V: np.ndarray) -> np.ndarray:
    """R17 int8 P.V of one head: P bf16 [S, S] (uint16), V bf16 [S, hd] -> O fp32 [S, hd]."""
    P = np.ascontiguousarray(P, dtype=np.uint16)
    V = np.ascontiguousarray(V, dtype=np.uint16)
    S, hd = V.shape
    assert P.shape == (S, S)
    O = np.empty((S, hd), np.float32)
    _check(_load().cref_attn_pv_i8(S, hd, _p(P), _p(V), _p(O)))
    return O


def attn_dq_fixed(dS: np.ndarray, K: np.ndarray, frac_bits: int, window: int = 0) -> np.ndarray:
    """R18 fixed-point dQ of one head: dS bf16 [S, S], K bf16 [S, hd] -> dQ fp32 [S, hd] (causal, window)."""
    dS = np.ascontiguousarray(dS, dtype=np.uint16)
    K = np.ascontiguousarray(K, dtype=np.uint16)
    S, hd = K.shape
    assert dS.shape == (S, S)
    dQ = np.empty((S, hd), np.float32)
    _check(_load().cref_attn_dq_fixed(S, hd, window, frac_bits, _p(dS), _p(K), _p(dQ)))
    return dQ


def fx_product(a: int, b: int, frac_bits: int) -> int:
    """R18 fixed-point value (as an unsigned 64-bit pattern) of the product of two bf16 bit patterns."""
    return int(_load().cref_fx_product(a, b, frac_bits))


def fx_to_f32(total: int, frac_bits: int) -> np.float32:
    """R18 rounding of a wrapped 64-bit sum (unsigned pattern) times 2^-F to binary32."""
    return np.float32(_load().cref_fx_to_f32(total % (1 << 64), frac_bits))


def lsq_step_grad(x: np.ndarray, s, dx: np.ndarray) -> np.float32:
    """R19 LSQ gradient of a per-tensor step: x bf16 [T, K] (uint16), dx fp32 [T, K]."""
    x = np.ascontiguousarray(x, dtype=np.uint16)
    dx = np.ascontiguousarray(dx, dtype=np.float32)
    T, K = x.shape
    return np.float32(_load().cref_lsq_step_grad(T, K, _p(x), np.float32(s), _p(dx)))


def embed_bwd(tokens: np.ndarray, dx: np.ndarray, vocab: int) -> np.ndarray:
    """R11: dE [vocab, d] from dx [T, d] (fp32) and the int32 tokens [T] of the microbatch."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32).reshape(-1)
    dx = np.ascontiguousarray(dx, dtype=np.float32)
    T, d = dx.shape
    assert tokens.size == T
    dE = np.empty((vocab, d), dtype=np.float32)
    _check(_load().cref_embed_bwd(T, vocab, d, _p(tokens), _p(dx), _p(dE)))
    return dE


def swiglu(g: np.ndarray, u: np.ndarray, da: np.ndarray):
    """SwiGLU per element: (a, dg, du) as bf16 bit patterns (uint16) from fp32 g, u and da."""
    g = np.ascontiguousarray(g, dtype=np.float32).reshape(-1)
    u = np.ascontiguousarray(u, dtype=np.float32).reshape(-1)
    da = np.ascontiguousarray(da, dtype=np.float32).reshape(-1)
    a, dg, du = (np.empty(g.size, np.uint16) for _ in range(3))
    _check(_load().cref_swiglu(g.size, _p(g), _p(u), _p(da), _p(a), _p(dg), _p(du)))
    return a, dg, du


def inv_sqrt_int(n: int) -> np.float32:
    """RN32(1/sqrt(n)) for an integer n >= 1, as the oracle evaluates the attention and LSQ scales."""
    return np.float32(_load().cref_inv_sqrt_int(int(n)))


def set_threads(n: int) -> None:
    """Threads of the oracle's parallel loops (independent outputs only; the arithmetic is the same)."""
    _load().cref_set_threads(int(n))


def num_threads() -> int:
    return int(_load().cref_num_threads())
