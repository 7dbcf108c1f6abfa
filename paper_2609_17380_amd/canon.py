"""ctypes binding of libcanon (include/canon.h): argument marshalling only.

Every computation runs in the HIP library; this module passes device pointers, sizes and the current
HIP stream, and raises on a non-OK status.  There is no fallback: if the library is not built, loading
fails with an error.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcanon.so")

OK, EINVAL, EUNSUPPORTED, EDEVICE, EWORKSPACE = 0, -1, -2, -3, -4
FWD, BWD, FWD_F32 = 0, 1, 2
SOFTMAX_CAUSAL, XENT = 0, 1


class CanonError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {_lib().canon_status_str(status).decode()} ({status})")


class Order(ctypes.Structure):
    _fields_ = [("version", ctypes.c_int32), ("chunk", ctypes.c_int32), ("tree", ctypes.c_int32),
                ("ftz", ctypes.c_int32)]


class DPPlan(ctypes.Structure):
    _fields_ = [("accum", ctypes.c_int32), ("dp_shard", ctypes.c_int32), ("dp_replicate", ctypes.c_int32)]


PLAN_MAX_DEPTH = 31


class PlanCursor(ctypes.Structure):
    """The gradient plan's position and Algorithm 2 stack (plain data: bytes(cursor) persists it)."""
    _fields_ = [("plan", DPPlan), ("next", ctypes.c_int32), ("n", ctypes.c_int64), ("inner", ctypes.c_int32),
                ("depth", ctypes.c_int32), ("level", ctypes.c_int32 * PLAN_MAX_DEPTH),
                ("slot", ctypes.c_int32 * PLAN_MAX_DEPTH)]


class ModelCfg(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("seq", ctypes.c_int32), ("micro_seqs", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("n_kv_heads", ctypes.c_int32), ("qk_norm", ctypes.c_int32), ("embed_norm", ctypes.c_int32),
                ("swa_window", ctypes.c_int32), ("swa_full_every", ctypes.c_int32), ("z_loss", ctypes.c_float),
                ("pv_int8", ctypes.c_int32), ("dq_fixed_bits", ctypes.c_int32), ("int8_linear", ctypes.c_int32)]


class AdamWConsts(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("lr", "beta1", "one_minus_beta1", "beta2", "one_minus_beta2",
                                              "inv_bc1", "inv_bc2", "eps", "decay_factor")]


class Clip(ctypes.Structure):
    """R15 settings and device outputs (pointers are device addresses, 0 for none)."""
    _fields_ = [("max_norm", ctypes.c_float), ("spike_norm", ctypes.c_float), ("skip_steps", ctypes.c_int32),
                ("norm_out", ctypes.c_void_p), ("skip_state", ctypes.c_void_p), ("skipped_out", ctypes.c_void_p)]


def make_clip(max_norm, spike_norm, skip_steps, norm_out=None, skip_state=None, skipped_out=None) -> Clip:
    return Clip(max_norm, spike_norm, skip_steps, _ptr(norm_out), _ptr(skip_state), _ptr(skipped_out))


ORDER_V1 = Order(1, 32, 0, 1)
_L = None


def _lib():
    global _L
    if _L is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
        sigs = {
            "canon_gemm": (i32, [vp, i32, i32, i64, i64, i64, vp, i64, vp, i64, vp, i64, vp, vp]),
            "canon_gemm_strided_batched": (i32, [vp, i32, i32, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64,
                                                 i64, i64, vp]),
            "canon_rownorm": (i32, [vp, i32, i64, i64, vp, vp, f32, vp, vp, vp, vp, vp, vp]),
            "canon_softmax_xent": (i32, [vp, i32, i64, i64, vp, f32, i64, vp, f32, f32, vp, vp, vp, vp]),
            "canon_grad_accum": (i32, [vp, vp, i64, vp, vp, vp]),
            "canon_plan_state_bytes": (sz, [vp, i64]),
            "canon_plan_begin": (i32, [vp, i64, vp]),
            "canon_plan_push": (i32, [vp, vp, vp, vp, sz, vp]),
            "canon_plan_finish": (i32, [vp, vp, vp, sz, vp, vp]),
            "canon_adamw": (i32, [i64, vp, vp, vp, vp, vp, vp, vp, vp]),
            "canon_block_fwd_bwd": (i32, [vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
            "canon_block_workspace_bytes": (sz, [vp, i32]),
            "canon_step": (i32, [vp, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, sz, vp, vp, vp, vp]),
            "canon_clip_grad_norm": (i32, [vp, i64, vp, vp, vp, vp, sz, vp]),
            "canon_clip_grad_norm_workspace_bytes": (sz, [i64, vp]),
            "canon_step_workspace_bytes": (sz, [vp, vp]),
            "canon_devmath": (i32, [i32, i64, vp, vp, vp, vp, vp]),
            "canon_quant_scales": (i32, [vp, i64, i64, vp, vp, vp]),
            "canon_quantize": (i32, [i64, i64, i32, vp, vp, i32, vp, vp]),
            "canon_gemm_i8": (i32, [i64, i64, i64, vp, i64, vp, i64, vp, vp, i64, vp, vp, vp]),
            "canon_qlinear_bwd": (i32, [vp, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
            "canon_qlinear_bwd_workspace_bytes": (sz, [i64, i64, i64]),
            "canon_state_hash": (i32, [i64, vp, vp, vp, vp, sz, vp]),
            "canon_state_hash_workspace_bytes": (sz, [i64, vp]),
            "canon_attn_pv_i8": (i32, [i64, i64, i64, i64, i64, i64, vp, vp, vp, vp, vp, sz, vp]),
            "canon_attn_pv_i8_workspace_bytes": (sz, [i64, i64, i64, i64]),
            "canon_attn_dq_fixed": (i32, [i64, i64, i64, i64, i64, i64, i32, vp, vp, vp, vp]),
            "canon_lsq_step_grad": (i32, [vp, i64, i64, vp, vp, vp, vp, vp, sz, vp]),
            "canon_lsq_step_grad_workspace_bytes": (sz, [i64, i64]),
            "canon_lsq_step_grad_noalloc": (i32, [vp, i64, i64, vp, vp, vp, vp, vp]),
            "canon_embed_bwd": (i32, [vp, i64, i64, i64, vp, vp, vp, vp, sz, vp]),
            "canon_embed_bwd_workspace_bytes": (sz, [i64, i64]),
            "canon_lsq_step_grad_noalloc_max_terms": (i64, []),
            "canon_status_str": (ctypes.c_char_p, [i32]),
            "canon_version": (i32, []),
        }
        for name, (res, args) in sigs.items():
            fn = getattr(lib, name)
            fn.restype, fn.argtypes = res, args
        _L = lib
    return _L


def lib():
    return _lib()


def _check(st: int, where: str):
    if st != OK:
        raise CanonError(st, where)


def _ptr(t) -> int:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    assert t.is_cuda and t.is_contiguous(), "device tensors must be contiguous CUDA/HIP tensors"
    return t.data_ptr()


def _ptrs(ts):
    return (ctypes.c_void_p * len(ts))(*[_ptr(t) for t in ts])


def _stream(stream=None) -> int:
    if isinstance(stream, int):  # a raw hipStream_t (0: the null stream)
        return stream
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


# ---- entry points (same names as the C ABI, without the prefix) -------------------------------------

EPI_NONE, EPI_ACCUM_PLAN = 0, 1


class GemmEpilogue(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("scale", ctypes.c_float)]


def gemm(m, n, k, a, lda, b, ldb, c, ldc, trans_a=0, trans_b=0, order=ORDER_V1, stream=None, accum_scale=None):
    """C = A B, or with accum_scale the plan's accumulation C = RN(C + RN(A B * accum_scale))."""
    epi = None if accum_scale is None else ctypes.byref(GemmEpilogue(EPI_ACCUM_PLAN, accum_scale))
    _check(_lib().canon_gemm(ctypes.byref(order), int(trans_a), int(trans_b), m, n, k, _ptr(a), lda, _ptr(b), ldb,
                             _ptr(c), ldc, epi, _stream(stream)), "canon_gemm")


def gemm_strided_batched(m, n, k, a, lda, stride_a, b, ldb, stride_b, c, ldc, stride_c, batch, trans_a=0, trans_b=0,
                         order=ORDER_V1, stream=None):
    _check(_lib().canon_gemm_strided_batched(ctypes.byref(order), int(trans_a), int(trans_b), m, n, k, _ptr(a), lda,
                                             stride_a, _ptr(b), ldb, stride_b, _ptr(c), ldc, stride_c, batch,
                                             _stream(stream)), "canon_gemm_strided_batched")


def rownorm(direction, rows, cols, x, gain, eps, y=None, rstd=None, dy=None, dx=None, dgain=None, order=ORDER_V1,
            stream=None):
    _check(_lib().canon_rownorm(ctypes.byref(order), direction, rows, cols, _ptr(x), _ptr(gain), eps, _ptr(y),
                                _ptr(rstd), _ptr(dy), _ptr(dx), _ptr(dgain), _stream(stream)), "canon_rownorm")


def softmax_xent(mode, rows, cols, x, out, scale=1.0, targets=None, inv_tokens=1.0, row_loss=None, mean_loss=None,
                 order=ORDER_V1, stream=None, window=0, z_loss=0.0):
    _check(_lib().canon_softmax_xent(ctypes.byref(order), mode, rows, cols, _ptr(x), scale, window, _ptr(targets),
                                     inv_tokens, z_loss, _ptr(out), _ptr(row_loss), _ptr(mean_loss),
                                     _stream(stream)), "canon_softmax_xent")


def grad_accum(plan: DPPlan, n, grads, out, order=ORDER_V1, stream=None):
    _check(_lib().canon_grad_accum(ctypes.byref(order), ctypes.byref(plan), n, _ptrs(grads), _ptr(out),
                                   _stream(stream)), "canon_grad_accum")


def plan_state_bytes(plan: DPPlan, n: int) -> int:
    return int(_lib().canon_plan_state_bytes(ctypes.byref(plan), n))


def plan_begin(plan: DPPlan, n: int) -> PlanCursor:
    cur = PlanCursor()
    _check(_lib().canon_plan_begin(ctypes.byref(plan), n, ctypes.byref(cur)), "canon_plan_begin")
    return cur


def _state_bytes(state, state_bytes):
    if state_bytes is not None:
        return state_bytes
    return 0 if state is None or isinstance(state, int) else state.numel() * state.element_size()


def plan_push(cursor: PlanCursor, grad, state, order=ORDER_V1, stream=None, state_bytes=None):
    """Feed the next microbatch's gradient (Algorithm 1's order); updates cursor in place."""
    _check(_lib().canon_plan_push(ctypes.byref(order), ctypes.byref(cursor), _ptr(grad), _ptr(state),
                                  _state_bytes(state, state_bytes), _stream(stream)), "canon_plan_push")


def plan_finish(cursor: PlanCursor, state, out, order=ORDER_V1, stream=None, state_bytes=None):
    _check(_lib().canon_plan_finish(ctypes.byref(order), ctypes.byref(cursor), _ptr(state),
                                    _state_bytes(state, state_bytes), _ptr(out), _stream(stream)),
           "canon_plan_finish")


def adamw(params, m, v, grads, decay_mask, consts: AdamWConsts, stream=None):
    n = len(params)
    sizes = (ctypes.c_int64 * n)(*[p.numel() for p in params])
    mask = (ctypes.c_uint8 * n)(*[int(x) for x in decay_mask])
    _check(_lib().canon_adamw(n, sizes, _ptrs(params), _ptrs(m), _ptrs(v), _ptrs(grads), mask, ctypes.byref(consts),
                              _stream(stream)), "canon_adamw")


def attn_pv_i8_workspace_bytes(batch, n_kv_heads, seq, head_dim) -> int:
    return int(_lib().canon_attn_pv_i8_workspace_bytes(batch, n_kv_heads, seq, head_dim))


def attn_pv_i8(batch, n_heads, n_kv_heads, seq, head_dim, window, P, V, workspace, o_f32=None, o_bf16=None,
               stream=None):
    _check(_lib().canon_attn_pv_i8(batch, n_heads, n_kv_heads, seq, head_dim, window, _ptr(P), _ptr(V), _ptr(o_f32),
                                   _ptr(o_bf16), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                   _stream(stream)), "canon_attn_pv_i8")


def attn_dq_fixed(batch, n_heads, n_kv_heads, seq, head_dim, window, frac_bits, dS, K, dQ, stream=None):
    _check(_lib().canon_attn_dq_fixed(batch, n_heads, n_kv_heads, seq, head_dim, window, frac_bits, _ptr(dS), _ptr(K),
                                      _ptr(dQ), _stream(stream)), "canon_attn_dq_fixed")


def lsq_step_grad_workspace_bytes(T, K) -> int:
    return int(_lib().canon_lsq_step_grad_workspace_bytes(T, K))


def lsq_step_grad(T, K, x, s, dx, grad, workspace, order=ORDER_V1, stream=None):
    _check(_lib().canon_lsq_step_grad(ctypes.byref(order), T, K, _ptr(x), _ptr(s), _ptr(dx), _ptr(grad),
                                      _ptr(workspace), workspace.numel() * workspace.element_size(),
                                      _stream(stream)), "canon_lsq_step_grad")


def embed_bwd_workspace_bytes(T, d) -> int:
    return int(_lib().canon_embed_bwd_workspace_bytes(T, d))


def embed_bwd(T, V, d, tokens, dx, dE, workspace, order=ORDER_V1, stream=None):
    """R11: dE [V, d] from the int32 tokens [T] and dx [T, d] (device tensors)."""
    _check(_lib().canon_embed_bwd(ctypes.byref(order), T, V, d, _ptr(tokens), _ptr(dx), _ptr(dE), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)), "canon_embed_bwd")


def lsq_step_grad_noalloc(T, K, x, s, dx, grad, order=ORDER_V1, stream=None):
    """canon_lsq_step_grad with the block sums in the library's own device array (no workspace)."""
    _check(_lib().canon_lsq_step_grad_noalloc(ctypes.byref(order), T, K, _ptr(x), _ptr(s), _ptr(dx), _ptr(grad),
                                              _stream(stream)), "canon_lsq_step_grad_noalloc")


def lsq_step_grad_noalloc_max_terms() -> int:
    return int(_lib().canon_lsq_step_grad_noalloc_max_terms())


def block_workspace_bytes(cfg: ModelCfg, batch: int) -> int:
    return int(_lib().canon_block_workspace_bytes(ctypes.byref(cfg), batch))


def block_fwd_bwd(cfg: ModelCfg, batch, x, dy, w, rope_cos, rope_sin, y, dx, dw, workspace, order=ORDER_V1,
                  stream=None):
    _check(_lib().canon_block_fwd_bwd(ctypes.byref(order), ctypes.byref(cfg), batch, _ptr(x), _ptr(dy), _ptrs(w),
                                      _ptr(rope_cos), _ptr(rope_sin), _ptr(y), _ptr(dx), _ptrs(dw), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), _stream(stream)),
           "canon_block_fwd_bwd")


def step_workspace_bytes(cfg: ModelCfg, plan: DPPlan) -> int:
    return int(_lib().canon_step_workspace_bytes(ctypes.byref(cfg), ctypes.byref(plan)))


def step(cfg: ModelCfg, plan: DPPlan, params, m, v, windows, rope_cos, rope_sin, consts: AdamWConsts, workspace,
         loss_out, grads_out=None, step_t=1, order=ORDER_V1, stream=None, clip: Clip | None = None,
         state_digest=None):
    """state_digest: None, or a 32-byte device tensor for the per-step audit hash (H1 of the windows, the
    parameters, m and v after the step, and the reduced gradient)."""
    _check(_lib().canon_step(ctypes.byref(order), ctypes.byref(cfg), ctypes.byref(plan), _ptrs(params), _ptrs(m),
                             _ptrs(v), step_t, _ptr(windows), _ptr(rope_cos), _ptr(rope_sin), ctypes.byref(consts),
                             ctypes.byref(clip) if clip is not None else None,
                             _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(loss_out),
                             _ptrs(grads_out) if grads_out is not None else None, _ptr(state_digest),
                             _stream(stream)), "canon_step")


def _sizes(tensors):
    return (ctypes.c_int64 * len(tensors))(*[t.numel() for t in tensors])


def clip_grad_norm_workspace_bytes(grads) -> int:
    return int(_lib().canon_clip_grad_norm_workspace_bytes(len(grads), _sizes(grads)))


def clip_grad_norm(grads, clip: Clip, workspace, order=ORDER_V1, stream=None):
    """R15 norm, spike decision and in-place clip of fp32 device tensors taken end to end in list order."""
    _check(_lib().canon_clip_grad_norm(ctypes.byref(order), len(grads), _sizes(grads), _ptrs(grads),
                                       ctypes.byref(clip), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream(stream)),
           "canon_clip_grad_norm")


DEVMATH_OPS = {"add": 0, "sub": 1, "mul": 2, "fma": 3, "div": 4, "sqrt": 5, "exp": 6, "log": 7, "sigmoid": 8,
               "silu": 9, "bf16": 10}


F32, BF16 = 0, 1


def quant_scales(rows, cols, w, scale, order=ORDER_V1, stream=None):
    _check(_lib().canon_quant_scales(ctypes.byref(order), rows, cols, _ptr(w), _ptr(scale), _stream(stream)),
           "canon_quant_scales")


def quantize(rows, cols, x, scale, per_row, q, stream=None):
    dtype = F32 if x.dtype == torch.float32 else BF16
    _check(_lib().canon_quantize(rows, cols, dtype, _ptr(x), _ptr(scale), int(per_row), _ptr(q), _stream(stream)),
           "canon_quantize")


def gemm_i8(m, n, k, a, lda, b, ldb, acc=None, y=None, ldc=None, sa=None, sb=None, stream=None):
    _check(_lib().canon_gemm_i8(m, n, k, _ptr(a), lda, _ptr(b), ldb, _ptr(acc), _ptr(y), n if ldc is None else ldc,
                                _ptr(sa), _ptr(sb), _stream(stream)), "canon_gemm_i8")


def qlinear_bwd_workspace_bytes(T, N, K) -> int:
    return int(_lib().canon_qlinear_bwd_workspace_bytes(T, N, K))


def qlinear_bwd(T, N, K, dy, qx, sx, qw, sw, dx, dw, workspace, order=ORDER_V1, stream=None):
    _check(_lib().canon_qlinear_bwd(ctypes.byref(order), T, N, K, _ptr(dy), _ptr(qx), _ptr(sx), _ptr(qw), _ptr(sw),
                                    _ptr(dx), _ptr(dw), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                    _stream(stream)), "canon_qlinear_bwd")


def _nbytes(tensors):
    return (ctypes.c_int64 * len(tensors))(*[t.numel() * t.element_size() for t in tensors])


def state_hash_workspace_bytes(tensors) -> int:
    return int(_lib().canon_state_hash_workspace_bytes(len(tensors), _nbytes(tensors)))


def state_hash(tensors, digest, workspace, stream=None):
    """Canonical state hash H1 of the tensors (declared order) into digest (device uint8 [32])."""
    _check(_lib().canon_state_hash(len(tensors), _ptrs(tensors), _nbytes(tensors), _ptr(digest), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)),
           "canon_state_hash")


def devmath(op: str, n, a, b=None, c=None, out=None, stream=None):
    _check(_lib().canon_devmath(DEVMATH_OPS[op], n, _ptr(a), _ptr(b), _ptr(c), _ptr(out), _stream(stream)),
           "canon_devmath")


def version() -> int:
    return int(_lib().canon_version())
