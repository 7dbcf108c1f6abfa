"""Seeded synthetic inputs (Philox4x32-10 counter-based stream).

This module is the only code shared by the CPU oracle and the GPU path: it
produces input buffers and holds none of the method's arithmetic.  A value is a
pure function of (seed, tensor id, element index), so any slice of a tensor can
be regenerated independently (the paper's counter-based generator rule).

The tensor-id table used by the synthetic workloads lives in ``TENSOR_IDS``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "philox_inputs.c")
_LIB = os.path.join(_HERE, "libcanon_inputs.so")
_lib = None

# Tensor ids: the Philox key's second word.  Per-layer tensors add 16 * layer.
TENSOR_IDS = {
    "gemm_a": 1, "gemm_b": 2,
    "x_in": 3, "dy_in": 4,
    "logits": 5, "targets": 6, "scores": 7,
    "grads": 8,            # + rank index
    "adam_p": 40, "adam_g": 41,
    "windows": 50,
    "embed": 100, "head": 101, "final_norm": 102, "embed_norm": 103,
    "attn_norm": 200, "w_qkv": 201, "w_o": 202, "ffn_norm": 203, "w_gate_up": 204, "w_down": 205,
}
LAYER_STRIDE = 16


def build() -> str:
    """Compile the generator with gcc (OpenMP across elements)."""
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-o", _LIB, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            raise RuntimeError(f"{_LIB} is not built; run __graft_entry__.build() first")
        lib = ctypes.CDLL(_LIB)
        u64, u32, i64, dbl, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
        lib.canon_in_normal_f32.argtypes = [u64, u32, u64, i64, dbl, dbl, vp]
        lib.canon_in_normal_bf16.argtypes = [u64, u32, u64, i64, dbl, dbl, vp]
        lib.canon_in_uniform_int.argtypes = [u64, u32, u64, i64, u32, vp]
        lib.canon_in_philox4x32_10.argtypes = [vp, vp, vp]
        for f in (lib.canon_in_normal_f32, lib.canon_in_normal_bf16, lib.canon_in_uniform_int,
                  lib.canon_in_philox4x32_10):
            f.restype = None
        _lib = lib
    return _lib


def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    out = np.zeros(4, dtype=np.uint32)
    _load().canon_in_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def _ptr(arr) -> int:
    if isinstance(arr, np.ndarray):
        assert arr.flags.c_contiguous
        return arr.ctypes.data
    return int(arr.data_ptr())  # a contiguous host torch tensor


def normal_f32(shape, seed: int, tid: int, std: float = 1.0, mean: float = 0.0, start: int = 0, out=None):
    n = int(np.prod(shape))
    if out is None:
        out = np.empty(shape, dtype=np.float32)
    _load().canon_in_normal_f32(seed, tid, start, n, mean, std, _ptr(out))
    return out


def normal_bf16(shape, seed: int, tid: int, std: float = 1.0, mean: float = 0.0, start: int = 0, out=None):
    """bf16 values as raw uint16 bit patterns."""
    n = int(np.prod(shape))
    if out is None:
        out = np.empty(shape, dtype=np.uint16)
    _load().canon_in_normal_bf16(seed, tid, start, n, mean, std, _ptr(out))
    return out


def uniform_int(shape, seed: int, tid: int, bound: int, start: int = 0, out=None):
    n = int(np.prod(shape))
    if out is None:
        out = np.empty(shape, dtype=np.int32)
    _load().canon_in_uniform_int(seed, tid, start, n, bound, _ptr(out))
    return out


def bf16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (no arithmetic: a 16-bit shift)."""
    return (u16.astype(np.uint32) << 16).view(np.float32)


def rope_tables(seq: int, head_dim: int, theta: float = 500000.0):
    """cos/sin tables [seq, head_dim/2] in fp32: angle(s, i) = s * theta^(-2i/head_dim), evaluated in
    double and rounded once (the paper lists RoPE tables among the reproducible operators; here they are an
    input shared by both sides)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / head_dim)
    ang = np.arange(seq, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


ADAMW_FIELDS = ("lr", "beta1", "one_minus_beta1", "beta2", "one_minus_beta2", "inv_bc1", "inv_bc2", "eps",
                "decay_factor")


def adamw_constants(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, wd=0.1, t=1):
    """AdamW constants evaluated in double and rounded once to fp32, in ``ADAMW_FIELDS`` order."""
    vals = (lr, beta1, 1.0 - beta1, beta2, 1.0 - beta2, 1.0 / (1.0 - beta1 ** t), 1.0 / (1.0 - beta2 ** t), eps,
            1.0 - lr * wd)
    return tuple(float(np.float32(v)) for v in vals)


# Initial activation steps of the int8 projections: 2 E|x| / sqrt(127) for unit-RMS normalised inputs
# (E|x| = sqrt(2/pi)) and for the smaller attention and SwiGLU outputs (E|x| about 0.3).
ACT_STEPS = {"sx_qkv": 0.1416, "sx_o": 0.0532, "sx_gate_up": 0.1416, "sx_down": 0.0532}


def model_param_shapes(n_layers, d_model, d_ffn, vocab, kv_dim=None, embed_norm=False, int8_linear=False):
    """Parameter tensors in the declared order, with (name, shape, init, weight-decay flag); init is the
    normal's std, None for a norm gain (1.0), or ("step", value) for an activation step.
    kv_dim: width of the key (and of the value) projection, n_kv_heads * head_dim (default d_model);
    embed_norm: a gain tensor after the embedding; int8_linear: four activation steps per layer after
    w_down (sx_qkv, sx_o, sx_gate_up, sx_down)."""
    kv = d_model if kv_dim is None else kv_dim
    out = [("embed", (vocab, d_model), 0.02, 0)]
    if embed_norm:
        out.append(("embed_norm", (d_model,), None, 0))
    for l in range(n_layers):
        out += [(f"l{l}.attn_norm", (d_model,), None, 0), (f"l{l}.w_qkv", (d_model + 2 * kv, d_model), 0.02, 1),
                (f"l{l}.w_o", (d_model, d_model), 0.02, 1), (f"l{l}.ffn_norm", (d_model,), None, 0),
                (f"l{l}.w_gate_up", (2 * d_ffn, d_model), 0.02, 1), (f"l{l}.w_down", (d_model, d_ffn), 0.02, 1)]
        if int8_linear:
            out += [(f"l{l}.{k}", (1,), ("step", v), 0) for k, v in ACT_STEPS.items()]
    out += [("final_norm", (d_model,), None, 0), ("head", (vocab, d_model), 0.02, 1)]
    return out


def bf16_pattern(value: float) -> int:
    """bf16 bit pattern of a float (round to nearest even)."""
    u = int(np.array([value], np.float32).view(np.uint32)[0])
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) & 0xFFFF


def model_params(n_layers, d_model, d_ffn, vocab, seed=0, std=0.02, out=None, kv_dim=None, embed_norm=False,
                 int8_linear=False):
    """bf16 parameters: N(0, std) for matrices, 1.0 for norm gains, the ACT_STEPS values for activation
    steps.  ``out`` may hold preallocated uint16 buffers (e.g. pinned host tensors) to fill instead of new
    numpy arrays."""
    res = []
    base = {"embed": TENSOR_IDS["embed"], "head": TENSOR_IDS["head"], "final_norm": TENSOR_IDS["final_norm"],
            "embed_norm": TENSOR_IDS["embed_norm"]}
    for idx, (name, shape, s, _) in enumerate(model_param_shapes(n_layers, d_model, d_ffn, vocab, kv_dim,
                                                                 embed_norm, int8_linear)):
        buf = None if out is None else out[idx]
        if isinstance(s, tuple):
            pat = bf16_pattern(s[1])
            arr = np.full(shape, pat, dtype=np.uint16) if buf is None else buf
            if buf is not None:
                np.asarray(arr).fill(pat) if isinstance(arr, np.ndarray) else arr.fill_(pat)
        elif s is None:
            arr = np.full(shape, 0x3F80, dtype=np.uint16) if buf is None else buf
            if buf is not None:
                np.asarray(arr).fill(0x3F80) if isinstance(arr, np.ndarray) else arr.fill_(0x3F80)
        else:
            if name in base:
                tid = base[name]
            else:
                layer, kind = name.split(".")
                tid = TENSOR_IDS[kind] + LAYER_STRIDE * (int(layer[1:]) + 1)
            arr = normal_bf16(shape, seed, tid, std=std if std is not None else s, out=buf)
        res.append(arr)
    return res
