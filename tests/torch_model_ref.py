"""Float64 autograd model of the decoder, used only to pin the oracle's block and step.

Independent of the oracle and of the GPU library: the forward pass is written
with plain PyTorch float64 ops and the backward pass comes from autograd.  The
bf16 storage points of the dataflow (every GEMM operand, and the bf16 logits)
are modelled with two autograd functions:

* ``rf``: rounds a GEMM input to bf16 in the forward pass; its gradient passes through.
* ``rb``: identity forward; rounds the gradient arriving at a GEMM output to bf16,
  since that gradient is the bf16 operand of both backward GEMMs.

Reductions run in float64, so oracle results agree only to a tolerance.
"""
import numpy as np
import torch

DT = torch.float64


class _RoundFwd(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        return x.to(torch.bfloat16).to(DT)

    @staticmethod
    def backward(ctx, g):
        return g


class _RoundBwd(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return g.to(torch.bfloat16).to(DT)


rf = _RoundFwd.apply
rb = _RoundBwd.apply


def bf16_tensor(u16: np.ndarray, requires_grad=False) -> torch.Tensor:
    f = (u16.astype(np.uint32) << 16).view(np.float32)
    return torch.tensor(f, dtype=DT, requires_grad=requires_grad)


def linear(x, w):
    """y = bf16(x) @ w^T with the gradient of y rounded to bf16 (w holds bf16 values)."""
    return rb(rf(x) @ w.T)


def rmsnorm(x, g, eps):
    return x * torch.rsqrt((x * x).mean(dim=-1, keepdim=True) + eps) * g


def rope(x, cos, sin):
    """x [..., S, hd] rotated in two halves; cos/sin [S, hd/2]."""
    h = x.shape[-1] // 2
    x1, x2 = x[..., :h], x[..., h:]
    return torch.cat([x1 * cos - x2 * sin, x2 * cos + x1 * sin], dim=-1)


def block(x, w, B, S, H, hd, F, eps, cos, sin, scale):
    """w: dict of float64 tensors attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down."""
    d = H * hd
    xn = rmsnorm(x, w["attn_norm"], eps)
    qkv = linear(xn, w["w_qkv"])                                     # [T, 3d]
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]

    def heads(t):
        return t.reshape(B, S, H, hd).permute(0, 2, 1, 3)            # [B, H, S, hd]

    qh = rf(rope(heads(q), cos, sin))
    kh = rf(rope(heads(k), cos, sin))
    vh = rf(heads(v))
    raw = rb(qh @ kh.transpose(-1, -2))                              # [B, H, S, S]
    sc = raw * scale
    mask = torch.tril(torch.ones(S, S, dtype=torch.bool))
    sc = sc.masked_fill(~mask, float("-inf"))
    p = rf(torch.softmax(sc, dim=-1))
    o = rb(p @ vh)                                                   # [B, H, S, hd]
    o = o.permute(0, 2, 1, 3).reshape(B * S, d)
    h = x + linear(o, w["w_o"])
    hn = rmsnorm(h, w["ffn_norm"], eps)
    gu = linear(hn, w["w_gate_up"])
    g, u = gu[:, :F], gu[:, F:]
    a = g * torch.sigmoid(g) * u
    return h + linear(a, w["w_down"])


def model_loss(params, tok, cfg, cos, sin, scale):
    """params: list of float64 leaf tensors in declared order; tok: int64 [B, S+1]."""
    B, S1 = tok.shape
    S = S1 - 1
    d, H, hd, F, L = cfg["d"], cfg["H"], cfg["hd"], cfg["F"], cfg["L"]
    inp, lab = tok[:, :S].reshape(-1), tok[:, 1:].reshape(-1)
    x = params[0][inp]
    names = ["attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down"]
    for l in range(L):
        w = {n: params[1 + 6 * l + i] for i, n in enumerate(names)}
        x = block(x, w, B, S, H, hd, F, cfg["eps"], cos, sin, scale)
    xf = rmsnorm(x, params[1 + 6 * L], cfg["eps"])
    logits = rf(linear(xf, params[2 + 6 * L]))
    return torch.nn.functional.cross_entropy(logits, lab, reduction="mean")
