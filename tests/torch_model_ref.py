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


def qlinear(x, w, s):
    """int8 projection: y = X^ W^^T with X^ = s clamp(rne(bf16(x) / s), -128, 127) and W^ the same with the
    per-row step 2 mean|w| / sqrt(127) (not trained).  Straight-through for x and w (no clipping mask); the
    step s gets LSQ's gradient: round(v) - v inside the range, the bound outside (v = x / s), times
    1/sqrt(127 K).  The gradient of y is rounded to bf16, the operand of the int8 backward."""
    xb = rf(x)
    K = w.shape[1]
    sw = 2.0 * w.detach().abs().mean(dim=1, keepdim=True) / np.sqrt(127.0)
    qw = torch.clamp(torch.round(w.detach() / sw), -128, 127)
    w_hat = w + (qw * sw - w).detach()
    g = 1.0 / np.sqrt(127.0 * K)
    s_eff = s * g + (s - s * g).detach()
    v = xb.detach() / s.detach()
    q = torch.clamp(torch.round(v), -128, 127)
    delta = torch.where(v < -128, torch.full_like(v, -128.0),
                        torch.where(v > 127, torch.full_like(v, 127.0), torch.round(v) - v))
    x_hat = xb + (q * s.detach() - xb).detach() + (s_eff - s_eff.detach()) * delta
    return rb(x_hat @ w_hat.T)


def rmsnorm(x, g, eps):
    return x * torch.rsqrt((x * x).mean(dim=-1, keepdim=True) + eps) * g


def rope(x, cos, sin):
    """x [..., S, hd] rotated in two halves; cos/sin [S, hd/2]."""
    h = x.shape[-1] // 2
    x1, x2 = x[..., :h], x[..., h:]
    return torch.cat([x1 * cos - x2 * sin, x2 * cos + x1 * sin], dim=-1)


def headnorm(x, eps):
    """Gain-free RMSNorm of each head row (last dimension)."""
    return x * torch.rsqrt((x * x).mean(dim=-1, keepdim=True) + eps)


def block(x, w, B, S, H, hd, F, eps, cos, sin, scale, Hkv=None, qk_norm=False, window=0, int8=False):
    """w: dict of float64 tensors attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down (and with int8 the
    activation steps sx_qkv, sx_o, sx_gate_up, sx_down).  Hkv: key/value heads (query head h reads head
    h // (H // Hkv)); qk_norm: gain-free per-head RMSNorm of q and k before the rotation; window: query i
    sees keys i - window < j <= i (0: all j <= i); int8: the four projections by qlinear."""
    Hkv = H if Hkv is None else Hkv
    if int8:
        def proj(t, name):
            return qlinear(t, w[name], w["sx" + name[1:]])
    else:
        def proj(t, name):
            return linear(t, w[name])
    d, kvw = H * hd, Hkv * hd
    xn = rmsnorm(x, w["attn_norm"], eps)
    qkv = proj(xn, "w_qkv")                                          # [T, d + 2 kvw]
    q, k, v = qkv[:, :d], qkv[:, d:d + kvw], qkv[:, d + kvw:]

    def heads(t, n):
        return t.reshape(B, S, n, hd).permute(0, 2, 1, 3)            # [B, n, S, hd]

    qh, kh = heads(q, H), heads(k, Hkv)
    if qk_norm:
        qh, kh = headnorm(qh, eps), headnorm(kh, eps)
    qh = rf(rope(qh, cos, sin))
    kh = rf(rope(kh, cos, sin))
    vh = rf(heads(v, Hkv))
    G = H // Hkv
    kh = kh.repeat_interleave(G, dim=1)                              # [B, H, S, hd]
    vh = vh.repeat_interleave(G, dim=1)
    raw = rb(qh @ kh.transpose(-1, -2))                              # [B, H, S, S]
    sc = raw * scale
    i = torch.arange(S).unsqueeze(1)
    j = torch.arange(S).unsqueeze(0)
    mask = j <= i
    if window:
        mask = mask & (j > i - window)
    sc = sc.masked_fill(~mask, float("-inf"))
    p = rf(torch.softmax(sc, dim=-1))
    o = rb(p @ vh)                                                   # [B, H, S, hd]
    o = o.permute(0, 2, 1, 3).reshape(B * S, d)
    h = x + proj(o, "w_o")
    hn = rmsnorm(h, w["ffn_norm"], eps)
    gu = proj(hn, "w_gate_up")
    g, u = gu[:, :F], gu[:, F:]
    a = g * torch.sigmoid(g) * u
    return h + proj(a, "w_down")


def layer_window(cfg, l):
    win = cfg.get("swa_window", 0)
    every = cfg.get("swa_full_every", 0)
    if not win or (every and (l + 1) % every == 0) or l == cfg["L"] - 1:
        return 0
    return win


def model_loss(params, tok, cfg, cos, sin, scale):
    """params: list of float64 leaf tensors in declared order; tok: int64 [B, S+1].  cfg may name the
    variants Hkv, qk_norm, embed_norm, swa_window, swa_full_every, z_loss."""
    B, S1 = tok.shape
    S = S1 - 1
    d, H, hd, F, L = cfg["d"], cfg["H"], cfg["hd"], cfg["F"], cfg["L"]
    en = 1 if cfg.get("embed_norm") else 0
    inp, lab = tok[:, :S].reshape(-1), tok[:, 1:].reshape(-1)
    x = params[0][inp]
    if en:
        x = rmsnorm(x, params[1], cfg["eps"])
    names = ["attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down"]
    q8 = bool(cfg.get("int8_linear"))
    if q8:
        names += ["sx_qkv", "sx_o", "sx_gate_up", "sx_down"]
    PL = len(names)
    for l in range(L):
        w = {n: params[1 + en + PL * l + i] for i, n in enumerate(names)}
        x = block(x, w, B, S, H, hd, F, cfg["eps"], cos, sin, scale, cfg.get("Hkv"), cfg.get("qk_norm", False),
                  layer_window(cfg, l), int8=q8)
    xf = rmsnorm(x, params[1 + en + PL * L], cfg["eps"])
    logits = rf(linear(xf, params[2 + en + PL * L]))
    loss = torch.nn.functional.cross_entropy(logits, lab, reduction="mean")
    zw = cfg.get("z_loss", 0.0)
    if zw:
        loss = loss + zw * (torch.logsumexp(logits, dim=-1) ** 2).mean()
    return loss
