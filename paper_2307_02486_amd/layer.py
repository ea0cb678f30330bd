"""A LongNet attention layer: dilated attention as the attention sublayer of
the paper's language model (Sec. 4.1: Magneto with xPos relative positions,
the standard attention replaced by dilated attention).

    u  = LN_in(x)                                   x: [B, N, E]
    q, k, v = projections of u, as [B, N, H, D]
    q, k = xPos(q, +1), xPos(k, -1)                 (dilated_attn_xpos)
    a  = dilated attention of q, k, v               (dilated_attn_fwd / _bwd)
    y  = out_proj(LN_sub(a as [B, N, E]))           (Magneto's sub-LayerNorm)

The residual connection belongs to the block around the layer.  The
attention and xPos run in the library's HIP kernels (their backward passes
too), and so do, in bf16, the LayerNorms (dilated_attn_layernorm_fwd / _bwd)
and the projections' weight gradients (dilated_attn_wgrad: a long reduction
over B * N rows into a small E x E matrix, a shape that general GEMM
libraries split poorly); the other products are plain library GEMMs from
torch.
"""
from __future__ import annotations

from typing import Sequence, Tuple

import torch

from .ops import dilated_attn, dilated_attn_bwd, layer_norm, layer_norm_bwd, wgrad, xpos


class DilatedAttentionFunction(torch.autograd.Function):
    """Differentiable dilated attention over [B, N, H, D] tensors."""

    @staticmethod
    def forward(ctx, q, k, v, patterns, causal, scale):
        q, k, v = q.contiguous(), k.contiguous(), v.contiguous()
        out, lse = dilated_attn(q, k, v, patterns, causal, scale)
        ctx.save_for_backward(q, k, v, out, lse)
        ctx.patterns, ctx.causal, ctx.scale = list(patterns), causal, scale
        return out

    @staticmethod
    def backward(ctx, dout):
        q, k, v, out, lse = ctx.saved_tensors
        dq, dk, dv = dilated_attn_bwd(q, k, v, out, lse, dout.contiguous(), ctx.patterns, ctx.causal,
                                      ctx.scale)
        return dq, dk, dv, None, None, None


class XPosFunction(torch.autograd.Function):
    """Differentiable xPos: the backward applies the transpose of the map."""

    @staticmethod
    def forward(ctx, x, sign, center, base, gamma, scale_base):
        ctx.args = (sign, center, base, gamma, scale_base)
        return xpos(x.contiguous(), sign, False, center, base, gamma, scale_base)

    @staticmethod
    def backward(ctx, dy):
        sign, center, base, gamma, scale_base = ctx.args
        return xpos(dy.contiguous(), sign, True, center, base, gamma, scale_base), None, None, None, None, None


class LinearFunction(torch.autograd.Function):
    """y = x w^T + b over the last dimension, with dw = dy^T x and db (the
    column sums of dy) from the library's weight-gradient kernels when they
    apply (bf16, both dimensions multiples of 128) and from torch otherwise."""

    @staticmethod
    def forward(ctx, x, w, b):
        ctx.save_for_backward(x, w)
        return torch.nn.functional.linear(x, w, b)

    @staticmethod
    def backward(ctx, dy):
        x, w = ctx.saved_tensors
        dy2 = dy.reshape(-1, dy.shape[-1]).contiguous()
        x2 = x.reshape(-1, x.shape[-1]).contiguous()
        dx = (dy2 @ w).view(x.shape) if ctx.needs_input_grad[0] else None
        if not (ctx.needs_input_grad[1] or ctx.needs_input_grad[2]):
            return dx, None, None
        if dy2.dtype == torch.bfloat16 and dy2.shape[1] % 128 == 0 and x2.shape[1] % 128 == 0:
            dw, db = wgrad(dy2, x2, bias_grad=True)
        else:
            dw, db = dy2.t() @ x2, dy2.sum(0)
        return dx, dw, db


def _linear(mod: torch.nn.Linear, x: torch.Tensor) -> torch.Tensor:
    return LinearFunction.apply(x, mod.weight, mod.bias)


class LayerNormFunction(torch.autograd.Function):
    """LayerNorm over the last dimension through the library's kernels."""

    @staticmethod
    def forward(ctx, x, weight, bias, eps):
        x = x.contiguous()
        y, mean, rstd = layer_norm(x, weight, bias, eps)
        ctx.save_for_backward(x, weight, mean, rstd)
        return y

    @staticmethod
    def backward(ctx, dy):
        x, weight, mean, rstd = ctx.saved_tensors
        dx, dw, db = layer_norm_bwd(dy.contiguous(), x, weight, mean, rstd)
        return dx, dw, db, None


def _layer_norm(mod: torch.nn.LayerNorm, x: torch.Tensor) -> torch.Tensor:
    """The library's LayerNorm for bf16 rows of E <= 2048 (E % 8 == 0), torch's otherwise."""
    E = x.shape[-1]
    if x.dtype == torch.bfloat16 and E % 8 == 0 and E <= 2048:
        return LayerNormFunction.apply(x, mod.weight, mod.bias, mod.eps)
    return mod(x)


class LongNetAttention(torch.nn.Module):
    """Attention sublayer with dilated attention (see the module docstring).

    embed_dim = num_heads * head_dim with head_dim in {32, 64, 128};
    patterns is the list of (segment length w, dilation r).  xPos uses
    rotation base `xpos_base`, gamma `xpos_gamma`, scale base
    `xpos_scale_base` and the sequence's middle position as its centre.
    """

    def __init__(self, embed_dim: int, num_heads: int, patterns: Sequence[Tuple[int, int]],
                 causal: bool = True, use_xpos: bool = True, xpos_base: float = 10000.0,
                 xpos_gamma: float = 0.4, xpos_scale_base: float = 512.0, eps: float = 1e-5,
                 device=None, dtype=torch.bfloat16):
        super().__init__()
        if embed_dim % num_heads:
            raise ValueError("embed_dim must be a multiple of num_heads")
        self.embed_dim, self.num_heads = embed_dim, num_heads
        self.head_dim = embed_dim // num_heads
        self.patterns, self.causal = list(patterns), causal
        self.use_xpos = use_xpos
        self.xpos_args = (xpos_base, xpos_gamma, xpos_scale_base)
        kw = dict(device=device, dtype=dtype)
        self.ln_in = torch.nn.LayerNorm(embed_dim, eps=eps, **kw)
        self.q_proj = torch.nn.Linear(embed_dim, embed_dim, **kw)
        self.k_proj = torch.nn.Linear(embed_dim, embed_dim, **kw)
        self.v_proj = torch.nn.Linear(embed_dim, embed_dim, **kw)
        self.ln_sub = torch.nn.LayerNorm(embed_dim, eps=eps, **kw)
        self.out_proj = torch.nn.Linear(embed_dim, embed_dim, **kw)

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        B, N, E = x.shape
        H, D = self.num_heads, self.head_dim
        u = _layer_norm(self.ln_in, x)
        q = _linear(self.q_proj, u).view(B, N, H, D)
        k = _linear(self.k_proj, u).view(B, N, H, D)
        v = _linear(self.v_proj, u).view(B, N, H, D)
        if self.use_xpos:
            base, gamma, scale_base = self.xpos_args
            q = XPosFunction.apply(q, 1, N // 2, base, gamma, scale_base)
            k = XPosFunction.apply(k, -1, N // 2, base, gamma, scale_base)
        a = DilatedAttentionFunction.apply(q, k, v, self.patterns, self.causal, None)
        return _linear(self.out_proj, _layer_norm(self.ln_sub, a.reshape(B, N, E)))

    def float64_params(self) -> dict:
        """The parameters as float64 NumPy arrays, keyed ln_in_g, ln_in_b, wq,
        bq, wk, bk, wv, bv, ln_sub_g, ln_sub_b, wo, bo."""
        p = {"ln_in_g": self.ln_in.weight, "ln_in_b": self.ln_in.bias,
             "wq": self.q_proj.weight, "bq": self.q_proj.bias, "wk": self.k_proj.weight, "bk": self.k_proj.bias,
             "wv": self.v_proj.weight, "bv": self.v_proj.bias,
             "ln_sub_g": self.ln_sub.weight, "ln_sub_b": self.ln_sub.bias,
             "wo": self.out_proj.weight, "bo": self.out_proj.bias}
        return {kk: vv.detach().to("cpu", torch.float64).numpy() for kk, vv in p.items()}
