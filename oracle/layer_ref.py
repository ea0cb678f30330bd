"""fp64 oracle of a LongNet attention layer.  TEST INFRASTRUCTURE ONLY.

Only tests/ (and the benchmark's CPU-baseline leg) may import this module;
the product path never uses it.

The paper builds its language model on the Magneto architecture with xPos
relative positions and replaces the standard attention with dilated attention
(Sec. 4.1).  The layer here is that attention sublayer, without the residual
connection, which belongs to the block around it:

    u  = LN_in(x)                                   x: [B, N, E]
    q, k, v = u Wq^T + bq, u Wk^T + bk, u Wv^T + bv  reshaped to [B, N, H, D]
    q', k' = xPos(q, +1), xPos(k, -1)
    a  = DilatedAttention(q', k', v)                 Sec. 2.2-2.3
    y  = LN_sub(a reshaped to [B, N, E]) Wo^T + bo   (Magneto's sub-LayerNorm)

xPos (Sun et al., "A Length-Extrapolatable Transformer", 2022) rotates each
pair of head-dimension elements (2i, 2i+1) of the row at position n by the
angle n * theta_i, theta_i = base^(-2i/D), and scales it by
zeta_i^(+-(n - c)/lambda), zeta_i = (2i/D + gamma) / (1 + gamma), with +
for queries and - for keys.  A query at n and a key at m then meet with
sum_i zeta_i^((n - m)/lambda) (q_i^T R((m - n) theta_i) k_i): the score
depends on the offset n - m only, and decays with it.  The centre c only
keeps the separate factors in floating-point range (it cancels in every
score); it is the middle position N // 2 by default.

LayerNorm is the usual one: (x - mean) / sqrt(var + eps) * g + b over the
last dimension, var the biased variance.

The backward (`layer_bwd_ref`) chains the textbook derivatives of the
projections and LayerNorms, the transpose of xPos (a rotation by -n theta_i
with the same scale) and the dilated-attention backward of
`dilated_bwd.dilated_attention_bwd_ref`.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Sequence, Tuple

import numpy as np

from .dilated_bwd import dilated_attention_bwd_ref
from .dilated_ref import dilated_attention_ref

Pattern = Tuple[int, int]


@dataclass
class XPosConfig:
    base: float = 10000.0    # rotation frequencies theta_i = base^(-2i/D)
    gamma: float = 0.4       # zeta_i = (2i/D + gamma) / (1 + gamma)
    scale_base: float = 512.0  # lambda
    center: int | None = None  # c; None: N // 2


def xpos_ref(x, sign: int, cfg: XPosConfig = XPosConfig(), transpose: bool = False):
    """xPos of x [B, N, H, D] (float64): sign +1 for queries, -1 for keys.
    transpose=True applies the transpose of the map (rotation by -n theta,
    same scale), which is what its backward multiplies the gradient by."""
    x = np.asarray(x, dtype=np.float64)
    B, N, H, D = x.shape
    assert D % 2 == 0
    c = N // 2 if cfg.center is None else cfg.center
    i = np.arange(D // 2, dtype=np.float64)
    theta = cfg.base ** (-2.0 * i / D)                      # [D/2]
    zeta = (2.0 * i / D + cfg.gamma) / (1.0 + cfg.gamma)    # [D/2]
    n = np.arange(N, dtype=np.float64)[:, None]             # [N, 1]
    ang = n * theta[None, :]                                # [N, D/2]
    if transpose:
        ang = -ang
    scl = zeta[None, :] ** (sign * (n - c) / cfg.scale_base)
    cs, sn = np.cos(ang) * scl, np.sin(ang) * scl           # [N, D/2]
    x0, x1 = x[..., 0::2], x[..., 1::2]                     # [B, N, H, D/2]
    y = np.empty_like(x)
    y[..., 0::2] = x0 * cs[None, :, None, :] - x1 * sn[None, :, None, :]
    y[..., 1::2] = x0 * sn[None, :, None, :] + x1 * cs[None, :, None, :]
    return y


def layer_norm_ref(x, g, b, eps: float = 1e-5):
    """LayerNorm over the last dimension; returns (y, xhat, rstd)."""
    x = np.asarray(x, dtype=np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    return xhat * np.asarray(g, np.float64) + np.asarray(b, np.float64), xhat, rstd


def layer_norm_bwd_ref(dy, xhat, rstd, g):
    """Gradients (dx, dg, db) of LayerNorm given its saved xhat and rstd."""
    dy = np.asarray(dy, dtype=np.float64)
    dxhat = dy * np.asarray(g, np.float64)
    dx = rstd * (dxhat - dxhat.mean(axis=-1, keepdims=True)
                 - xhat * (dxhat * xhat).mean(axis=-1, keepdims=True))
    red = tuple(range(dy.ndim - 1))
    return dx, (dy * xhat).sum(axis=red), dy.sum(axis=red)


PARAM_NAMES = ("ln_in_g", "ln_in_b", "wq", "bq", "wk", "bk", "wv", "bv",
               "ln_sub_g", "ln_sub_b", "wo", "bo")


def layer_ref(x, params: dict, H: int, patterns: Sequence[Pattern], causal: bool = True,
              xpos: XPosConfig | None = XPosConfig(), eps: float = 1e-5):
    """Forward of the layer; returns y [B, N, E] and the intermediates the
    backward needs."""
    p = {kk: np.asarray(vv, np.float64) for kk, vv in params.items()}
    x = np.asarray(x, dtype=np.float64)
    B, N, E = x.shape
    D = E // H
    u, uhat, urstd = layer_norm_ref(x, p["ln_in_g"], p["ln_in_b"], eps)
    q = (u @ p["wq"].T + p["bq"]).reshape(B, N, H, D)
    k = (u @ p["wk"].T + p["bk"]).reshape(B, N, H, D)
    v = (u @ p["wv"].T + p["bv"]).reshape(B, N, H, D)
    if xpos is not None:
        qx, kx = xpos_ref(q, +1, xpos), xpos_ref(k, -1, xpos)
    else:
        qx, kx = q, k
    a, lse = dilated_attention_ref(qx, kx, v, patterns, causal)
    a2 = a.reshape(B, N, E)
    z, zhat, zrstd = layer_norm_ref(a2, p["ln_sub_g"], p["ln_sub_b"], eps)
    y = z @ p["wo"].T + p["bo"]
    saved = dict(u=u, uhat=uhat, urstd=urstd, qx=qx, kx=kx, v=v, a=a2, z=z, zhat=zhat, zrstd=zrstd)
    return y, saved


def layer_bwd_ref(x, dy, params: dict, H: int, patterns: Sequence[Pattern], causal: bool = True,
                  xpos: XPosConfig | None = XPosConfig(), eps: float = 1e-5):
    """Gradients of sum(dy * layer(x)) with respect to x and every parameter."""
    p = {kk: np.asarray(vv, np.float64) for kk, vv in params.items()}
    dy = np.asarray(dy, dtype=np.float64)
    y, s = layer_ref(x, params, H, patterns, causal, xpos, eps)
    B, N, E = dy.shape
    D = E // H
    g = {}
    g["wo"] = np.einsum("bne,bnf->ef", dy, s["z"])
    g["bo"] = dy.sum(axis=(0, 1))
    dz = dy @ p["wo"]
    da, g["ln_sub_g"], g["ln_sub_b"] = layer_norm_bwd_ref(dz, s["zhat"], s["zrstd"], p["ln_sub_g"])
    dqx, dkx, dv, _, _ = dilated_attention_bwd_ref(s["qx"], s["kx"], s["v"], da.reshape(B, N, H, D),
                                                   patterns, causal)
    if xpos is not None:
        dq, dk = xpos_ref(dqx, +1, xpos, transpose=True), xpos_ref(dkx, -1, xpos, transpose=True)
    else:
        dq, dk = dqx, dkx
    dq, dk, dv = dq.reshape(B, N, E), dk.reshape(B, N, E), dv.reshape(B, N, E)
    u = s["u"]
    for name, dd in (("q", dq), ("k", dk), ("v", dv)):
        g["w" + name] = np.einsum("bne,bnf->ef", dd, u)
        g["b" + name] = dd.sum(axis=(0, 1))
    du = dq @ p["wq"] + dk @ p["wk"] + dv @ p["wv"]
    dx, g["ln_in_g"], g["ln_in_b"] = layer_norm_bwd_ref(du, s["uhat"], s["urstd"], p["ln_in_g"])
    return dx, g, y
