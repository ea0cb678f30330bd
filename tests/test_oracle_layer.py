"""Pins of the LongNet-layer oracle (CPU only).

xPos is pinned by properties that its definition fixes and a plausible slip
breaks: scores that depend on the offset n - m only (a wrong sign of the key
scale or of one rotation breaks it), a hand-written one-pair case, the
rotation's norm preservation with the stated scale, and the adjoint identity
of the transpose used by the backward.  LayerNorm is checked against
torch.nn.functional.layer_norm in float64 and its backward against torch's
autograd.  The whole layer is checked against a float64 torch composition
with scaled_dot_product_attention for a single dense pattern, and its
backward against central finite differences of the layer's forward.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.layer_ref import (PARAM_NAMES, XPosConfig, layer_bwd_ref, layer_norm_bwd_ref, layer_norm_ref,
                              layer_ref, xpos_ref)


def _scores(qx, kx):
    """[B, H, N, N] dot products of every query row with every key row."""
    return np.einsum("bnhd,bmhd->bhnm", qx, kx)


@pytest.mark.parametrize("D", [2, 8, 64])
def test_xpos_scores_depend_on_offset_only(D):
    rng = np.random.default_rng(D)
    B, N, H, s = 1, 24, 2, 7
    q, k = rng.standard_normal((2, B, N, H, D))
    cfg = XPosConfig(scale_base=16.0, center=5)
    S = _scores(xpos_ref(q, +1, cfg), xpos_ref(k, -1, cfg))
    # the same rows placed s positions later in a longer sequence (another centre)
    q2, k2 = np.zeros((2, B, N + s, H, D))
    q2[:, s:], k2[:, s:] = q, k
    cfg2 = XPosConfig(scale_base=16.0, center=11)
    S2 = _scores(xpos_ref(q2, +1, cfg2), xpos_ref(k2, -1, cfg2))[:, :, s:, s:]
    np.testing.assert_allclose(S2, S, rtol=1e-9, atol=1e-9)


def test_xpos_one_pair_by_hand():
    """D = 2: theta_0 = 1, zeta_0 = gamma / (1 + gamma)."""
    cfg = XPosConfig(gamma=0.5, scale_base=4.0, center=1)
    x = np.array([0.3, -1.2])
    X = np.zeros((1, 3, 1, 2))
    X[0, :, 0] = x
    Y = xpos_ref(X, -1, cfg)
    zeta = 0.5 / 1.5
    for n in range(3):
        s = zeta ** (-(n - 1) / 4.0)
        c, sn = np.cos(n), np.sin(n)
        want = s * np.array([c * x[0] - sn * x[1], sn * x[0] + c * x[1]])
        np.testing.assert_allclose(Y[0, n, 0], want, rtol=1e-13)


def test_xpos_pair_norms_and_adjoint():
    rng = np.random.default_rng(3)
    B, N, H, D = 2, 9, 3, 16
    cfg = XPosConfig(scale_base=8.0)
    x, y = rng.standard_normal((2, B, N, H, D))
    for sign in (1, -1):
        fx = xpos_ref(x, sign, cfg)
        i = np.arange(D // 2)
        zeta = (2 * i / D + cfg.gamma) / (1 + cfg.gamma)
        n = np.arange(N)[:, None]
        scl = zeta[None, :] ** (sign * (n - N // 2) / cfg.scale_base)
        pn = lambda t: np.hypot(t[..., 0::2], t[..., 1::2])  # noqa: E731
        np.testing.assert_allclose(pn(fx), pn(x) * scl[None, :, None, :], rtol=1e-12)
        # <f(x), y> = <x, f^T(y)>
        lhs = float((fx * y).sum())
        rhs = float((x * xpos_ref(y, sign, cfg, transpose=True)).sum())
        assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs))


def test_layer_norm_matches_torch():
    rng = np.random.default_rng(4)
    x, dy = rng.standard_normal((2, 3, 5, 12))
    g, b = rng.standard_normal((2, 12))
    y, xhat, rstd = layer_norm_ref(x, g, b)
    xt = torch.tensor(x, requires_grad=True)
    gt, bt = torch.tensor(g, requires_grad=True), torch.tensor(b, requires_grad=True)
    yt = torch.nn.functional.layer_norm(xt, (12,), gt, bt, 1e-5)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    (yt * torch.tensor(dy)).sum().backward()
    dx, dg, db = layer_norm_bwd_ref(dy, xhat, rstd, g)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-10, atol=1e-10)


def _params(E, seed):
    rng = np.random.default_rng(seed)
    p = {}
    for name in PARAM_NAMES:
        shape = (E, E) if name.startswith("w") else (E,)
        scale = 1.0 / np.sqrt(E) if name.startswith("w") else 0.3
        p[name] = rng.standard_normal(shape) * scale
    p["ln_in_g"] += 1.0
    p["ln_sub_g"] += 1.0
    return p


@pytest.mark.parametrize("use_xpos", [False, True])
def test_layer_dense_pattern_matches_torch_sdpa(use_xpos):
    """One pattern with w = N, r = 1 is standard causal attention."""
    B, N, H, D = 2, 16, 2, 4
    E = H * D
    p = _params(E, 5)
    x = np.random.default_rng(6).standard_normal((B, N, E))
    cfg = XPosConfig(scale_base=8.0) if use_xpos else None
    y, _ = layer_ref(x, p, H, [(N, 1)], True, cfg)
    T = {kk: torch.tensor(vv) for kk, vv in p.items()}
    ln = torch.nn.functional.layer_norm
    u = ln(torch.tensor(x), (E,), T["ln_in_g"], T["ln_in_b"], 1e-5)
    q, k, v = ((u @ T["w" + c].T + T["b" + c]).reshape(B, N, H, D) for c in "qkv")
    if use_xpos:
        q = torch.tensor(xpos_ref(q.numpy(), +1, cfg))
        k = torch.tensor(xpos_ref(k.numpy(), -1, cfg))
    a = torch.nn.functional.scaled_dot_product_attention(q.transpose(1, 2), k.transpose(1, 2),
                                                         v.transpose(1, 2), is_causal=True)
    a = a.transpose(1, 2).reshape(B, N, E)
    want = ln(a, (E,), T["ln_sub_g"], T["ln_sub_b"], 1e-5) @ T["wo"].T + T["bo"]
    np.testing.assert_allclose(y, want.numpy(), rtol=1e-10, atol=1e-10)


LAYER_CASES = [
    # (B, N, H, D, patterns, causal, xpos)
    (1, 10, 2, 4, [(4, 1), (10, 2)], True, True),
    (2, 9, 2, 2, [(9, 1), (5, 3)], False, True),   # ragged segments, non-causal
    (1, 8, 1, 4, [(8, 2), (4, 1)], True, False),
]


@pytest.mark.parametrize("case", LAYER_CASES)
def test_layer_backward_matches_finite_differences(case):
    B, N, H, D, pats, causal, use_xpos = case
    E = H * D
    p = _params(E, N + H)
    rng = np.random.default_rng(N * 7 + D)
    x, dy = rng.standard_normal((2, B, N, E))
    cfg = XPosConfig(scale_base=8.0) if use_xpos else None
    dx, grads, _ = layer_bwd_ref(x, dy, p, H, pats, causal, cfg)

    def loss(xx, pp):
        return float((dy * layer_ref(xx, pp, H, pats, causal, cfg)[0]).sum())

    eps = 1e-6
    for _ in range(3):
        u = rng.standard_normal(x.shape)
        fd = (loss(x + eps * u, p) - loss(x - eps * u, p)) / (2 * eps)
        assert abs(fd - float((dx * u).sum())) <= 1e-6 * max(1.0, abs(fd))
    for name in PARAM_NAMES:
        u = rng.standard_normal(p[name].shape)
        pp, pm = dict(p), dict(p)
        pp[name], pm[name] = p[name] + eps * u, p[name] - eps * u
        fd = (loss(x, pp) - loss(x, pm)) / (2 * eps)
        assert abs(fd - float((grads[name] * u).sum())) <= 1e-6 * max(1.0, abs(fd)), name


def test_layer_planted_mistakes_are_caught():
    """A key scale with the query's sign, or a rotation of the transpose in
    the wrong direction, fails the pins above."""
    rng = np.random.default_rng(9)
    q, k = rng.standard_normal((2, 1, 12, 1, 8))
    cfg = XPosConfig(scale_base=4.0)
    S = _scores(xpos_ref(q, +1, cfg), xpos_ref(k, +1, cfg))          # wrong key sign
    q2, k2 = np.zeros((2, 1, 15, 1, 8))
    q2[:, 3:], k2[:, 3:] = q, k
    S2 = _scores(xpos_ref(q2, +1, cfg), xpos_ref(k2, +1, cfg))[:, :, 3:, 3:]
    assert not np.allclose(S, S2, rtol=1e-6)
    x, y = rng.standard_normal((2, 1, 12, 1, 8))
    lhs = float((xpos_ref(x, 1, cfg) * y).sum())
    wrong = float((x * xpos_ref(y, 1, cfg, transpose=False)).sum())  # not the transpose
    assert abs(lhs - wrong) > 1e-6
