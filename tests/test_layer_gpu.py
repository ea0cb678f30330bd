"""GPU parity of the xPos kernel and the LongNet attention layer against the
fp64 layer oracle, on the exact values the GPU sees.

Bars (derived from the arithmetic):
  * xPos: per pair of elements, |y - ref| <= tol * |ref pair| with tol
    4e-5 for float32 (float32 sine, cosine and exp2 of an exponent up to
    about 60) and 4e-3 for bf16 (output rounding 2^-9 per element, plus the
    float32 error).
  * Layer, float32 (float32 attention kernel, float32 GEMMs): max-abs 1e-4
    on outputs of size about 1 (float32 rounding through a handful of
    sums of at most E terms).
  * Layer, bf16: every intermediate (LayerNorm outputs, projections, xPos,
    attention output) is rounded to bf16 (2^-9 relative each) and the
    projections sum E products of such values, so the output error is a few
    times 2^-9 of its size: max-abs <= 4e-2 on outputs of size about 1.
    Gradients pass through the same roundings twice (forward intermediates
    and backward products): max-abs <= 3e-2 of each gradient's largest
    reference entry.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle.layer_ref import XPosConfig, layer_bwd_ref, layer_ref, xpos_ref
from tests.gpu_util import note, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _pair_rel_err(y, ref):
    y, ref = np.asarray(y, np.float64), np.asarray(ref, np.float64)
    e = np.hypot(y[..., 0::2] - ref[..., 0::2], y[..., 1::2] - ref[..., 1::2])
    n = np.hypot(ref[..., 0::2], ref[..., 1::2])
    return float((e / np.maximum(n, 1e-30)).max())


XPOS_CASES = [
    # (B, N, H, D, center or None, dtype)
    (1, 100, 3, 64, None, torch.float32),
    (2, 2049, 2, 32, 0, torch.float32),
    (1, 32768, 2, 64, None, torch.float32),    # angles up to 32767 rad, scale exponents up to 58
    (1, 5, 1, 256, 4, torch.float32),
    (1, 100, 3, 64, None, torch.bfloat16),
    (1, 32768, 2, 128, None, torch.bfloat16),
]


@pytest.mark.parametrize("case", XPOS_CASES, ids=lambda c: str(c)[:40])
def test_xpos_matches_oracle(case):
    from paper_2307_02486_amd import xpos
    B, N, H, D, center, dtype = case
    note(f"[xpos] {case}")
    x = workloads.make_random((B, N, H, D), dtype, 1.0, 700 + N, "cuda", 0)
    x64 = x.to("cpu", torch.float64).numpy()
    tol = 4e-5 if dtype == torch.float32 else 4e-3
    cfg = XPosConfig(center=center)
    for sign in (1, -1):
        for transpose in (False, True):
            y = xpos(x, sign, transpose, center)
            torch.cuda.synchronize()
            ref = xpos_ref(x64, sign, cfg, transpose)
            err = _pair_rel_err(y.to("cpu", torch.float64).numpy(), ref)
            assert err <= tol, f"sign {sign} transpose {transpose}: rel err {err}"
    # in place gives the same values
    y = xpos(x, -1, False, center)
    x2 = x.clone()
    xpos(x2, -1, False, center, out=x2)
    torch.cuda.synchronize()
    assert torch.equal(x2, y)


def test_xpos_errors_launch_nothing():
    from paper_2307_02486_amd import DilatedAttnError, xpos
    x = torch.ones((1, 16, 2, 64), dtype=torch.bfloat16, device="cuda")
    note("[xpos errors]")
    with pytest.raises(DilatedAttnError) as e:
        xpos(x, 0)
    assert e.value.name == "DA_EINVAL"
    with pytest.raises(DilatedAttnError) as e:
        xpos(x, 1, center=16)
    assert e.value.name == "DA_EINVAL"
    with pytest.raises(DilatedAttnError):   # scale exponents beyond the stated range
        xpos(torch.ones((1, 40000, 1, 32), dtype=torch.bfloat16, device="cuda"), 1)
    with pytest.raises(DilatedAttnError) as e:
        xpos(torch.ones((1, 16, 2, 12), dtype=torch.float32, device="cuda"), 1)
    assert e.value.name == "DA_EINVAL"
    torch.cuda.synchronize()
    assert (x == 1).all().item()


LAYER_CASES = [
    # (B, N, H, D, patterns, causal)
    (1, 512, 2, 64, [(128, 1), (256, 2), (512, 4)], True),
    (2, 300, 4, 32, [(128, 1), (300, 3)], True),
    # E = 96: the weight gradients take torch's GEMM (the library's kernel
    # needs multiples of 128), the LayerNorms still the library's; non-causal
    (1, 256, 3, 32, [(64, 1), (256, 4)], False),
]


def _make_layer(B, N, H, D, pats, causal, dtype, seed):
    from paper_2307_02486_amd.layer import LongNetAttention
    E = H * D
    torch.manual_seed(seed)
    layer = LongNetAttention(E, H, pats, causal, device="cuda", dtype=dtype)
    with torch.no_grad():   # non-trivial LayerNorm parameters
        for ln in (layer.ln_in, layer.ln_sub):
            ln.weight.add_(0.2 * torch.randn_like(ln.weight))
            ln.bias.add_(0.2 * torch.randn_like(ln.bias))
    x = workloads.make_random((B, N, E), dtype, 1.0, seed, "cuda", 0)
    return layer, x


@pytest.mark.parametrize("case", LAYER_CASES, ids=lambda c: str(c)[:30])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_layer_forward_matches_oracle(case, dtype):
    B, N, H, D, pats, causal = case
    note(f"[layer fwd] {case} {dtype}")
    layer, x = _make_layer(B, N, H, D, pats, causal, dtype, 11)
    with torch.no_grad():
        y = layer(x)
    torch.cuda.synchronize()
    ref, _ = layer_ref(x.to("cpu", torch.float64).numpy(), layer.float64_params(), H, pats, causal,
                       XPosConfig())
    err = float(np.abs(y.to("cpu", torch.float64).numpy() - ref).max())
    note(f"[layer fwd] max-abs err {err:.3e} (|ref| max {np.abs(ref).max():.2f})")
    assert err <= (1e-4 if dtype == torch.float32 else 4e-2)


@pytest.mark.parametrize("case", LAYER_CASES, ids=lambda c: str(c)[:30])
def test_layer_backward_matches_oracle(case):
    B, N, H, D, pats, causal = case
    note(f"[layer bwd] {case}")
    layer, x = _make_layer(B, N, H, D, pats, causal, torch.bfloat16, 12)
    x.requires_grad_(True)
    dy = workloads.make_random((B, N, H * D), torch.bfloat16, 1.0, 13, "cuda", 0)
    y = layer(x)
    y.backward(dy)
    torch.cuda.synchronize()
    dx, grads, _ = layer_bwd_ref(x.detach().to("cpu", torch.float64).numpy(),
                                 dy.to("cpu", torch.float64).numpy(), layer.float64_params(), H, pats,
                                 causal, XPosConfig())
    got = {"ln_in_g": layer.ln_in.weight.grad, "ln_in_b": layer.ln_in.bias.grad,
           "wq": layer.q_proj.weight.grad, "bq": layer.q_proj.bias.grad,
           "wk": layer.k_proj.weight.grad, "bk": layer.k_proj.bias.grad,
           "wv": layer.v_proj.weight.grad, "bv": layer.v_proj.bias.grad,
           "ln_sub_g": layer.ln_sub.weight.grad, "ln_sub_b": layer.ln_sub.bias.grad,
           "wo": layer.out_proj.weight.grad, "bo": layer.out_proj.bias.grad}
    pairs = [("x", x.grad, dx)] + [(kk, got[kk], grads[kk]) for kk in got]
    for name, g, ref in pairs:
        g = g.to("cpu", torch.float64).numpy()
        rel = float(np.abs(g - ref).max() / max(np.abs(ref).max(), 1e-30))
        note(f"[layer bwd] d{name}: max-abs err / max|ref| = {rel:.3e}")
        assert rel <= 3e-2, f"d{name}: {rel}"


def test_layer_backward_computes_only_requested_gradients():
    """Frozen parameters get no gradient, an input without requires_grad
    none either, and the input gradient alone equals the one computed with
    every parameter's."""
    B, N, H, D, pats, causal = LAYER_CASES[0]
    note("[layer bwd] requested gradients only")
    layer, x = _make_layer(B, N, H, D, pats, causal, torch.bfloat16, 14)
    dy = workloads.make_random((B, N, H * D), torch.bfloat16, 1.0, 15, "cuda", 0)
    layer(x).backward(dy)                       # x needs no gradient
    assert x.grad is None and layer.q_proj.weight.grad is not None
    x.requires_grad_(True)
    layer.zero_grad(set_to_none=True)
    layer(x).backward(dy)
    dx_full = x.grad.clone()
    layer.zero_grad(set_to_none=True)
    for p in layer.parameters():
        p.requires_grad_(False)
    x.grad = None
    layer(x).backward(dy)                       # only x needs a gradient
    torch.cuda.synchronize()
    assert all(p.grad is None for p in layer.parameters())
    assert torch.equal(x.grad, dx_full)
