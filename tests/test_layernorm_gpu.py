"""GPU parity of the LayerNorm kernels (dilated_attn_layernorm_fwd / _bwd)
against torch's float32 LayerNorm and its autograd on the same bf16 values.

Bars, elementwise and derived from the arithmetic: outputs are rounded to
bf16 once (unit roundoff 2^-8); before that both sides compute in float32,
differing by a few float32 roundings in the row statistics and in the order
of the sums, which 2^-14 of the row's (or column's) largest term covers.
  * y:  |y - ref| <= 2^-8 |ref| + 2^-14 (|xhat| |g| + |b|) max over the row
  * dx: |dx - ref| <= 2^-8 |ref| + 2^-14 rstd (|dy g| max over the row) (1 + |xhat|)
  * dg, db: sums over all rows, |err| <= 2^-8 |ref| + 2^-14 sum_rows |term|
"""
import pytest
import torch

import workloads
from tests.gpu_util import note, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


CASES = [
    # (rows, E, x sigma, x offset): the layer's shape, widths on every kernel
    # variant (E / 8 up to 64, 128 and 256 chunks) with ragged lane use, a
    # ragged last workgroup, and a large offset (cancellation in the mean)
    (32768, 768, 1.0, 0.0),
    (1000, 64, 1.0, 0.0),
    (77, 520, 2.0, 0.0),
    (130, 1024, 1.0, 0.0),
    (65, 2048, 1.0, 0.0),
    (300, 768, 0.5, 40.0),
    (1, 8, 1.0, 0.0),
]


def _data(rows, E, sigma, offset, seed):
    x = workloads.make_random((rows, E), torch.float32, sigma, seed, "cuda", 0) + offset
    x = x.to(torch.bfloat16)
    g = (1.0 + 0.3 * workloads.make_random((E,), torch.float32, 1.0, seed, "cuda", 1)).to(torch.bfloat16)
    b = (0.3 * workloads.make_random((E,), torch.float32, 1.0, seed, "cuda", 2)).to(torch.bfloat16)
    dy = workloads.make_random((rows, E), torch.bfloat16, 1.0, seed, "cuda", 3)
    return x, g, b, dy


def _ratio(err, bound):
    return float((err / bound.clamp_min(1e-30)).max()) if err.numel() else 0.0


@pytest.mark.parametrize("case", CASES, ids=str)
def test_layernorm_matches_float32(case):
    from paper_2307_02486_amd import layer_norm, layer_norm_bwd
    rows, E, sigma, offset = case
    note(f"[layernorm] rows={rows} E={E}")
    x, g, b, dy = _data(rows, E, sigma, offset, 40 + E)
    y, mean, rstd = layer_norm(x, g, b, 1e-5)
    dx, dg, db = layer_norm_bwd(dy, x, g, mean, rstd)
    torch.cuda.synchronize()

    xf = x.float().requires_grad_(True)
    gf, bf = g.float().requires_grad_(True), b.float().requires_grad_(True)
    ref = torch.nn.functional.layer_norm(xf, (E,), gf, bf, 1e-5)
    ref.backward(dy.float())
    mu = x.float().mean(-1, keepdim=True)
    rs = torch.rsqrt(((x.float() - mu) ** 2).mean(-1, keepdim=True) + 1e-5)
    xhat = (x.float() - mu) * rs
    assert torch.allclose(mean, mu[:, 0], rtol=1e-5, atol=1e-5 * (1 + abs(offset)))
    assert torch.allclose(rstd, rs[:, 0], rtol=1e-4)

    tiny = 2.0 ** -14
    row_y = (xhat.abs() * g.float().abs() + b.float().abs()).amax(-1, keepdim=True)
    r_y = _ratio((y.float() - ref.detach()).abs(), 2.0 ** -8 * ref.detach().abs() + tiny * row_y)
    dyg = (dy.float() * g.float()).abs().amax(-1, keepdim=True)
    r_dx = _ratio((dx.float() - xf.grad).abs(), 2.0 ** -8 * xf.grad.abs() + tiny * rs * dyg * (1 + xhat.abs()))
    mag_g = (dy.float() * xhat).abs().sum(0)
    mag_b = dy.float().abs().sum(0)
    r_dg = _ratio((dg.float() - gf.grad).abs(), 2.0 ** -8 * gf.grad.abs() + tiny * mag_g)
    r_db = _ratio((db.float() - bf.grad).abs(), 2.0 ** -8 * bf.grad.abs() + tiny * mag_b)
    note(f"[layernorm] err/bar: y {r_y:.3f} dx {r_dx:.3f} dg {r_dg:.3f} db {r_db:.3f}")
    assert max(r_y, r_dx, r_dg, r_db) <= 1.0


def test_layernorm_in_place_and_zero_rows():
    from paper_2307_02486_amd import layer_norm_bwd
    from paper_2307_02486_amd import _lib
    from paper_2307_02486_amd.ops import layer_norm
    note("[layernorm] in place, rows = 0")
    x, g, b, _ = _data(50, 256, 1.0, 0.0, 5)
    y, _, _ = layer_norm(x, g, b)
    x2 = x.clone()
    mean = torch.empty(50, device="cuda")
    rstd = torch.empty(50, device="cuda")
    lib = _lib.load()
    rc = lib.dilated_attn_layernorm_fwd(x2.data_ptr(), g.data_ptr(), b.data_ptr(), x2.data_ptr(), mean.data_ptr(),
                                        rstd.data_ptr(), 50, 256, 1e-5, 1, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == 0 and torch.equal(x2, y)
    e = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    s = torch.empty((0,), device="cuda")
    dx, dg, db = layer_norm_bwd(e, e, g, s, s)
    torch.cuda.synchronize()
    assert dx.shape == (0, 256) and (dg == 0).all().item() and (db == 0).all().item()


def test_layernorm_errors_launch_nothing():
    from paper_2307_02486_amd import DilatedAttnError, layer_norm
    note("[layernorm errors]")
    x = torch.ones((4, 12), dtype=torch.bfloat16, device="cuda")
    w = torch.ones(12, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(DilatedAttnError) as e:
        layer_norm(x, w, w)
    assert e.value.name == "DA_EINVAL"
    x = torch.ones((4, 64), device="cuda")
    w = torch.ones(64, device="cuda")
    with pytest.raises(DilatedAttnError) as e:
        layer_norm(x, w, w)
    assert e.value.name == "DA_EUNSUPPORTED"
