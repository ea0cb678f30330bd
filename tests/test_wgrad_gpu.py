"""GPU parity of the projections' weight-gradient kernel (dilated_attn_wgrad):
dw = dy^T x for bf16 dy [K, M] and x [K, N], and the bias gradient db (the
column sums of dy), against float32 results of the same bf16 values on the
GPU.

Bar, elementwise and derived from the arithmetic: the kernel rounds its
float32 sum to bf16 once (unit roundoff 2^-8), and it and the reference sum
the exact bf16 x bf16 products in float32 in different orders.  That sum
error is at most K 2^-24 of the sum of the products' magnitudes in the worst
case and grows like sqrt(K) 2^-24 of it in practice (both sides sum in
blocks); 2^-12 of the magnitude sum covers it for every K here:
    |dw - ref| <= 2^-8 |ref| + 2^-12 * (|dy|^T |x|).
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
    # (K, M, N): the layer's shape (B * N = 32768 rows, E = 768), a ragged k
    # tail, one k tile, non-square outputs, a reduction longer than one split
    (32768, 768, 768),
    (300, 128, 256),
    (64 * 3 + 5, 256, 128),
    (1, 128, 128),
    (65536, 128, 384),
    (4097, 1024, 1024),
]


def _check(dw, dy, x):
    ref = dy.float().t() @ x.float()
    mag = dy.float().abs().t() @ x.float().abs()
    err = (dw.float() - ref).abs()
    bound = 2.0 ** -8 * ref.abs() + 2.0 ** -12 * mag
    worst = float((err / bound.clamp_min(1e-30)).max())
    note(f"[wgrad] max |err| {float(err.max()):.3e}, max err/bound {worst:.3f}")
    assert worst <= 1.0


@pytest.mark.parametrize("case", CASES, ids=str)
def test_wgrad_matches_float32_product(case):
    from paper_2307_02486_amd import wgrad
    K, M, N = case
    note(f"[wgrad] K={K} M={M} N={N}")
    dy = workloads.make_random((K, M), torch.bfloat16, 1.0, 900 + M, "cuda", 0)
    x = workloads.make_random((K, N), torch.bfloat16, 1.0, 901 + N, "cuda", 0)
    dw = wgrad(dy, x)
    torch.cuda.synchronize()
    _check(dw, dy, x)
    # a second call into a caller-supplied output that held other values
    out = torch.full((M, N), 7.0, dtype=torch.bfloat16, device="cuda")
    wgrad(dy, x, out=out)
    torch.cuda.synchronize()
    assert torch.equal(out, dw)
    # with the bias gradient: the same dw, and db within the same kind of bar
    dw2, db = wgrad(dy, x, bias_grad=True)
    torch.cuda.synchronize()
    assert torch.equal(dw2, dw)
    ref = dy.float().sum(0)
    bound = 2.0 ** -8 * ref.abs() + 2.0 ** -12 * dy.float().abs().sum(0)
    worst = float(((db.float() - ref).abs() / bound).max())
    note(f"[wgrad] db err/bound {worst:.3f}")
    assert worst <= 1.0


def test_wgrad_empty_reduction_gives_zeros():
    from paper_2307_02486_amd import wgrad
    note("[wgrad] K=0")
    dy = torch.empty((0, 128), dtype=torch.bfloat16, device="cuda")
    x = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    out = torch.full((128, 256), 3.0, dtype=torch.bfloat16, device="cuda")
    wgrad(dy, x, out=out)
    _, db = wgrad(dy, x, bias_grad=True)
    torch.cuda.synchronize()
    assert (out == 0).all().item() and (db == 0).all().item()


def test_wgrad_errors_launch_nothing():
    from paper_2307_02486_amd import DilatedAttnError, wgrad
    note("[wgrad errors]")
    dy = torch.ones((64, 100), dtype=torch.bfloat16, device="cuda")
    x = torch.ones((64, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.full((100, 128), 5.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(DilatedAttnError) as e:
        wgrad(dy, x, out=out)
    assert e.value.name == "DA_EINVAL"
    with pytest.raises(DilatedAttnError) as e:
        wgrad(torch.ones((64, 128), device="cuda"), torch.ones((64, 128), device="cuda"))
    assert e.value.name == "DA_EUNSUPPORTED"
    torch.cuda.synchronize()
    assert (out == 5).all().item()
