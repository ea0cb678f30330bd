"""GPU test of dilated_attn_fwd_noalloc (the forward pass with the library's
own fixed workspace): called through the C ABI, its results must equal those
of dilated_attn_fwd on the same inputs, for two calls in a row, the second on
a smaller problem (the array keeps the first call's contents); a problem whose
workspace exceeds the fixed size is rejected before any launch."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests.gpu_util import TOL, note, require_gpu, to64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    require_gpu()
    from paper_2307_02486_amd import _lib
    return _lib.load()


def _noalloc(lib, q, k, v, patterns, causal=True):
    from paper_2307_02486_amd import _lib
    B, N, H, D = q.shape
    out = torch.full_like(q, float("nan"))
    lse = torch.full((B, H, N), float("nan"), dtype=torch.float32, device=q.device)
    arr, n = _lib.pattern_array(patterns)
    dt = _lib.DA_BF16 if q.dtype == torch.bfloat16 else _lib.DA_F32
    rc = lib.dilated_attn_fwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                                      B, N, H, D, arr, n, int(causal), dt, 0.0,
                                      torch.cuda.current_stream().cuda_stream)
    return rc, out, lse


def test_noalloc_matches_fwd_two_calls(lib):
    from paper_2307_02486_amd import dilated_attn, plan
    cases = [workloads.BY_NAME["n32k_h12_d64_5pat"], workloads.BY_NAME["n8k_b2_h12_d64_3pat"]]
    for wl in cases:
        info = plan(wl.B, wl.N, wl.H, wl.D, wl.patterns, wl.causal, wl.torch_dtype)
        assert info["workspace_bytes"] <= 128 << 20
        note(f"[noalloc] {wl.name}: workspace {info['workspace_bytes']} bytes")
        q, k, v = workloads.make_qkv(wl, device="cuda")
        rc, o1, l1 = _noalloc(lib, q, k, v, list(wl.patterns), wl.causal)
        assert rc == 0, rc
        o2, l2 = dilated_attn(q, k, v, list(wl.patterns), wl.causal)
        torch.cuda.synchronize()
        assert torch.equal(o1, o2), f"{wl.name}: out differs from dilated_attn_fwd"
        assert torch.equal(l1, l2), f"{wl.name}: lse differs from dilated_attn_fwd"


def test_noalloc_small_ragged_against_oracle(lib):
    """A third call, smaller again, with ragged segments: equal to
    dilated_attn_fwd and within the bf16 bars of the oracle."""
    from paper_2307_02486_amd import dilated_attn
    B, N, H, D = 1, 777, 5, 64
    pats = [(256, 1), (512, 7), (777, 3)]
    q, k, v = (workloads.make_random((B, N, H, D), torch.bfloat16, 1.0, 77, "cuda", t) for t in range(3))
    rc, o1, l1 = _noalloc(lib, q, k, v, pats)
    assert rc == 0, rc
    o2, l2 = dilated_attn(q, k, v, pats)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    ro, rl = oracle.dilated_attention_ref(to64(q), to64(k), to64(v), pats, True)
    assert float(np.abs(to64(o1) - ro).max()) <= TOL["bf16"][0]
    assert float(np.abs(to64(l1) - rl).max()) <= TOL["bf16"][1]


def test_noalloc_rejects_problem_beyond_fixed_workspace(lib):
    """The 256K-token workload needs about 1.1 GB of workspace: rejected with
    DA_ETOOLARGE from the plan alone, buffers untouched."""
    from paper_2307_02486_amd import _lib
    wl = workloads.BY_NAME["n256k_h16_d64_8pat_geo"]
    out = torch.full((16,), 7.0, device="cuda")
    lse = torch.full((16,), 7.0, device="cuda")
    x = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    arr, n = _lib.pattern_array(wl.patterns)
    rc = lib.dilated_attn_fwd_noalloc(x.data_ptr(), x.data_ptr(), x.data_ptr(), out.data_ptr(), lse.data_ptr(),
                                      wl.B, wl.N, wl.H, wl.D, arr, n, 1, _lib.DA_BF16, 0.0, None)
    assert _lib.ERRORS[rc] == "DA_ETOOLARGE"
    torch.cuda.synchronize()
    assert (out == 7.0).all().item() and (lse == 7.0).all().item()
