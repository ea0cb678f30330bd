"""GPU parity of the backward pass against the fp64 backward oracle.

The GPU path runs its own forward (out, lse) and then the backward; the
oracle computes everything from the same q, k, v, dout.  Bar for bf16
gradients (none is stated for them): max-abs error <= 2e-2 * max(1, max|ref|)
per tensor, the forward's bf16 bar for values of order one, scaled for
larger gradients.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from tests.gpu_util import note, require_gpu, to64

pytestmark = pytest.mark.gpu
REL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _gpu_bwd(q, k, v, dout, pats, causal, scale=None):
    from paper_2307_02486_amd import dilated_attn, dilated_attn_bwd
    out, lse = dilated_attn(q, k, v, pats, causal, scale)
    nan = float("nan")
    dq, dk, dv = (torch.full_like(q, nan) for _ in range(3))
    dilated_attn_bwd(q, k, v, out, lse, dout, pats, causal, scale, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    return dq, dk, dv


def _check(name, got, ref, tag):
    assert not np.isnan(got).any(), f"{tag}: NaN in {name} (element not written?)"
    bar = REL * max(1.0, float(np.abs(ref).max()))
    err = float(np.abs(got - ref).max())
    assert err <= bar, f"{tag}: {name} max-abs err {err:.3e} > {bar:.3e}"
    return err


def _inputs(B, N, H, D, seed):
    return [workloads.make_random((B, N, H, D), torch.bfloat16, 1.0, seed, "cuda", t) for t in range(4)]


CASES = [
    # (B, N, H, D, patterns, causal)
    (1, 256, 2, 32, [(64, 1), (128, 2), (256, 4)], True),
    (1, 777, 3, 64, [(256, 1), (512, 7), (1000, 9)], True),
    (2, 777, 3, 64, [(256, 1), (512, 7), (1000, 9)], False),
    (1, 1000, 2, 64, [(1000, 1)], True),                 # dense, ragged tiles
    (1, 300, 4, 64, [(128, 1), (128, 1), (300, 3)], True),  # duplicate pattern
    (1, 200, 5, 32, [(50, 3)], True),                    # rows no pattern keeps: zero gradients
    (1, 1031, 6, 64, [(2048, 1), (4096, 3), (333, 2)], True),  # w > N
    (1, 64, 16, 64, [(64, 64), (64, 1)], True),          # r = w
    (1, 513, 17, 128, [(512, 1), (513, 20)], True),      # D = 128 (two column halves)
    (2, 777, 3, 128, [(256, 1), (512, 7), (1000, 9)], False),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"B{c[0]}N{c[1]}H{c[2]}D{c[3]}{'c' if c[5] else 'nc'}{len(c[4])}p")
def test_backward_all_rows(case):
    B, N, H, D, pats, causal = case
    note(f"[bwd] {case}")
    q, k, v, dout = _inputs(B, N, H, D, seed=500 + N + H * 7 + D)
    dq, dk, dv = _gpu_bwd(q, k, v, dout, pats, causal)
    rq, rk, rv, _, _ = oracle.dilated_attention_bwd_ref(to64(q), to64(k), to64(v), to64(dout), pats, causal)
    errs = [_check(n, to64(g), r, str(case)) for n, g, r in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv))]
    note(f"[bwd] {case}: errors dq {errs[0]:.2e} dk {errs[1]:.2e} dv {errs[2]:.2e}")


def test_backward_n8k_two_heads():
    """The 8K workload's shapes (2 x 8192 x 12 x 64, patterns up to w = 8192),
    every row of heads 0 and 5."""
    wl = workloads.BY_NAME["n8k_b2_h12_d64_3pat"]
    note("[bwd] n8k heads 0,5")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    dout = workloads.make_random(q.shape, torch.bfloat16, 1.0, wl.seed, "cuda", 3)
    dq, dk, dv = _gpu_bwd(q, k, v, dout, list(wl.patterns), wl.causal)
    hs = [0, 5]
    rq, rk, rv, _, _ = oracle.dilated_attention_bwd_ref(to64(q), to64(k), to64(v), to64(dout),
                                                        list(wl.patterns), wl.causal, heads=hs)
    for n, g, r in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        e = _check(n, to64(g)[:, :, hs], r[:, :, hs], "n8k")
        note(f"[bwd] n8k {n} err {e:.2e}")


def test_backward_n32k_sampled_rows():
    """The benchmark workload (32768 x 12 x 64, five patterns): sampled rows
    of heads 0 and 5 against the row-restricted backward oracle."""
    wl = workloads.BY_NAME["n32k_h12_d64_5pat"]
    note("[bwd] n32k sampled rows")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    dout = workloads.make_random(q.shape, torch.bfloat16, 1.0, wl.seed, "cuda", 3)
    pats = list(wl.patterns)
    dq, dk, dv = _gpu_bwd(q, k, v, dout, pats, wl.causal)
    assert torch.isfinite(dq).all() and torch.isfinite(dk).all() and torch.isfinite(dv).all()
    rng = np.random.default_rng(7)
    rows = [(0, int(p), h) for h in (0, 5) for p in sorted(set(rng.integers(0, wl.N, 10).tolist()) |
                                                          {0, 2047, 2048, 16383, wl.N - 1})]
    qc, kc, vc, oc = q.cpu(), k.cpu(), v.cpu(), dout.cpu()
    rq = oracle.dq_rows_ref(qc, kc, vc, oc, pats, True, None, rows)
    rk, rv = oracle.dkdv_rows_ref(qc, kc, vc, oc, pats, True, None, rows)
    idx = (torch.tensor([r[0] for r in rows]), torch.tensor([r[1] for r in rows]), torch.tensor([r[2] for r in rows]))
    for n, g, r in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        e = _check(n, g.cpu()[idx].double().numpy(), r, "n32k")
        note(f"[bwd] n32k {n}: {len(rows)} rows, err {e:.2e}")


def test_backward_deterministic():
    q, k, v, dout = _inputs(1, 777, 3, 64, seed=11)
    pats = [(256, 1), (512, 7)]
    a = _gpu_bwd(q, k, v, dout, pats, True)
    b = _gpu_bwd(q, k, v, dout, pats, True)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_backward_error_leaves_buffers_untouched():
    from paper_2307_02486_amd import DilatedAttnError, dilated_attn, dilated_attn_bwd
    q, k, v, dout = _inputs(1, 128, 2, 64, seed=12)
    out, lse = dilated_attn(q, k, v, [(64, 1)], True)
    dq = torch.full_like(q, 7.0)
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(DilatedAttnError):
        dilated_attn_bwd(q, k, v, out, lse, dout, [(64, 1)], True, dq=dq, workspace=small)
    torch.cuda.synchronize()
    assert (dq == 7.0).all()


def test_backward_n1m_sampled_rows():
    """The 1M-token, D = 128 workload (six patterns up to w = N): dq on random
    rows, dk and dv on rows at the end of the sequence (the queries seeing a
    key there are few, which keeps the oracle cheap), heads 0 and 15."""
    wl = workloads.BY_NAME["n1m_h16_d128_6pat"]
    note("[bwd] n1m sampled rows")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    dout = workloads.make_random(q.shape, torch.bfloat16, 1.0, wl.seed, "cuda", 3)
    pats = list(wl.patterns)
    dq, dk, dv = _gpu_bwd(q, k, v, dout, pats, wl.causal)
    for t in (dq, dk, dv):
        assert torch.isfinite(t).all().item()
    rng = np.random.default_rng(9)
    qrows = [(0, int(p), h) for h in (0, 15) for p in sorted(set(rng.integers(0, wl.N, 8).tolist()) | {0, wl.N - 1})]
    krows = [(0, wl.N - 1 - i, h) for h in (0, 15) for i in range(0, 64, 9)]
    qc, kc, vc, oc = q.cpu(), k.cpu(), v.cpu(), dout.cpu()
    rq = oracle.dq_rows_ref(qc, kc, vc, oc, pats, True, None, qrows)
    rk, rv = oracle.dkdv_rows_ref(qc, kc, vc, oc, pats, True, None, krows)
    def pick(t, rows):
        return t[tuple(torch.tensor([r[i] for r in rows]) for i in range(3))].double().numpy()
    e = _check("dq", pick(dq.cpu(), qrows), rq, "n1m")
    note(f"[bwd] n1m dq: {len(qrows)} rows, err {e:.2e}")
    for n, g, r in (("dk", dk, rk), ("dv", dv, rv)):
        e = _check(n, pick(g.cpu(), krows), r, "n1m")
        note(f"[bwd] n1m {n}: {len(krows)} rows, err {e:.2e}")


@pytest.mark.parametrize("scale_kind", ["default", "generic"])
def test_backward_large_scores(scale_kind):
    """Scores four times the workloads' (q, k ~ N(0, 2^2)) with the default
    scale at the 8K workload's shapes (every row of heads 0 and 5), and with a
    scale whose product with log2(e) is not a short binary fraction on a
    smaller ragged case: q and k enter the score MFMAs unrounded."""
    if scale_kind == "default":
        wl = workloads.BY_NAME["n8k_b2_h12_d64_3pat"]
        shape, pats, hs, scale = (wl.B, wl.N, wl.H, wl.D), list(wl.patterns), [0, 5], None
    else:
        shape, pats, hs, scale = (1, 777, 3, 64), [(256, 1), (512, 7), (777, 3)], None, 0.1301 / 1.4426950408889634
    note(f"[bwd] large scores {scale_kind} {shape}")
    q = workloads.make_random(shape, torch.bfloat16, 2.0, 4343, "cuda", 0)
    k = workloads.make_random(shape, torch.bfloat16, 2.0, 4343, "cuda", 1)
    v = workloads.make_random(shape, torch.bfloat16, 1.0, 4343, "cuda", 2)
    dout = workloads.make_random(shape, torch.bfloat16, 1.0, 4343, "cuda", 3)
    dq, dk, dv = _gpu_bwd(q, k, v, dout, pats, True, scale)
    rq, rk, rv, _, _ = oracle.dilated_attention_bwd_ref(to64(q), to64(k), to64(v), to64(dout), pats, True,
                                                        scale, heads=hs)
    for n, g, r in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        gg, rr = to64(g), r
        if hs is not None:
            gg, rr = gg[:, :, hs], rr[:, :, hs]
        e = _check(n, gg, rr, f"large scores {scale_kind}")
        note(f"[bwd] large scores {scale_kind} {n} err {e:.2e}")


@pytest.mark.parametrize("gmax", [1e5, 1e-8])
@pytest.mark.parametrize("shape,pats", [((1, 777, 3, 64), [(256, 1), (512, 7), (777, 3)]),
                                        ((1, 513, 2, 128), [(512, 1), (513, 20)])],
                         ids=["D64", "D128"])
def test_backward_value_range(gmax, shape, pats):
    """dout scaled so that the gradients reach about `gmax`: the per-pattern
    gradients are stored as fp16 rows scaled by a power of two per 64-column
    chunk, so neither 1e5 (above fp16's 65504) nor 1e-8 (below fp16's
    smallest subnormal, 6e-8) loses relative precision.  Bar: 2e-2 of each tensor's largest magnitude
    (the gradient bar, taken relative at every scale)."""
    note(f"[bwd] value range {gmax:g} {shape} {pats}")
    q = workloads.make_random(shape, torch.bfloat16, 1.0, 4545, "cuda", 0)
    k = workloads.make_random(shape, torch.bfloat16, 1.0, 4545, "cuda", 1)
    v = workloads.make_random(shape, torch.bfloat16, 1.0, 4545, "cuda", 2)
    dout = (workloads.make_random(shape, torch.float32, 1.0, 4545, "cuda", 3) * gmax).to(torch.bfloat16)
    dq, dk, dv = _gpu_bwd(q, k, v, dout, pats, True)
    rq, rk, rv, _, _ = oracle.dilated_attention_bwd_ref(to64(q), to64(k), to64(v), to64(dout), pats, True)
    for n, g, r in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        got = to64(g)
        assert np.isfinite(got).all(), f"{n}: not finite"
        top = float(np.abs(r).max())
        err = float(np.abs(got - r).max())
        assert err <= REL * top, f"{n}: max-abs err {err:.3e} > {REL * top:.3e} (max |ref| {top:.3e})"
        note(f"[bwd] value range {gmax:g} {shape}: {n} err/max {err / top:.2e}")
