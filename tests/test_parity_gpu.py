"""GPU parity: the HIP path against the CPU oracle on the same seeded inputs.

Bars: bf16 inputs max-abs 2e-2 on out and 1e-2 on lse; float32 inputs 1e-4.
The oracle sees the exact float64 values of the tensors handed to the GPU.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests.gpu_util import (TOL, compare_full, compare_rows, note, require_gpu, run_gpu,
                            sample_rows, to64)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


# ---- the workloads -----------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny_n256_h2_d32_f32", "n8k_b2_h12_d64_3pat"])
def test_workload_all_rows(name):
    wl = workloads.BY_NAME[name]
    note(f"[parity] {name} all rows")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    eo, el = compare_full(q, k, v, list(wl.patterns), wl.causal, wl.dtype, tag=name)
    note(f"[parity] {name}: out err {eo:.3e} lse err {el:.3e}")


def test_n32k_all_rows_of_two_heads():
    """The benchmark workload: every row of head 0 (segment lengths 2731) and
    head 5 (2730 for the r = 6 and r = 12 patterns)."""
    wl = workloads.BY_NAME["n32k_h12_d64_5pat"]
    note("[parity] n32k heads 0,5 all rows")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    eo, el = compare_full(q, k, v, list(wl.patterns), wl.causal, wl.dtype, tag=wl.name, heads=[0, 5])
    note(f"[parity] n32k heads 0,5: out err {eo:.3e} lse err {el:.3e}")


@pytest.mark.parametrize("name", ["n32k_h12_d64_5pat", "n256k_h16_d64_8pat_geo", "n1m_h16_d128_6pat"])
def test_workload_sampled_rows(name):
    wl = workloads.BY_NAME[name]
    note(f"[parity] {name} sampled rows")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    out, lse = run_gpu(q, k, v, list(wl.patterns), wl.causal)
    # every row written, none NaN/Inf (all rows are covered: the first pattern has r = 1)
    assert torch.isfinite(lse).all().item()
    assert torch.isfinite(out).all().item()
    rows = sample_rows(wl, np.random.default_rng(wl.seed), per_head=48)
    eo, el = compare_rows(q, k, v, out, lse, wl, rows, tag=name)
    note(f"[parity] {name}: {len(rows)} rows, out err {eo:.3e} lse err {el:.3e}")


@pytest.mark.parametrize("name", ["n32k_h12_d64_5pat", "n8k_b2_h12_d64_3pat"])
def test_non_causal_sampled_rows(name):
    """The workloads' shapes with causal = False (Eq. 6 literally: every kept
    key of the segment is visible)."""
    import dataclasses
    wl = dataclasses.replace(workloads.BY_NAME[name], causal=False)
    note(f"[parity] {name} non-causal sampled rows")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    out, lse = run_gpu(q, k, v, list(wl.patterns), False)
    assert torch.isfinite(lse).all().item() and torch.isfinite(out).all().item()
    rows = sample_rows(wl, np.random.default_rng(wl.seed + 1), per_head=24)
    eo, el = compare_rows(q, k, v, out, lse, wl, rows, tag=name + " non-causal")
    note(f"[parity] {name} non-causal: {len(rows)} rows, out err {eo:.3e} lse err {el:.3e}")


WIDER = [
    # (B, N, H, D, dtype, patterns, causal): longer segments than the edge cases
    (1, 4096, 4, 64, "f32", [(2048, 1), (4096, 4)], True),      # float32 kernel, 32 query tiles per segment
    (2, 8192, 8, 32, "bf16", [(2048, 1), (4096, 2), (8192, 4)], True),  # D = 32 at the 8K shape
]


@pytest.mark.parametrize("case", WIDER, ids=lambda c: f"B{c[0]}N{c[1]}H{c[2]}D{c[3]}{c[4]}")
def test_wider_cases_all_rows(case):
    B, N, H, D, dt, pats, causal = case
    note(f"[wider] {case}")
    dtype = torch.bfloat16 if dt == "bf16" else torch.float32
    q, k, v = (workloads.make_random((B, N, H, D), dtype, 1.0, 2000 + N + D, "cuda", t) for t in range(3))
    eo, el = compare_full(q, k, v, pats, causal, dt, tag=str(case))
    note(f"[wider] {case}: out err {eo:.3e} lse err {el:.3e}")


# ---- edge cases at small sizes ------------------------------------------------

EDGE = [
    # (B, N, H, D, dtype, patterns, causal)
    (1, 1, 1, 64, "bf16", [(1, 1)], True),
    (1, 1, 3, 32, "f32", [(4, 2)], True),
    (1, 300, 3, 64, "bf16", [(128, 1), (300, 3), (64, 5)], True),
    (2, 777, 5, 32, "bf16", [(256, 1), (512, 7), (1000, 9)], False),
    (1, 513, 17, 128, "bf16", [(512, 1), (513, 20)], True),
    (1, 200, 2, 64, "bf16", [(50, 3)], True),            # rows no pattern keeps
    (1, 256, 4, 64, "bf16", [(64, 1), (64, 1), (256, 4)], True),   # duplicate pattern
    (1, 1000, 2, 64, "bf16", [(1000, 1)], True),         # dense: 8 query tiles, ragged
    (1, 1000, 2, 64, "bf16", [(1000, 1)], False),
    (1, 1031, 6, 64, "bf16", [(2048, 1), (4096, 3), (333, 2)], True),  # w > N
    (2, 129, 3, 64, "f32", [(64, 1), (129, 2), (100, 7)], True),
    (1, 300, 2, 128, "f32", [(128, 1), (300, 3)], False),
    (1, 160, 2, 32, "f32", [(160, 1)], True),
    (1, 4096, 2, 128, "bf16", [(4096, 1), (2048, 2)], True),
    (1, 64, 16, 64, "bf16", [(64, 64), (64, 1)], True),   # r = w
    # r*H*D so large that a key tile spans >= 2 GiB of rows: 64-bit addressing path
    (1, 1024, 64, 128, "bf16", [(1024, 1), (1024, 1024)], True),
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: f"B{c[0]}N{c[1]}H{c[2]}D{c[3]}{c[4]}{'c' if c[6] else 'nc'}{len(c[5])}p")
def test_edge_cases(case):
    B, N, H, D, dt, pats, causal = case
    note(f"[edge] {case}")
    dtype = torch.bfloat16 if dt == "bf16" else torch.float32
    seed = 1000 + N * 7 + H * 13 + D
    q, k, v = (workloads.make_random((B, N, H, D), dtype, 1.0, seed, "cuda", t) for t in range(3))
    compare_full(q, k, v, pats, causal, dt, tag=str(case))


# ---- online-softmax regimes: scores that grow along the sequence --------------

LOG2E = 1.4426950408889634


def _integer_qkv(B, N, H, D, seed, jump_at, jump):
    """q, k with small integer entries (exact in bf16) and keys from position
    `jump_at` on multiplied by `jump`; v ~ N(0, 1) in bf16.  With the scale
    2^-3 / log2(e) the kernel's scaled scores (log2 units) are q.k / 8 exactly."""
    g = torch.Generator().manual_seed(seed)
    q = torch.randint(-2, 3, (B, N, H, D), generator=g).to(torch.float32)
    k = torch.randint(-2, 3, (B, N, H, D), generator=g).to(torch.float32)
    k[:, jump_at:] *= jump
    v = torch.randn((B, N, H, D), generator=g)
    return (x.to(torch.bfloat16).cuda() for x in (q, k, v))


def _max_excess(q, k, causal, tile=64):
    """Largest amount (log2 units) by which a visible score of a query exceeds
    the max over the visible keys of the first 64-key tile, dense pattern."""
    qf, kf = q[0, :, 0].float().cpu(), k[0, :, 0].float().cpu()
    s = (qf @ kf.T) / 8.0
    N = s.shape[0]
    if causal:
        s = s.masked_fill(torch.ones(N, N, dtype=torch.bool).triu(1), float("-inf"))
    first = s[:, :tile].max(dim=1).values
    return float((s.max(dim=1).values - first).max())


# scale * log2(e) of the regime tests: 1/8 makes every scaled score exact in
# float32 and in bf16; 0.1301 (not a short binary fraction) makes q * scale *
# log2(e) inexact in bf16, so a kernel that rounded the scaled q would show it
# in scores of this size (hundreds of log2 units).
REGIME_SCALES = {"exact": 0.125, "generic": 0.1301}


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("regime,jump,lo,hi", [("rescale", 2.0, 10.0, 26.0), ("rerun", 8.0, 40.0, 120.0),
                                               ("overflow", 16.0, 140.0, 1e9)])
@pytest.mark.parametrize("scale_kind", ["exact", "generic"])
def test_growing_scores(D, causal, regime, jump, lo, hi, scale_kind):
    """Later keys score far above the first key tile.  'rescale': the
    reference max is moved after a tile (tile sums above the slack, below the
    limit); 'rerun': tile sums pass the limit, so the work item runs again
    with a row max for every tile; 'overflow': probabilities overflow to
    infinity before that rerun.  All must match the oracle."""
    B, N, H = 1, 1000, 2
    note(f"[softmax regime] {regime} D={D} causal={causal} scale={scale_kind}")
    q, k, v = _integer_qkv(B, N, H, D, seed=31 + D, jump_at=300, jump=jump)
    sl2 = REGIME_SCALES[scale_kind]
    ex = _max_excess(q, k, causal) * sl2 / 0.125
    assert lo <= ex <= hi, f"construction gives a max excess of {ex} (wanted [{lo}, {hi}])"
    scale = sl2 / LOG2E
    eo, el = compare_full(q, k, v, [(1000, 1), (500, 2)], causal, "bf16", scale=scale,
                          tag=f"{regime} D{D} {scale_kind}")
    note(f"[softmax regime] {regime}: excess {ex:.1f}, out err {eo:.3e} lse err {el:.3e}")


def test_n32k_large_scores_default_scale():
    """The benchmark shape with q, k ~ N(0, 2^2) (scores four times as large
    as the workload's) and the default scale 1/sqrt(D): every row of heads 0
    and 5.  v stays N(0, 1): its size only scales out, whose bf16 rounding
    the range tests below cover."""
    wl = workloads.BY_NAME["n32k_h12_d64_5pat"]
    note("[parity] n32k sigma=2 heads 0,5")
    shape = (wl.B, wl.N, wl.H, wl.D)
    q = workloads.make_random(shape, torch.bfloat16, 2.0, 4242, "cuda", 0)
    k = workloads.make_random(shape, torch.bfloat16, 2.0, 4242, "cuda", 1)
    v = workloads.make_random(shape, torch.bfloat16, 1.0, 4242, "cuda", 2)
    eo, el = compare_full(q, k, v, list(wl.patterns), True, "bf16", tag="n32k sigma=2", heads=[0, 5])
    note(f"[parity] n32k sigma=2: out err {eo:.3e} lse err {el:.3e}")


# Bound on |out - oracle| relative to max|v| for bf16 inputs: probabilities
# rounded to bf16 before the product with v (2^-9 relative), the per-pattern
# rows kept to 2^-11 of their largest magnitude, out rounded to bf16 (2^-9),
# plus float32 sums: 2^-9 + 2^-11 + 2^-9 + 2^-12 < 4.7e-3.
REL_OUT_BAR = 4.7e-3


@pytest.mark.parametrize("vmax", [1e5, 1e-6])
def test_n32k_value_range(vmax):
    """The benchmark shape with v scaled so that max|v| is about `vmax`:
    per-pattern rows far outside fp16's normal range (above 65504, below
    6.1e-5) must keep their relative precision.  Every row of heads 0 and 5;
    out against the oracle within REL_OUT_BAR * max|v|, lse within 1e-2."""
    wl = workloads.BY_NAME["n32k_h12_d64_5pat"]
    note(f"[parity] n32k value range max|v| ~ {vmax:g}")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    v = (v.float() * (vmax / float(v.float().abs().max()))).to(torch.bfloat16)
    vm = float(v.float().abs().max())
    assert 0.5 * vmax <= vm <= 2.0 * vmax
    eo, el = compare_full(q, k, v, list(wl.patterns), True, "bf16", tag=f"n32k max|v|={vm:g}", heads=[0, 5],
                          tol=(REL_OUT_BAR * vm, 1e-2))
    note(f"[parity] n32k max|v|={vm:g}: out err {eo:.3e} ({eo / vm:.2e} of max|v|) lse err {el:.3e}")


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_q_zero_closed_form(dt):
    """q = 0: lse = ln(count of visible keys over all patterns), out = their mean."""
    B, N, H, D = 1, 333, 4, 64
    pats = [(64, 1), (128, 3), (333, 5)]
    dtype = torch.bfloat16 if dt == "bf16" else torch.float32
    note(f"[q0] {dt}")
    q = torch.zeros((B, N, H, D), dtype=dtype, device="cuda")
    k = workloads.make_random((B, N, H, D), dtype, 1.0, 77, "cuda", 1)
    v = workloads.make_random((B, N, H, D), dtype, 1.0, 77, "cuda", 2)
    out, lse = run_gpu(q, k, v, pats, True)
    v64 = to64(v)
    go, gl = to64(out), to64(lse)
    for h in range(H):
        for p in range(N):
            cnt, acc = 0, np.zeros(D)
            for (w, r) in pats:
                st = (p // w) * w
                if (p - st) % r != h % r:
                    continue
                prefix = list(range(st + h % r, p + 1, r))
                cnt += len(prefix)
                acc += v64[0, prefix, h].sum(axis=0)
            assert abs(gl[0, h, p] - math.log(cnt)) < 1e-5
            assert np.abs(go[0, p, h] - acc / cnt).max() < TOL[dt][0]


def test_scale_argument():
    B, N, H, D = 1, 200, 2, 64
    q, k, v = (workloads.make_random((B, N, H, D), torch.bfloat16, 1.0, 5, "cuda", t) for t in range(3))
    note("[scale]")
    compare_full(q, k, v, [(64, 1), (200, 2)], True, "bf16", scale=0.3, tag="scale=0.3")


def test_deterministic():
    wl = workloads.BY_NAME["n8k_b2_h12_d64_3pat"]
    note("[determinism] n8k")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    o1, l1 = run_gpu(q, k, v, list(wl.patterns))
    o2, l2 = run_gpu(q, k, v, list(wl.patterns))
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_error_leaves_buffers_untouched():
    from paper_2307_02486_amd import DilatedAttnError, dilated_attn
    q, k, v = (workloads.make_random((1, 64, 2, 64), torch.bfloat16, 1.0, 9, "cuda", t) for t in range(3))
    out = torch.full_like(q, 7.0)
    lse = torch.full((1, 2, 64), 7.0, device="cuda")
    ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    note("[errors]")
    with pytest.raises(DilatedAttnError) as e:
        dilated_attn(q, k, v, [(32, 1)], out=out, lse=lse, workspace=ws)
    assert e.value.name == "DA_EWORKSPACE"
    with pytest.raises(DilatedAttnError) as e:
        dilated_attn(q, k, v, [(32, 33)], out=out, lse=lse)
    assert e.value.name == "DA_EINVAL"
    torch.cuda.synchronize()
    assert (out == 7.0).all().item() and (lse == 7.0).all().item()


def test_stream_argument():
    """Work goes to the stream given, in order with the caller's other work."""
    from paper_2307_02486_amd import dilated_attn
    B, N, H, D = 1, 512, 2, 64
    q, k, v = (workloads.make_random((B, N, H, D), torch.bfloat16, 1.0, 11, "cuda", t) for t in range(3))
    ref_o, ref_l = run_gpu(q, k, v, [(128, 1), (512, 4)])
    s = torch.cuda.Stream()
    note("[stream]")
    with torch.cuda.stream(s):
        o, l = dilated_attn(q, k, v, [(128, 1), (512, 4)], stream=s)
    s.synchronize()
    assert torch.equal(o, ref_o) and torch.equal(l, ref_l)


# ---- the dense-versus-dilated sweep's configurations ----------------------------

@pytest.mark.parametrize("variant", ["dense", "dilated"])
@pytest.mark.parametrize("N", [8192, 131072])
def test_sweep_config_sampled_rows(N, variant):
    """The sweep's shapes (2^20 tokens, H=16, D=128): every row finite, and
    sampled rows of the first and last (b, h) against the oracle."""
    wl = workloads.sweep_workload(N, variant)
    note(f"[parity] {wl.name} sampled rows")
    q, k, v = workloads.make_qkv(wl, device="cuda")
    out, lse = run_gpu(q, k, v, list(wl.patterns), wl.causal)
    assert torch.isfinite(lse).all().item()
    assert torch.isfinite(out).all().item()
    rng = np.random.default_rng(wl.seed)
    rows = []
    for b in sorted({0, wl.B - 1}):
        for h in sorted({0, wl.H - 1}):
            ps = set(rng.integers(0, N, 24).tolist()) | {0, 2047, 2048, N - 1}
            rows += [(b, int(p), h) for p in sorted(ps)]
    eo, el = compare_rows(q, k, v, out, lse, wl, rows, tag=wl.name)
    note(f"[parity] {wl.name}: {len(rows)} rows, out err {eo:.3e} lse err {el:.3e}")
