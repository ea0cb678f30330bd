"""Host-side logic: plan helpers built with g++ (also under ASan/UBSan), the
C ABI's exported symbols, plan accounting and argument errors.  No GPU."""
import ctypes
import math
import os
import re
import shutil
import subprocess

import numpy as np
import pytest
import torch

import oracle
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2307_02486_amd", "csrc")
HEADER = os.path.join(ROOT, "include", "dilated_attn.h")


def _gxx_run(tmp_path, extra):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "t")
    cmd = [gxx, "-std=c++17", "-O1", *extra, "-I", CSRC, "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "cpp", "test_plan_host.cpp"), os.path.join(CSRC, "plan.cpp"), "-o", exe]
    subprocess.run(cmd, check=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "OK" in res.stdout


def test_plan_helpers_host(tmp_path):
    _gxx_run(tmp_path, [])


def test_plan_helpers_sanitized(tmp_path):
    _gxx_run(tmp_path, ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-g"])


@pytest.fixture(scope="module")
def lib():
    from paper_2307_02486_amd import _lib
    return _lib.load()


def test_exports_every_declared_symbol(lib):
    text = open(HEADER).read()
    names = re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(dilated_attn_\w+)\s*\(", text, re.M)
    assert set(names) == {"dilated_attn_plan", "dilated_attn_fwd", "dilated_attn_fwd_noalloc", "dilated_attn_strerror",
                          "dilated_attn_profile_begin", "dilated_attn_profile_end",
                          "dilated_attn_bwd_plan", "dilated_attn_bwd", "dilated_attn_xpos",
                          "dilated_attn_wgrad_workspace", "dilated_attn_wgrad",
                          "dilated_attn_layernorm_fwd", "dilated_attn_layernorm_bwd_workspace",
                          "dilated_attn_layernorm_bwd"}
    for n in names:
        assert hasattr(lib, n), n
    nm = subprocess.run(["nm", "-D", "--defined-only", os.path.join(ROOT, "paper_2307_02486_amd",
                                                                     "libdilated_attn.so")],
                        capture_output=True, text=True).stdout
    for n in names:
        assert re.search(rf"\bT {n}$", nm, re.M), n


def test_strerror(lib):
    for code in (0, -1, -2, -3, -4, -5, -6, 7):
        assert lib.dilated_attn_strerror(code)


@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda w: w.name)
def test_plan_accounting_matches_enumeration(wl):
    from paper_2307_02486_amd import plan
    info = plan(wl.B, wl.N, wl.H, wl.D, wl.patterns, wl.causal, wl.torch_dtype)
    flops = oracle.sparse_flops(wl.B, wl.N, wl.H, wl.D, wl.patterns, wl.causal)
    rows = wl.B * oracle.covered_rows(wl.N, wl.H, wl.patterns)
    assert info["covered_rows"] == rows
    assert info["sparse_flops"] == pytest.approx(flops, rel=1e-12)
    es = 2 if wl.dtype == "bf16" else 4     # element size of q, k, v, out
    ws = 2 if wl.dtype == "bf16" else 4     # per-pattern outputs: scaled fp16 or fp32
    rec = 8                                 # per-row record: lse and scale (float32 each)
    assert info["bytes_attn"] == rows * (3 * wl.D * es + wl.D * ws + rec)
    assert info["bytes_combine"] == rows * (wl.D * ws + rec) + wl.B * wl.N * wl.H * (wl.D * es + 4)


def test_plan_workspace_layout():
    """Workspace per pattern: compact output rows (fp16 for bf16 inputs, fp32
    for fp32 inputs) and an 8-byte record per row, each block 256-byte aligned."""
    from paper_2307_02486_amd import plan
    pats = [(2048, 1), (4096, 2), (8192, 4), (16384, 6), (32768, 12)]
    for dtype, es in ((torch.bfloat16, 2), (torch.float32, 4)):
        info = plan(1, 32768, 12, 64, pats, True, dtype)
        want = 0
        for (w, r) in pats:
            rows = 12 * (32768 // w) * (-(-w // r))
            want += -(-rows * 64 * es // 256) * 256
            want += -(-rows * 8 // 256) * 256
        assert info["workspace_bytes"] == want


def test_plan_takes_no_environment_switch(monkeypatch):
    """What a call computes and launches depends on its arguments only."""
    from paper_2307_02486_amd.ops import plan_raw
    pats = [(2048, 1), (4096, 2)]
    rc0, i0 = plan_raw(1, 8192, 12, 64, pats, 1, 1, 0.0)
    monkeypatch.setenv("DILATED_ATTN_FUSE_COMBINE", "1")
    rc1, i1 = plan_raw(1, 8192, 12, 64, pats, 1, 1, 0.0)
    assert rc0 == rc1 == 0 and i0 == i1
    assert "combine_fused" not in i0


def test_plan_accounting_random_small():
    from paper_2307_02486_amd import plan
    rng = np.random.default_rng(7)
    for _ in range(150):
        N = int(rng.integers(1, 300))
        H = int(rng.integers(1, 9))
        pats = []
        for _ in range(int(rng.integers(1, 6))):
            w = int(rng.integers(1, 2 * N + 3))
            pats.append((w, int(rng.integers(1, w + 1))))
        causal = bool(rng.random() < 0.6)
        info = plan(1, N, H, 32, pats, causal, torch.float32)
        assert info["covered_rows"] == oracle.covered_rows(N, H, pats)
        assert info["sparse_flops"] == oracle.sparse_flops(1, N, H, 32, pats, causal)


def test_plan_paper_flop_formula():
    """Sec. 2.4: 2*N*d*sum(w/r^2) per head, plus 2*d per kept row (diagonal)."""
    from paper_2307_02486_amd import plan
    wl = workloads.BY_NAME["n256k_h16_d64_8pat_geo"]
    info = plan(wl.B, wl.N, wl.H, wl.D, wl.patterns)
    paper = wl.H * 2 * wl.N * wl.D * sum(w / r ** 2 for w, r in wl.patterns)
    assert info["sparse_flops"] == pytest.approx(paper + 2 * wl.D * info["covered_rows"], rel=1e-12)
    # geometric bound with alpha = 2, w0 = 2048
    assert info["sparse_flops"] - 2 * wl.D * info["covered_rows"] <= wl.H * 4 * 2048 * wl.N * wl.D


BAD_PLANS = [
    # (B, N, H, D, patterns, causal, dtype, scale) -> code
    ((0, 16, 2, 64, [(8, 1)], 1, 1, 0.0), "DA_EINVAL"),
    ((1, 0, 2, 64, [(8, 1)], 1, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 0, 64, [(8, 1)], 1, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 2, 64, [], 1, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 2, 64, [(8, 1)] * 17, 1, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 2, 64, [(8, 9)], 1, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 2, 64, [(8, 0)], 1, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 2, 64, [(0, 1)], 1, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 2, 64, [(8, 1)], 2, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 2, 64, [(8, 1)], 1, 1, -1.0), "DA_EINVAL"),
    ((1, 16, 2, 64, [(8, 1)], 1, 1, float("nan")), "DA_EINVAL"),
    ((1, 2 ** 31, 2, 64, [(8, 1)], 1, 1, 0.0), "DA_EINVAL"),
    ((1, 16, 2, 48, [(8, 1)], 1, 1, 0.0), "DA_EUNSUPPORTED"),
    ((1, 16, 2, 64, [(8, 1)], 1, 7, 0.0), "DA_EUNSUPPORTED"),
]


@pytest.mark.parametrize("args,code", BAD_PLANS)
def test_plan_rejects(args, code):
    from paper_2307_02486_amd import _lib, plan_raw
    rc, _ = plan_raw(*args)
    assert _lib.ERRORS[rc] == code


def test_fwd_rejects_before_touching_device(lib):
    """Argument errors return before any HIP call (fake, never dereferenced pointers)."""
    from paper_2307_02486_amd import _lib
    arr, n = _lib.pattern_array([(8, 1)])
    good = [0x10000, 0x20000, 0x30000, 0x40000, 0x50000]
    def call(ptrs, ws=0x100000, ws_bytes=1 << 20, B=1, N=16, H=2, D=64, dtype=1, pats=(arr, n)):
        return lib.dilated_attn_fwd(*ptrs, B, N, H, D, pats[0], pats[1], 1, dtype, 0.0, ws, ws_bytes, None)
    assert _lib.ERRORS[call([0] + good[1:])] == "DA_EINVAL"
    assert _lib.ERRORS[call(good, ws=0)] == "DA_EINVAL"
    assert _lib.ERRORS[call([good[0] + 8] + good[1:])] == "DA_EALIGN"
    assert _lib.ERRORS[call(good, ws=0x100008)] == "DA_EALIGN"
    assert _lib.ERRORS[call(good, ws_bytes=16)] == "DA_EWORKSPACE"
    assert _lib.ERRORS[call([good[0], good[1], good[2], good[0], good[4]])] == "DA_EINVAL"   # out aliases q
    assert _lib.ERRORS[call(good, ws=good[1])] == "DA_EINVAL"                               # workspace aliases k
    assert _lib.ERRORS[call(good, D=40)] == "DA_EUNSUPPORTED"
    bad_arr, bn = _lib.pattern_array([(4, 5)])
    assert _lib.ERRORS[call(good, pats=(bad_arr, bn))] == "DA_EINVAL"


def test_profile_window_arguments(lib):
    assert lib.dilated_attn_profile_begin(0) == -1
    assert lib.dilated_attn_profile_begin(1 << 21) == -1
    assert lib.dilated_attn_profile_end(None, None, None) == -1   # no window open


def test_bwd_plan_accounting():
    """Backward workspace = two [B,H,N] float32 arrays plus, per pattern, three
    fp16 [units][lmax][D] blocks and three float32 [units][lmax][ceil(D/64)]
    scale blocks, each 256-byte aligned; flops = 10 D per pair."""
    from paper_2307_02486_amd import plan, plan_bwd
    import torch
    for (B, N, H, D, pats) in [(1, 32768, 12, 64, [(2048, 1), (4096, 2), (8192, 4), (16384, 6), (32768, 12)]),
                               (2, 777, 5, 32, [(256, 1), (512, 7), (1000, 9)]),
                               (1, 513, 17, 128, [(512, 1), (513, 20)])]:
        f = plan(B, N, H, D, pats, True, torch.bfloat16)
        b = plan_bwd(B, N, H, D, pats, True, torch.bfloat16)
        al = lambda x: (x + 255) // 256 * 256
        ws = al(al(B * H * N * 4) + B * H * N * 4)
        for (w, r) in pats:
            w = min(w, N)
            rows = B * H * (-(-N // w)) * (-(-w // r))
            for _ in range(3):
                ws = al(ws + rows * D * 2)
            for _ in range(3):
                ws = al(ws + rows * (-(-D // 64)) * 4)
        assert b["workspace_bytes"] == ws
        assert b["sparse_flops"] == pytest.approx(2.5 * f["sparse_flops"], rel=1e-12)
        assert b["covered_rows"] == f["covered_rows"]
        assert b["num_work_items"] == 2 * f["num_work_items"]


def test_bwd_unsupported_and_errors(lib):
    """The backward covers bf16 (D in {32, 64, 128}); argument errors return
    before any HIP call (fake, never dereferenced pointers)."""
    from paper_2307_02486_amd import _lib, plan_raw
    arr, n = _lib.pattern_array([(8, 1)])
    info = _lib.PlanInfo()
    import ctypes
    assert lib.dilated_attn_bwd_plan(1, 16, 2, 128, arr, n, 1, 1, 0.0, ctypes.byref(info)) == 0
    huge, hn = _lib.pattern_array([(1 << 20, 1 << 19)])      # a 65-row tile spans > 2 GiB
    assert _lib.ERRORS[lib.dilated_attn_bwd_plan(1, 1 << 20, 64, 128, huge, hn, 1, 1, 0.0,
                                                 ctypes.byref(info))] == "DA_EUNSUPPORTED"
    assert _lib.ERRORS[lib.dilated_attn_bwd_plan(1, 16, 2, 64, arr, n, 1, 0, 0.0, ctypes.byref(info))] == \
        "DA_EUNSUPPORTED"
    assert lib.dilated_attn_bwd_plan(1, 16, 2, 64, arr, n, 1, 1, 0.0, ctypes.byref(info)) == 0
    good = [0x10000 * (i + 1) for i in range(9)]   # q k v out lse dout dq dk dv
    def call(ptrs, ws=0x1000000, ws_bytes=1 << 20, D=64, dtype=1):
        return lib.dilated_attn_bwd(*ptrs, 1, 16, 2, D, arr, n, 1, dtype, 0.0, ws, ws_bytes, None)
    assert _lib.ERRORS[call([0] + good[1:])] == "DA_EINVAL"
    assert _lib.ERRORS[call(good[:8] + [0])] == "DA_EINVAL"
    assert _lib.ERRORS[call(good, ws=0)] == "DA_EINVAL"
    assert _lib.ERRORS[call(good[:6] + [good[6] + 4] + good[7:])] == "DA_EALIGN"
    assert _lib.ERRORS[call(good, ws_bytes=16)] == "DA_EWORKSPACE"
    assert _lib.ERRORS[call(good[:6] + [good[0]] + good[7:])] == "DA_EINVAL"     # dq aliases q
    assert _lib.ERRORS[call(good[:7] + [good[6]] + good[8:])] == "DA_EINVAL"     # dk aliases dq
    assert _lib.ERRORS[call(good, ws=good[5])] == "DA_EINVAL"                     # workspace aliases dout
    assert _lib.ERRORS[call(good, D=40)] == "DA_EUNSUPPORTED"
    assert _lib.ERRORS[call(good, dtype=0)] == "DA_EUNSUPPORTED"


@pytest.mark.parametrize("args,code", [
    # (B, N, H, D, sign, transpose, center, base, gamma, scale_base, dtype)
    ((1, 16, 2, 12, 1, 0, 8, 1e4, 0.4, 512.0, 1), -1),      # D not a multiple of 8
    ((1, 16, 2, 264, 1, 0, 8, 1e4, 0.4, 512.0, 1), -1),     # D above 256
    ((1, 16, 2, 64, 0, 0, 8, 1e4, 0.4, 512.0, 1), -1),      # sign 0
    ((1, 16, 2, 64, 1, 2, 8, 1e4, 0.4, 512.0, 1), -1),      # transpose 2
    ((1, 16, 2, 64, 1, 0, 16, 1e4, 0.4, 512.0, 1), -1),     # center outside [0, N)
    ((1, 16, 2, 64, 1, 0, 8, 1.0, 0.4, 512.0, 1), -1),      # base <= 1
    ((1, 16, 2, 64, 1, 0, 8, 1e4, 0.0, 512.0, 1), -1),      # gamma <= 0
    ((1, 16, 2, 64, 1, 0, 8, 1e4, 0.4, float("nan"), 1), -1),
    ((1, 40000, 1, 64, 1, 0, 20000, 1e4, 0.4, 512.0, 1), -1),  # scale exponents beyond 64
    ((1, 16, 2, 64, 1, 0, 8, 1e4, 0.4, 512.0, 7), -2),      # unknown dtype
    ((0, 16, 2, 64, 1, 0, 8, 1e4, 0.4, 512.0, 1), -1),
    ((2, 1 << 30, 2, 8, 1, 0, 8, 1e4, 0.4, 512.0, 1), -1),  # 2^35 elements: beyond a 32-bit grid
])
def test_xpos_rejects_bad_arguments(lib, args, code):
    """Argument checks come before any launch: dummy pointers are never used."""
    assert lib.dilated_attn_xpos(256, 512, *args, None) == code


def test_wgrad_workspace_sizes(lib):
    """Splits of the reduction: at most 512 workgroups of 128 x 128 output
    tiles, whole 64-row k tiles per split, none for an empty reduction."""
    import ctypes
    out = ctypes.c_uint64(0)

    def ws(K, M, N):
        rc = lib.dilated_attn_wgrad_workspace(K, M, N, ctypes.byref(out))
        return rc if rc else out.value

    # float32 partials of dw per split, then of db per slice of 256 rows (at most 1024 slices)
    assert ws(0, 768, 768) == 0
    assert ws(1, 768, 768) == (768 + 1) * 768 * 4                # one k tile: one split, one slice
    assert ws(32768, 768, 768) == (14 * 768 + 128) * 768 * 4     # 36 tiles x 14 splits = 504 workgroups
    assert ws(64 * 100, 128, 128) == (100 * 128 + 25) * 128 * 4  # 512 splits capped at the 100 k tiles
    assert ws(1 << 20, 16384, 16384) == (16384 + 1024) * 16384 * 4  # more tiles than 512: one split
    for bad in ((-1, 128, 128), (64, 100, 128), (64, 128, 0), (64, 128, 16512), ((1 << 30) + 1, 128, 128)):
        assert ws(*bad) == -1, bad


@pytest.mark.parametrize("args,code", [
    # (K, M, N, dtype, workspace, workspace_bytes)
    ((64, 100, 128, 1, 4096, 1 << 20), -1),          # M not a multiple of 128
    ((64, 128, 128, 0, 4096, 1 << 20), -2),          # float32: no kernel
    ((64, 128, 128, 1, 4096, 16), -3),               # workspace too small
    ((64, 128, 128, 1, None, 1 << 20), -1),          # no workspace
    ((64, 128, 128, 1, 4100, 1 << 20), -4),          # workspace misaligned
    ((64, 128, 128, 1, 512, 1 << 20), -1),           # workspace overlaps x
])
def test_wgrad_rejects_bad_arguments(lib, args, code):
    """Argument checks come before any launch: dummy pointers are never used.
    dy at 256, x at 512, dw at 1 << 24 and db at 1 << 25 (sizes small enough
    not to meet)."""
    K, M, N, dtype, ws, wsb = args
    assert lib.dilated_attn_wgrad(256, 512, 1 << 24, 1 << 25, K, M, N, dtype, ws, wsb, None) == code


def test_wgrad_rejects_overlapping_bias_gradient(lib):
    assert lib.dilated_attn_wgrad(256, 512, 1 << 24, (1 << 24) + 64, 64, 128, 128, 1, 1 << 26, 1 << 20, None) == -1
    assert lib.dilated_attn_wgrad(256, 512, 1 << 24, 1 << 25, 64, 128, 128, 1, 1 << 25, 1 << 20, None) == -1
    assert lib.dilated_attn_wgrad(256, 512, 1 << 24, (1 << 25) + 8, 64, 128, 128, 1, 1 << 26, 1 << 20, None) == -4


@pytest.mark.parametrize("args,code", [
    # (x, g, b, y, mean, rstd, rows, E, eps, dtype)
    ((256, 1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, 4, 12, 1e-5, 1), -1),      # E not a multiple of 8
    ((256, 1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, 4, 2056, 1e-5, 1), -1),    # E above 2048
    ((256, 1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, 4, 64, 0.0, 1), -1),       # eps 0
    ((256, 1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, 4, 64, 1e-5, 0), -2),      # float32: no kernel
    ((264, 1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, 4, 64, 1e-5, 1), -4),      # x misaligned
    ((256, 1 << 20, 1 << 21, 512, 1 << 23, 1 << 24, 4, 64, 1e-5, 1), -1),          # y overlaps x
    ((256, 1 << 20, 1 << 21, 1 << 22, 1 << 22, 1 << 24, 4, 64, 1e-5, 1), -1),      # mean overlaps y
    ((256, 1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, -1, 64, 1e-5, 1), -1),     # negative rows
    ((256, 1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, (1 << 26) + 1, 8, 1e-5, 1), -1),  # beyond 2^26 rows
])
def test_layernorm_fwd_rejects_bad_arguments(lib, args, code):
    """Argument checks come before any launch: dummy pointers are never used."""
    assert lib.dilated_attn_layernorm_fwd(*args, None) == code


def test_layernorm_bwd_workspace_and_errors(lib):
    import ctypes
    out = ctypes.c_uint64(0)
    assert lib.dilated_attn_layernorm_bwd_workspace(32768, 768, ctypes.byref(out)) == 0
    assert out.value == (1024 + 32) * 2 * 768 * 4         # 1024 workgroups of 32 rows, 32 slices of 32
    assert lib.dilated_attn_layernorm_bwd_workspace(0, 768, ctypes.byref(out)) == 0 and out.value == 0
    assert lib.dilated_attn_layernorm_bwd_workspace(64, 20, ctypes.byref(out)) == -1
    # dy, x, g, mean, rstd, dx, dg, db at disjoint dummy addresses; rows 4, E 64
    ptrs = [1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, 1 << 25, 1 << 26, 1 << 27]
    ws = 1 << 28
    call = lambda p, w=ws, wb=1 << 20, dtype=1: lib.dilated_attn_layernorm_bwd(*p, 4, 64, dtype, w, wb, None)  # noqa: E731
    assert call(ptrs, wb=16) == -3                                      # workspace too small
    assert call(ptrs, dtype=0) == -2
    assert call(ptrs[:5] + [ptrs[0]] + ptrs[6:]) == -1                  # dx aliases dy
    assert call(ptrs, w=ptrs[6]) == -1                                  # workspace aliases dg
    assert call(ptrs, w=None) == -1
