"""Helpers shared by the GPU tests: running the HIP path and the oracle on the
same seeded inputs and comparing them."""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle
import workloads

TOL = {"bf16": (2e-2, 1e-2), "f32": (1e-4, 1e-4)}   # (out max-abs, lse max-abs)


def note(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("this test needs the MI355X: no HIP device visible")
    from paper_2307_02486_amd import _lib
    _lib.load()


def run_gpu(q, k, v, patterns, causal=True, scale=None, canary=True):
    from paper_2307_02486_amd import dilated_attn
    B, N, H, D = q.shape
    out = lse = None
    if canary:
        out = torch.full_like(q, float("nan"))
        lse = torch.full((B, H, N), float("nan"), dtype=torch.float32, device=q.device)
    out, lse = dilated_attn(q, k, v, patterns, causal, scale, out=out, lse=lse)
    torch.cuda.synchronize()
    return out, lse


def to64(x: torch.Tensor) -> np.ndarray:
    return x.detach().to("cpu", torch.float64).numpy()


def compare_full(q, k, v, patterns, causal, dtype_key, scale=None, tag="", heads=None, gpu=None, tol=None):
    """GPU vs oracle on every row (of `heads`, default all); returns (max out
    err, max lse err).  `tol` = (out bar, lse bar) replaces the dtype's bars."""
    out, lse = gpu if gpu is not None else run_gpu(q, k, v, patterns, causal, scale)
    ro, rl = oracle.dilated_attention_ref(to64(q), to64(k), to64(v), patterns, causal, scale, heads=heads)
    go, gl = to64(out), to64(lse)
    if heads is not None:
        hs = list(heads)
        ro, rl, go, gl = ro[:, :, hs], rl[:, hs], go[:, :, hs], gl[:, hs]
    assert not np.isnan(go).any(), f"{tag}: NaN in out (row not written?)"
    assert not np.isnan(gl).any(), f"{tag}: NaN in lse (row not written?)"
    fin = np.isfinite(rl)
    assert np.array_equal(fin, np.isfinite(gl)), f"{tag}: covered-row sets differ"
    assert np.all(go[~np.transpose(fin, (0, 2, 1))] == 0), f"{tag}: uncovered rows must be 0"
    eo = float(np.abs(go - ro).max()) if go.size else 0.0
    el = float(np.abs(gl[fin] - rl[fin]).max()) if fin.any() else 0.0
    to, tl = TOL[dtype_key] if tol is None else tol
    assert eo <= to, f"{tag}: out max-abs err {eo} > {to}"
    assert el <= tl, f"{tag}: lse max-abs err {el} > {tl}"
    return eo, el


def sample_rows(wl, rng: np.random.Generator, per_head: int):
    """Rows (b, p, h) to check at full size: random rows plus the first and
    last row, the ends of the largest pattern's segments and rows kept by the
    most patterns."""
    N, H = wl.N, wl.H
    wmax = max(w for w, _ in wl.patterns)
    rows = set()
    for b in range(wl.B):
        for h in range(H):
            ps = set(rng.integers(0, N, per_head).tolist())
            ps.update({0, N - 1})
            for st in range(0, N, min(wmax, N)):
                ps.update({st, min(st + wmax, N) - 1})
            lo = int(rng.integers(0, max(1, N - 4096)))
            cand = np.arange(lo, min(N, lo + 4096))
            cnt = np.zeros(cand.size, int)
            for (w, r) in wl.patterns:
                cnt += ((cand % w) % r) == (h % r)
            best = cand[cnt == cnt.max()][:8]
            ps.update(best.tolist())
            rows.update((b, int(p), h) for p in ps)
    return sorted(rows)


def compare_rows(q, k, v, out, lse, wl, rows, scale=None, tag=""):
    qc, kc, vc = q.cpu(), k.cpu(), v.cpu()
    ro, rl = oracle.dilated_attention_rows_ref(qc, kc, vc, wl.patterns, wl.causal, scale, rows)
    bi = torch.tensor([r[0] for r in rows])
    pi = torch.tensor([r[1] for r in rows])
    hi = torch.tensor([r[2] for r in rows])
    go = out[bi.cuda(), pi.cuda(), hi.cuda()].to(torch.float64).cpu().numpy()
    gl = lse[bi.cuda(), hi.cuda(), pi.cuda()].to(torch.float64).cpu().numpy()
    to, tl = TOL[wl.dtype]
    eo = float(np.abs(go - ro).max())
    el = float(np.abs(gl - rl).max())
    assert eo <= to, f"{tag}: sampled out max-abs err {eo} > {to}"
    assert el <= tl, f"{tag}: sampled lse max-abs err {el} > {tl}"
    return eo, el
