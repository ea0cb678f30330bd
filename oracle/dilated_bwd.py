"""Step-by-step fp64 oracle of the dilated-attention backward pass.

TEST INFRASTRUCTURE ONLY: imported by tests/ and the benchmark's CPU-baseline
leg; the product path never uses it.

The forward mixes the patterns by their softmax denominators (Sec. 2.2,
Eqs. 9-10), which is the same as one softmax over the multiset of (pattern,
key) pairs a query sees (Sec. 2.2, after Eq. 10).  With s = scale q.k, the
combined lse of the query and P = exp(s - lse), the output is the sum of P v
over that multiset.  The gradient of a loss with upstream gradient dout is
therefore the softmax-attention derivative taken over the multiset, one
pattern at a time (the paper's distributed algorithm has a backward pass,
Sec. 3.1):

  delta_p = sum_d dout[p, d] out[p, d]                       (per query row)
  for each pattern i, head h, segment g with kept rows idx:
      S  = scale Qt Kt^T, masked as in the forward (causal: key <= query)
      P  = exp(S - lse[idx])          (lse is the COMBINED lse of the row)
      dP = dOt Vt^T
      dS = P * (dP - delta[idx])
      dq[idx] += scale dS Kt,  dk[idx] += scale dS^T Qt,  dv[idx] += P^T dOt

Rows a pattern does not keep receive nothing from it (Eq. 7), and a key seen
through several patterns collects one contribution per pattern.  These are
the closed-form derivatives of the forward's definition; the tests pin them
against finite differences of the forward oracle and, for the dense case,
against PyTorch's autograd of scaled-dot-product attention.
"""
from __future__ import annotations

from typing import Iterable, List, Sequence, Tuple

import numpy as np

from .dilated_ref import (Pattern, _rows, default_scale, dilated_attention_ref, dilated_attention_rows_ref,
                          head_offset, index_set, num_segments, segment_bounds)


def delta_ref(dout: np.ndarray, out: np.ndarray) -> np.ndarray:
    """delta[b, h, p] = sum_d dout[b, p, h, d] * out[b, p, h, d]  ->  [B, H, N]."""
    return np.transpose((np.asarray(dout, np.float64) * np.asarray(out, np.float64)).sum(axis=3), (0, 2, 1))


def attend_bwd(qt, kt, vt, dot, lse_t, delta_t, causal: bool, scale: float):
    """Gradients of one sparsified segment (rows in sequence order).

    qt, kt, vt, dot: [L, D]; lse_t, delta_t: [L] (the query rows' combined
    lse and delta).  Returns (dq, dk, dv), each [L, D].
    """
    L = qt.shape[0]
    S = scale * (qt @ kt.T)
    if causal:
        S = np.where(np.tril(np.ones((L, L), dtype=bool)), S, -np.inf)
    P = np.exp(S - lse_t[:, None])
    dP = dot @ vt.T
    dS = P * (dP - delta_t[:, None])
    return scale * (dS @ kt), scale * (dS.T @ qt), P.T @ dot


def dilated_attention_bwd_ref(q, k, v, dout, patterns: Sequence[Pattern], causal: bool = True,
                              scale: float | None = None, heads: Iterable[int] | None = None):
    """Backward of the full dilated attention.

    Returns (dq, dk, dv) [B,N,H,D] float64 and the forward's (out, lse).
    `heads` restricts the work to a subset of heads (the others stay 0).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    B, N, H, D = q.shape
    if scale is None:
        scale = default_scale(D)
    out, lse = dilated_attention_ref(q, k, v, patterns, causal, scale, heads)
    delta = delta_ref(dout, out)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    hs = range(H) if heads is None else heads
    for (w, r) in patterns:
        for b in range(B):
            for h in hs:
                for g in range(num_segments(N, w)):
                    idx = index_set(N, w, r, h, g)
                    if idx.size == 0:
                        continue
                    gq, gk, gv = attend_bwd(q[b, idx, h], k[b, idx, h], v[b, idx, h], dout[b, idx, h],
                                            lse[b, h, idx], delta[b, h, idx], causal, scale)
                    dq[b, idx, h] += gq
                    dk[b, idx, h] += gk
                    dv[b, idx, h] += gv
    return dq, dk, dv, out, lse


def _rows_of(x, b, idx, h):
    """Rows x[b, idx, h, :] as float64 NumPy (x a NumPy array or a CPU tensor)."""
    return _rows(x, b, np.asarray(idx, dtype=np.int64), h)


def _kept_position(p: int, w: int, r: int, h: int):
    """(segment, index within the kept rows) of position p under pattern
    (w, r) for head h, or None when the pattern does not keep p."""
    g = p // w
    start, _ = segment_bounds(g, w, 1 << 62)
    if (p - start) % r != head_offset(h, r):
        return None
    return g, (p - start) // r


def dq_rows_ref(q, k, v, dout, patterns: Sequence[Pattern], causal: bool, scale: float | None,
                rows: Sequence[Tuple[int, int, int]]) -> np.ndarray:
    """dq for selected query rows (b, p, h) only: [R, D] float64."""
    B, N, H, D = q.shape
    if scale is None:
        scale = default_scale(D)
    out, lse = dilated_attention_rows_ref(q, k, v, patterns, causal, scale, rows)
    res = np.zeros((len(rows), D), dtype=np.float64)
    for ri, (b, p, h) in enumerate(rows):
        qp = _rows_of(q, b, [p], h)[0]
        dop = _rows_of(dout, b, [p], h)[0]
        delta = float(dop @ out[ri])
        for (w, r) in patterns:
            kp = _kept_position(p, w, r, h)
            if kp is None:
                continue
            g, t = kp
            idx = index_set(N, w, r, h, g)
            vis = idx[:t + 1] if causal else idx
            kt, vt = _rows_of(k, b, vis, h), _rows_of(v, b, vis, h)
            P = np.exp(scale * (kt @ qp) - lse[ri])
            dS = P * (vt @ dop - delta)
            res[ri] += scale * (dS @ kt)
    return res


def dkdv_rows_ref(q, k, v, dout, patterns: Sequence[Pattern], causal: bool, scale: float | None,
                  rows: Sequence[Tuple[int, int, int]]):
    """dk and dv for selected key rows (b, p, h) only: two [R, D] float64.

    A key row collects, for every pattern keeping it, the contributions of
    the queries of its sparsified segment that see it; their combined lse
    and delta come from the forward oracle on those query rows.
    """
    B, N, H, D = q.shape
    if scale is None:
        scale = default_scale(D)
    # every (pattern, key row) -> the query rows that see it
    plan: List[Tuple[int, int, np.ndarray]] = []
    needed = set()
    for ri, (b, p, h) in enumerate(rows):
        for (w, r) in patterns:
            kp = _kept_position(p, w, r, h)
            if kp is None:
                continue
            g, t = kp
            idx = index_set(N, w, r, h, g)
            qs = idx[t:] if causal else idx
            plan.append((ri, b, h, qs))
            needed.update((b, int(x), h) for x in qs)
    needed = sorted(needed)
    out, lse = dilated_attention_rows_ref(q, k, v, patterns, causal, scale, needed)
    where = {row: i for i, row in enumerate(needed)}
    dk = np.zeros((len(rows), D), dtype=np.float64)
    dv = np.zeros((len(rows), D), dtype=np.float64)
    for ri, b, h, qs in plan:
        p = rows[ri][1]
        kp = _rows_of(k, b, [p], h)[0]
        vp = _rows_of(v, b, [p], h)[0]
        sel = np.array([where[(b, int(x), h)] for x in qs])
        qt = _rows_of(q, b, qs, h)
        dot = _rows_of(dout, b, qs, h)
        delta = np.einsum("rd,rd->r", dot, out[sel])
        P = np.exp(scale * (qt @ kp) - lse[sel])
        dS = P * (dot @ vp - delta)
        dk[ri] += scale * (dS @ qt)
        dv[ri] += P @ dot
    return dk, dv
