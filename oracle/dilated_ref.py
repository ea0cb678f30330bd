"""Step-by-step fp64 oracle of dilated attention (LongNet, Sec. 2.2-2.3).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg; the product path never uses it.

Tensors are laid out [B, N, H, D] (batch, sequence position, head, head dim),
and the combined log-sum-exp is [B, H, N].  Each function follows one step of
the method in the paper's order:

  1. segment the sequence into pieces of length w      (Sec. 2.2, Eqs. 3-5, 8)
  2. keep every r-th row, starting at the head offset  (Sec. 2.3, offset s_j)
  3. dense softmax attention inside each sparsified    (Sec. 2.2, Eq. 6)
     segment, producing the output and log-sum-exp
  4. scatter back (zeros on unselected rows) and mix   (Sec. 2.2, Eqs. 7, 9, 10)
     the patterns with weights proportional to each
     pattern's softmax denominator

Readings of points the paper leaves open (each one is also listed with its
reason in the design notes):
  * scale: scores are multiplied by 1/sqrt(D) unless a scale is given (the
    paper's Eq. 1 and Eq. 6 print no scale; the operator is a drop-in for
    standard attention, which uses 1/sqrt(D));
  * causal: when causal, a query sees the keys of its sparsified segment at or
    before its own position (the model is a decoder language model, Sec. 4.1);
  * the offset is segment-local: segment g of pattern (w, r) keeps rows
    p in [g*w, min((g+1)*w, N)) with (p - g*w) mod r == h mod r (the first
    selected row is Q_{iw+s_j}, Sec. 2.3); heads are numbered from 0;
  * a last segment shorter than w (N not a multiple of w) is truncated;
  * the weight s_i is the unshifted softmax denominator, exp(lse_i); a pattern
    that does not select a row contributes s_i = 0 there;
  * keys seen through several patterns count once per pattern (the mixture is
    one softmax over the multiset of keys, Sec. 2.2 after Eq. 10);
  * a row that no pattern selects gets out = 0 and lse = -inf.
"""
from __future__ import annotations

import math
from typing import Iterable, List, Sequence, Tuple

import numpy as np

Pattern = Tuple[int, int]   # (w, r): segment length, dilation rate


def default_scale(D: int) -> float:
    """Softmax scale used when none is given: 1/sqrt(D)."""
    return 1.0 / math.sqrt(D)


def head_offset(h: int, r: int) -> int:
    """Row offset of head h inside each segment: s_h = h mod r (Sec. 2.3)."""
    return h % r


def num_segments(N: int, w: int) -> int:
    """Number of segments of length w covering N rows (Sec. 2.2, Eq. 8)."""
    return -(-N // w)


def segment_bounds(g: int, w: int, N: int) -> Tuple[int, int]:
    """Half-open row range [start, end) of segment g (Sec. 2.2, Eqs. 3-5)."""
    start = g * w
    return start, min(start + w, N)


def index_set(N: int, w: int, r: int, h: int, g: int) -> np.ndarray:
    """Sequence positions kept by pattern (w, r) for head h in segment g.

    Every r-th row of the segment, starting at the head's offset (Sec. 2.2
    Eqs. 3-5 with the offset of Sec. 2.3).  May be empty when the offset is
    past the end of a short last segment.
    """
    start, end = segment_bounds(g, w, N)
    return np.arange(start + head_offset(h, r), end, r, dtype=np.int64)


def attend(qt: np.ndarray, kt: np.ndarray, vt: np.ndarray, causal: bool,
           scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Dense softmax attention on one sparsified segment (Sec. 2.2, Eq. 6).

    qt, kt, vt are [L, D] float64 (the gathered rows, in sequence order).
    Returns (o, lse): o = softmax(scale * qt kt^T) vt as [L, D] and the
    natural-log log-sum-exp of each row's scores as [L].  With causal=True
    key t' is visible to query t only when t' <= t.
    """
    L = qt.shape[0]
    S = scale * (qt @ kt.T)
    if causal:
        S = np.where(np.tril(np.ones((L, L), dtype=bool)), S, -np.inf)
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    denom = E.sum(axis=1, keepdims=True)
    o = (E @ vt) / denom
    lse = m[:, 0] + np.log(denom[:, 0])
    return o, lse


def per_pattern_ref(q, k, v, pattern: Pattern, causal: bool, scale: float,
                    heads: Iterable[int] | None = None):
    """Output of one dilated pattern, scattered back to full length.

    Returns (O_i [B,N,H,D], LSE_i [B,H,N], cov_i [B,N,H] bool).  Rows the
    pattern does not select hold 0 in O_i (Sec. 2.2, Eq. 7) and -inf in
    LSE_i (their softmax denominator is 0).  `heads` restricts the work to a
    subset of heads (the others stay uncovered).
    """
    w, r = pattern
    B, N, H, D = q.shape
    O = np.zeros((B, N, H, D), dtype=np.float64)
    LSE = np.full((B, H, N), -np.inf, dtype=np.float64)
    cov = np.zeros((B, N, H), dtype=bool)
    hs = range(H) if heads is None else heads
    for b in range(B):
        for h in hs:
            for g in range(num_segments(N, w)):
                idx = index_set(N, w, r, h, g)
                if idx.size == 0:
                    continue
                o, lse = attend(q[b, idx, h, :], k[b, idx, h, :],
                                v[b, idx, h, :], causal, scale)
                O[b, idx, h, :] = o
                LSE[b, h, idx] = lse
                cov[b, idx, h] = True
    return O, LSE, cov


def combine_ref(Os: Sequence[np.ndarray], LSEs: Sequence[np.ndarray]):
    """Mix per-pattern outputs by their softmax denominators (Eqs. 9-10).

    Os[i] is [B,N,H,D] with zeros on rows pattern i does not select; LSEs[i]
    is [B,H,N] with -inf there.  With s_i = exp(LSE_i), the weights are
    alpha_i = s_i / sum_j s_j, out = sum_i alpha_i O_i and the combined
    lse = log(sum_i s_i).  Rows with every s_i = 0 give out = 0, lse = -inf.
    """
    L = np.stack(LSEs, axis=0)                         # [k, B, H, N]
    m = L.max(axis=0)                                  # [B, H, N]
    covered = np.isfinite(m)
    m_safe = np.where(covered, m, 0.0)
    w = np.exp(L - m_safe[None])                       # s_i / exp(m); 0 if uncovered
    total = w.sum(axis=0)                              # sum_j s_j / exp(m)
    lse = np.where(covered, m_safe + np.log(np.where(covered, total, 1.0)), -np.inf)
    alpha = np.where(covered[None], w / np.where(covered, total, 1.0)[None], 0.0)
    out = np.zeros_like(Os[0])
    for i, O in enumerate(Os):
        out += np.transpose(alpha[i], (0, 2, 1))[..., None] * O   # [B,N,H,1]
    return out, lse


def dilated_attention_ref(q, k, v, patterns: Sequence[Pattern], causal: bool = True,
                          scale: float | None = None, heads: Iterable[int] | None = None):
    """Full dilated-attention forward: every pattern, then the mixture.

    q, k, v: [B, N, H, D] arrays (converted to float64).  Returns
    (out [B,N,H,D] float64, lse [B,H,N] float64).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    if scale is None:
        scale = default_scale(q.shape[3])
    Os, LSEs = [], []
    for pat in patterns:
        O, LSE, _ = per_pattern_ref(q, k, v, pat, causal, scale, heads)
        Os.append(O)
        LSEs.append(LSE)
    return combine_ref(Os, LSEs)


def dilated_attention_rows_ref(q, k, v, patterns: Sequence[Pattern], causal: bool,
                               scale: float | None, rows: Sequence[Tuple[int, int, int]]):
    """Oracle output for selected (b, p, h) rows only.

    The same steps as dilated_attention_ref, restricted to the queries named in
    `rows`: for each pattern the row's segment and index set are formed, the
    row's scores against the visible keys of that set give (o_i, lse_i), and
    the patterns are mixed by their denominators.  q, k, v may be any array
    type indexable as [b, p, h, :] (for example torch CPU tensors); rows are
    gathered one segment at a time.  Returns (out [R, D], lse [R]) float64.
    """
    B, N, H, D = q.shape
    if scale is None:
        scale = default_scale(D)
    R = len(rows)
    out = np.zeros((R, D), dtype=np.float64)
    lse = np.full(R, -np.inf, dtype=np.float64)
    per_row: List[List[Tuple[float, np.ndarray]]] = [[] for _ in range(R)]
    # group requested rows by (pattern, b, h, segment) so each segment is gathered once
    groups = {}
    for ridx, (b, p, h) in enumerate(rows):
        for pi, (w, r) in enumerate(patterns):
            g = p // w
            start, _ = segment_bounds(g, w, N)
            if (p - start) % r != head_offset(h, r):
                continue
            groups.setdefault((pi, b, h, g), []).append(ridx)
    for (pi, b, h, g), ridxs in groups.items():
        w, r = patterns[pi]
        idx = index_set(N, w, r, h, g)
        kt = _rows(k, b, idx, h)
        vt = _rows(v, b, idx, h)
        for ridx in ridxs:
            p = rows[ridx][1]
            t = int(np.searchsorted(idx, p))
            qt = _rows(q, b, idx[t:t + 1], h)
            n_vis = t + 1 if causal else idx.size
            srow = scale * (qt @ kt[:n_vis].T)[0]
            m = srow.max()
            e = np.exp(srow - m)
            den = e.sum()
            per_row[ridx].append((m + math.log(den), (e @ vt[:n_vis]) / den))
    for ridx, parts in enumerate(per_row):
        if not parts:
            continue
        ls = np.array([p[0] for p in parts])
        m = ls.max()
        tot = np.exp(ls - m).sum()
        lse[ridx] = m + math.log(tot)
        for l_i, o_i in parts:
            out[ridx] += math.exp(l_i - lse[ridx]) * o_i
    return out, lse


def _rows(x, b, idx, h):
    """Gather rows x[b, idx, h, :] as float64 NumPy."""
    sel = x[b, idx, h, :] if isinstance(x, np.ndarray) else x[b, idx.tolist(), h, :]
    if not isinstance(sel, np.ndarray):
        sel = sel.double().numpy() if hasattr(sel, "double") else np.asarray(sel)
    return np.asarray(sel, dtype=np.float64)
