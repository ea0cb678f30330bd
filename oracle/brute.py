"""Brute-force constructions of dilated attention, for tiny inputs only.

TEST INFRASTRUCTURE ONLY (imported by tests/ and nothing in the product path).

These two functions compute the same operator as dilated_ref by different
routes, so the three can be checked against each other:

* brute_mask_ref builds, for every pattern and head, the N x N 0/1 pattern
  matrix of the sparse-attention form (Sec. 2.1, Eq. 2) from a membership
  predicate, runs masked softmax attention over all N keys, and mixes the
  patterns with s_i = exp(lse_i) directly (no max shifting);
* brute_multiset_ref follows the remark after Eq. 10 (Sec. 2.2): for each
  query it lists the keys of every pattern that selects it, keeping
  duplicates, and takes one softmax over that list.

Neither uses the segment/arange enumeration of dilated_ref.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np


def _selected(p: int, w: int, r: int, h: int) -> bool:
    """Does pattern (w, r) keep row p for head h?  (segment-local offset h mod r)"""
    return (p % w) % r == h % r


def _visible(p: int, kp: int, w: int, r: int, h: int, causal: bool) -> bool:
    """Is key row kp visible to query row p under pattern (w, r), head h?"""
    return (p // w == kp // w and _selected(p, w, r, h) and _selected(kp, w, r, h)
            and (not causal or kp <= p))


def visible_multiset(N: int, patterns: Sequence[Tuple[int, int]], h: int, p: int,
                     causal: bool) -> List[int]:
    """Key positions query p of head h attends to, one entry per pattern that sees it."""
    keys: List[int] = []
    for (w, r) in patterns:
        for kp in range(N):
            if _visible(p, kp, w, r, h, causal):
                keys.append(kp)
    return keys


def brute_mask_ref(q, k, v, patterns, causal=True, scale=None):
    """Mask-matrix construction (Sec. 2.1 Eq. 2 per pattern, then Eqs. 9-10)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, N, H, D = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    num = np.zeros((B, N, H, D))
    den = np.zeros((B, N, H))
    pos = np.arange(N)
    for (w, r) in patterns:
        for h in range(H):
            sel = (pos % w) % r == h % r
            same_seg = (pos[:, None] // w) == (pos[None, :] // w)
            M = same_seg & sel[:, None] & sel[None, :]
            if causal:
                M &= pos[None, :] <= pos[:, None]
            for b in range(B):
                S = scale * q[b, :, h, :] @ k[b, :, h, :].T
                for p in range(N):
                    if not M[p].any():
                        continue
                    e = np.exp(S[p][M[p]])            # unshifted: s_i = sum e
                    s_i = e.sum()
                    o_i = (e @ v[b, M[p], h, :]) / s_i
                    num[b, p, h] += s_i * o_i
                    den[b, p, h] += s_i
    out = np.where(den[..., None] > 0, num / np.where(den > 0, den, 1.0)[..., None], 0.0)
    lse = np.where(den > 0, np.log(np.where(den > 0, den, 1.0)), -np.inf)
    return out, np.transpose(lse, (0, 2, 1))


def brute_multiset_ref(q, k, v, patterns, causal=True, scale=None):
    """One softmax per query over the multiset of keys of all patterns (Sec. 2.2)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, N, H, D = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    out = np.zeros((B, N, H, D))
    lse = np.full((B, H, N), -np.inf)
    for h in range(H):
        for p in range(N):
            keys = visible_multiset(N, patterns, h, p, causal)
            if not keys:
                continue
            for b in range(B):
                scores = [scale * float(np.dot(q[b, p, h], k[b, kp, h])) for kp in keys]
                m = max(scores)
                ws = [math.exp(s - m) for s in scores]
                tot = sum(ws)
                acc = np.zeros(D)
                for wgt, kp in zip(ws, keys):
                    acc += wgt * v[b, kp, h]
                out[b, p, h] = acc / tot
                lse[b, h, p] = m + math.log(tot)
    return out, lse
