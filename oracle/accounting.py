"""Work accounting of dilated attention by explicit enumeration.

TEST INFRASTRUCTURE ONLY.

Counts what the method must compute (Sec. 2.4): every (query, key) pair that
is unmasked inside a sparsified segment costs 2*D flops for the scores and
2*D for the weighted sum of values, i.e. 4*D per pair.  With a causal mask a
segment of L kept rows has L(L+1)/2 pairs, without one L^2.  Used to pin the
library's own accounting and the paper's closed-form FLOP estimates.
"""
from __future__ import annotations

from typing import Sequence, Tuple

from .dilated_ref import index_set, num_segments


def exact_causal_pairs(N: int, H: int, patterns: Sequence[Tuple[int, int]],
                       causal: bool = True) -> int:
    """Number of unmasked (query, key) pairs over all heads, patterns, segments (B=1)."""
    total = 0
    for (w, r) in patterns:
        for h in range(H):
            for g in range(num_segments(N, w)):
                L = index_set(N, w, r, h, g).size
                total += L * (L + 1) // 2 if causal else L * L
    return total


def covered_rows(N: int, H: int, patterns: Sequence[Tuple[int, int]]) -> int:
    """Sum over patterns of the number of (row, head) results they produce (B=1)."""
    total = 0
    for (w, r) in patterns:
        for h in range(H):
            for g in range(num_segments(N, w)):
                total += index_set(N, w, r, h, g).size
    return total


def sparse_flops(B: int, N: int, H: int, D: int, patterns, causal=True) -> int:
    """Exact flops of the method: 4*D per unmasked pair.

    Sec. 2.4 estimates one pattern at 2*N*w*d/r^2, i.e. 2*L^2*d per segment of
    L = w/r rows, which is the causal count L^2/2 pairs x 4*d without the
    diagonal; the exact causal count adds 2*d per kept row."""
    return 4 * D * B * exact_causal_pairs(N, H, patterns, causal)
