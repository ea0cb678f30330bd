"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these compares the oracle with itself: each check uses an independent
construction (hand-derived fixture, library attention, closed form, invariant,
or brute force over explicit pattern matrices).
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import (brute_mask_ref, brute_multiset_ref, combine_ref,
                    dilated_attention_ref, index_set, per_pattern_ref)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# --- P1: index sets --------------------------------------------------------

def _load_multisets():
    rows = {}
    with open(os.path.join(GOLDEN, "tiny_multisets.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            left, right = line.split(":")
            h, p = map(int, left.split())
            rows[(h, p)] = sorted(map(int, right.split()))
    return rows


TINY_PATTERNS = [(4, 1), (6, 2), (10, 3)]


def test_golden_multisets_brute_predicate():
    """The membership predicate reproduces the hand-derived multisets."""
    gold = _load_multisets()
    assert len(gold) == 30
    for (h, p), keys in gold.items():
        assert sorted(oracle.visible_multiset(10, TINY_PATTERNS, h, p, True)) == keys


def test_golden_multisets_q_zero_oracle():
    """q = 0 and one-hot v: out is the multiplicity of each key over the
    multiset size and lse = ln(size), exactly as the fixture says."""
    gold = _load_multisets()
    N, H, D = 10, 3, 10
    q = np.zeros((1, N, H, D))
    k = rnd((1, N, H, D), 1)
    v = np.zeros((1, N, H, D))
    for p in range(N):
        v[0, p, :, p] = 1.0
    out, lse = dilated_attention_ref(q, k, v, TINY_PATTERNS, causal=True)
    for (h, p), keys in gold.items():
        expect = np.bincount(keys, minlength=N) / len(keys)
        np.testing.assert_allclose(out[0, p, h], expect, atol=1e-14)
        assert abs(lse[0, h, p] - math.log(len(keys))) < 1e-14


def test_index_sets_match_predicate():
    """arange-based index sets == brute-force membership predicate."""
    rng = np.random.default_rng(3)
    for _ in range(200):
        N = int(rng.integers(1, 40))
        w = int(rng.integers(1, 50))
        r = int(rng.integers(1, w + 1))
        h = int(rng.integers(0, 20))
        g_all = set()
        for g in range(oracle.num_segments(N, w)):
            idx = index_set(N, w, r, h, g)
            assert np.all(np.diff(idx) == r)
            brute = [p for p in range(N) if p // w == g and (p % w) % r == h % r]
            assert idx.tolist() == brute
            g_all.update(idx.tolist())
        # over r consecutive heads every row is selected exactly once
    for N, w, r in [(37, 12, 5), (64, 16, 4), (20, 20, 7)]:
        count = np.zeros(N, int)
        for h in range(r):
            for g in range(oracle.num_segments(N, w)):
                count[index_set(N, w, r, h, g)] += 1
        assert np.all(count == 1)


def test_ragged_length_counts():
    """(16384, 6) with 12 heads: lengths 2731 for offsets 0..3 and 2730 for
    4..5; a full cycle of offsets covers the segment once."""
    N, w, r = 32768, 16384, 6
    Ls = [index_set(N, w, r, h, 0).size for h in range(12)]
    assert Ls == [2731, 2731, 2731, 2731, 2730, 2730] * 2
    assert sum(Ls[:6]) == w


# --- P2/P3: attention core ------------------------------------------------

def _sdpa(q, k, v, causal, scale):
    """torch float64 SDPA on [L, D] arrays (library routine, independent)."""
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x))[None, None]
    o = torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), is_causal=causal, scale=scale)
    return o[0, 0].numpy()


@pytest.mark.parametrize("causal", [True, False])
def test_dense_special_case(causal):
    """One pattern with w = N, r = 1 is ordinary softmax attention (Eq. 1)."""
    B, N, H, D = 2, 33, 3, 8
    q, k, v = rnd((B, N, H, D), 10), rnd((B, N, H, D), 11), rnd((B, N, H, D), 12)
    out, lse = dilated_attention_ref(q, k, v, [(N, 1)], causal=causal)
    scale = 1 / math.sqrt(D)
    for b in range(B):
        for h in range(H):
            ref = _sdpa(q[b, :, h], k[b, :, h], v[b, :, h], causal, scale)
            np.testing.assert_allclose(out[b, :, h], ref, atol=1e-12)
            s = torch.from_numpy(scale * q[b, :, h] @ k[b, :, h].T)
            if causal:
                s = s.masked_fill(torch.triu(torch.ones(N, N, dtype=torch.bool), 1), -math.inf)
            np.testing.assert_allclose(lse[b, h], torch.logsumexp(s, dim=1).numpy(), atol=1e-12)


def test_segment_special_case():
    """(w, 1) is block-diagonal causal attention (Sparse Transformer local
    pattern of Sec. 2.1), including a truncated last block."""
    B, N, H, D, w = 1, 45, 2, 4, 16
    q, k, v = rnd((B, N, H, D), 20), rnd((B, N, H, D), 21), rnd((B, N, H, D), 22)
    out, _ = dilated_attention_ref(q, k, v, [(w, 1)], causal=True, scale=0.7)
    for h in range(H):
        for st in range(0, N, w):
            en = min(st + w, N)
            ref = _sdpa(q[0, st:en, h], k[0, st:en, h], v[0, st:en, h], True, 0.7)
            np.testing.assert_allclose(out[0, st:en, h], ref, atol=1e-12)


def test_dilated_single_pattern_against_sdpa_on_gathered_rows():
    """(w, r) equals SDPA applied to the rows picked by the predicate."""
    B, N, H, D, w, r = 1, 50, 5, 6, 20, 3
    q, k, v = rnd((B, N, H, D), 30), rnd((B, N, H, D), 31), rnd((B, N, H, D), 32)
    out, lse = dilated_attention_ref(q, k, v, [(w, r)], causal=True)
    for h in range(H):
        for g in range(3):
            rows = [p for p in range(N) if p // w == g and (p % w) % r == h % r]
            ref = _sdpa(q[0, rows, h], k[0, rows, h], v[0, rows, h], True, 1 / math.sqrt(D))
            np.testing.assert_allclose(out[0, rows, h], ref, atol=1e-12)
        unsel = [p for p in range(N) if (p % w) % r != h % r]
        assert np.all(out[0, unsel, h] == 0) and np.all(np.isneginf(lse[0, h, unsel]))


# --- P4: combine ------------------------------------------------------------

def test_combine_disjoint_partition():
    """Attend over disjoint parts of a key list and mix by denominators ==
    softmax attention over the whole list."""
    rng = np.random.default_rng(40)
    D, nk = 7, 23
    qv = rng.standard_normal(D)
    K = rng.standard_normal((nk, D))
    V = rng.standard_normal((nk, D))
    scores = K @ qv
    full_w = np.exp(scores - scores.max())
    full_out = (full_w / full_w.sum()) @ V
    full_lse = np.log(np.exp(scores).sum())
    for parts in (2, 3, 5):
        perm = rng.permutation(nk)
        chunks = np.array_split(perm, parts)
        Os, Ls = [], []
        for c in chunks:
            s = scores[c]
            e = np.exp(s - s.max())
            Os.append(((e / e.sum()) @ V[c]).reshape(1, 1, 1, D))
            Ls.append(np.array([[[s.max() + np.log(e.sum())]]]))
        # one pattern that covers nothing
        Os.append(np.zeros((1, 1, 1, D)))
        Ls.append(np.array([[[-np.inf]]]))
        out, lse = combine_ref(Os, Ls)
        np.testing.assert_allclose(out[0, 0, 0], full_out, atol=1e-12)
        assert abs(lse[0, 0, 0] - full_lse) < 1e-12


def test_combine_uncovered_row():
    out, lse = combine_ref([np.ones((1, 1, 1, 3)) * 0, np.zeros((1, 1, 1, 3))],
                           [np.full((1, 1, 1), -np.inf)] * 2)
    assert np.all(out == 0) and np.isneginf(lse).all()


# --- P5/P8: three constructions agree -------------------------------------

def _random_case(rng):
    N = int(rng.integers(1, 40))
    H = int(rng.integers(1, 5))
    D = int(rng.integers(1, 6))
    k = int(rng.integers(1, 5))
    pats = []
    for _ in range(k):
        w = int(rng.integers(1, 2 * N + 2))
        r = int(rng.integers(1, min(w, 9) + 1))
        pats.append((w, r))
    if rng.random() < 0.3:
        pats.append(pats[0])      # duplicate pattern counts twice
    causal = bool(rng.random() < 0.7)
    return N, H, D, pats, causal


def test_three_constructions_agree():
    rng = np.random.default_rng(50)
    for trial in range(40):
        N, H, D, pats, causal = _random_case(rng)
        B = 1 + trial % 2
        q, k, v = rnd((B, N, H, D), 100 + trial), rnd((B, N, H, D), 200 + trial), rnd((B, N, H, D), 300 + trial)
        o1, l1 = dilated_attention_ref(q, k, v, pats, causal)
        o2, l2 = brute_mask_ref(q, k, v, pats, causal)
        o3, l3 = brute_multiset_ref(q, k, v, pats, causal)
        for o, l in ((o2, l2), (o3, l3)):
            np.testing.assert_allclose(o1, o, atol=1e-11, err_msg=f"{pats} causal={causal}")
            fin = np.isfinite(l1)
            assert np.array_equal(fin, np.isfinite(l))
            np.testing.assert_allclose(l1[fin], l[fin], atol=1e-11)


# --- P6: q = 0 closed form at a larger size ---------------------------------

def test_q_zero_closed_form():
    """q = 0: each pattern is a uniform average over its causal prefix, so
    lse = ln(sum_i (t_i + 1)) and out = (sum of visible v) / that count."""
    B, N, H, D = 1, 97, 4, 3
    pats = [(16, 1), (32, 3), (97, 5), (50, 7)]
    v = rnd((B, N, H, D), 60)
    out, lse = dilated_attention_ref(np.zeros((B, N, H, D)), rnd((B, N, H, D), 61), v, pats)
    for h in range(H):
        for p in range(N):
            cnt, acc = 0, np.zeros(D)
            for (w, r) in pats:
                st = (p // w) * w
                if (p - st) % r != h % r:
                    continue
                prefix = list(range(st + h % r, p + 1, r))
                cnt += len(prefix)
                acc += v[0, prefix, h].sum(axis=0)
            assert cnt > 0
            assert abs(lse[0, h, p] - math.log(cnt)) < 1e-13
            np.testing.assert_allclose(out[0, p, h], acc / cnt, atol=1e-13)


# --- P7: invariants ---------------------------------------------------------

def test_weights_sum_to_one_and_linearity():
    B, N, H, D = 1, 40, 3, 5
    pats = [(8, 1), (16, 2), (40, 4)]
    q, k = rnd((B, N, H, D), 70), rnd((B, N, H, D), 71)
    c = rnd((D,), 72)
    vconst = np.broadcast_to(c, (B, N, H, D)).copy()
    out, _ = dilated_attention_ref(q, k, vconst, pats)
    np.testing.assert_allclose(out, vconst, atol=1e-12)
    v1, v2 = rnd((B, N, H, D), 73), rnd((B, N, H, D), 74)
    o1, _ = dilated_attention_ref(q, k, v1, pats)
    o2, _ = dilated_attention_ref(q, k, v2, pats)
    o12, _ = dilated_attention_ref(q, k, 2 * v1 - 3 * v2, pats)
    np.testing.assert_allclose(o12, 2 * o1 - 3 * o2, atol=1e-11)
    assert np.abs(o1).max() <= np.abs(v1).max() + 1e-12


def test_scale_is_applied():
    """Scaling q by a is the same as scale a/sqrt(D)."""
    B, N, H, D = 1, 30, 2, 4
    q, k, v = rnd((B, N, H, D), 80), rnd((B, N, H, D), 81), rnd((B, N, H, D), 82)
    pats = [(10, 2), (30, 3)]
    o1, l1 = dilated_attention_ref(2.5 * q, k, v, pats)
    o2, l2 = dilated_attention_ref(q, k, v, pats, scale=2.5 / math.sqrt(D))
    np.testing.assert_allclose(o1, o2, atol=1e-12)
    np.testing.assert_allclose(l1, l2, atol=1e-12)


# --- rows oracle vs full oracle ----------------------------------------------

def test_rows_oracle_matches_brute():
    """The row-restricted oracle agrees with the mask-matrix construction."""
    rng = np.random.default_rng(90)
    for trial in range(10):
        N, H, D, pats, causal = _random_case(rng)
        B = 2
        q, k, v = rnd((B, N, H, D), 400 + trial), rnd((B, N, H, D), 500 + trial), rnd((B, N, H, D), 600 + trial)
        o2, l2 = brute_mask_ref(q, k, v, pats, causal)
        rows = [(b, p, h) for b in range(B) for p in range(N) for h in range(H)]
        o, l = oracle.dilated_attention_rows_ref(torch.from_numpy(q), torch.from_numpy(k),
                                                 torch.from_numpy(v), pats, causal, None, rows)
        for i, (b, p, h) in enumerate(rows):
            np.testing.assert_allclose(o[i], o2[b, p, h], atol=1e-11)
            if np.isfinite(l2[b, h, p]):
                assert abs(l[i] - l2[b, h, p]) < 1e-11
            else:
                assert np.isneginf(l[i])


# --- accounting ---------------------------------------------------------------

def test_flops_against_paper_formula():
    """Exact causal flops == the Sec. 2.4 estimate 2*N*d*sum(w/r^2) per head
    plus the diagonal term 2*d per kept row, when r | w and w | N."""
    N, H, D = 4096, 4, 64
    pats = [(256, 1), (512, 2), (1024, 4), (4096, 8)]
    exact = oracle.sparse_flops(1, N, H, D, pats)
    paper = H * 2 * N * D * sum(w / r ** 2 for w, r in pats)
    diag = 2 * D * oracle.covered_rows(N, H, pats)
    assert exact == paper + diag
    # geometric schedule bound of Sec. 2.4 with alpha = 2, w0 = 256
    pats_geo = [(256 * 2 ** i, 2 ** i) for i in range(5)]
    per_head = oracle.sparse_flops(1, 4096, 1, D, pats_geo) - 2 * D * oracle.covered_rows(4096, 1, pats_geo)
    assert per_head <= 2 * 2 / (2 - 1) * 256 * 4096 * D
