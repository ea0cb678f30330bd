"""Pins of the backward oracle (CPU only).

The backward oracle writes out the closed-form derivative of the forward's
definition.  It is pinned against things it does not share code with:
  * central finite differences of the forward oracle (a scalar loss
    sum(dout * out)), on tiny inputs with ragged segments, r not dividing w,
    duplicate patterns, causal and not;
  * the dense special case (one pattern w = N, r = 1) against PyTorch's
    autograd of float64 scaled-dot-product attention;
  * the row-restricted helpers against the full backward.
"""
import numpy as np
import pytest
import torch

import oracle

CASES = [
    # (B, N, H, D, patterns, causal)
    (1, 12, 2, 4, [(4, 1), (6, 2), (12, 3)], True),
    (1, 11, 3, 3, [(5, 1), (11, 2), (7, 4)], True),     # ragged last segments, r not dividing w
    (2, 9, 2, 2, [(9, 1), (3, 1), (9, 1)], False),      # duplicate pattern, non-causal
    (1, 10, 4, 3, [(10, 3), (4, 2)], True),             # rows no pattern keeps
]


def _inputs(B, N, H, D, seed):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((B, N, H, D)) for _ in range(4)]


def _loss(q, k, v, dout, pats, causal, scale):
    out, _ = oracle.dilated_attention_ref(q, k, v, pats, causal, scale)
    return float((dout * out).sum())


@pytest.mark.parametrize("case", CASES)
def test_backward_matches_finite_differences(case):
    B, N, H, D, pats, causal = case
    q, k, v, dout = _inputs(B, N, H, D, seed=N * 31 + H)
    scale = 0.7
    dq, dk, dv, _, _ = oracle.dilated_attention_bwd_ref(q, k, v, dout, pats, causal, scale)
    eps = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        it = np.nditer(x, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            old = x[i]
            x[i] = old + eps
            lp = _loss(q, k, v, dout, pats, causal, scale)
            x[i] = old - eps
            lm = _loss(q, k, v, dout, pats, causal, scale)
            x[i] = old
            num[i] = (lp - lm) / (2 * eps)
        err = np.abs(num - g).max()
        assert err < 1e-6, f"d{name}: finite differences differ by {err}"


def test_dense_case_matches_sdpa_autograd():
    B, N, H, D = 2, 24, 3, 8
    q, k, v, dout = _inputs(B, N, H, D, seed=5)
    dq, dk, dv, _, _ = oracle.dilated_attention_bwd_ref(q, k, v, dout, [(N, 1)], True, None)
    tq, tk, tv = (torch.tensor(x.transpose(0, 2, 1, 3), dtype=torch.float64, requires_grad=True)
                  for x in (q, k, v))
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    out.backward(torch.tensor(dout.transpose(0, 2, 1, 3), dtype=torch.float64))
    for name, mine, ref in (("q", dq, tq.grad), ("k", dk, tk.grad), ("v", dv, tv.grad)):
        err = np.abs(mine - ref.numpy().transpose(0, 2, 1, 3)).max()
        assert err < 1e-10, f"d{name}: {err}"


def test_delta_is_rowsum_of_dout_times_out():
    rng = np.random.default_rng(1)
    dout, out = rng.standard_normal((2, 5, 3, 4)), rng.standard_normal((2, 5, 3, 4))
    d = oracle.delta_ref(dout, out)
    for b in range(2):
        for p in range(5):
            for h in range(3):
                assert abs(d[b, h, p] - sum(dout[b, p, h, i] * out[b, p, h, i] for i in range(4))) < 1e-12


def test_row_helpers_match_full_backward():
    B, N, H, D = 1, 40, 3, 5
    pats = [(8, 1), (16, 2), (40, 3)]
    q, k, v, dout = _inputs(B, N, H, D, seed=9)
    dq, dk, dv, _, _ = oracle.dilated_attention_bwd_ref(q, k, v, dout, pats, True, None)
    rows = [(0, p, h) for p in (0, 1, 7, 8, 23, 38, 39) for h in range(H)]
    rq = oracle.dq_rows_ref(q, k, v, dout, pats, True, None, rows)
    rk, rv = oracle.dkdv_rows_ref(q, k, v, dout, pats, True, None, rows)
    for ri, (b, p, h) in enumerate(rows):
        assert np.abs(rq[ri] - dq[b, p, h]).max() < 1e-12
        assert np.abs(rk[ri] - dk[b, p, h]).max() < 1e-12
        assert np.abs(rv[ri] - dv[b, p, h]).max() < 1e-12


def test_uncovered_rows_get_zero_gradient():
    B, N, H, D = 1, 10, 4, 3
    q, k, v, dout = _inputs(B, N, H, D, seed=3)
    pats = [(10, 3)]            # head h keeps rows h mod 3, +3, ...; head 3 keeps rows 0,3,6,9
    dq, dk, dv, _, _ = oracle.dilated_attention_bwd_ref(q, k, v, dout, pats, True, None)
    for h in range(H):
        kept = set(range(h % 3, N, 3))
        for p in range(N):
            if p not in kept:
                assert not dq[0, p, h].any() and not dk[0, p, h].any() and not dv[0, p, h].any()


# ---- planted mistakes must be caught by the finite-difference pin -------------

import oracle.dilated_bwd as bwd  # noqa: E402

ORIG_ATTEND_BWD = bwd.attend_bwd


def _m_local_lse(qt, kt, vt, dot, lse_t, delta_t, causal, scale):
    # the pattern's own lse instead of the combined one
    L = qt.shape[0]
    S = scale * (qt @ kt.T)
    if causal:
        S = np.where(np.tril(np.ones((L, L), dtype=bool)), S, -np.inf)
    m = S.max(axis=1)
    own = m + np.log(np.exp(S - m[:, None]).sum(axis=1))
    return ORIG_ATTEND_BWD(qt, kt, vt, dot, own, delta_t, causal, scale)


def _m_no_delta(qt, kt, vt, dot, lse_t, delta_t, causal, scale):
    return ORIG_ATTEND_BWD(qt, kt, vt, dot, lse_t, 0 * delta_t, causal, scale)


def _m_dk_unscaled(qt, kt, vt, dot, lse_t, delta_t, causal, scale):
    dq, dk, dv = ORIG_ATTEND_BWD(qt, kt, vt, dot, lse_t, delta_t, causal, scale)
    return dq, dk / scale, dv


def _m_dk_transposed(qt, kt, vt, dot, lse_t, delta_t, causal, scale):
    L = qt.shape[0]
    S = scale * (qt @ kt.T)
    if causal:
        S = np.where(np.tril(np.ones((L, L), dtype=bool)), S, -np.inf)
    P = np.exp(S - lse_t[:, None])
    dS = P * (dot @ vt.T - delta_t[:, None])
    return scale * (dS @ kt), scale * (dS @ qt), P.T @ dot


def _m_dv_from_ds(qt, kt, vt, dot, lse_t, delta_t, causal, scale):
    dq, dk, _ = ORIG_ATTEND_BWD(qt, kt, vt, dot, lse_t, delta_t, causal, scale)
    L = qt.shape[0]
    S = scale * (qt @ kt.T)
    if causal:
        S = np.where(np.tril(np.ones((L, L), dtype=bool)), S, -np.inf)
    P = np.exp(S - lse_t[:, None])
    dS = P * (dot @ vt.T - delta_t[:, None])
    return dq, dk, dS.T @ dot


@pytest.mark.parametrize("mutant", [_m_local_lse, _m_no_delta, _m_dk_unscaled, _m_dk_transposed, _m_dv_from_ds],
                         ids=lambda f: f.__name__)
def test_mutant_is_caught(mutant, monkeypatch):
    monkeypatch.setattr(bwd, "attend_bwd", mutant)
    with pytest.raises(AssertionError):
        test_backward_matches_finite_differences(CASES[0])
