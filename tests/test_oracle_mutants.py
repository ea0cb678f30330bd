"""Planted mistakes in the oracle must be caught by its pins.

Each mutant replaces one step of the CPU oracle with a plausible error (a
dropped term, a wrong offset, a transposed operand, an off-by-one mask) and
checks that at least one pin test fails.  Mutants live only inside this test,
on the CPU.
"""
import numpy as np
import pytest

import oracle.dilated_ref as ref
from tests import test_oracle as pins

PIN_TESTS = [
    pins.test_golden_multisets_q_zero_oracle,
    lambda: pins.test_dense_special_case(True),
    pins.test_segment_special_case,
    pins.test_dilated_single_pattern_against_sdpa_on_gathered_rows,
    pins.test_three_constructions_agree,
    pins.test_q_zero_closed_form,
    pins.test_scale_is_applied,
]


def _attend_mask_strict(qt, kt, vt, causal, scale):
    L = qt.shape[0]
    S = scale * (qt @ kt.T)
    if causal:
        S = np.where(np.tril(np.ones((L, L), dtype=bool), -1), S, -1e300)
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    d = E.sum(axis=1, keepdims=True)
    return (E @ vt) / d, m[:, 0] + np.log(d[:, 0])


def _attend_no_scale(qt, kt, vt, causal, scale):
    return ORIG["attend"](qt, kt, vt, causal, 1.0)


def _attend_transposed(qt, kt, vt, causal, scale):
    L = qt.shape[0]
    S = scale * (kt @ qt.T)
    if causal:
        S = np.where(np.tril(np.ones((L, L), dtype=bool)), S, -np.inf)
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    d = E.sum(axis=1, keepdims=True)
    return (E @ vt) / d, m[:, 0] + np.log(d[:, 0])



def _combine_plain_mean(Os, LSEs):
    out, lse = ORIG["combine_ref"](Os, LSEs)
    cov = np.stack([np.isfinite(l) for l in LSEs]).sum(axis=0)      # [B,H,N]
    mean = sum(Os) / np.maximum(np.transpose(cov, (0, 2, 1))[..., None], 1)
    return mean, lse


def _combine_lse_max(Os, LSEs):
    out, lse = ORIG["combine_ref"](Os, LSEs)
    return out, np.stack(LSEs).max(axis=0)


ORIG = {"attend": ref.attend, "combine_ref": ref.combine_ref}

MUTANTS = {
    "offset_ignored": ("head_offset", lambda h, r: 0),
    "offset_plus_one": ("head_offset", lambda h, r: (h + 1) % r),
    "global_residue": ("index_set", lambda N, w, r, h, g: np.arange(
        g * w + ((h % r) - g * w) % r, min(g * w + w, N), r, dtype=np.int64)),
    "mask_excludes_diagonal": ("attend", _attend_mask_strict),
    "scale_dropped": ("attend", _attend_no_scale),
    "operands_transposed": ("attend", _attend_transposed),
    "mix_plain_mean": ("combine_ref", _combine_plain_mean),
    "lse_max_only": ("combine_ref", _combine_lse_max),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(ref, attr, fn)
    caught = 0
    for t in PIN_TESTS:
        try:
            t()
        except (AssertionError, IndexError, ValueError, FloatingPointError):
            caught += 1
    assert caught > 0, f"mutant {name} survived every pin"
