"""Negative controls of the parity checker (CPU only).

Every GPU parity claim rests on tests/checker.py.  These tests feed it a
correct result (the oracle's own, outputs rounded to bf16 as the GPU rounds
them) and perturbed copies of it, and require each perturbation to be
rejected: a zeroed output, an output scaled by 1.05, a swap of two tokens
whose scores differ by more than the tie tolerance, a dropped window token,
an unsorted or duplicated row, a wrong count, a token past the query's
position.  A permitted tie swap must still pass.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import hs2_oracle as O
from paper_2609_26368_amd import workloads as W
from tests import checker as CK


@pytest.fixture(scope="module")
def case():
    w = W.Workload("checker_neg", 2, 900, 2, 16, 2, 128, 64, 16, 1, ctx_min=500)
    inp = W.make_inputs(w, seed=21)
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window)
    return w, inp, ref


def _bf16_round(x):
    return CK.bf16_bits_to_f64(W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32)))


def _row(ref, w, inp, b=0, g=1, c=1):
    pos = int(inp.lens[b]) - w.n_queries + c
    return ref["idx"][b, g, c].copy(), ref["P"][b, g, c], pos, max(0, pos - w.window + 1)


# ---------------------------------------------------------------- attention outputs
def test_correct_output_passes(case):
    _, _, ref = case
    r = CK.check_out(_bf16_round(ref["out"]), ref["out"])
    assert r["max_normwise"] < 5e-3


def test_zeroed_output_is_rejected(case):
    _, _, ref = case
    with pytest.raises(AssertionError):
        CK.check_out(np.zeros_like(ref["out"]), ref["out"])


@pytest.mark.slow
def test_zeroed_long_context_output_needs_the_normwise_guard():
    """At 128K tokens of N(0, 1) data the outputs are so small that an all-zero
    output passes the elementwise bound; the normwise guard rejects it."""
    w = W.Workload("checker_long", 1, 131072, 1, 4, 1, 128, 64, 16, 1)
    inp = W.make_inputs(w, seed=22)
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window)["out"]
    zero = np.zeros_like(ref)
    assert (np.abs(zero - ref) <= CK.OUT_ATOL + CK.OUT_RTOL * np.abs(ref)).all()
    with pytest.raises(AssertionError, match="normwise"):
        CK.check_out(zero, ref)
    CK.check_out(_bf16_round(ref), ref)


def test_output_scaled_by_1_05_is_rejected(case):
    _, _, ref = case
    with pytest.raises(AssertionError, match="normwise"):
        CK.check_out(_bf16_round(ref["out"] * 1.05), ref["out"])


def test_one_head_zeroed_is_rejected(case):
    _, _, ref = case
    bad = _bf16_round(ref["out"])
    bad[1, 0, 5] = 0.0
    with pytest.raises(AssertionError):
        CK.check_out(bad, ref["out"])


def test_sampled_rows_only_see_their_rows(case):
    """rows= restricts the comparison: a broken head outside the mask passes,
    inside it fails."""
    _, _, ref = case
    bad = _bf16_round(ref["out"])
    bad[1, 0, 5] = 0.0
    rows = np.zeros(ref["out"].shape[:3], dtype=bool)
    rows[0] = True
    CK.check_out(bad, ref["out"], rows=rows)
    rows[1, 0, 5] = True
    with pytest.raises(AssertionError):
        CK.check_out(bad, ref["out"], rows=rows)


# ---------------------------------------------------------------- index rows against the oracle
def test_correct_rows_pass(case):
    w, inp, ref = case
    assert CK.check_idx(ref["idx"].copy(), ref["idx"], ref["P"], inp.lens, w.n_queries, w.window)["swaps"] == 0
    CK.check_idx_structure(ref["idx"], inp.lens, w.n_queries, w.k, w.window)


def _swap_candidates(row, P, wlo):
    """The lowest-scoring selected top-k token and the best unselected candidate."""
    sel = row[(row >= 0) & (row < wlo)]
    uns = np.setdiff1d(np.arange(wlo), sel)
    t_out = sel[np.argmin(P[sel])]
    t_in = uns[np.argmax(P[uns])]
    return int(t_out), int(t_in)


def test_non_tie_swap_is_rejected(case):
    w, inp, ref = case
    row, P, pos, wlo = _row(ref, w, inp)
    t_out, t_in = _swap_candidates(row, P, wlo)
    assert abs(P[t_out] - P[t_in]) / P[t_out] > CK.TIE_RTOL  # a real (non-tie) swap
    bad = np.sort(np.where(row == t_out, t_in, row)[row >= 0])
    bad = np.concatenate([bad, row[row < 0]])
    with pytest.raises(AssertionError, match="swap of tokens"):
        CK.check_idx_row(bad, row, P, wlo)
    CK.check_idx_structure(bad[None, None, None].repeat(1, 0), [pos + 1], 1, w.k, w.window)  # structure alone is fine


def test_tie_swap_is_tolerated(case):
    """The same swap passes when the two scores are within the tie tolerance."""
    w, inp, ref = case
    row, P, pos, wlo = _row(ref, w, inp)
    t_out, t_in = _swap_candidates(row, P, wlo)
    P2 = P.copy()
    P2[t_in] = np.float32(P2[t_out] * (1 + 2e-7))
    good = np.sort(np.where(row == t_out, t_in, row)[row >= 0])
    good = np.concatenate([good, row[row < 0]])
    assert CK.check_idx_row(good, row, P2, wlo) == 1


def test_dropped_window_token_is_rejected(case):
    w, inp, ref = case
    row, P, pos, wlo = _row(ref, w, inp)
    # replace window token pos - 3 by the best unselected candidate (same count)
    _, t_in = _swap_candidates(row, P, wlo)
    v = row[row >= 0]
    v = np.sort(np.where(v == pos - 3, t_in, v))
    bad = np.concatenate([v, row[row < 0]])
    with pytest.raises(AssertionError, match="window token"):
        CK.check_idx_row(bad, row, P, wlo)
    with pytest.raises(AssertionError, match="window"):
        CK.check_idx_structure(bad[None, None, None], [pos + 1], 1, w.k, w.window)


def test_unsorted_row_is_rejected(case):
    w, inp, ref = case
    row, P, pos, wlo = _row(ref, w, inp)
    bad = row.copy()
    bad[[3, 4]] = bad[[4, 3]]
    with pytest.raises(AssertionError, match="ascending"):
        CK.check_idx_row(bad, row, P, wlo)
    with pytest.raises(AssertionError, match="ascending"):
        CK.check_idx_structure(bad[None, None, None], [pos + 1], 1, w.k, w.window)


def test_duplicated_index_is_rejected(case):
    w, inp, ref = case
    row, P, pos, wlo = _row(ref, w, inp)
    bad = row.copy()
    bad[5] = bad[4]
    with pytest.raises(AssertionError):
        CK.check_idx_row(bad, row, P, wlo)
    with pytest.raises(AssertionError, match="ascending"):
        CK.check_idx_structure(bad[None, None, None], [pos + 1], 1, w.k, w.window)


def test_wrong_count_is_rejected(case):
    w, inp, ref = case
    row, P, pos, wlo = _row(ref, w, inp)
    n = int((row >= 0).sum())
    short = row.copy()
    short[0:n - 1] = row[1:n]
    short[n - 1] = -1  # one top-k token dropped
    with pytest.raises(AssertionError, match="selects"):
        CK.check_idx_row(short, row, P, wlo)
    with pytest.raises(AssertionError, match="tokens, expected"):
        CK.check_idx_structure(short[None, None, None], [pos + 1], 1, w.k, w.window)


def test_padding_gap_is_rejected(case):
    w, inp, ref = case
    row, P, pos, wlo = _row(ref, w, inp)
    bad = row.copy()
    bad[2] = -1  # a hole inside the valid prefix
    with pytest.raises(AssertionError):
        CK.check_idx_row(bad, row, P, wlo)
    with pytest.raises(AssertionError):
        CK.check_idx_structure(bad[None, None, None], [pos + 1], 1, w.k, w.window)


def test_token_past_position_is_rejected():
    """Structure: a row whose window is shifted one past the query's position."""
    k, win, pos = 4, 3, 20
    good = np.array([1, 5, 7, 9, 18, 19, 20], dtype=np.int32)
    CK.check_idx_structure(good[None, None, None], [pos + 1], 1, k, win)
    bad = np.array([1, 5, 7, 9, 19, 20, 21], dtype=np.int32)
    with pytest.raises(AssertionError):
        CK.check_idx_structure(bad[None, None, None], [pos + 1], 1, k, win)


def test_negative_position_row_must_be_empty():
    k, win = 4, 3
    C = 3
    rows = np.full((1, 1, C, k + win), -1, dtype=np.int32)
    rows[0, 0, 2, :2] = [0, 1]  # len 2: queries 0 (pos -1) is empty, 1 (pos 0) holds token 0, 2 (pos 1) tokens 0, 1
    rows[0, 0, 1, 0] = 0
    CK.check_idx_structure(rows, [2], C, k, win)
    rows[0, 0, 0, 0] = 0
    with pytest.raises(AssertionError, match="tokens, expected"):
        CK.check_idx_structure(rows, [2], C, k, win)


# ---------------------------------------------------------------- pooled scores
def test_scores_perturbed_beyond_tolerance_are_rejected(case):
    w, inp, ref = case
    P = ref["P"].copy()
    CK.check_scores(P, ref["P"], inp.lens, w.n_queries, w.window)
    P[0, 0, 0, 10] *= 1 + 5 * CK.SCORE_RTOL
    with pytest.raises(AssertionError, match="outside tolerance"):
        CK.check_scores(P, ref["P"], inp.lens, w.n_queries, w.window)
