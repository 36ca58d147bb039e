"""The GPU-versus-oracle comparison rules themselves (tests/parity.py), exercised on the CPU with
index rows built from the oracle, so that a rule that is too lax fails here before it is trusted
on the GPU.

The page-tie case: two eligible pages hold the same keys in reverse order, so their mean keys and
coarse scores (Eq. 9) are equal and either may be recalled (Eq. 10 under the tie rule), but their
fine scores (Eq. 11) put the top tokens at different positions. A selection made on the other
tied page is correct only when the checker re-runs the oracle's fine stage on that page; a wrong
fine selection on it must still be rejected.
"""
from types import SimpleNamespace

import numpy as np
import pytest

import oracle.lsa_oracle as orc
from tests import parity as P

# P = B = 4, M = 1 recalled page, K_sparse = 2, no sink, a window of 4, one head, d = 2
W = SimpleNamespace(page=4, sub_block=4, keep_pages=1, k_sparse=2, k_sink=0, k_swa=4, run_align=4,
                    pooling="mean")
T = 15                                   # eligible range [0, 11]: pages 0, 1, 2


def _case():
    k = np.zeros((T + 1, 2))
    k[0:4, 0] = [1.0, 2.0, 3.0, 4.0]      # page 0
    k[4:8, 0] = [4.0, 3.0, 2.0, 1.0]      # page 1: the same keys reversed (equal mean)
    k[8:12, 0] = 0.5                      # page 2: lower mean
    k[12:16, 0] = 1.0                     # window
    q = np.array([[1.0, 0.0]])
    w = np.array([1.0])
    prm = P.oracle_params(W)
    k_mean = orc.sub_block_mean_keys(k, W.sub_block)
    return P.oracle_index_row(T, q, w, k, k_mean, prm)


def _gpu_row(S):
    S = np.asarray(S, np.int64)
    cap = W.k_sink + W.k_swa + W.k_sparse
    row = np.full(cap, -1, np.int64)
    row[:S.size] = S
    return row[None, :], np.array([S.size])


def test_case_has_a_page_tie():
    r = _case()
    assert r["page_score"][0] == r["page_score"][1] > r["page_score"][2]
    assert np.array_equal(r["pages"], [0])                   # the tie goes to the smaller page
    assert np.array_equal(r["sparse"], [2, 3])


def test_selection_on_the_other_tied_page_is_accepted():
    r = _case()
    idx, cnt = _gpu_row([4, 5, 12, 13, 14, 15])              # page 1 recalled, its top two tokens
    stats = P.check_index_rows(W, [T], idx, cnt, np.array([[1]]), [r])
    assert stats["page_tie_rows"] == 1 and stats["exact"] == 1


def test_wrong_fine_selection_on_the_other_tied_page_is_rejected():
    r = _case()
    idx, cnt = _gpu_row([4, 6, 12, 13, 14, 15])              # token 6 (score 2) instead of 5 (score 3)
    with pytest.raises(AssertionError):
        P.check_index_rows(W, [T], idx, cnt, np.array([[1]]), [r])


def test_tokens_outside_the_recalled_page_are_rejected():
    r = _case()
    idx, cnt = _gpu_row([2, 3, 12, 13, 14, 15])              # page 0's tokens while reporting page 1
    with pytest.raises(AssertionError):
        P.check_index_rows(W, [T], idx, cnt, np.array([[1]]), [r])


def test_a_page_that_is_no_tie_is_rejected():
    r = _case()
    idx, cnt = _gpu_row([8, 9, 12, 13, 14, 15])              # page 2 scores below the threshold
    with pytest.raises(AssertionError):
        P.check_index_rows(W, [T], idx, cnt, np.array([[2]]), [r])


def test_page_tie_without_an_oracle_rerun_is_rejected():
    r = _case()
    del r["rerun"]
    idx, cnt = _gpu_row([4, 5, 12, 13, 14, 15])
    with pytest.raises(AssertionError):
        P.check_index_rows(W, [T], idx, cnt, np.array([[1]]), [r])


def test_same_pages_exact_and_token_tie():
    r = _case()
    idx, cnt = _gpu_row([2, 3, 12, 13, 14, 15])
    assert P.check_index_rows(W, [T], idx, cnt, np.array([[0]]), [r])["exact"] == 1
    idx, cnt = _gpu_row([1, 3, 12, 13, 14, 15])              # not a tie: token 1 scores 2 < 3
    with pytest.raises(AssertionError):
        P.check_index_rows(W, [T], idx, cnt, np.array([[0]]), [r])
