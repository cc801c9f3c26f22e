"""The parity checker itself, on the CPU: exact lists where the oracle's
margin exceeds 1e-6, and on near-tie rows any valid top-k of the oracle's
ranking, but nothing else (a planted wrong block fails)."""
import numpy as np
import pytest

import oracle as O
from tests import parity as PT


def _res(rows, cap):
    """A fake GPU result with one head: rows of ascending block indices."""
    nb = len(rows)
    idx = np.full((1, nb, cap), -1, np.int32)
    cnt = np.zeros((1, nb), np.int32)
    for i, r in enumerate(rows):
        idx[0, i, :len(r)] = r
        cnt[0, i] = len(r)
    return {"idx": idx, "cnt": cnt}


def test_near_tie_row_accepts_either_tied_block_and_rejects_a_wrong_one():
    # blocks 2 and 3 differ by 1e-7 at the boundary of the top 3
    s = np.array([5.0, 4.0, 3.0 + 1e-7, 3.0, 1.0, 0.0])
    lst, margin = O.topk_row(s, 3)
    assert list(lst) == [0, 1, 2] and margin <= PT.NEAR_TIE
    rank = PT.ranking(O.TOPK, 3, s)
    for got, ok in (([0, 1, 2], True), ([0, 1, 3], True), ([0, 1, 4], False), ([0, 2, 3], False),
                    ([1, 2, 3], False)):
        res = _res([got] * 6, 4)
        if ok:
            assert PT.check_lists(res, 0, 0, O.TOPK, lst, margin, 6, 4, rank=rank) in ("ok", "near_tie")
        else:
            with pytest.raises(AssertionError, match="not a valid top-k"):
                PT.check_lists(res, 0, 0, O.TOPK, lst, margin, 6, 4, rank=rank)
    # a short list fails too
    with pytest.raises(AssertionError):
        PT.check_lists(_res([[0, 1]] * 6, 4), 0, 0, O.TOPK, lst, margin, 6, 4, rank=rank)
    # a near-tie row without the oracle's ranking is refused outright
    with pytest.raises(AssertionError, match="without the oracle's ranking"):
        PT.check_lists(_res([[0, 1, 3]] * 6, 4), 0, 0, O.TOPK, lst, margin, 6, 4)


def test_rows_with_a_clear_margin_must_equal_the_oracle():
    s = np.array([5.0, 4.0, 3.5, 3.0, 1.0, 0.0])
    lst, margin = O.topk_row(s, 3)
    assert margin > PT.NEAR_TIE
    rank = PT.ranking(O.TOPK, 3, s)
    assert PT.check_lists(_res([[0, 1, 2]] * 6, 4), 0, 0, O.TOPK, lst, margin, 6, 4, rank=rank) == "ok"
    with pytest.raises(AssertionError, match="!= oracle"):
        PT.check_lists(_res([[0, 1, 3]] * 6, 4), 0, 0, O.TOPK, lst, margin, 6, 4, rank=rank)


def test_valid_topk_against_subset_enumeration():
    """valid_topk accepts exactly the k-subsets whose every kept score is
    within 1e-6 of the k-th and every dropped one within 1e-6 of the
    (k+1)-th: brute force over all subsets of small rows with planted
    near-ties."""
    from itertools import combinations

    g = np.random.default_rng(3)
    for _ in range(40):
        nb = int(g.integers(2, 8))
        s = np.round(g.standard_normal(nb), 1)
        s[g.integers(nb)] += g.choice([0.0, 5e-7, 2e-6])
        k = int(g.integers(1, nb + 1))
        ranked = np.sort(s)[::-1]
        for sub in combinations(range(nb), k):
            kept = np.zeros(nb, bool)
            kept[list(sub)] = True
            want = s[kept].min() >= ranked[k - 1] - 1e-6 and (k == nb or s[~kept].max() <= ranked[k] + 1e-6)
            assert PT.valid_topk(list(sub), s, k) == want, (s, k, sub)
        # the oracle's own choice is always valid
        assert PT.valid_topk(O.topk_row(s, k)[0], s, k)


def test_cosine_near_tie_is_checked_per_frame():
    # frames of 128 tokens: blocks {0, 1} frame 0, {2, 3} frame 1, {4, 5} frame 2
    sim = np.array([0.9, 0.9 + 5e-7, 0.1, 0.5, 0.3, 0.2])
    lst, margin = O.cosine_topk_row(sim, 1, 128, 64)
    assert list(lst) == [1, 3, 4] and margin <= PT.NEAR_TIE
    rank = PT.ranking(O.COSINE_TOPK, 1, sim, 128)
    ok = _res([[0, 3, 4]] * 6, 3)  # frame 0's tied block
    assert PT.check_lists(ok, 0, 0, O.COSINE_TOPK, lst, margin, 6, 3, rank=rank) == "near_tie"
    for bad in ([1, 2, 4], [1, 3, 5], [0, 1, 3]):  # a wrong block in a frame without a tie
        with pytest.raises(AssertionError, match="not a valid top-k"):
            PT.check_lists(_res([bad] * 6, 3), 0, 0, O.COSINE_TOPK, lst, margin, 6, 3, rank=rank)
