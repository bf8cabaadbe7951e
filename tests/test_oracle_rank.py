"""Pins for the oracle's filtered ranking metrics (the paper evaluates answer
quality by MRR; Experiments). The oracle counts, for each answer, the
non-answer entities that rank before it. These tests check it against a
different computation (a full sort of the row, then positions) and against
hand-worked examples and special cases."""

import math

import numpy as np
import pytest

from oracle import oracle as O


def _csr(lists):
    off = np.zeros(len(lists) + 1, np.int32)
    for i, l in enumerate(lists):
        off[i + 1] = off[i] + len(l)
    ids = np.array([e for l in lists for e in l], np.int32)
    return off, ids


def test_worked_example_with_ties():
    # row 0: scores  e0 0.9, e1 0.5, e2 0.9, e3 0.1, e4 0.7
    # ranking order: e0 (0.9, lower index first), e2, e4, e1, e3
    # answers {2 (hard), 0 (easy)}: e2 is preceded only by e0, an answer -> rank 1;
    #                               e0 is first -> rank 1
    # row 1: same scores, answers {3 (hard), 4 (hard)}:
    #   e4 is preceded by e0, e2 (non-answers) -> rank 3
    #   e3 is preceded by e0, e2, e1 (non-answers) and e4 (answer, filtered) -> rank 4
    s = np.array([[0.9, 0.5, 0.9, 0.1, 0.7]] * 2, np.float32)
    off, ids = _csr([[2, 0], [3, 4]])
    hard = np.array([1, 0, 1, 1], np.int32)
    rank, met = O.rank_answers(s, off, ids, hard)
    assert rank.tolist() == [1, 1, 4, 3]
    assert met[0].tolist() == [1.0, 1.0, 1.0, 1.0]           # only e2 is hard, rank 1
    assert met[1][0] == pytest.approx((1 / 4 + 1 / 3) / 2)   # MRR
    assert met[1][1:].tolist() == [0.0, 0.5, 1.0]            # Hits@1, @3, @10


def test_against_full_sort():
    """Filtered rank = 1 + position in the full ranking - answers placed
    before it, computed by sorting each row (score descending, index
    ascending): a different algorithm from the oracle's counting."""
    rng = np.random.default_rng(3)
    B, N = 40, 500
    s = (rng.integers(0, 60, size=(B, N)) / 7.0).astype(np.float32)     # many exact ties
    s[5] = 1.0                                                           # a row of all-equal scores
    s[7, ::3] = -0.0
    s[7, 1::3] = 0.0                                                     # -0 and +0 rank equal
    lists = []
    for q in range(B):
        n = int(rng.integers(1, 30)) if q != 9 else N                    # row 9: every entity is an answer
        lists.append(rng.permutation(N)[:n].tolist())
    off, ids = _csr(lists)
    hard = (rng.random(ids.shape[0]) < 0.6).astype(np.int32)
    rank, met = O.rank_answers(s, off, ids, hard)
    for q in range(B):
        row = s[q].astype(np.float64) + 0.0                              # -0 -> +0 for the sort key
        order = np.lexsort((np.arange(N), -row))                         # score desc, then index asc
        pos = np.empty(N, np.int64)
        pos[order] = np.arange(N)
        ans = np.array(lists[q])
        ans_pos = np.sort(pos[ans])
        for i, a in enumerate(lists[q]):
            n_ans_before = int(np.searchsorted(ans_pos, pos[a]))
            assert rank[off[q] + i] == pos[a] - n_ans_before + 1
        h = [rank[off[q] + i] for i in range(len(lists[q])) if hard[off[q] + i]]
        if h:
            assert met[q][0] == pytest.approx(np.mean([1.0 / r for r in h]), rel=1e-15)
            for j, k in enumerate((1, 3, 10)):
                assert met[q][1 + j] == pytest.approx(np.mean([r <= k for r in h]))
        else:
            assert all(math.isnan(x) for x in met[q])
    assert (rank[off[9]:off[10]] == 1).all()                             # all answers: nothing left to rank


def test_special_cases():
    N = 64
    s = np.linspace(1.0, 0.0, N, dtype=np.float32)[None, :].repeat(3, axis=0)
    # top entity alone -> rank 1; bottom entity alone -> rank N; bottom with the
    # top 10 entities also answers -> rank N - 10
    off, ids = _csr([[0], [N - 1], [N - 1] + list(range(10))])
    rank, met = O.rank_answers(s, off, ids)
    assert rank[0] == 1 and rank[1] == N and rank[2] == N - 10
    assert met[0].tolist() == [1.0, 1.0, 1.0, 1.0]
    assert met[1][0] == pytest.approx(1.0 / N) and met[1][1:].tolist() == [0.0, 0.0, 0.0]
    # no hard answers -> NaN metrics
    _, met = O.rank_answers(s[:1], *_csr([[3]]), hard=np.array([0], np.int32))
    assert all(math.isnan(x) for x in met[0])
    # an id outside the table is rejected
    with pytest.raises(ValueError):
        O.rank_answers(s[:1], *_csr([[N]]))
