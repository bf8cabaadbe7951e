"""Comparison rules between the GPU library and the CPU oracle.

Scores: |gpu - oracle| <= rtol * max(|oracle|, gamma) element by element.
The gamma floor keeps the bound meaningful where scores cross zero.

Top-k (score descending, equal scores by index ascending):
  1. the GPU list is itself in that order, judged on its own scores;
  2. the GPU's reported score of every returned index matches the oracle's
     score of that index;
  3. position by position the two sorted score lists agree;
  4. where the index at a position differs from the oracle's, the oracle
     score of the GPU's index is within the tolerance of the oracle's score
     at that position (a near-tie swap); indices in one list but not the
     other have oracle scores within the tolerance of the oracle's k-th score.
Everything else must be identical.
"""

from __future__ import annotations

import numpy as np

from oracle import oracle as O

# One line per full-size workload checked: how many score rows and top-k
# lists were compared (printed in pytest's terminal summary).
COVERAGE: list = []


def tol_of(o: np.ndarray, rtol: float, gamma: float) -> np.ndarray:
    return rtol * np.maximum(np.abs(o), abs(gamma))


def check_scores(gpu: np.ndarray, ora: np.ndarray, rtol: float, gamma: float, what: str = ""):
    gpu = np.asarray(gpu, np.float64)
    ora = np.asarray(ora, np.float64)
    assert gpu.shape == ora.shape, (gpu.shape, ora.shape)
    err = np.abs(gpu - ora)
    bound = tol_of(ora, rtol, gamma)
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} scores outside tolerance; worst at {i}: "
                             f"gpu={gpu[i]!r} oracle={ora[i]!r} bound={bound[i]:.3g}")
    return float((err / bound).max()) if err.size else 0.0


def check_topk(idx: np.ndarray, val: np.ndarray, ora_rows: np.ndarray, k: int, rtol: float,
               gamma: float, what: str = ""):
    """idx/val: GPU top-k [B x k]; ora_rows: oracle scores [B x N] of the same queries."""
    idx = np.asarray(idx, np.int64)
    val = np.asarray(val, np.float64)
    ora_rows = np.asarray(ora_rows, np.float64)
    B, N = ora_rows.shape
    oi, ov = O.topk(ora_rows, k)
    n_swaps = 0
    for q in range(B):
        gi, gv, row = idx[q], val[q], ora_rows[q]
        assert np.all((gi >= 0) & (gi < N)), f"{what} q={q}: index out of range {gi}"
        assert len(set(gi.tolist())) == k, f"{what} q={q}: duplicate indices"
        # 1. own order
        for p in range(k - 1):
            ok = gv[p] > gv[p + 1] or (gv[p] == gv[p + 1] and gi[p] < gi[p + 1])
            assert ok, f"{what} q={q}: GPU list out of order at {p}: {gv[p]} {gi[p]} / {gv[p+1]} {gi[p+1]}"
        t = tol_of(row[gi], rtol, gamma)
        # 2. reported scores
        bad = np.abs(gv - row[gi]) > t
        assert not bad.any(), f"{what} q={q}: reported score off at positions {np.nonzero(bad)[0][:5]}"
        # 3. sorted lists agree
        tp = tol_of(ov[q], rtol, gamma)
        bad = np.abs(gv - ov[q]) > tp
        assert not bad.any(), f"{what} q={q}: sorted score lists differ at {np.nonzero(bad)[0][:5]}"
        # 4. index differences only among near-ties
        for p in np.nonzero(gi != oi[q])[0]:
            n_swaps += 1
            assert abs(row[gi[p]] - ov[q][p]) <= tp[p], \
                f"{what} q={q} pos {p}: gpu idx {gi[p]} (oracle {row[gi[p]]}) vs oracle idx {oi[q][p]} ({ov[q][p]})"
        kth = ov[q][k - 1]
        for e in set(gi.tolist()) ^ set(oi[q].tolist()):
            assert abs(row[e] - kth) <= tol_of(np.array([kth]), rtol, gamma)[0], \
                f"{what} q={q}: entity {e} in one list only, oracle score {row[e]} vs k-th {kth}"
    return n_swaps
