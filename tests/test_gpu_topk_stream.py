"""Top-k selection at large batches (the streaming path: one wavefront per
row, rows split when there are too few) on adversarial score matrices:
masses of exact ties, all scores equal, most scores -inf, k from 1 to 256,
and rows split into segments whose lists are merged in a second round.

The selection is checked bit for bit against a plain sort of the GPU's own
score rows (score descending, equal scores by index ascending), so these
tests see the selection alone, free of the scorer's rounding; the scores
themselves are checked against the oracle elsewhere.
"""

import numpy as np
import pytest

from paper_2503_02172_amd import synth

pytestmark = pytest.mark.gpu
S = synth.STRUCTURE_ID


def _exact_topk(scores: np.ndarray, k: int):
    """Per row: the first k of (score descending, index ascending)."""
    B, N = scores.shape
    idx = np.empty((B, k), np.int64)
    for q in range(B):
        o = np.lexsort((np.arange(N), -scores[q].astype(np.float64)))
        idx[q] = o[:k]
    return idx, np.take_along_axis(scores, idx, 1)


def _run(w, B, k, seed, anchor_below=None):
    import torch
    from paper_2503_02172_amd import kgq
    qb = synth.draw_queries("1p", B, w.n_entities, w.n_relations, seed=seed)
    if anchor_below is not None:
        qb.anchors[:] = qb.anchors % anchor_below
    with kgq.engine_for(w, max_batch=B) as eng:
        out = eng.execute(S["1p"], qb.anchors, qb.relations, k=k, scores=True)
        top = eng.execute(S["1p"], qb.anchors, qb.relations, k=k)
        torch.cuda.synchronize()
        sc = out["scores"].cpu().numpy()
        gi, gv = out["idx"].cpu().numpy(), out["score"].cpu().numpy()
        assert np.array_equal(gi, top["idx"].cpu().numpy()), "top-k with and without scores differ"
    ei, ev = _exact_topk(sc, k)
    bad = np.nonzero((gi != ei).any(1))[0]
    assert bad.size == 0, (f"B={B} N={w.n_entities} k={k}: {bad.size} rows differ; first row {bad[0]}: "
                           f"gpu {gi[bad[0]][:8]} exact {ei[bad[0]][:8]}")
    assert np.array_equal(gv.view(np.uint32), ev.astype(np.float32).view(np.uint32))
    return sc


def _gqe(n_ent, dim, seed, entity):
    w = synth.make_tiny(synth.MODEL_GQE, n_ent=n_ent, n_rel=7, dim=dim, seed=seed)
    w.params["entity"] = entity(np.random.Generator(np.random.PCG64(seed)), n_ent, dim).astype(np.float32)
    return w


@pytest.mark.parametrize("k", [1, 100, 256])
def test_gpu_topk_stream_quantised_ties(k):
    """Entity coordinates in {-0.5, 0, 0.5}: few distinct scores, so every
    threshold the selection takes falls inside a mass of equal scores."""
    w = _gqe(5000, 4, 900 + k, lambda g, n, d: g.integers(-1, 2, size=(n, d)) * 0.5)
    w.params["relation"] = (np.random.Generator(np.random.PCG64(7)).integers(-1, 2, size=(7, 4)) * 0.5).astype(np.float32)
    sc = _run(w, 2048, k, seed=901)
    assert len(np.unique(sc[0])) < 100       # the ties are real


def test_gpu_topk_stream_all_equal():
    """Every entity identical: each row is one value repeated, and the top k
    are the first k indices."""
    row = np.random.Generator(np.random.PCG64(3)).uniform(-0.5, 0.5, size=4)
    w = _gqe(3000, 4, 910, lambda g, n, d: np.tile(row, (n, 1)))
    sc = _run(w, 2048, 100, seed=911)
    assert np.all(sc == sc[:, :1])


def test_gpu_topk_stream_mostly_minus_infinity():
    """All but the first 50 entities infinitely far: their scores are -inf
    and tie, so the top 100 hold the 50 finite ones, then indices 50 .. 99.
    Anchors are finite entities (an infinite anchor would make NaN scores)."""
    def ent(g, n, d):
        e = np.full((n, d), np.inf)
        e[:50] = g.uniform(-0.5, 0.5, size=(50, d))
        return e
    w = _gqe(3000, 4, 920, ent)
    sc = _run(w, 2048, 100, seed=921, anchor_below=50)
    assert np.isneginf(sc[:, 50:]).all() and np.isfinite(sc[:, :50]).all()


def test_gpu_topk_stream_split_rows_with_ties():
    """1,024 rows of 40,000 scores: each row is split into two streamed
    segments, and a second round merges the per-segment lists; quantised
    entities make ties that cross the segment boundary."""
    w = _gqe(40000, 4, 930, lambda g, n, d: g.integers(-1, 2, size=(n, d)) * 0.5)
    _run(w, 1024, 100, seed=931)


def test_gpu_topk_stream_random_scores():
    """A plain random table at the streaming shape, k = 100 and k = 7."""
    w = synth.make_tiny(synth.MODEL_GQE, n_ent=14505, n_rel=7, dim=8, seed=940)
    _run(w, 2304, 100, seed=941)
    _run(w, 2304, 7, seed=942)


# ---------------------------------------------------------------------------
# BetaE at 65 or more scored rows with 2d a multiple of 32: the bf16 scorer
# also writes each output row's chunk keys (the largest score key of every
# 64 entities), and the first streaming round starts its threshold at the
# k-th largest chunk key and skips chunks below it. The same bit-for-bit
# check against a plain sort of the GPU's own score rows shows that skipping
# loses nothing: wrong keys (too low, or on the wrong row or chunk) would
# drop elements of the top k.
# ---------------------------------------------------------------------------

def _betae(n_ent, dim, seed, entity=None):
    w = synth.make_tiny(synth.MODEL_BETAE, n_ent=n_ent, n_rel=7, dim=dim, seed=seed)
    if entity is not None:
        w.params["entity.alpha_beta"] = entity(np.random.Generator(np.random.PCG64(seed)), n_ent, 2 * dim)
    return w


def _run_structure(w, structure, B, k, seed):
    import torch
    from paper_2503_02172_amd import kgq
    qb = synth.draw_queries(structure, B, w.n_entities, w.n_relations, seed=seed)
    with kgq.engine_for(w, max_batch=B) as eng:
        out = eng.execute(S[structure], qb.anchors, qb.relations, k=k, scores=True)
        top = eng.execute(S[structure], qb.anchors, qb.relations, k=k)
        torch.cuda.synchronize()
        sc = out["scores"].cpu().numpy()
        gi, gv = out["idx"].cpu().numpy(), out["score"].cpu().numpy()
        assert np.array_equal(gi, top["idx"].cpu().numpy()), "top-k with and without scores differ"
    ei, ev = _exact_topk(sc, k)
    bad = np.nonzero((gi != ei).any(1))[0]
    assert bad.size == 0, (f"{structure} B={B} N={w.n_entities} k={k}: {bad.size} rows differ; first row "
                           f"{bad[0]}: gpu {gi[bad[0]][:8]} exact {ei[bad[0]][:8]}")
    assert np.array_equal(gv.view(np.uint32), ev.astype(np.float32).view(np.uint32))
    return sc


@pytest.mark.parametrize("k", [1, 100, 256])
def test_gpu_topk_pruned_betae_ragged(k):
    """9,001 entities: 141 chunk keys per row, the last covering 41
    entities; k = 1 and 100 seed the threshold from the keys, k = 256 (more
    than the chunks) streams every chunk."""
    _run_structure(_betae(9001, 16, 950), "1p", 2048, k, seed=951 + k)


def test_gpu_topk_pruned_betae_ties():
    """Entities drawn from 40 distinct embeddings: each row holds at most
    40 distinct scores, so the k-th largest chunk key ties with many
    elements in many chunks, and the tie rule (index ascending) decides."""
    def ent(g, n, d2):
        base = np.maximum(1.0 + g.uniform(-1.0, 1.0, size=(40, d2)), 0.05)
        return base[g.integers(0, 40, size=n)].astype(np.float32)
    sc = _run_structure(_betae(9001, 16, 960, ent), "1p", 2048, 100, seed=961)
    assert len(np.unique(sc[0])) <= 40


@pytest.mark.parametrize("structure", ["2u", "up"])
def test_gpu_topk_pruned_betae_union(structure):
    """Union structures: an output row is the maximum of two scored rows,
    and its chunk keys must be those of the maximum."""
    _run_structure(_betae(9001, 16, 970), structure, 2048, 100, seed=971)


def test_gpu_topk_pruned_betae_segments():
    """1,024 rows of 20,000 scores: each row streams as two segments (the
    first round pruned by each segment's own chunk keys), then a merge
    round over the per-segment lists."""
    _run_structure(_betae(20000, 16, 980), "1p", 1024, 100, seed=981)
