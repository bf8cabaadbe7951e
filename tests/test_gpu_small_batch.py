"""Parity at small batches with full-size embeddings (d = 400), where the
library changes strategy: dense layers split K over a workspace and add the
slices in a second kernel, the BetaE scorer uses 64 x 64 tiles, and the GQE /
Query2Box scorers split the dimensions over slices whose partials a second
kernel sums (with the union max). The oracle evaluates the same queries node
by node."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_02172_amd import synth
from tests.parity import check_scores, check_topk

pytestmark = pytest.mark.gpu
S = synth.STRUCTURE_ID


def _run(model, structures, batches, n_ent=1500, n_rel=11, dim=400, seed=31):
    import torch
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(model, n_ent=n_ent, n_rel=n_rel, dim=dim, seed=seed)
    eng = kgq.engine_for(w, max_batch=max(batches) + 8)
    m = O.Model(model, w.params, w.gamma)
    for st in structures:
        for B in batches:
            q = synth.draw_queries(st, B, n_ent, n_rel, seed=seed + 100 * B + S[st])
            out = eng.execute(S[st], q.anchors, q.relations, k=10, scores=True)
            torch.cuda.synchronize()
            ref = m.scores(np.full(B, S[st]), q.anchors, q.relations)
            what = f"model {model} {st} B={B}"
            check_scores(out["scores"].cpu().numpy(), ref, w.rtol, w.gamma, what)
            check_topk(out["idx"].cpu().numpy(), out["score"].cpu().numpy(), ref, 10, w.rtol, w.gamma, what)


def test_gpu_small_batches_betae():
    _run(O.BETAE, ["1p", "3p", "2in", "inp", "pni", "up"], [1, 2, 5])


def test_gpu_small_batches_q2b():
    _run(O.Q2B, ["1p", "2i", "ip", "2u", "up"], [1, 3, 17])


def test_gpu_small_batches_gqe():
    _run(O.GQE, ["2p", "3i", "up"], [1, 4])


def test_gpu_small_batch_mixed_matches_large_batch():
    """The same queries executed alone (small-batch paths) and inside a large
    mixed batch (full paths) agree within the tolerance."""
    import torch
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(O.Q2B, n_ent=2000, n_rel=9, dim=400, seed=41)
    eng = kgq.engine_for(w, max_batch=1100)
    mixed = synth.draw_mixed(synth.EPFO, 1100, 2000, 9, seed=42)
    big = eng.execute(mixed.structure_ids, mixed.anchors, mixed.relations, k=10, scores=True)
    torch.cuda.synchronize()
    for q in (0, 7, 1099):
        one = eng.execute(mixed.structure_ids[q:q + 1], mixed.anchors[q:q + 1], mixed.relations[q:q + 1], k=10,
                          scores=True)
        torch.cuda.synchronize()
        check_scores(one["scores"].cpu().numpy(), big["scores"].cpu().numpy()[q:q + 1].astype(np.float64),
                     w.rtol, w.gamma, f"query {q}")


@pytest.mark.parametrize("n_ent,batches", [(33000, [64, 65, 128, 129]), (20000, [65, 129])])
def test_gpu_betae_scorer_path_boundary(n_ent, batches):
    """The BetaE scorer takes the FP32 64 x 64 tile up to 64 scored rows, or up
    to 128 when 128-row tiles would give fewer than 256 workgroups, and the
    bf16 split tile above (2d = 64). 33,000 entities give 258 entity tiles of
    128: 64 rows on the FP32 tile, 65, 128 and 129 on the bf16 one; 20,000
    give 157: 65 rows on the FP32 tile, 129 on the bf16 one. Both sides of
    each boundary against the oracle."""
    _run(O.BETAE, ["1p"], batches, n_ent=n_ent, n_rel=7, dim=32, seed=57)
