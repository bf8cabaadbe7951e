"""GPU parity on small tables with odd sizes: every structure of every model,
single-structure and mixed batches, full score rows and top-k, through the
C ABI, against the CPU oracle."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_02172_amd import synth
from tests.parity import check_scores, check_topk

pytestmark = pytest.mark.gpu

EPFO = list(range(9))
ALL = list(range(14))


def _engine(w, max_batch=64):
    from paper_2503_02172_amd import kgq
    return kgq.engine_for(w, max_batch=max_batch)


def _run_and_check(eng, w, m, sid, anchors, rels, k, mixed=False):
    import torch
    out = eng.execute(sid, anchors, rels, k=k, scores=True)
    torch.cuda.synchronize()
    ora = m.scores(sid if mixed else int(sid), anchors, rels)
    what = f"{w.name} s={sid if not mixed else 'mixed'}"
    check_scores(out["scores"].cpu().numpy(), ora, w.rtol, w.gamma, what)
    check_topk(out["idx"].cpu().numpy(), out["score"].cpu().numpy(), ora, k, w.rtol, w.gamma, what)
    return out


@pytest.mark.parametrize("model,structures", [(O.GQE, EPFO), (O.Q2B, EPFO), (O.BETAE, ALL)],
                         ids=["gqe", "q2b", "betae"])
@pytest.mark.parametrize("n_ent,dim,B", [(37, 8, 5), (600, 12, 37)], ids=["N37d8", "N600d12"])
def test_gpu_tiny_every_structure(model, structures, n_ent, dim, B):
    w = synth.make_tiny(model, n_ent=n_ent, n_rel=7, dim=dim, seed=100 + model)
    m = O.Model(model, w.params, w.gamma)
    eng = _engine(w)
    for s in structures:
        name = synth.STRUCTURES[s]
        print(f"[tiny] model={model} N={n_ent} d={dim} B={B} structure={name}", flush=True)
        qb = synth.draw_queries(name, B, n_ent, 7, seed=1000 + s)
        _run_and_check(eng, w, m, s, qb.anchors, qb.relations, min(5, n_ent))
    eng.close()


@pytest.mark.parametrize("model", [O.GQE, O.Q2B, O.BETAE], ids=["gqe", "q2b", "betae"])
def test_gpu_tiny_mixed(model):
    w = synth.make_tiny(model, n_ent=300, n_rel=9, dim=16, seed=200 + model)
    m = O.Model(model, w.params, w.gamma)
    eng = _engine(w, max_batch=64)
    structs = synth.STRUCTURES[:9] if model != O.BETAE else synth.STRUCTURES
    qb = synth.draw_mixed(structs, 53, 300, 9, seed=7)
    print(f"[tiny-mixed] model={model} B=53", flush=True)
    _run_and_check(eng, w, m, qb.structure_ids, qb.anchors, qb.relations, 10, mixed=True)
    eng.close()


@pytest.mark.parametrize("model", [O.GQE, O.Q2B], ids=["gqe", "q2b"])
@pytest.mark.parametrize("dim,B", [(344, 1100), (684, 1100), (1028, 53)],
                         ids=["d344-large", "d684-large", "d1028-small"])
def test_gpu_pack_chunk_tails(model, dim, B):
    """The query pack transposes a block of TQ rows through LDS, KC
    dimensions at a time: KC = 340 for the large form (12 Query2Box or 24 GQE
    rows per wavefront, more than 1,024 scored rows) and KC = 1,024 for the
    small form (4 or 8 rows). d = 344 and d = 684 at B = 1,100 (more than
    1,024 scored rows: large form) end in a 4-dimension tail after one and
    two full chunks; d = 1,028 at B = 53 (small form) after one. Mixed
    batches with unions, so groups and pairs of rows are packed across the
    chunk boundaries too."""
    w = synth.make_tiny(model, n_ent=300, n_rel=5, dim=dim, seed=300 + dim + model)
    m = O.Model(model, w.params, w.gamma)
    eng = _engine(w, max_batch=B)
    qb = synth.draw_mixed(synth.STRUCTURES[:9], B, 300, 5, seed=11)
    rows = eng.describe_plan(qb.structure_ids)["scored_rows"]
    assert (rows > 1024) == (B > 1024), rows
    print(f"[pack-tails] model={model} d={dim} B={B} scored rows={rows}", flush=True)
    _run_and_check(eng, w, m, qb.structure_ids, qb.anchors, qb.relations, 10, mixed=True)
    eng.close()


@pytest.mark.parametrize("model", [O.GQE, O.Q2B], ids=["gqe", "q2b"])
@pytest.mark.parametrize("B", [1024, 1025])
def test_gpu_small_form_switch(model, B):
    """Up to 1,024 scored rows the pack and scorer use fewer rows per
    wavefront; 1p queries score one row each, so B = 1024 runs the small form
    and B = 1025 the large one, on the same tables. At N = 300 (two entity
    blocks) and d = 48, B = 1025 makes fewer than 128 scorer workgroups
    (22 Query2Box or 11 GQE query groups x 2 blocks), so the large form also
    runs its split-dimension path (partials summed by a second kernel). At
    B = 1024 the small form makes 128 workgroups for Query2Box (no split) and
    64 for GQE (split)."""
    w = synth.make_tiny(model, n_ent=300, n_rel=5, dim=48, seed=400 + model)
    m = O.Model(model, w.params, w.gamma)
    eng = _engine(w, max_batch=B)
    qb = synth.draw_queries("1p", B, 300, 5, seed=13)
    print(f"[small-switch] model={model} B={B} d=48", flush=True)
    _run_and_check(eng, w, m, 0, qb.anchors, qb.relations, 10)
    eng.close()


@pytest.mark.parametrize("dim", [32, 40])
@pytest.mark.parametrize("model", [O.GQE, O.Q2B, O.BETAE], ids=["gqe", "q2b", "betae"])
def test_gpu_tiny_dense_bf16x3(model, dim):
    """Every dense layer forced onto the bf16 matrix-core path (weights and
    inputs split into three bf16 parts, six part products): every structure,
    then a mixed batch, at d = 32 (every layer's K a multiple of 32) and
    d = 40 (K = 40 or 80: a last stage of 8 or 16 columns against
    zero-padded weight planes), with 70 entities (a ragged entity tile) and
    37 queries (ragged row tiles)."""
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(model, n_ent=70, n_rel=7, dim=dim, seed=130 + model)
    m = O.Model(model, w.params, w.gamma)
    eng = _engine(w)
    eng.set_dense_path(kgq.DENSE_BF16X3)
    structures = EPFO if model != O.BETAE else ALL
    for s in structures:
        name = synth.STRUCTURES[s]
        print(f"[bf16x3] model={model} d={dim} structure={name}", flush=True)
        qb = synth.draw_queries(name, 37, 70, 7, seed=1300 + s)
        _run_and_check(eng, w, m, s, qb.anchors, qb.relations, 5)
    qb = synth.draw_mixed([synth.STRUCTURES[s] for s in structures], 53, 70, 7, seed=1399)
    _run_and_check(eng, w, m, qb.structure_ids, qb.anchors, qb.relations, 10, mixed=True)
    eng.close()
