"""GPU parity of compiled query structures: graphs (Eq. 2) that the library
rewrites into normal form and fuses (Algorithm 1), executed through the C
ABI and compared element by element with the oracle's node-by-node
evaluation of the same graph on the same seeded inputs."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_02172_amd import synth
from tests.parity import check_scores, check_topk

pytestmark = pytest.mark.gpu
S = synth.STRUCTURE_ID
NEG = ("2in", "3in", "inp", "pin", "pni")


def setup(model, n_ent=301, n_rel=13, dim=8, seed=7, max_batch=96):
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(model, n_ent=n_ent, n_rel=n_rel, dim=dim, seed=seed)
    return w, kgq.engine_for(w, max_batch=max_batch), O.Model(model, w.params, w.gamma)


def run_graph(eng, m, w, text, B, seed, k=10):
    import torch
    nodes = synth.graph_nodes(text)
    sid = eng.compile(text)
    B = min(B, eng.structure_info(sid)["max_batch"])   # larger structures hold fewer queries
    q = synth.draw_graph_queries(nodes, B, w.n_entities, w.n_relations, seed)
    print(f"[graph] model={w.model} B={B} {text}", flush=True)
    out = eng.execute(sid, q.anchors, q.relations, k=k, scores=True)
    torch.cuda.synchronize()
    ref = m.graph_scores(nodes, q.anchors, q.relations)
    what = f"model {w.model} B={B} {text}"
    check_scores(out["scores"].cpu().numpy(), ref, w.rtol, w.gamma, what)
    check_topk(out["idx"].cpu().numpy(), out["score"].cpu().numpy(), ref, k, w.rtol, w.gamma, what)


@pytest.mark.parametrize("model", [O.GQE, O.Q2B, O.BETAE], ids=["gqe", "q2b", "betae"])
def test_gpu_builtin_text_equals_builtin_id(model):
    """A built-in structure compiled from its text runs the same fused plan
    as the built-in id: identical scores and top-k."""
    import torch
    w, eng, m = setup(model)
    for name in synth.STRUCTURES:
        if model != O.BETAE and name in NEG:
            continue
        q = synth.draw_queries(name, 37, w.n_entities, w.n_relations, seed=50 + S[name])
        a = eng.execute(S[name], q.anchors, q.relations, k=10, scores=True)
        b = eng.execute(eng.compile(synth.STRUCTURE_TEXT[name]), q.anchors, q.relations, k=10, scores=True)
        torch.cuda.synchronize()
        assert torch.equal(a["scores"], b["scores"]), name
        assert torch.equal(a["idx"], b["idx"]) and torch.equal(a["score"], b["score"]), name


@pytest.mark.parametrize("model", [O.GQE, O.Q2B, O.BETAE], ids=["gqe", "q2b", "betae"])
def test_gpu_random_structures(model):
    w, eng, m = setup(model, seed=11 + model)
    for i in range(16):
        seed = 1000 * model + i
        text = synth.random_structure(seed, negation=model == O.BETAE)
        run_graph(eng, m, w, text, B=[1, 7, 33, 70][i % 4], seed=seed)


EDGE = [
    "p(p(p(p(p(p(p(p(e0,r0),r1),r2),r3),r4),r5),r6),r7)",          # one chain of 8 hops
    "i(p(i(p(i(p(e0,r0),p(e1,r1)),r2),p(e2,r3)),r4),p(e3,r5))",      # three intersection stages
    "i(p(e0,r0),p(e1,r1),p(e2,r2),p(e3,r3))",                        # four-way intersection
    "u(p(e0,r0),p(e1,r1),p(e2,r2))",                                 # three terms: a padded group of four
    "i(u(p(e0,r0),p(e1,r1)),u(p(e2,r2),p(e3,r3)))",                  # four terms
    "p(p(i(u(p(e0,r0),p(e1,r1)),p(e2,r2)),r3),r4)",                  # union below an intersection and a chain
    "i(p(i(p(e0,r0),p(e1,r1)),r2),p(i(p(e2,r3),p(e3,r4)),r5))",      # two groups in one later stage
]
EDGE_NEG = [
    "n(p(e0,r0))",                                                   # negated answer
    "i(n(n(p(e0,r0))),p(e1,r1))",                                    # double negation folds
    "n(u(p(e0,r0),p(e1,r1)))",                                       # De Morgan
    "p(n(i(p(e0,r0),p(e1,r1))),r2)",                                 # projection of a negated intersection
    "u(n(p(e0,r0)),i(p(e1,r1),n(p(e2,r2))),p(e3,r3))",               # negated terms in a group of four
    "i(n(u(p(e0,r0),p(e1,r1),p(e2,r2))),p(e3,r3))",                  # three negations in one intersection
]


@pytest.mark.parametrize("model", [O.GQE, O.Q2B, O.BETAE], ids=["gqe", "q2b", "betae"])
@pytest.mark.parametrize("B", [5, 67])
def test_gpu_graph_edge_cases(model, B):
    w, eng, m = setup(model, n_ent=523, seed=21 + model)
    cases = EDGE + (EDGE_NEG if model == O.BETAE else [])
    for i, text in enumerate(cases):
        run_graph(eng, m, w, text, B, seed=300 + i)


@pytest.mark.parametrize("model", [O.GQE, O.Q2B, O.BETAE], ids=["gqe", "q2b", "betae"])
def test_gpu_graph_mixed_with_builtins(model):
    """Built-in and compiled structures in one mixed batch (one plan, one
    launch per fused-operator kind and stage)."""
    import torch
    w, eng, m = setup(model, n_ent=409, seed=31 + model, max_batch=256)
    texts = ["i(p(i(p(e0,r0),p(e1,r1)),r2),p(e2,r2))", "u(p(e0,r0),p(e1,r1),p(p(e2,r2),r2))",
             "p(p(i(u(p(e0,r0),p(e1,r1)),p(e2,r2)),r1),r0)"]
    if model == O.BETAE:
        texts.append("i(n(u(p(e0,r0),p(e1,r1))),p(e2,r2))")
    own = [eng.compile(t) for t in texts]
    names = [n for n in synth.STRUCTURES if model == O.BETAE or n not in NEG]
    pool = [S[n] for n in names] + own
    rng = np.random.default_rng(5 + model)
    B = 200
    sid = np.asarray(rng.choice(pool, size=B), np.int32)
    a = np.full((B, 3), -1, np.int32)
    r = np.full((B, 3), -1, np.int32)
    graphs = {S[n]: synth.graph_nodes(synth.STRUCTURE_TEXT[n]) for n in names}
    graphs.update({s: synth.graph_nodes(t) for s, t in zip(own, texts)})
    for q in range(B):
        na, nr = synth.graph_arity(graphs[int(sid[q])])
        a[q, :na] = rng.integers(0, w.n_entities, na)
        r[q, :nr] = rng.integers(0, w.n_relations, nr)
    print(f"[graph] mixed model={model} B={B}", flush=True)
    out = eng.execute(sid, a, r, k=10, scores=True)
    torch.cuda.synchronize()
    ref = np.empty((B, w.n_entities))
    for s, g in graphs.items():
        rows = np.nonzero(sid == s)[0]
        if rows.size:
            na, nr = synth.graph_arity(g)
            ref[rows] = m.graph_scores(g, a[rows, :na], r[rows, :nr])
    check_scores(out["scores"].cpu().numpy(), ref, w.rtol, w.gamma, f"mixed model {model}")
    check_topk(out["idx"].cpu().numpy(), out["score"].cpu().numpy(), ref, 10, w.rtol, w.gamma, "mixed")


@pytest.mark.parametrize("model", [O.GQE, O.Q2B, O.BETAE], ids=["gqe", "q2b", "betae"])
def test_gpu_graph_full_dim_small_batches(model):
    """d = 400 at batches of 1-3: the small-batch paths (split-K dense layers,
    split-d VALU scoring with its second pass, 64 x 64 matrix-core tiles)
    with groups of four scored rows and several intersection stages."""
    w, eng, m = setup(model, n_ent=1500, n_rel=11, dim=400, seed=41, max_batch=8)
    texts = ["u(p(e0,r0),p(e1,r1),p(e2,r2))", "i(p(i(p(e0,r0),p(e1,r1)),r2),p(e2,r3))"]
    if model == O.BETAE:
        texts.append("u(n(p(e0,r0)),i(p(e1,r1),n(p(e2,r2))),p(e3,r3))")
    for text in texts:
        for B in (1, 3):
            run_graph(eng, m, w, text, B, seed=700 + B)


def test_gpu_graph_at_its_batch_bound():
    """A structure bigger than the built-ins runs at the batch bound the
    handle reports for it, and is refused above it."""
    from paper_2503_02172_amd import kgq
    w, eng, m = setup(O.Q2B, n_ent=257, max_batch=24)
    text = "u(i(p(e0,r0),p(e1,r1),p(e2,r2)),i(p(e3,r3),p(e4,r4),p(e5,r5)),p(e6,r6))"
    sid = eng.compile(text)
    mb = eng.structure_info(sid)["max_batch"]
    assert 1 <= mb < 24
    run_graph(eng, m, w, text, mb, seed=9)
    nodes = synth.graph_nodes(text)
    q = synth.draw_graph_queries(nodes, mb + 1, w.n_entities, w.n_relations, 9)
    with pytest.raises(kgq.KgqError) as ei:
        eng.execute(sid, q.anchors, q.relations, k=10)
    assert ei.value.name == "INVALID_ARG"
