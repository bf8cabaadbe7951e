"""GPU edge cases: exact ties, k limits, batch of one, checked mode, bad
padding, determinism, non-default streams, and the dense layer on its own."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_02172_amd import synth
from tests.parity import check_scores, check_topk

pytestmark = pytest.mark.gpu
S = synth.STRUCTURE_ID


def _eng(w, **kw):
    from paper_2503_02172_amd import kgq
    return kgq.engine_for(w, **kw)


def test_gpu_exact_ties_order_by_index():
    import torch
    for model in (O.GQE, O.Q2B, O.BETAE):
        w = synth.make_tiny(model, n_ent=700, n_rel=5, dim=16, seed=40 + model)
        key = "entity.alpha_beta" if model == O.BETAE else "entity"
        if model != O.BETAE:   # relation 0 moves nothing: the anchor row scores best
            rk = "relation" if model == O.GQE else "relation.center"
            rel = w.params[rk].copy()
            rel[0] = 0.0
            w.params[rk] = rel
        ent = w.params[key].copy()
        dup = [3, 260, 511, 699]          # rows copied from entity 100, across blocks
        ent[dup] = ent[100]
        w.params[key] = ent
        eng = _eng(w, max_batch=8)
        m = O.Model(model, w.params, w.gamma)
        # the 1p query anchored at 100 with the relation that keeps it closest
        a = np.full((4, 1), 100, np.int32)
        r = np.arange(4, dtype=np.int32)[:, None]
        out = eng.execute(S["1p"], a, r, k=50, scores=True)
        torch.cuda.synchronize()
        sc = out["scores"].cpu().numpy()
        idx = out["idx"].cpu().numpy()
        for q in range(4):
            tied = sc[q, [100] + dup]
            assert np.all(tied == tied[0]), "identical rows must score identically"
            pos = [int(np.nonzero(idx[q] == e)[0][0]) for e in sorted([100] + dup) if e in idx[q]]
            assert pos == sorted(pos), "tied entities must appear in index order"
        ora = m.scores(S["1p"], a, r)
        check_topk(idx, out["score"].cpu().numpy(), ora, 50, w.rtol, w.gamma, f"ties model {model}")
        if model != O.BETAE:
            # relation 0: the five identical rows tie for first place; k = 3 cuts
            # through the tie, so the three lowest indices are taken, in order
            small = eng.execute(S["1p"], a[:1], r[:1], k=3)
            torch.cuda.synchronize()
            assert small["idx"].cpu().numpy()[0].tolist() == [3, 100, 260]
        eng.close()


@pytest.mark.parametrize("N,k", [(37, 1), (37, 37), (1500, 1024), (1500, 1), (5000, 100), (16384, 7),
                                 (16385, 300), (40000, 1024), (40000, 100)])
def test_gpu_k_limits(N, k):
    import torch
    w = synth.make_tiny(O.Q2B, n_ent=N, n_rel=5, dim=8, seed=50)
    eng = _eng(w, max_batch=8)
    m = O.Model(O.Q2B, w.params, w.gamma)
    qb = synth.draw_queries("2u", 3, N, 5, seed=51)
    out = eng.execute(S["2u"], qb.anchors, qb.relations, k=k)
    torch.cuda.synchronize()
    ora = m.scores(S["2u"], qb.anchors, qb.relations)
    check_topk(out["idx"].cpu().numpy(), out["score"].cpu().numpy(), ora, k, w.rtol, w.gamma, f"N={N} k={k}")
    eng.close()


def test_gpu_ties_across_topk_segments():
    """Rows longer than one top-k segment are reduced in rounds; exact ties in
    different segments must still come out lowest index first."""
    import torch
    w = synth.make_tiny(O.GQE, n_ent=40000, n_rel=3, dim=8, seed=90)
    rel = w.params["relation"].copy()
    rel[0] = 0.0
    w.params["relation"] = rel
    ent = w.params["entity"].copy()
    dup = [5, 16383, 16384, 32768, 39999]
    ent[dup] = ent[20000]
    w.params["entity"] = ent
    eng = _eng(w, max_batch=4)
    a = np.full((2, 1), 20000, np.int32)
    r = np.zeros((2, 1), np.int32)
    for k, want in ((3, [5, 16383, 16384]), (6, [5, 16383, 16384, 20000, 32768, 39999]), (100, None)):
        out = eng.execute(S["1p"], a, r, k=k)
        torch.cuda.synchronize()
        got = out["idx"].cpu().numpy()
        if want is not None:
            assert got[0].tolist() == want and got[1].tolist() == want
        else:
            assert got[0, :6].tolist() == sorted(dup + [20000])
            m = O.Model(O.GQE, w.params, w.gamma)
            check_topk(got, out["score"].cpu().numpy(), m.scores(S["1p"], a, r), k, w.rtol, w.gamma)
    eng.close()


def test_gpu_batch_of_one_and_reuse_of_cached_plans():
    import torch
    w = synth.make_tiny(O.BETAE, n_ent=333, n_rel=6, dim=8, seed=60)
    eng = _eng(w, max_batch=40)
    m = O.Model(O.BETAE, w.params, w.gamma)
    for B in (1, 40, 7, 1):   # batch size changes re-lower the cached plan
        for s in (S["ip"], S["pni"], S["up"]):
            qb = synth.draw_queries(synth.STRUCTURES[s], B, 333, 6, seed=61 + B + s)
            out = eng.execute(s, qb.anchors, qb.relations, k=7, scores=True)
            torch.cuda.synchronize()
            ora = m.scores(s, qb.anchors, qb.relations)
            check_scores(out["scores"].cpu().numpy(), ora, w.rtol, w.gamma, f"B={B} s={s}")
            check_topk(out["idx"].cpu().numpy(), out["score"].cpu().numpy(), ora, 7, w.rtol, w.gamma)
    eng.close()


def test_gpu_checked_mode_reports_bad_ids():
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(O.GQE, n_ent=64, n_rel=5, dim=8, seed=70)
    eng = _eng(w, max_batch=8)
    eng.set_checked(True)
    a = np.array([[1, 2], [3, 64]], np.int32)          # 64 is out of range
    r = np.array([[0, 1], [2, 3]], np.int32)
    with pytest.raises(kgq.KgqError) as e:
        eng.execute(S["2i"], a, r, k=3)
    assert e.value.status == -2
    r_bad = np.array([[0, 1], [2, -7]], np.int32)
    with pytest.raises(kgq.KgqError) as e:
        eng.execute(S["2i"], np.array([[1, 2], [3, 4]], np.int32), r_bad, k=3)
    assert e.value.status == -2
    # mixed batch: an unused slot that is not -1
    sid = np.array([S["1p"], S["2i"]], np.int32)
    a = np.array([[5, 0, -1], [1, 2, -1]], np.int32)     # query 0 slot 1 should be -1
    r = np.array([[0, -1, -1], [1, 2, -1]], np.int32)
    with pytest.raises(kgq.KgqError) as e:
        eng.execute(sid, a, r, k=3)
    assert e.value.status == -1
    # a valid batch still runs in checked mode, and unchecked mode never faults
    a[0, 1] = -1
    eng.execute(sid, a, r, k=3)
    eng.set_checked(False)
    eng.execute(S["2i"], np.array([[1, 2], [3, 9999]], np.int32), np.array([[0, 1], [2, 3]], np.int32), k=3)
    import torch
    torch.cuda.synchronize()
    eng.close()


def test_gpu_deterministic_and_stream():
    import torch
    w = synth.make_tiny(O.Q2B, n_ent=3000, n_rel=9, dim=32, seed=80)
    eng = _eng(w, max_batch=64)
    qb = synth.draw_mixed(synth.STRUCTURES[:9], 60, 3000, 9, seed=81)
    a = eng.execute(qb.structure_ids, qb.anchors, qb.relations, k=20, scores=True)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b = eng.execute(qb.structure_ids, qb.anchors, qb.relations, k=20, scores=True)
    s.synchronize()
    torch.cuda.synchronize()
    for key in ("scores", "idx", "score"):
        assert torch.equal(a[key], b[key]), key
    eng.close()


@pytest.mark.parametrize("path", [0, 1, 2], ids=["auto", "fp32", "bf16x3"])
@pytest.mark.parametrize("M,N,K,act", [(1, 1, 4, 0), (37, 50, 12, 1), (130, 1600, 800, 1), (700, 800, 1600, 2),
                                       (64, 64, 64, 0), (1029, 400, 400, 0),
                                       # direct-to-LDS loop: one half stage, stages fewer than / equal to
                                       # the ring, a half last stage after full ones, ragged M and N
                                       (65, 70, 16, 1), (200, 33, 48, 0), (129, 127, 80, 2), (66, 190, 96, 1),
                                       (3, 400, 400, 1),
                                       # bf16 path: one or two stages, ragged tiles, 64 x 128 tiles
                                       (65, 70, 32, 1), (200, 33, 64, 0), (129, 127, 96, 2),
                                       (1100, 800, 800, 1), (4100, 1100, 160, 0), (4097, 1030, 1600, 1),
                                       # bf16 path, K not a multiple of 32: a last stage of 4, 16 or 8
                                       # columns against zero-padded weight planes (64 x 64 and
                                       # 128 x 64 tiles)
                                       (65, 70, 36, 1), (129, 127, 48, 0), (1100, 800, 400, 1),
                                       (300, 1600, 1200, 1), (4100, 1100, 400, 0), (2050, 1030, 1000, 2)])
def test_gpu_dense_matches_fp64(M, N, K, act, path):
    """One dense layer against an fp64 matmul on each path: automatic choice,
    FP32 matrix cores only, and the bf16 path wherever K allows it (a
    multiple of 4, at least 32; x split into three bf16 parts in registers,
    w into zero-padded planes when the layer is set up)."""
    import torch
    from paper_2503_02172_amd import kgq
    rng = np.random.default_rng(M * 7 + N)
    x = rng.uniform(-1, 1, (M, K)).astype(np.float32)
    wt = (rng.uniform(-1, 1, (N, K)) / np.sqrt(K)).astype(np.float32)
    b = rng.uniform(-0.5, 0.5, N).astype(np.float32)
    eng = kgq.Engine(kgq.GQE, 10, 2, 4, 1.0, 1, device=0)
    eng.set_dense_path(path)
    y = eng.dense(torch.tensor(x, device="cuda"), torch.tensor(wt, device="cuda"),
                  torch.tensor(b, device="cuda"), act)
    torch.cuda.synchronize()
    ref = x.astype(np.float64) @ wt.astype(np.float64).T + b
    if act == 1:
        ref = np.maximum(ref, 0)
    elif act == 2:
        ref = np.clip(ref + 1, 0.05, 1e9)
    # fp32 accumulation of K products of magnitude <= 1/sqrt(K)
    np.testing.assert_allclose(y.cpu().numpy(), ref, rtol=1e-5, atol=1e-5 * np.sqrt(K) / 10 + 1e-6)
    eng.close()


def test_gpu_concurrent_streams_match_sequential():
    """Executes on different streams use separate scratch sets and may overlap;
    their results equal those of the same calls on one stream."""
    import torch
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(O.Q2B, n_ent=5000, n_rel=11, dim=16, seed=95)
    seq = kgq.engine_for(w, max_batch=64, concurrency=1)
    con = kgq.engine_for(w, max_batch=64, concurrency=2)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    qs = [synth.draw_queries(n, 40 + i, 5000, 11, seed=96 + i) for i, n in enumerate(["2i", "up", "3p", "pi"])]
    ref = []
    for qb in qs:
        ref.append(seq.execute(S[qb.structure], qb.anchors, qb.relations, k=25, scores=True))
    torch.cuda.synchronize()
    outs = []
    for i, qb in enumerate(qs):
        with torch.cuda.stream(streams[i % 2]):
            outs.append(con.execute(S[qb.structure], qb.anchors, qb.relations, k=25, scores=True))
    torch.cuda.synchronize()
    for r, o in zip(ref, outs):
        for key in ("scores", "idx", "score"):
            assert torch.equal(r[key], o[key]), key
    seq.close()
    con.close()



@pytest.mark.parametrize("model", [O.Q2B, O.BETAE])
def test_gpu_concurrent_mixed_calls_match_sequential(model):
    """Mixed-structure executes alternating between two streams on a handle
    with two scratch lanes (more calls than lanes, no host sync between them,
    so lanes and plan-upload slots are reused while earlier calls may still
    run) equal the same calls made one at a time on one stream."""
    import torch
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(model, n_ent=3000, n_rel=9, dim=32, seed=120 + model)
    structs = synth.STRUCTURES if model == O.BETAE else synth.STRUCTURES[:9]
    seq = kgq.engine_for(w, max_batch=64, concurrency=1)
    con = kgq.engine_for(w, max_batch=64, concurrency=2)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    qs = [synth.draw_mixed(structs, n, 3000, 9, seed=130 + i) for i, n in enumerate([60, 17, 64, 5, 33, 48])]
    ref = [seq.execute(qb.structure_ids, qb.anchors, qb.relations, k=20, scores=True) for qb in qs]
    torch.cuda.synchronize()
    outs = []
    for i, qb in enumerate(qs):
        with torch.cuda.stream(streams[i % 2]):
            outs.append(con.execute(qb.structure_ids, qb.anchors, qb.relations, k=20, scores=True))
    torch.cuda.synchronize()
    for r, o in zip(ref, outs):
        for key in ("scores", "idx", "score"):
            assert torch.equal(r[key], o[key]), key
    seq.close()
    con.close()

def test_gpu_memory_accounting():
    """Parameters do not depend on max_batch; the execute scratch grows with
    max_batch and scales with the number of concurrency lanes; BetaE holds the
    first-layer tables ([N x 4d] + [R x 4d] floats) among its parameters."""
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(O.BETAE, n_ent=300, n_rel=7, dim=16, seed=5)
    m8 = _eng(w, max_batch=8).memory()
    m64 = _eng(w, max_batch=64).memory()
    m8x2 = _eng(w, max_batch=8, concurrency=2).memory()
    assert m8["param_bytes"] == m64["param_bytes"] == m8x2["param_bytes"] > 0
    assert m64["scratch_bytes"] > m8["scratch_bytes"] > 0
    assert m8x2["scratch_bytes"] == 2 * m8["scratch_bytes"]
    d, N, R = 16, 300, 7
    assert m8["param_bytes"] >= 4 * (N * 4 * d + R * 4 * d)
    g = synth.make_tiny(O.GQE, n_ent=300, n_rel=7, dim=16, seed=5)
    assert _eng(g, max_batch=8).memory()["param_bytes"] < m8["param_bytes"]
    assert kgq.BETAE == O.BETAE


def test_gpu_batch_above_65535():
    """A batch larger than the 65,535 limit of a grid's y and z dimensions:
    every kernel launches over a one-dimensional grid (or y within limits)."""
    import torch
    B = 70000
    w = synth.make_tiny(O.GQE, n_ent=37, n_rel=5, dim=8, seed=21)
    eng = _eng(w, max_batch=B)
    q = synth.draw_queries("2i", B, 37, 5, seed=22)
    out = eng.execute(S["2i"], q.anchors, q.relations, k=5, scores=True)
    torch.cuda.synchronize()
    m = O.Model(O.GQE, w.params, w.gamma)
    rows = np.r_[0:50, B - 50:B, 30000:30050]
    ref = m.scores(np.full(rows.size, S["2i"]), q.anchors[rows], q.relations[rows])
    check_scores(out["scores"].cpu().numpy()[rows], ref, w.rtol, w.gamma, "2i B=70000")
    check_topk(out["idx"].cpu().numpy()[rows], out["score"].cpu().numpy()[rows], ref, 5, w.rtol, w.gamma,
               "2i B=70000")


def test_gpu_execute_on_a_non_current_stream():
    """Engine.execute(stream=s) with s not the current stream allocates its
    device copies of the inputs and its outputs on s, so memory handed out on
    the current stream right after the call cannot alias buffers the library
    still reads or writes on s. The results equal a plain call's."""
    import torch
    from oracle import oracle as O
    from paper_2503_02172_amd import kgq, synth

    w = synth.make_tiny(O.Q2B, n_ent=5000, n_rel=7, dim=256, seed=61)
    qb = synth.draw_mixed(synth.STRUCTURES[:9], 300, 5000, 7, seed=62)
    with kgq.engine_for(w, max_batch=300) as eng:
        ref = eng.execute(qb.structure_ids, qb.anchors, qb.relations, k=20, scores=True)
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        for it in range(3):
            out = eng.execute(qb.structure_ids, qb.anchors, qb.relations, k=20, scores=True, stream=s)
            # immediately allocate and overwrite memory on the current stream
            junk = [torch.full((300, 5000), -7.0, device="cuda") for _ in range(4)]
            junk2 = torch.full((300, 3), -1, dtype=torch.int32, device="cuda")
            s.synchronize()
            torch.cuda.synchronize()
            assert torch.equal(out["scores"], ref["scores"]), f"iteration {it}"
            assert torch.equal(out["idx"], ref["idx"]) and torch.equal(out["score"], ref["score"])
            del junk, junk2, out
