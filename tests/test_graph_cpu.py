"""Structure compilation without a GPU: the text reader, the graph rules, and
the fused plan the compiler produces (Algorithm 1's groups), observed
through kgq_structure_info and kgq_describe_plan on a validation-only
handle (device = -1)."""

import numpy as np
import pytest

from paper_2503_02172_amd import kgq, synth

INVALID, UNSUP, NO_DEV = -1, -4, -5
S = synth.STRUCTURE_ID
NEG = ("2in", "3in", "inp", "pin", "pni")


def dry(model=kgq.GQE, max_batch=16, N=50, R=6, d=8):
    return kgq.Engine(model, N, R, d, 12.0, max_batch, 0.02, kgq.F32, device=-1)


def rc_of(fn):
    with pytest.raises(kgq.KgqError) as ei:
        fn()
    return ei.value.status


def nodes(rows):
    return np.asarray(rows, np.int32).reshape(-1, 6)


def test_parse_matches_the_input_module_reader():
    for seed in range(40):
        t = synth.random_structure(seed, negation=seed % 3 == 0)
        assert np.array_equal(kgq.parse_structure(t), synth.graph_nodes(t)), t
    assert np.array_equal(kgq.parse_structure(" p ( e0 , r0 ) "), synth.graph_nodes("p(e0,r0)"))


def test_parse_errors():
    for t in ["", "p(e0)", "i(p(e0,r0))", "x(e0)", "p(e0,r0) p(e1,r1)", "p(e0,q0)",
              "u(p(e0,r0),p(e1,r1),p(e2,r2),p(e3,r3),p(e4,r4))", "n(p(e0,r0)", "e"]:
        assert rc_of(lambda: kgq.parse_structure(t)) == INVALID, t
    deep = "e0"
    for h in range(70):
        deep = f"p({deep},r0)"
    assert rc_of(lambda: kgq.parse_structure(deep)) == INVALID   # 71 nodes > 64


def test_compile_rules():
    e = dry(kgq.BETAE)
    A, P, AND, OR, NOT = 0, 1, 2, 3, 4
    bad = {
        "forward input": [[P, 0, 1, -1, -1, -1], [A, 0, -1, -1, -1, -1]],
        "unused node": [[A, 0, -1, -1, -1, -1], [P, 0, 0, -1, -1, -1], [A, 1, -1, -1, -1, -1]],
        "anchor into intersection": [[A, 0, -1, -1, -1, -1], [P, 0, 0, -1, -1, -1], [AND, -1, 0, 1, -1, -1]],
        "anchor answer": [[A, 0, -1, -1, -1, -1]],
        "slot gap": [[A, 1, -1, -1, -1, -1], [P, 0, 0, -1, -1, -1]],
        "slot too large": [[A, 0, -1, -1, -1, -1], [P, 8, 0, -1, -1, -1]],
        "one-input union": [[A, 0, -1, -1, -1, -1], [P, 0, 0, -1, -1, -1], [OR, -1, 1, -1, -1, -1]],
        "unpacked inputs": [[A, 0, -1, -1, -1, -1], [P, 0, 0, -1, -1, -1], [A, 1, -1, -1, -1, -1],
                            [P, 1, 2, -1, -1, -1], [AND, -1, 1, -1, 3, -1]],
        "unknown op": [[A, 0, -1, -1, -1, -1], [9, 0, 0, -1, -1, -1]],
    }
    for what, g in bad.items():
        assert rc_of(lambda: e.compile(nodes(g))) == INVALID, what
    # more than four terms at a node once unions are distributed
    eight = "i(u(p(e0,r0),p(e1,r1)),u(p(e2,r2),p(e3,r3)),u(p(e4,r4),p(e5,r5)))"
    assert rc_of(lambda: e.compile(eight)) == INVALID
    # negation only on BetaE
    for m in (kgq.GQE, kgq.Q2B):
        assert rc_of(lambda: dry(m).compile("i(p(e0,r0),n(p(e1,r1)))")) == UNSUP
    # the per-handle limit
    f = dry(kgq.GQE)
    ids = [f.compile("p(e0,r0)") for _ in range(64)]
    assert ids == list(range(14, 78))
    assert rc_of(lambda: f.compile("p(e0,r0)")) == INVALID


@pytest.mark.parametrize("model", [kgq.GQE, kgq.Q2B, kgq.BETAE, kgq.CONE, kgq.LOGICE])
def test_builtins_compile_like_their_text(model):
    """A built-in structure and its text form compiled on the handle lower to
    the same plan, alone and mixed."""
    e = dry(model, max_batch=64)
    names = [n for n in synth.STRUCTURES if model in synth.NEGATION_MODELS or n not in NEG]
    own = {n: e.compile(synth.STRUCTURE_TEXT[n]) for n in names}
    for n in names:
        assert e.describe_plan([S[n]] * 3) == e.describe_plan([own[n]] * 3), n
        info = e.structure_info(own[n])
        assert (info["anchors"], info["relations"]) == synth.ARITY[n]
        assert info["launches"] == e.describe_plan([S[n]])["launches"]
        assert e.structure_info(S[n]) == info
    mix = [S[n] for n in names] * 2
    assert e.describe_plan(mix) == e.describe_plan([own[synth.STRUCTURES[s]] for s in mix])
    if model not in synth.NEGATION_MODELS:
        assert rc_of(lambda: e.structure_info(S["2in"])) == UNSUP


def test_horizontal_fusion_one_chain_per_path():
    """GQE / Query2Box: a run of projections is one fused chain, whatever its
    length; BetaE runs one projection level per hop."""
    for model in (kgq.GQE, kgq.Q2B):
        e = dry(model)
        for hops in range(1, 9):
            t = "e0"
            for h in range(hops):
                t = f"p({t},r{h})"
            info = e.structure_info(e.compile(t))
            assert info["fused_ops"] == 1 and info["launches"] == 4, (model, hops, info)
    for model in (kgq.BETAE, kgq.CONE):
        e = dry(model)
        info = e.structure_info(e.compile("p(p(p(p(e0,r0),r1),r2),r3)"))
        assert info["fused_ops"] == 4
        assert info["launches"] == 3 + 3 * 4 + 3   # table-path first hop, three full hops, pack/score/top-k
    # LogicE: one more launch per hop (the bound map after the sigmoid layer)
    e = dry(kgq.LOGICE)
    info = e.structure_info(e.compile("p(p(p(p(e0,r0),r1),r2),r3)"))
    assert info["fused_ops"] == 4 and info["launches"] == 4 + 3 * 5 + 3


def test_vertical_and_hybrid_fusion():
    """An intersection is one group; projections after it fold into its
    combine on GQE / Query2Box and run as projection levels on BetaE."""
    t = "p(p(i(p(e0,r0),p(e1,r1),p(p(e2,r2),r3)),r4),r5)"
    g = dry(kgq.GQE)
    info = g.structure_info(g.compile(t))
    assert info["fused_ops"] == 4 and info["intersection_stages"] == 1
    assert info["launches"] == 1 + 3 + 3
    q = dry(kgq.Q2B)
    assert q.structure_info(q.compile(t))["launches"] == 1 + 6 + 3
    b = dry(kgq.BETAE)
    sid = b.compile(t)
    p = b.describe_plan([sid, sid])
    assert (p["level1"], p["level2"], p["post"], p["groups"], p["intersection_inputs"]) == (6, 2, 4, 2, 6)
    assert b.structure_info(sid)["fused_ops"] == 4 + 1 + 2
    # ConE and LogicE plan like BetaE; an intersection stage is 6 launches
    # for ConE (prep, stacked first layers, attention layer, axis combine,
    # gate layer, aperture combine) and 1 for LogicE (the t-norm)
    for model, per_and, per_level in ((kgq.CONE, 6, 4), (kgq.LOGICE, 1, 5)):
        e = dry(model)
        sid = e.compile(t)
        pm = e.describe_plan([sid, sid])
        assert {k: v for k, v in pm.items() if k != "launches"} == {k: v for k, v in p.items() if k != "launches"}
        info = e.structure_info(sid)
        assert info["fused_ops"] == 4 + 1 + 2
        # levels: first hop (table path), the second hop of the 2p branch, two post hops
        assert info["launches"] == (per_level - 1) + 3 * per_level + per_and + 3


def test_nested_intersections_run_in_stages():
    """An intersection over another intersection's result runs one stage
    later; all intersections of a stage run together across the batch."""
    t = "i(p(i(p(e0,r0),p(e1,r1)),r2),p(e2,r3))"
    for model in (kgq.GQE, kgq.Q2B, kgq.BETAE, kgq.CONE, kgq.LOGICE):
        e = dry(model, max_batch=32)
        sid = e.compile(t)
        p = e.describe_plan([sid, S["2i"], sid])
        assert p["intersection_stages"] == 2
        assert p["groups"] == 2 + 1 + 2
        assert p["intersection_inputs"] == 4 + 2 + 4


def test_normal_form_rows():
    """Unions move to the top (Eq. 1): 2 terms score as a pair, 3 or 4 terms
    as a group of four rows; the negation of a union is one intersection."""
    e = dry(kgq.BETAE, max_batch=32)
    cases = {
        "u(p(e0,r0),p(e1,r1),p(e2,r2))": (3, 4, 0, 1),
        "i(u(p(e0,r0),p(e1,r1)),u(p(e2,r2),p(e3,r3)))": (4, 4, 4, 1),
        "i(u(p(e0,r0),p(e1,r1)),p(e2,r2))": (2, 2, 2, 0),
        "n(u(p(e0,r0),p(e1,r1)))": (1, 1, 1, 0),
        "i(n(n(p(e0,r0))),p(e1,r1))": (1, 1, 1, 0),
    }
    for t, (terms, rows, groups, quads) in cases.items():
        sid = e.compile(t)
        assert e.structure_info(sid)["terms"] == terms, t
        p = e.describe_plan([sid])
        assert (p["scored_rows"], p["groups"], p["union_quads"]) == (rows, groups, quads), t
    # double negation folds: same plan as 2i
    assert e.describe_plan([e.compile("i(n(n(p(e0,r0))),p(e1,r1))")]) == e.describe_plan([S["2i"]])


def test_capacity_bounds_and_mixed_arity():
    """A structure larger than the built-ins reports a smaller batch bound,
    and a batch above it is refused before anything runs; structures with
    more than 3 slots cannot join a mixed batch."""
    e = dry(kgq.Q2B, max_batch=16)
    e.load_all(synth.make_tiny(kgq.Q2B, n_ent=50, n_rel=6, dim=8).params)
    big = "u(i(p(e0,r0),p(e1,r1),p(e2,r2)),i(p(e3,r3),p(e4,r4),p(e5,r5)),p(e6,r6))"
    sid = e.compile(big)
    mb = e.structure_info(sid)["max_batch"]
    assert 1 <= mb < 16
    a = np.zeros((mb + 1, 7), np.int32)
    assert rc_of(lambda: e.execute_into(sid, mb + 1, a, a, 5, None, a, a.astype(np.float32), 0)) == INVALID
    assert rc_of(lambda: e.execute_into(sid, mb, a, a, 5, None, a, a.astype(np.float32), 0)) == NO_DEV
    four = e.compile("p(p(p(p(e0,r0),r1),r2),r3)")
    ids = np.array([S["1p"], four], np.int32)
    m3 = np.zeros((2, 3), np.int32)
    assert rc_of(lambda: e.execute_mixed_into(ids, m3, m3, 5, None, m3, m3.astype(np.float32), 0)) == INVALID
