"""C ABI checks that need no GPU: exported symbols, argument validation on a
validation-only handle (device = -1), and the plan lowering's row counts."""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2503_02172_amd import kgq, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kgq.h")

INVALID, RANGE, NOT_LOADED, UNSUP, NO_DEV = -1, -2, -3, -4, -5


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:kgq_status|const char\*)\s+(kgq_\w+)\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    lib = kgq.lib()
    names = declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", kgq.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (kgq_\w+)", out))
    assert set(names) <= exported
    assert exported <= set(names), f"undeclared exports: {exported - set(names)}"


def dry(model=kgq.GQE, N=50, R=6, d=8, max_batch=16, dtype=kgq.F32):
    return kgq.Engine(model, N, R, d, 12.0, max_batch, 0.02, dtype, device=-1)


def fake(n):   # a host address; a validation-only handle never dereferences it
    return np.zeros(max(n, 1), np.int32)


def full_load(e, model, N=50, R=6, d=8):
    w = synth.make_tiny(model, n_ent=N, n_rel=R, dim=d)
    e.load_all(w.params)


def rc_of(fn):
    with pytest.raises(kgq.KgqError) as ei:
        fn()
    return ei.value.status


def test_create_validation():
    bad = [dict(model=5), dict(model=-1), dict(dim=6), dict(dim=0), dict(n_entities=0), dict(n_relations=0),
           dict(max_batch=0), dict(device=-2), dict(model=kgq.LOGICE, tnorm=3), dict(model=kgq.LOGICE, tnorm=-1),
           dict(model=kgq.CONE, entity_dtype=kgq.BF16), dict(model=kgq.CONE, center_reg=1.5)]
    for kw in bad:
        args = dict(model=kgq.GQE, n_entities=10, n_relations=2, dim=8, gamma=1.0, max_batch=4, device=-1)
        args.update(kw)
        assert rc_of(lambda: kgq.Engine(**args)) == INVALID, kw
    assert kgq.lib().kgq_create(None, None) == INVALID
    assert kgq.lib().kgq_destroy(None) == 0
    # the two cone / fuzzy-logic models create, with every t-norm
    for tn in (kgq.TNORM_PRODUCT, kgq.TNORM_MIN, kgq.TNORM_LUKASIEWICZ):
        kgq.Engine(kgq.LOGICE, 10, 2, 8, 1.0, 4, device=-1, tnorm=tn).close()
    kgq.Engine(kgq.CONE, 10, 2, 8, 30.0, 4, device=-1).close()


def test_arity_table():
    for s, name in enumerate(synth.STRUCTURES):
        assert kgq.arity(s) == synth.ARITY[name]
    assert rc_of(lambda: kgq.arity(14)) == INVALID
    assert rc_of(lambda: kgq.arity(-1)) == INVALID


def test_load_params_validation():
    e = dry()
    d = 8
    assert rc_of(lambda: e.load("nope", np.zeros(4, np.float32))) == INVALID
    assert rc_of(lambda: e.load("relation", np.zeros((6, d + 1), np.float32))) == INVALID   # wrong size
    assert rc_of(lambda: e.load("entity", np.zeros((50, d), np.uint16), kgq.BF16)) == INVALID  # dtype
    e.load("relation", np.zeros((6, d), np.float32))
    eb = dry(dtype=kgq.BF16)
    eb.load("entity", np.zeros((50, d), np.uint16), kgq.BF16)
    assert rc_of(lambda: eb.load("entity", np.zeros((50, d), np.float32))) == INVALID


def test_execute_validation_order():
    e = dry()
    a, r = fake(32), fake(32)
    idx, val = fake(64), np.zeros(64, np.float32)
    # not loaded
    assert rc_of(lambda: e.execute_into(0, 2, a, r, 5, None, idx, val, stream=0)) == NOT_LOADED
    full_load(e, kgq.GQE)
    assert rc_of(lambda: e.execute_into(14, 2, a, r, 5, None, idx, val, stream=0)) == INVALID
    assert rc_of(lambda: e.execute_into(9, 2, a, r, 5, None, idx, val, stream=0)) == UNSUP   # 2in on GQE
    assert rc_of(lambda: e.execute_into(0, 0, a, r, 5, None, idx, val, stream=0)) == INVALID  # batch 0
    assert rc_of(lambda: e.execute_into(0, 17, a, r, 5, None, idx, val, stream=0)) == INVALID  # > max_batch
    assert rc_of(lambda: e.execute_into(0, 2, a, r, 0, None, idx, val, stream=0)) == INVALID  # k = 0
    assert rc_of(lambda: e.execute_into(0, 2, a, r, 51, None, idx, val, stream=0)) == INVALID  # k > N
    assert rc_of(lambda: e.execute_into(0, 2, a, r, 5, None, idx, None, stream=0)) == INVALID  # half top-k
    assert rc_of(lambda: e.execute_into(0, 2, a, r, 5, None, None, None, stream=0)) == INVALID  # no output
    assert rc_of(lambda: e.execute_into(0, 2, None, r, 5, None, idx, val, stream=0)) == INVALID
    # every argument valid: a validation-only handle stops at the device
    assert rc_of(lambda: e.execute_into(0, 2, a, r, 5, None, idx, val, stream=0)) == NO_DEV
    sc = np.zeros(100, np.float32)
    assert rc_of(lambda: e.execute_into(3, 2, a, r, 0, sc, None, None, stream=0)) == NO_DEV


def test_execute_mixed_validation():
    e = dry(model=kgq.Q2B)
    full_load(e, kgq.Q2B)
    a, r = fake(48), fake(48)
    idx, val = fake(64), np.zeros(64, np.float32)
    ok = np.array([0, 3, 8, 5], np.int32)
    assert rc_of(lambda: e.execute_mixed_into(ok, a, r, 3, None, idx, val, stream=0)) == NO_DEV
    assert rc_of(lambda: e.execute_mixed_into(np.array([0, 12], np.int32), a, r, 3, None, idx, val,
                                              stream=0)) == UNSUP
    assert rc_of(lambda: e.execute_mixed_into(np.array([0, 99], np.int32), a, r, 3, None, idx, val,
                                              stream=0)) == INVALID
    for model in (kgq.CONE, kgq.LOGICE):
        ec = dry(model=model)
        full_load(ec, model)
    eb = dry(model=kgq.BETAE)
    full_load(eb, kgq.BETAE)
    allq = np.arange(14, dtype=np.int32)
    assert rc_of(lambda: eb.execute_mixed_into(allq, a, r, 3, None, idx, val, stream=0)) == NO_DEV


def test_dense_validation():
    e = dry()
    x = np.zeros(64, np.float32)
    assert rc_of(lambda: e._check(   # K not a multiple of 4
        kgq.lib().kgq_dense(e.h, x.ctypes.data, 4, 6, x.ctypes.data, 0, 4, 0, x.ctypes.data, 0))) == INVALID
    assert rc_of(lambda: e._check(
        kgq.lib().kgq_dense(e.h, x.ctypes.data, 4, 8, x.ctypes.data, 0, 4, 3, x.ctypes.data, 0))) == INVALID
    assert rc_of(lambda: e._check(
        kgq.lib().kgq_dense(e.h, x.ctypes.data, 4, 8, x.ctypes.data, 0, 4, 1, x.ctypes.data, 0))) == NO_DEV


def test_dense_path_selection():
    """kgq_set_dense_path takes the three paths and refuses others; a layer on
    a validation-only handle still reports that there is no device."""
    e = dry()
    for path in (kgq.DENSE_AUTO, kgq.DENSE_FP32, kgq.DENSE_BF16X3):
        e.set_dense_path(path)
    for bad in (-1, 3, 1 << 20):
        assert rc_of(lambda: e.set_dense_path(bad)) == INVALID
    assert rc_of(lambda: e._check(kgq.lib().kgq_set_dense_path(None, 0))) == INVALID
    x = np.zeros(64, np.float32)
    e.set_dense_path(kgq.DENSE_BF16X3)
    assert rc_of(lambda: e._check(
        kgq.lib().kgq_dense(e.h, x.ctypes.data, 4, 32, x.ctypes.data, 0, 4, 1, x.ctypes.data, 0))) == NO_DEV


def plan(model, sids):
    e = dry(model=model, max_batch=max(16, len(sids)))
    return e.describe_plan(sids)


def test_plan_counts_per_structure():
    S = synth.STRUCTURE_ID
    # GQE: chains = branches, one group per intersection, union -> 2 scored rows
    p = plan(kgq.GQE, [S["1p"]])
    assert (p["chains"], p["groups"], p["scored_rows"], p["union_pairs"]) == (1, 0, 1, 0)
    assert p["launches"] == 4   # chain, pack, score, top-k
    p = plan(kgq.GQE, [S["3i"], S["2i"]])
    assert (p["chains"], p["groups"], p["intersection_inputs"], p["scored_rows"]) == (5, 2, 5, 2)
    assert p["launches"] == 7
    p = plan(kgq.Q2B, [S["2u"], S["up"], S["1p"]])
    assert (p["chains"], p["scored_rows"], p["union_pairs"]) == (5, 5, 2)
    assert plan(kgq.Q2B, [S["ip"]])["launches"] == 10
    # BetaE hop levels: 3p -> 1,1,1; up -> 2,2; pi -> 2,1; ip/inp -> post level
    p = plan(kgq.BETAE, [S["3p"]])
    assert (p["level1"], p["level2"], p["level3"], p["post"]) == (1, 1, 1, 0)
    # first hop: table gather + 2 dense layers; later hops: prep + 3 dense
    # layers; then pack, score, top-k
    assert p["launches"] == 3 + 4 + 4 + 3
    p = plan(kgq.BETAE, [S["up"], S["pi"], S["inp"], S["pni"]])
    assert p["level1"] == 2 + 2 + 2 + 2
    assert p["level2"] == 2 + 1 + 0 + 1
    assert p["level3"] == 0
    assert p["post"] == 1
    assert p["groups"] == 3 and p["intersection_inputs"] == 6
    assert p["scored_rows"] == 5 and p["union_pairs"] == 1


def test_plan_mixed_c5_shape():
    w_ids = synth.draw_mixed(synth.STRUCTURES, 2048, 10, 10, seed=20250305).structure_ids
    p = plan(kgq.BETAE, w_ids)
    n = {s: int((w_ids == i).sum()) for i, s in enumerate(synth.STRUCTURES)}
    branches = sum(n[s] * {"2i": 2, "3i": 3, "pi": 2, "ip": 2, "2u": 2, "up": 2, "2in": 2, "3in": 3,
                           "inp": 2, "pin": 2, "pni": 2}.get(s, 1) for s in synth.STRUCTURES)
    assert p["chains"] == branches
    assert p["union_pairs"] == n["2u"] + n["up"]
    assert p["scored_rows"] == 2048 + n["2u"] + n["up"]
    assert p["post"] == n["ip"] + n["inp"]


def test_memory_of_validation_only_handle_is_zero():
    e = dry()
    assert e.memory() == {"param_bytes": 0, "scratch_bytes": 0}


def test_rank_answers_validation():
    import ctypes
    e = dry(N=50)
    L = kgq.lib()
    p = ctypes.c_void_p(16)
    bad = [(0, p, 50, p, p, p), (2, None, 50, p, p, p), (2, p, 49, p, p, p), (2, p, 50, None, p, p),
           (2, p, 50, p, None, p), (2, p, 50, p, p, None)]
    for batch, sc, ld, off, ids, out in bad:
        assert L.kgq_rank_answers(e.h, batch, sc, ld, off, ids, None, out, None, None) == -1
    assert L.kgq_rank_answers(e.h, 2, p, 50, p, p, None, p, None, None) == -5
    assert L.kgq_rank_answers(None, 2, p, 50, p, p, None, p, None, None) == -1
