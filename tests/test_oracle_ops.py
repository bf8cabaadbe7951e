"""Pins of the oracle's operators, query structures, scorers and top-k.

Each check compares the oracle with something other than itself: an
identity the method must satisfy, a hand-derived worked example, a special
choice of weights that reduces an operator to a closed form, a library
routine (numpy), or brute force.
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_02172_amd import synth

S = synth.STRUCTURE_ID


def tiny(model, **kw):
    w = synth.make_tiny(model, **kw)
    return w, O.Model(model, w.params, w.gamma)


# ---------------------------------------------------------------------------
# GQE
# ---------------------------------------------------------------------------

def test_oracle_gqe_score_identity_and_example():
    w, m = tiny(O.GQE)
    for e in [0, 5, 36]:
        st = m.anchor(e)
        assert m.score(st, e) == w.gamma  # q = E[e] -> distance 0
    # worked example: d = 2, q = (0, 0), e = (1, -2): gamma - (1 + 2)
    p = {"entity": np.array([[1.0, -2.0]], np.float32), "relation": np.zeros((1, 2), np.float32),
         "inter.w1": np.zeros((2, 2), np.float32), "inter.b1": np.zeros(2, np.float32),
         "inter.w2": np.zeros((2, 2), np.float32), "inter.b2": np.zeros(2, np.float32)}
    m2 = O.Model(O.GQE, p, 12.0)
    assert m2.score(np.zeros(2), 0) == 9.0


def test_oracle_gqe_score_vs_numpy():
    w, m = tiny(O.GQE)
    rng = np.random.default_rng(1)
    q = rng.uniform(-1, 1, w.dim)
    E = w.params["entity"].astype(np.float64)
    ref = w.gamma - np.abs(q[None, :] - E).sum(1)
    got = np.array([m.score(q, e) for e in range(w.n_entities)])
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-13)


def test_oracle_gqe_translation_chain():
    # 2p with Rel[r1] = -Rel[r0] returns to the anchor, so the anchor scores gamma.
    w = synth.make_tiny(O.GQE)
    p = dict(w.params)
    rel = p["relation"].copy()
    rel[1] = -rel[0]
    p["relation"] = rel
    m = O.Model(O.GQE, p, w.gamma)
    st = m.query_states(S["2p"], [4], [0, 1])[0]
    np.testing.assert_allclose(st, w.params["entity"][4].astype(np.float64), atol=0)
    # 3p with (r0, r0, r1) equals 1p with r0 exactly when the relation values
    # are dyadic, so that no rounding occurs.
    rel = (np.round(w.params["relation"] * 1024) / 1024).astype(np.float32)
    rel[1] = -rel[0]
    p["relation"] = rel
    m = O.Model(O.GQE, p, w.gamma)
    a = m.query_states(S["3p"], [3], [0, 0, 1])[0]
    b = m.query_states(S["1p"], [3], [0])[0]
    np.testing.assert_array_equal(a, b)


def _zero_att(p, d_in, d_hid, d_out, prefix):
    p[prefix + "w1"] = np.zeros((d_hid, d_in), np.float32)
    p[prefix + "b1"] = np.zeros(d_hid, np.float32)
    p[prefix + "w2"] = np.zeros((d_out, d_hid), np.float32)
    p[prefix + "b2"] = np.zeros(d_out, np.float32)


def test_oracle_intersection_identical_branches_gqe():
    w, m = tiny(O.GQE)
    rng = np.random.default_rng(3)
    x = rng.uniform(-1, 1, w.dim)
    for n in (2, 3):
        out = m.intersect([x] * n)
        np.testing.assert_allclose(out, x, rtol=1e-15, atol=1e-15)
    # 2i / 3i of identical branches = 1p
    a = m.query_states(S["2i"], [7, 7], [2, 2])[0]
    b = m.query_states(S["1p"], [7], [2])[0]
    np.testing.assert_allclose(a, b, atol=1e-15)
    a = m.query_states(S["3i"], [1, 1, 1], [4, 4, 4])[0]
    b = m.query_states(S["1p"], [1], [4])[0]
    np.testing.assert_allclose(a, b, atol=1e-15)


def test_oracle_intersection_zero_logits_is_mean():
    # With a zero second layer every branch has the same logit, so the
    # softmax across branches gives weight 1/n and the result is the mean.
    w = synth.make_tiny(O.GQE)
    p = dict(w.params)
    p["inter.w2"] = np.zeros_like(p["inter.w2"])
    p["inter.b2"] = np.full_like(p["inter.b2"], 0.375)
    m = O.Model(O.GQE, p, w.gamma)
    rng = np.random.default_rng(4)
    xs = [rng.uniform(-1, 1, w.dim) for _ in range(3)]
    np.testing.assert_allclose(m.intersect(xs[:2]), (xs[0] + xs[1]) / 2, atol=1e-15)
    np.testing.assert_allclose(m.intersect(xs), (xs[0] + xs[1] + xs[2]) / 3, atol=1e-15)


def test_oracle_intersection_softmax_is_per_dimension_across_branches():
    # W1 = I, W2 = I, zero biases: logit_j = ReLU(x_j), so for two branches the
    # weight of branch 0 in dimension i is sigmoid(ReLU(x0_i) - ReLU(x1_i)).
    d = 6
    eye = np.eye(d, dtype=np.float32)
    p = {"entity": np.zeros((2, d), np.float32), "relation": np.zeros((1, d), np.float32),
         "inter.w1": eye, "inter.b1": np.zeros(d, np.float32),
         "inter.w2": eye, "inter.b2": np.zeros(d, np.float32)}
    m = O.Model(O.GQE, p, 12.0)
    x0 = np.array([0.5, -1.0, 2.0, 0.0, 3.0, -0.25])
    x1 = np.array([1.5, 0.5, -2.0, 0.0, 3.0, 0.75])
    w0 = 1.0 / (1.0 + np.exp(-(np.maximum(x0, 0) - np.maximum(x1, 0))))
    np.testing.assert_allclose(m.intersect([x0, x1]), w0 * x0 + (1 - w0) * x1, rtol=1e-14, atol=1e-15)
    # the result is symmetric in the branch order
    np.testing.assert_allclose(m.intersect([x1, x0]), m.intersect([x0, x1]), atol=1e-15)


def test_oracle_union_is_max_of_branches():
    w, m = tiny(O.GQE)
    a = np.array([[3, 9], [0, 36]], np.int32)
    r = np.array([[1, 4], [2, 2]], np.int32)
    u = m.scores(S["2u"], a, r)
    p0 = m.scores(S["1p"], a[:, :1], r[:, :1])
    p1 = m.scores(S["1p"], a[:, 1:], r[:, 1:])
    np.testing.assert_array_equal(u, np.maximum(p0, p1))
    # up = (a0.r0.r2) v (a1.r1.r2): max of two 2p queries
    r3 = np.array([[1, 4, 3], [2, 2, 0]], np.int32)
    up = m.scores(S["up"], a, r3)
    q0 = m.scores(S["2p"], a[:, :1], r3[:, [0, 2]])
    q1 = m.scores(S["2p"], a[:, 1:], r3[:, [1, 2]])
    np.testing.assert_array_equal(up, np.maximum(q0, q1))


def test_oracle_structure_compositions():
    w, m = tiny(O.GQE)
    # ip = projection of 2i
    a, r = [3, 8], [0, 1, 4]
    ip = m.query_states(S["ip"], a, r)[0]
    two_i = m.query_states(S["2i"], a, r[:2])[0]
    np.testing.assert_allclose(ip, m.project(two_i, 4), atol=1e-15)
    # pi = intersection of a 2p branch (r0, r1) and a 1p branch (r2)
    pi = m.query_states(S["pi"], a, r)[0]
    b0 = m.query_states(S["2p"], [3], [0, 1])[0]
    b1 = m.query_states(S["1p"], [8], [4])[0]
    np.testing.assert_allclose(pi, m.intersect([b0, b1]), atol=1e-15)
    with pytest.raises(ValueError):
        m.query_states(S["2in"], [1, 2], [0, 1])  # GQE has no negation


# ---------------------------------------------------------------------------
# Query2Box
# ---------------------------------------------------------------------------

def _q2b_unit_model(entity, center, offset_raw, gamma=24.0):
    d = entity.shape[1]
    p = {"entity": np.asarray(entity, np.float32),
         "relation.center": np.asarray(center, np.float32),
         "relation.offset_raw": np.asarray(offset_raw, np.float32)}
    for grp in ("inter.center.", "inter.offset."):
        _zero_att(p, d, d, d, grp)
    return O.Model(O.Q2B, p, gamma)


def test_oracle_q2b_box_worked_example():
    # d = 2, box center (0, 0), offset (1, 1), gamma = 24, inside weight 0.02.
    #   v = (2, 0.5):  nearest box point (1, 0.5): outside 1, inside 1.5 -> 22.97
    #   v = (0.5,-0.5): inside the box: outside 0, inside 1.0           -> 23.98
    #   v = (0, 0):     the center: both distances 0                     -> 24
    ent = np.array([[0.0, 0.0], [2.0, 0.5], [0.5, -0.5]])
    raw = np.full((1, 2), np.log(np.expm1(1.0)))  # softplus(raw) = 1
    m = _q2b_unit_model(ent, np.zeros((1, 2)), raw)
    st = m.query_states(S["1p"], [0], [0])[0]
    np.testing.assert_allclose(st, [0, 0, 1, 1], atol=1e-7)
    s = m.scores(S["1p"], np.array([[0]]), np.array([[0]]))[0]
    # the offset is softplus(float32(raw)), within 1e-7 of 1
    np.testing.assert_allclose(s, [24.0, 22.97, 23.98], atol=1e-6)


def test_oracle_q2b_point_inside_box_has_no_outside_distance():
    rng = np.random.default_rng(8)
    d = 5
    c = rng.uniform(-1, 1, d)
    o = rng.uniform(0.1, 1, d)
    v = (c + rng.uniform(-0.9, 0.9, d) * o).astype(np.float32).astype(np.float64)  # inside
    assert np.all(np.abs(v - c) <= o)
    m = _q2b_unit_model(v[None, :], np.zeros((1, d)), np.zeros((1, d)))
    st = np.concatenate([c, o])
    assert m.score(st, 0) == pytest.approx(24.0 - 0.02 * np.abs(c - v).sum(), abs=1e-13)


def test_oracle_q2b_zero_offset_reduces_to_gqe():
    # softplus(-1000) = 0 in double: boxes degenerate to points, dist_in = 0,
    # and the score is GQE's gamma - ||v - c||_1.
    wq = synth.make_tiny(O.Q2B, seed=9)
    p = dict(wq.params)
    p["relation.offset_raw"] = np.full_like(p["relation.offset_raw"], -1000.0)
    mq = O.Model(O.Q2B, p, wq.gamma)
    pg = {"entity": p["entity"], "relation": p["relation.center"]}
    for k in ("w1", "b1", "w2", "b2"):
        pg["inter." + k] = p["inter.center." + k]
    mg = O.Model(O.GQE, pg, wq.gamma)
    a = np.array([[1, 2], [5, 30]], np.int32)
    r = np.array([[0, 3], [4, 4]], np.int32)
    np.testing.assert_allclose(mq.scores(S["2i"], a, r), mg.scores(S["2i"], a, r), rtol=0, atol=1e-13)
    np.testing.assert_allclose(mq.scores(S["2p"], a[:, :1], r), mg.scores(S["2p"], a[:, :1], r),
                               rtol=0, atol=1e-13)


def test_oracle_q2b_offset_intersection_gate():
    wq = synth.make_tiny(O.Q2B, seed=10)
    d = wq.dim
    rng = np.random.default_rng(10)
    br = [np.concatenate([rng.uniform(-1, 1, d), rng.uniform(0.01, 1, d)]) for _ in range(3)]
    mins = np.minimum(np.minimum(br[0][d:], br[1][d:]), br[2][d:])
    # gate saturated open: sigmoid(40) = 1 - 4e-18 -> offset = elementwise min
    p = dict(wq.params)
    p["inter.offset.w2"] = np.zeros_like(p["inter.offset.w2"])
    p["inter.offset.b2"] = np.full_like(p["inter.offset.b2"], 40.0)
    m = O.Model(O.Q2B, p, wq.gamma)
    np.testing.assert_allclose(m.intersect(br)[d:], mins, rtol=1e-15)
    # zero gate input: sigmoid(0) = 1/2
    p["inter.offset.b2"] = np.zeros_like(p["inter.offset.b2"])
    m = O.Model(O.Q2B, p, wq.gamma)
    np.testing.assert_allclose(m.intersect(br)[d:], 0.5 * mins, rtol=1e-15)
    # W3 = I, b3 = 0 (offsets are positive, so ReLU passes them), W4 = I,
    # b4 = 0: the gate input is the mean of the branch offsets, so the offset
    # is min_j o_j * sigmoid(mean_j o_j).
    eye = np.eye(d, dtype=np.float32)
    p["inter.offset.w1"], p["inter.offset.b1"] = eye, np.zeros(d, np.float32)
    p["inter.offset.w2"], p["inter.offset.b2"] = eye, np.zeros(d, np.float32)
    m = O.Model(O.Q2B, p, wq.gamma)
    mean = (br[0][d:] + br[1][d:] + br[2][d:]) / 3.0
    np.testing.assert_allclose(m.intersect(br)[d:], mins / (1.0 + np.exp(-mean)), rtol=1e-14)
    # identical branches with random weights: center unchanged, offset shrinks
    m = O.Model(O.Q2B, wq.params, wq.gamma)
    out = m.intersect([br[0]] * 2)
    np.testing.assert_allclose(out[:d], br[0][:d], atol=1e-15)
    assert np.all(out[d:] <= br[0][d:]) and np.all(out[d:] > 0)


def test_oracle_q2b_projection_accumulates_softplus_offsets():
    wq = synth.make_tiny(O.Q2B, seed=12)
    m = O.Model(O.Q2B, wq.params, wq.gamma)
    d = wq.dim
    st = m.query_states(S["2p"], [6], [1, 3])[0]
    sp = np.logaddexp(0, wq.params["relation.offset_raw"].astype(np.float64))
    np.testing.assert_allclose(st[d:], sp[1] + sp[3], rtol=1e-14)
    c = wq.params["entity"][6].astype(np.float64) + wq.params["relation.center"][1] + \
        wq.params["relation.center"][3].astype(np.float64)
    np.testing.assert_allclose(st[:d], c, rtol=1e-14, atol=1e-15)


# ---------------------------------------------------------------------------
# BetaE
# ---------------------------------------------------------------------------

def test_oracle_betae_projection_reduces_to_shift():
    # W1 = [P; -P], W2 = I, W3 = [P^T, -P^T] with a permutation P (not an
    # involution): ReLU(Px) and ReLU(-Px) pass unchanged through layer 2 and
    # layer 3 recombines them to P^T P x = x. The projection becomes
    # clamp([alpha; beta] + Rel[r] + 1, 0.05, 1e9). A transposed weight would
    # apply P twice and fail.
    d = 3
    w = 2 * d
    perm = np.roll(np.eye(w), 1, axis=0)  # cyclic shift, P @ P != I
    p = {"entity.alpha_beta": np.array([[0.5, 1.0, 2.0, 0.3, 0.7, 1.1], [1, 1, 1, 1, 1, 1]], np.float32),
         "relation": np.array([[0.25, -0.5, 0.125, -2.0, 0.0, 1.0]], np.float32),
         "proj.w1": np.vstack([perm, -perm]).astype(np.float32),
         "proj.b1": np.zeros(2 * w, np.float32),
         "proj.w2": np.eye(2 * w, dtype=np.float32),
         "proj.b2": np.zeros(2 * w, np.float32),
         "proj.w3": np.hstack([perm.T, -perm.T]).astype(np.float32),
         "proj.b3": np.zeros(w, np.float32)}
    _zero_att(p, w, w, d, "inter.")
    m = O.Model(O.BETAE, p, 60.0)
    st = m.query_states(S["1p"], [0], [0])[0]
    x = p["entity.alpha_beta"][0].astype(np.float64) + p["relation"][0]
    np.testing.assert_allclose(st, np.clip(x + 1.0, 0.05, 1e9), atol=1e-15)
    assert st[3] == 0.05  # clamp exercised: 0.3 - 2 + 1 < 0.05
    # W2 = W3 = 0: the output is reg(b3) whatever the input
    p["proj.w2"] = np.zeros_like(p["proj.w2"])
    p["proj.w3"] = np.zeros_like(p["proj.w3"])
    p["proj.b3"] = np.array([0.5, -2.0, 0.0, 1.0, -0.9, 3.0], np.float32)
    m = O.Model(O.BETAE, p, 60.0)
    st = m.query_states(S["1p"], [1], [0])[0]
    np.testing.assert_allclose(st, [1.5, 0.05, 1.0, 2.0, 0.1, 4.0], atol=1e-7)


def test_oracle_betae_projection_vs_numpy_matmul():
    wb = synth.make_tiny(O.BETAE, seed=13)
    m = O.Model(O.BETAE, wb.params, wb.gamma)
    p = {k: v.astype(np.float64) for k, v in wb.params.items()}
    x = p["entity.alpha_beta"][2] + p["relation"][3]
    h1 = np.maximum(p["proj.w1"] @ x + p["proj.b1"], 0)
    h2 = np.maximum(p["proj.w2"] @ h1 + p["proj.b2"], 0)
    y = p["proj.w3"] @ h2 + p["proj.b3"]
    ref = np.clip(y + 1, 0.05, 1e9)
    got = m.query_states(S["1p"], [2], [3])[0]
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-14)


def test_oracle_betae_negation_and_double_negation():
    wb, m = tiny(O.BETAE, seed=14)
    rng = np.random.default_rng(14)
    st = rng.uniform(0.05, 5.0, 2 * wb.dim)
    np.testing.assert_allclose(m.negate(st), 1.0 / st, rtol=0)
    np.testing.assert_allclose(m.negate(m.negate(st)), st, rtol=1e-15)
    assert np.array_equal(m.negate(np.array([2.0, 0.5] * wb.dim)), np.array([0.5, 2.0] * wb.dim))


def test_oracle_betae_negation_structures():
    wb, m = tiny(O.BETAE, seed=15)
    a, r = [4, 9], [0, 2, 3]
    p1 = lambda e, rr: m.query_states(S["1p"], [e], [rr])[0]
    p2 = lambda e, r0, r1: m.query_states(S["2p"], [e], [r0, r1])[0]
    two_in = m.query_states(S["2in"], a, r[:2])[0]
    np.testing.assert_allclose(two_in, m.intersect([p1(4, 0), m.negate(p1(9, 2))]), rtol=1e-15)
    three_in = m.query_states(S["3in"], [4, 9, 1], [0, 2, 3])[0]
    np.testing.assert_allclose(three_in, m.intersect([p1(4, 0), p1(9, 2), m.negate(p1(1, 3))]),
                               rtol=1e-15)
    inp = m.query_states(S["inp"], a, r)[0]
    np.testing.assert_allclose(inp, m.project(two_in, 3), rtol=1e-15)
    pin = m.query_states(S["pin"], a, r)[0]
    np.testing.assert_allclose(pin, m.intersect([p2(4, 0, 2), m.negate(p1(9, 3))]), rtol=1e-15)
    pni = m.query_states(S["pni"], a, r)[0]
    np.testing.assert_allclose(pni, m.intersect([m.negate(p2(4, 0, 2)), p1(9, 3)]), rtol=1e-15)
    assert not np.allclose(pin, pni)


def test_oracle_betae_intersection_identity_and_score():
    wb, m = tiny(O.BETAE, seed=16)
    rng = np.random.default_rng(16)
    st = rng.uniform(0.05, 3.0, 2 * wb.dim)
    for n in (2, 3):
        np.testing.assert_allclose(m.intersect([st] * n), st, rtol=1e-15)
    # an entity scored against its own Beta embedding has KL 0 -> score gamma
    for e in (0, 17, 36):
        assert m.score(m.anchor(e), e) == pytest.approx(wb.gamma, abs=1e-12)


def _betae_att_model(d, v1, v2):
    """BetaE model whose intersection attention has the given first and
    second layers (zero biases); the projection weights are unused."""
    w = 2 * d
    p = {"entity.alpha_beta": np.ones((1, w), np.float32), "relation": np.zeros((1, w), np.float32)}
    for k, shp in (("w1", (2 * w, w)), ("b1", (2 * w,)), ("w2", (2 * w, 2 * w)), ("b2", (2 * w,)),
                   ("w3", (w, 2 * w)), ("b3", (w,))):
        p["proj." + k] = np.zeros(shp, np.float32)
    p["inter.w1"], p["inter.b1"] = v1.astype(np.float32), np.zeros(w, np.float32)
    p["inter.w2"], p["inter.b2"] = v2.astype(np.float32), np.zeros(d, np.float32)
    return O.Model(O.BETAE, p, 60.0)


def test_oracle_betae_intersection_attention_reads_alpha_and_beta():
    """The attention MLP of the BetaE intersection takes the whole state
    [alpha; beta] (width 2d), has hidden width 2d and d logits, and its
    per-dimension weights apply to alpha and to beta alike (reading R-B4 of
    Eq. 3's parameters). Selector weights reduce the logits to ReLU(alpha)
    or ReLU(beta) of each branch, so the weight of branch 0 in dimension i is
    sigmoid(logit_0i - logit_1i). An oracle that fed only alpha to the MLP,
    used another hidden width or mixed up the two halves fails one of the
    two cases, because alpha and beta differ in every dimension."""
    d = 4
    eye, zero = np.eye(d), np.zeros((d, d))
    # V2 = [I | 0]: logits = first d hidden units
    v2 = np.hstack([eye, zero])
    a0 = np.array([0.5, 2.0, 0.125, 1.5])
    b0 = np.array([3.0, 0.25, 1.0, 0.75])
    a1 = np.array([1.25, 0.5, 2.5, 0.0625])
    b1 = np.array([0.5, 1.75, 0.375, 4.0])
    x0, x1 = np.concatenate([a0, b0]), np.concatenate([a1, b1])
    for v1, l0, l1 in ((np.block([[eye, zero], [zero, zero]]), a0, a1),    # hidden = [alpha; 0]
                       (np.block([[zero, eye], [zero, zero]]), b0, b1)):   # hidden = [beta; 0]
        m = _betae_att_model(d, v1, v2)
        w0 = 1.0 / (1.0 + np.exp(-(np.maximum(l0, 0) - np.maximum(l1, 0))))
        want = np.concatenate([w0 * a0 + (1 - w0) * a1, w0 * b0 + (1 - w0) * b1])
        np.testing.assert_allclose(m.intersect([x0, x1]), want, rtol=1e-14, atol=1e-15)
    # the hidden units beyond the first d feed nothing when V2's right half
    # is zero, and do feed the logits when it is not: V1 routes beta to the
    # upper half of the hidden layer, V2 = [0 | I] reads it back
    v1 = np.block([[zero, zero], [zero, eye]])
    m = _betae_att_model(d, v1, np.hstack([zero, eye]))
    w0 = 1.0 / (1.0 + np.exp(-(b0 - b1)))
    want = np.concatenate([w0 * a0 + (1 - w0) * a1, w0 * b0 + (1 - w0) * b1])
    np.testing.assert_allclose(m.intersect([x0, x1]), want, rtol=1e-14, atol=1e-15)


def test_oracle_betae_kl_direction_in_score():
    # d = 1, entity Beta(2,3), query Beta(1,1): the score is
    # gamma - KL(entity || query) = 60 - (ln 12 - 9/4).
    p = {"entity.alpha_beta": np.array([[2.0, 3.0]], np.float32),
         "relation": np.zeros((1, 2), np.float32)}
    for k, shp in (("w1", (4, 2)), ("b1", (4,)), ("w2", (4, 4)), ("b2", (4,)), ("w3", (2, 4)), ("b3", (2,))):
        p["proj." + k] = np.zeros(shp, np.float32)
    _zero_att(p, 2, 2, 1, "inter.")
    m = O.Model(O.BETAE, p, 60.0)
    assert m.score(np.array([1.0, 1.0]), 0) == pytest.approx(60.0 - (np.log(12.0) - 2.25), abs=1e-13)


# ---------------------------------------------------------------------------
# Top-k and batching
# ---------------------------------------------------------------------------

def _brute_topk(row, k):
    order = np.lexsort((np.arange(row.size), -row))  # score desc, then index asc
    return order[:k], row[order[:k]]


def test_oracle_topk_brute_force_with_ties():
    rng = np.random.default_rng(20)
    for N in (1, 7, 33, 64):
        for k in sorted({1, min(5, N), N}):
            sc = rng.integers(0, 6, size=(4, N)).astype(np.float64)  # many exact ties
            idx, val = O.topk(sc, k)
            for q in range(4):
                bi, bv = _brute_topk(sc[q], k)
                np.testing.assert_array_equal(idx[q], bi)
                np.testing.assert_array_equal(val[q], bv)
    with pytest.raises(ValueError):
        O.topk(np.zeros((1, 3)), 4)


def test_oracle_topk_duplicate_entities_order_by_index():
    w = synth.make_tiny(O.GQE, n_ent=40)
    p = dict(w.params)
    ent = p["entity"].copy()
    ent[[5, 12, 30]] = ent[20]  # four identical rows -> four exactly tied scores
    p["entity"] = ent
    m = O.Model(O.GQE, p, w.gamma)
    st = m.anchor(20)
    sc = np.array([[m.score(st, e) for e in range(40)]])
    idx, val = O.topk(sc, 6)
    np.testing.assert_array_equal(idx[0, :4], [5, 12, 20, 30])
    assert np.all(val[0, :4] == w.gamma)


def test_oracle_batched_scores_match_single_and_threads():
    w, m = tiny(O.GQE, n_ent=50)
    a = np.array([[1, 2, 3], [4, 5, 6], [7, 8, 9]], np.int32)
    r = np.array([[0, 1, 2], [3, 4, 0], [1, 1, 1]], np.int32)
    sid = np.array([S["3i"], S["pi"], S["up"]], np.int32)
    s1 = m.scores(sid, a, r, nthreads=1)
    s8 = m.scores(sid, a, r, nthreads=8)
    np.testing.assert_array_equal(s1, s8)
    st = m.query_states(S["pi"], a[1], r[1])[0]
    np.testing.assert_array_equal(s1[1], [m.score(st, e) for e in range(50)])


def test_oracle_rejects_bad_batches():
    w, m = tiny(O.GQE)
    with pytest.raises(ValueError):
        m.scores(S["1p"], np.array([[w.n_entities]]), np.array([[0]]))
    with pytest.raises(ValueError):
        m.scores(S["1p"], np.array([[0]]), np.array([[-1]]))
    with pytest.raises(ValueError):
        m.scores(S["2in"], np.array([[0, 1]]), np.array([[0, 1]]))
    with pytest.raises(ValueError):
        m.scores(14, np.array([[0]]), np.array([[0]]))
