"""Pins of the oracle's ConE and LogicE operators.

The paper names both models (Related Work; Experiments, Baselines; Table 1)
without writing their operators; the oracle follows the two models' own
definitions (readings listed in the oracle's header). Each check compares the
oracle with something other than itself: a hand-derived worked example, the
same geometry computed another way (unit vectors instead of half-angle
sines), an algebraic law the operator must satisfy (involution, complement,
t-norm axioms), special weights that reduce an MLP to a closed form, or a
numpy matmul.
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_02172_amd import synth

S = synth.STRUCTURE_ID
PI = np.pi


# ---------------------------------------------------------------------------
# ConE
# ---------------------------------------------------------------------------

def _cone_model(d, entity_axes, gamma=30.0, modulus=0.1, center_reg=0.02, n_rel=1, params=None):
    p = {"entity.axis": np.asarray(entity_axes, np.float32).reshape(-1, d),
         "relation": np.zeros((n_rel, 2 * d), np.float32),
         "modulus": np.array([modulus], np.float32)}
    for k, shp in (("w1", (4 * d, 2 * d)), ("b1", (4 * d,)), ("w2", (4 * d, 4 * d)), ("b2", (4 * d,)),
                   ("w3", (2 * d, 4 * d)), ("b3", (2 * d,))):
        p["proj." + k] = np.zeros(shp, np.float32)
    for grp in ("inter.axis.", "inter.arg."):
        p[grp + "w1"] = np.zeros((d, 2 * d), np.float32)
        p[grp + "b1"] = np.zeros(d, np.float32)
        p[grp + "w2"] = np.zeros((d, d), np.float32)
        p[grp + "b2"] = np.zeros(d, np.float32)
    if params:
        p.update({k: np.asarray(v, np.float32) for k, v in params.items()})
    return p, O.Model(O.CONE, p, gamma, center_reg=center_reg)


def test_oracle_cone_score_worked_example():
    # d = 2, query axis (0, pi/2), half-aperture (pi/2, pi/3); entity (pi/4, -pi/2).
    #   dim 0: t = pi/4: |sin(pi/8)| = 0.382683 < |sin(pi/4)| -> inside: out 0, in 0.382683
    #   dim 1: t = -pi: |sin(-pi/2)| = 1 >= |sin(pi/6)| = 0.5 -> outside:
    #          out = min(|sin((-pi + pi/3)/2)|, |sin((-pi - pi/3)/2)|) = sin(pi/3), in = 0.5
    # score = 30 - 0.1 (sin(pi/3) + 0.02 (sin(pi/8) + 0.5))
    # = 29.91163209276. The entity angles and the modulus are float32 values
    # (pi/4, -pi/2 and 0.1 rounded), which moves the score by a few 1e-9.
    e = np.float32([PI / 4, -PI / 2]).astype(np.float64)
    _, m = _cone_model(2, [e], gamma=30.0, modulus=0.1, center_reg=0.02)
    q = np.array([0.0, PI / 2, PI / 2, PI / 3])
    assert m.score(q, 0) == pytest.approx(29.91163209276, abs=1e-8)


def _cone_geometry(e, axis, psi):
    """Per-dimension (outside, inside) distances from unit vectors: the sector
    is the set of directions within angle psi of the axis; outside it, the
    distance is half the chord to the nearer boundary ray; the inside part is
    half the chord to the axis, capped at half the chord of psi."""
    ve = np.stack([np.cos(e), np.sin(e)], -1)
    va = np.stack([np.cos(axis), np.sin(axis)], -1)
    vl = np.stack([np.cos(axis - psi), np.sin(axis - psi)], -1)
    vu = np.stack([np.cos(axis + psi), np.sin(axis + psi)], -1)
    ang = np.arccos(np.clip((ve * va).sum(-1), -1.0, 1.0))          # angle to the axis, in [0, pi]
    inside = ang < psi
    chord_l = np.linalg.norm(ve - vl, axis=-1) / 2
    chord_u = np.linalg.norm(ve - vu, axis=-1) / 2
    out = np.where(inside, 0.0, np.minimum(chord_l, chord_u))
    half_chord_axis = np.linalg.norm(ve - va, axis=-1) / 2
    inn = np.minimum(half_chord_axis, np.sin(psi / 2))
    return out, inn


def test_oracle_cone_score_matches_unit_vector_geometry():
    rng = np.random.default_rng(71)
    d, n = 6, 40
    ent = rng.uniform(-PI, PI, size=(n, d)).astype(np.float32)
    _, m = _cone_model(d, ent, gamma=7.0, modulus=0.25, center_reg=0.3)
    for _ in range(20):
        axis = rng.uniform(-PI, PI, d)
        psi = rng.uniform(0.0, PI, d)
        q = np.concatenate([axis, psi])
        for e in range(n):
            out, inn = _cone_geometry(ent[e].astype(np.float64), axis, psi)
            want = 7.0 - 0.25 * (out.sum() + 0.3 * inn.sum())
            assert m.score(q, e) == pytest.approx(want, abs=1e-9)


def test_oracle_cone_point_cone_and_axis_score_gamma():
    rng = np.random.default_rng(72)
    ent = rng.uniform(-PI, PI, size=(5, 4)).astype(np.float32)
    _, m = _cone_model(4, ent)
    for e in range(5):
        # the entity's own cone (aperture 0) and any cone on its axis: distance 0
        assert m.score(m.anchor(e), e) == 30.0
        q = np.concatenate([ent[e].astype(np.float64), rng.uniform(0, PI, 4)])
        assert m.score(q, e) == pytest.approx(30.0, abs=1e-12)


def test_oracle_cone_negation_is_the_complement():
    """Per dimension, a direction lies in exactly one of a cone and its
    negation (away from the boundary rays), and negating twice returns the
    cone."""
    rng = np.random.default_rng(73)
    n = 400
    ent = rng.uniform(-PI, PI, size=(n, 1)).astype(np.float32)
    _, m = _cone_model(1, ent, center_reg=0.0, modulus=1.0, gamma=0.0)
    for _ in range(30):
        q = np.array([rng.uniform(-PI, PI), rng.uniform(0.05, PI - 0.05)])
        nq = m.negate(q)
        assert -PI <= nq[0] <= PI and 0.0 <= nq[1] <= PI
        np.testing.assert_allclose(m.negate(nq), q, rtol=0, atol=1e-15)
        for e in range(n):
            out_q, out_n = -m.score(q, e), -m.score(nq, e)    # gamma 0, lambda 0: the outside distance
            if min(abs(np.sin((ent[e, 0] - q[0] - q[1]) / 2)), abs(np.sin((ent[e, 0] - q[0] + q[1]) / 2))) < 1e-6:
                continue                                      # on a boundary ray
            assert (out_q == 0.0) != (out_n == 0.0), (q, nq, ent[e])
    # the axis moves by -pi or +pi by its sign
    np.testing.assert_allclose(m.negate(np.array([0.5, 1.0])), [0.5 - PI, PI - 1.0], atol=1e-15)
    np.testing.assert_allclose(m.negate(np.array([-0.5, 0.25])), [PI - 0.5, PI - 0.25], atol=1e-15)


def test_oracle_cone_projection_reduces_to_the_output_maps():
    # W1 = [P; -P], W2 = I, W3 = [P^T, -P^T]: the MLP is the identity on
    # x = state + Rel[r] (a transposed weight would apply P twice), so the
    # projection is theta = pi tanh(theta + theta_r), psi = pi/2 (tanh(2 (psi + psi_r)) + 1).
    d = 3
    w = 2 * d
    perm = np.roll(np.eye(w), 1, axis=0)
    rel = np.array([[0.25, -0.5, 1.0, 0.1, -0.2, 0.4]], np.float32)
    ent = np.array([[0.3, -1.2, 2.0]], np.float32)
    _, m = _cone_model(d, ent, n_rel=1, params={
        "relation": rel, "proj.w1": np.vstack([perm, -perm]), "proj.w2": np.eye(2 * w),
        "proj.w3": np.hstack([perm.T, -perm.T])})
    st = m.query_states(S["1p"], [0], [0])[0]
    x = np.concatenate([ent[0].astype(np.float64), np.zeros(d)]) + rel[0]
    np.testing.assert_allclose(st[:d], PI * np.tanh(x[:d]), atol=1e-15)
    np.testing.assert_allclose(st[d:], 0.5 * PI * (np.tanh(2 * x[d:]) + 1), atol=1e-15)


def test_oracle_cone_projection_vs_numpy_matmul():
    wc = synth.make_tiny(O.CONE, seed=74)
    m = O.Model(O.CONE, wc.params, wc.gamma)
    p = {k: v.astype(np.float64) for k, v in wc.params.items()}
    d = wc.dim
    x = np.concatenate([p["entity.axis"][5], np.zeros(d)]) + p["relation"][2]
    h1 = np.maximum(p["proj.w1"] @ x + p["proj.b1"], 0)
    h2 = np.maximum(p["proj.w2"] @ h1 + p["proj.b2"], 0)
    y = p["proj.w3"] @ h2 + p["proj.b3"]
    want = np.concatenate([PI * np.tanh(y[:d]), 0.5 * PI * (np.tanh(2 * y[d:]) + 1)])
    np.testing.assert_allclose(m.query_states(S["1p"], [5], [2])[0], want, rtol=1e-13, atol=1e-14)


def test_oracle_cone_intersection_identity_gate_and_mean():
    d = 4
    _, m = _cone_model(d, np.zeros((1, d)))
    rng = np.random.default_rng(75)
    st = np.concatenate([rng.uniform(-3, 3, d), rng.uniform(0.1, 3, d)])
    # identical branches: the axis is unchanged, the half-aperture scaled by
    # the gate sigmoid(b4) = 1/2 (all-zero weights)
    for n in (2, 3):
        out = m.intersect([st] * n)
        np.testing.assert_allclose(out[:d], st[:d], atol=1e-15)
        np.testing.assert_allclose(out[d:], st[d:] / 2, atol=1e-15)
    # zero logits: equal weights, so the axis bisects the two branch axes,
    # and a saturated gate (b4 = 40) leaves min(psi_j)
    _, m = _cone_model(d, np.zeros((1, d)), params={"inter.arg.b2": np.full(d, 40.0)})
    a = np.array([0.3, -2.9, 1.0, -0.5])
    b = np.array([1.1, 2.9, -1.0, 0.25])
    s0 = np.concatenate([a, [0.5, 1.0, 2.0, 0.1]])
    s1 = np.concatenate([b, [0.7, 0.2, 2.5, 0.3]])
    out = m.intersect([s0, s1])
    bis = np.angle(np.exp(1j * a) + np.exp(1j * b))       # direction of the sum of the unit vectors
    np.testing.assert_allclose(out[:d], bis, atol=1e-14)
    np.testing.assert_allclose(out[d:], np.minimum(s0[d:], s1[d:]), rtol=1e-15)
    assert abs(out[1]) > 3.0   # the mean of -2.9 and 2.9 is on the far side, at +-pi


def test_oracle_cone_intersection_attention_and_gate_wiring():
    """Selector weights make the attention logits ReLU(theta - psi) or
    ReLU(theta + psi) of each branch and the gate input twice the mean of one
    of them, so the wiring of u_j = [theta_j - psi_j; theta_j + psi_j] into
    both set functions, and which layers belong to which, is pinned."""
    d = 3
    I, Z = np.eye(d), np.zeros((d, d))
    s0 = np.array([0.4, 1.5, -0.3, 0.2, 0.6, 1.1])
    s1 = np.array([1.3, 0.1, 0.9, 0.5, 0.05, 0.3])

    def w0_of(l0, l1):
        return 1.0 / (1.0 + np.exp(-(np.maximum(l0, 0) - np.maximum(l1, 0))))

    lo = (np.hstack([I, Z]), lambda s: s[:d] - s[d:])     # reads theta - psi
    hi = (np.hstack([Z, I]), lambda s: s[:d] + s[d:])     # reads theta + psi
    # the two set functions get different selectors (and then the other way
    # round), so swapping their weights fails too
    for (sa, fa), (sg, fg) in ((lo, hi), (hi, lo), (lo, lo), (hi, hi)):
        _, m = _cone_model(d, np.zeros((1, d)), params={
            "inter.axis.w1": sa, "inter.axis.w2": I, "inter.arg.w1": sg, "inter.arg.w2": 2 * I})
        out = m.intersect([s0, s1])
        w0 = w0_of(fa(s0), fa(s1))
        x = w0 * np.cos(s0[:d]) + (1 - w0) * np.cos(s1[:d])
        y = w0 * np.sin(s0[:d]) + (1 - w0) * np.sin(s1[:d])
        np.testing.assert_allclose(out[:d], np.arctan2(y, x), atol=1e-14)
        gate = 1 / (1 + np.exp(-2 * (np.maximum(fg(s0), 0) + np.maximum(fg(s1), 0)) / 2))
        np.testing.assert_allclose(out[d:], np.minimum(s0[d:], s1[d:]) * gate, rtol=1e-14)


def test_oracle_cone_structures_and_margin():
    wc = synth.make_tiny(O.CONE, seed=76)
    m = O.Model(O.CONE, wc.params, wc.gamma)
    p1 = lambda e, r: m.query_states(S["1p"], [e], [r])[0]
    two_in = m.query_states(S["2in"], [4, 9], [0, 2])[0]
    np.testing.assert_allclose(two_in, m.intersect([p1(4, 0), m.negate(p1(9, 2))]), rtol=1e-15, atol=1e-15)
    inp = m.query_states(S["inp"], [4, 9], [0, 2, 3])[0]
    np.testing.assert_allclose(inp, m.project(two_in, 3), rtol=1e-15, atol=1e-15)
    # the margin: inf without negation or intersection; with a negation, at
    # most the smallest |axis| it complemented
    m.query_states(S["1p"], [4], [0])
    assert O.Model.last_margin() == np.inf
    m.query_states(S["2in"], [4, 9], [0, 2])
    assert O.Model.last_margin() <= np.abs(p1(9, 2)[:wc.dim]).min()
    u = m.scores(S["2u"], np.array([[3, 9]]), np.array([[1, 4]]))
    np.testing.assert_array_equal(u, np.maximum(m.scores(S["1p"], np.array([[3]]), np.array([[1]])),
                                                m.scores(S["1p"], np.array([[9]]), np.array([[4]]))))


# ---------------------------------------------------------------------------
# LogicE
# ---------------------------------------------------------------------------

def _logice_model(d, ent, gamma=1.0, tnorm=O.TNORM_PRODUCT, n_rel=1, params=None):
    p = {"entity.bounds": np.asarray(ent, np.float32).reshape(-1, 2 * d),
         "relation": np.zeros((n_rel, d), np.float32)}
    for k, shp in (("w1", (4 * d, 3 * d)), ("b1", (4 * d,)), ("w2", (4 * d, 4 * d)), ("b2", (4 * d,)),
                   ("w3", (2 * d, 4 * d)), ("b3", (2 * d,))):
        p["proj." + k] = np.zeros(shp, np.float32)
    if params:
        p.update({k: np.asarray(v, np.float32) for k, v in params.items()})
    return p, O.Model(O.LOGICE, p, gamma, tnorm=tnorm)


def test_oracle_logice_score_worked_example():
    # d = 2: q = [l 0.1, 0.2 | u 0.5, 0.7], e = [0.3, 0.2 | 0.4, 0.9]
    # sum |e - q| = 0.2 + 0 + 0.1 + 0.2 = 0.5, over 2d = 4 -> gamma - 0.125
    e = np.array([[0.3, 0.2, 0.4, 0.9]], np.float32)
    _, m = _logice_model(2, e, gamma=1.0)
    q = np.array([0.1, 0.2, 0.5, 0.7])
    want = 1.0 - np.abs(e[0].astype(np.float64) - q).sum() / 4
    assert m.score(q, 0) == pytest.approx(want, abs=1e-15)
    assert m.score(q, 0) == pytest.approx(0.875, abs=1e-7)
    assert m.score(m.anchor(0), 0) == 1.0


def test_oracle_logice_negation_complements_the_bounds():
    _, m = _logice_model(2, np.zeros((1, 4)))
    q = np.array([0.1, 0.25, 0.5, 0.75])
    np.testing.assert_allclose(m.negate(q), [0.5, 0.25, 0.9, 0.75], atol=1e-15)   # [1 - u; 1 - l]
    rng = np.random.default_rng(81)
    for _ in range(10):
        lo = rng.uniform(0, 1, 5)
        st = np.concatenate([lo, lo + rng.uniform(0, 1, 5) * (1 - lo)])
        _, m = _logice_model(5, np.zeros((1, 10)))
        nst = m.negate(st)
        assert np.all(nst[:5] <= nst[5:])
        np.testing.assert_allclose(m.negate(nst), st, atol=1e-15)


@pytest.mark.parametrize("tnorm", [O.TNORM_PRODUCT, O.TNORM_MIN, O.TNORM_LUKASIEWICZ],
                         ids=["product", "min", "lukasiewicz"])
def test_oracle_logice_tnorm_laws(tnorm):
    d = 6
    _, m = _logice_model(d, np.zeros((1, 2 * d)), tnorm=tnorm)
    rng = np.random.default_rng(82 + tnorm)
    xs = [rng.uniform(0, 1, 2 * d) for _ in range(3)]
    ones, zeros = np.ones(2 * d), np.zeros(2 * d)
    np.testing.assert_allclose(m.intersect([xs[0], ones]), xs[0], atol=1e-15)          # identity
    np.testing.assert_allclose(m.intersect([ones, xs[0]]), xs[0], atol=1e-15)
    np.testing.assert_array_equal(m.intersect([xs[0], zeros]), zeros)                   # annihilator
    np.testing.assert_allclose(m.intersect([xs[0], xs[1]]), m.intersect([xs[1], xs[0]]), atol=1e-15)
    np.testing.assert_allclose(m.intersect(xs), m.intersect([m.intersect(xs[:2]), xs[2]]), atol=1e-15)
    np.testing.assert_allclose(m.intersect(xs), m.intersect([xs[0], m.intersect(xs[1:])]), atol=1e-15)
    # the n-ary closed forms
    want = {O.TNORM_PRODUCT: xs[0] * xs[1] * xs[2],
            O.TNORM_MIN: np.minimum(np.minimum(xs[0], xs[1]), xs[2]),
            O.TNORM_LUKASIEWICZ: np.maximum(0.0, xs[0] + xs[1] + xs[2] - 2.0)}[tnorm]
    np.testing.assert_allclose(m.intersect(xs), want, atol=1e-15)
    # bounds stay ordered: t-norms are monotone
    lo = rng.uniform(0, 1, (3, d))
    sts = [np.concatenate([l, l + rng.uniform(0, 1, d) * (1 - l)]) for l in lo]
    out = m.intersect(sts)
    assert np.all(out[:d] <= out[d:] + 1e-15)
    if tnorm == O.TNORM_MIN:
        np.testing.assert_array_equal(m.intersect([xs[0], xs[0]]), xs[0])             # idempotent


def test_oracle_logice_projection_concatenates_state_then_relation():
    # x = [l; u; r]. W1 copies l and u, and splits r into ReLU(r), ReLU(-r);
    # W2 = I; W3 makes y_l = l + r, y_u = u. Then l' = sigmoid(l + r),
    # u' = l' + sigmoid(u) (1 - l'). Feeding [r; l; u] instead, or putting the
    # relation anywhere else, changes the result.
    d = 2
    I, Z = np.eye(d), np.zeros((d, d))
    w1 = np.block([[I, Z, Z], [Z, I, Z], [Z, Z, I], [Z, Z, -I]])
    w3 = np.block([[I, Z, I, -I], [Z, I, Z, Z]])
    ent = np.array([[0.2, 0.6, 0.5, 0.9]], np.float32)
    rel = np.array([[0.75, -1.5]], np.float32)
    _, m = _logice_model(d, ent, params={"relation": rel, "proj.w1": w1, "proj.w2": np.eye(4 * d),
                                         "proj.w3": w3})
    st = m.query_states(S["1p"], [0], [0])[0]
    e = ent[0].astype(np.float64)
    lo = 1 / (1 + np.exp(-(e[:d] + rel[0])))
    hi = lo + (1 - lo) / (1 + np.exp(-e[d:]))
    np.testing.assert_allclose(st, np.concatenate([lo, hi]), atol=1e-15)


def test_oracle_logice_projection_vs_numpy_matmul():
    wl = synth.make_tiny(O.LOGICE, seed=83)
    m = O.Model(O.LOGICE, wl.params, wl.gamma)
    p = {k: v.astype(np.float64) for k, v in wl.params.items()}
    d = wl.dim
    x = np.concatenate([p["entity.bounds"][7], p["relation"][1]])
    h1 = np.maximum(p["proj.w1"] @ x + p["proj.b1"], 0)
    h2 = np.maximum(p["proj.w2"] @ h1 + p["proj.b2"], 0)
    y = p["proj.w3"] @ h2 + p["proj.b3"]
    lo = 1 / (1 + np.exp(-y[:d]))
    want = np.concatenate([lo, lo + (1 - lo) / (1 + np.exp(-y[d:]))])
    np.testing.assert_allclose(m.query_states(S["1p"], [7], [1])[0], want, rtol=1e-13, atol=1e-14)


def test_oracle_logice_structures():
    wl = synth.make_tiny(O.LOGICE, seed=84)
    m = O.Model(O.LOGICE, wl.params, wl.gamma, tnorm=O.TNORM_LUKASIEWICZ)
    p1 = lambda e, r: m.query_states(S["1p"], [e], [r])[0]
    p2 = lambda e, r0, r1: m.query_states(S["2p"], [e], [r0, r1])[0]
    pin = m.query_states(S["pin"], [4, 9], [0, 2, 3])[0]
    np.testing.assert_allclose(pin, m.intersect([p2(4, 0, 2), m.negate(p1(9, 3))]), atol=1e-15)
    pni = m.query_states(S["pni"], [4, 9], [0, 2, 3])[0]
    np.testing.assert_allclose(pni, m.intersect([m.negate(p2(4, 0, 2)), p1(9, 3)]), atol=1e-15)
    three_in = m.query_states(S["3in"], [4, 9, 1], [0, 2, 3])[0]
    np.testing.assert_allclose(three_in, m.intersect([p1(4, 0), p1(9, 2), m.negate(p1(1, 3))]), atol=1e-15)
    # GQE and Query2Box reject negation; the three negation models accept it
    assert m.graph_info(synth.graph_nodes("n(p(e0,r0))")) == (1, 1, 1)
