"""Pins of the oracle's evaluation of query computation graphs (Eq. 2) in
disjunctive normal form (Eq. 1).

The graph evaluator is checked against things other than itself: the
oracle's separately written formulas of the 14 benchmark structures (pinned
in test_oracle_ops), closed forms under weights that reduce an intersection
to a plain mean, the distributive and De Morgan laws written out with those
formulas, and the identities double negation = identity and A or A = A.
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_02172_amd import synth

S = synth.STRUCTURE_ID
G = synth.graph_nodes
MODELS = [O.GQE, O.Q2B, O.BETAE]


def tiny(model, **kw):
    w = synth.make_tiny(model, **kw)
    return w, O.Model(model, w.params, w.gamma)


def uniform_attention(model, params):
    """Zero attention weights: every branch gets weight 1/n in every
    dimension (softmax of equal logits)."""
    p = dict(params)
    pre = "inter.center." if model == O.Q2B else "inter."
    for k in ("w1", "b1", "w2", "b2"):
        p[pre + k] = np.zeros_like(p[pre + k])
    return p


@pytest.mark.parametrize("model", MODELS)
def test_graph_equals_structure_formulas(model):
    """Each benchmark structure written as a graph evaluates exactly like the
    oracle's hand-written formula of that structure."""
    w, m = tiny(model)
    for name in synth.STRUCTURES:
        if model != O.BETAE and name in ("2in", "3in", "inp", "pin", "pni"):
            continue
        q = synth.draw_queries(name, 6, w.n_entities, w.n_relations, seed=100 + S[name])
        ref = m.scores(S[name], q.anchors, q.relations)
        got = m.graph_scores(G(synth.STRUCTURE_TEXT[name]), q.anchors, q.relations)
        assert np.array_equal(got, ref), name


def test_graph_deep_chain_closed_form():
    """GQE: a chain of projections is the anchor plus the sum of the relation
    vectors (translation composes), for chains longer than the benchmark's."""
    w, m = tiny(O.GQE)
    E = w.params["entity"].astype(np.float64)
    R = w.params["relation"].astype(np.float64)
    for hops in (4, 6):
        text = "e0"
        for h in range(hops):
            text = f"p({text},r{h})"
        a = np.array([[3], [17]], np.int32)
        r = np.array([[0, 1, 2, 3, 4, 0][:hops], [4, 4, 3, 2, 1, 0][:hops]], np.int32)
        got = m.graph_scores(G(text), a, r)
        for q in range(2):
            c = E[a[q, 0]] + R[r[q]].sum(0)
            ref = w.gamma - np.abs(c[None, :] - E).sum(1)
            np.testing.assert_allclose(got[q], ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("model", MODELS)
def test_graph_union_distributes_over_intersection(model):
    """(A or B) and C scores as max(A and C, B and C), with both sides taken
    from the oracle's 2i formula."""
    w, m = tiny(model)
    rng = np.random.default_rng(3)
    a = rng.integers(0, w.n_entities, (5, 3)).astype(np.int32)
    r = rng.integers(0, w.n_relations, (5, 3)).astype(np.int32)
    got = m.graph_scores(G("i(u(p(e0,r0),p(e1,r1)),p(e2,r2))"), a, r)
    ac = m.scores(S["2i"], a[:, [0, 2]], r[:, [0, 2]])
    bc = m.scores(S["2i"], a[:, [1, 2]], r[:, [1, 2]])
    np.testing.assert_array_equal(got, np.maximum(ac, bc))


@pytest.mark.parametrize("model", MODELS)
def test_graph_product_of_unions_term_order(model):
    """(A or B) and (C or D) has the four terms A&C, A&D, B&C, B&D (first
    input varying slowest), each equal to the 2i formula's state."""
    w, m = tiny(model)
    a = np.array([1, 5, 9, 30], np.int32)
    r = np.array([0, 1, 2, 3], np.int32)
    st = m.graph_states(G("i(u(p(e0,r0),p(e1,r1)),u(p(e2,r2),p(e3,r3)))"), a, r)
    assert st.shape[0] == 4
    for t, (x, y) in enumerate([(0, 2), (0, 3), (1, 2), (1, 3)]):
        ref = m.query_states(S["2i"], a[[x, y]], r[[x, y]])[0]
        np.testing.assert_array_equal(st[t], ref)


def test_graph_nested_and_four_way_intersection_uniform_weights():
    """GQE with zero attention weights: an intersection is the plain mean of
    its branches, so ((A and B) and C) = (A + B) / 4 + C / 2 and a four-way
    intersection is the mean of four."""
    w = synth.make_tiny(O.GQE)
    p = uniform_attention(O.GQE, w.params)
    m = O.Model(O.GQE, p, w.gamma)
    E = p["entity"].astype(np.float64)
    R = p["relation"].astype(np.float64)
    a = np.array([2, 11, 29, 7], np.int32)
    r = np.array([3, 0, 4, 1], np.int32)
    br = [E[a[j]] + R[r[j]] for j in range(4)]
    st = m.graph_states(G("i(i(p(e0,r0),p(e1,r1)),p(e2,r2))"), a[:3], r[:3])[0]
    np.testing.assert_allclose(st, (br[0] + br[1]) / 4 + br[2] / 2, rtol=0, atol=1e-15)
    st = m.graph_states(G("i(p(e0,r0),p(e1,r1),p(e2,r2),p(e3,r3))"), a, r)[0]
    np.testing.assert_allclose(st, sum(br) / 4, rtol=0, atol=1e-15)


def test_graph_de_morgan_negated_union():
    """BetaE with zero attention weights: not(A or B) is the intersection of
    the negations, i.e. the mean of the reciprocal shape parameters of the
    two 1p states."""
    w = synth.make_tiny(O.BETAE)
    p = uniform_attention(O.BETAE, w.params)
    m = O.Model(O.BETAE, p, w.gamma)
    a = np.array([4, 20], np.int32)
    r = np.array([1, 3], np.int32)
    A = m.query_states(S["1p"], a[:1], r[:1])[0]
    B = m.query_states(S["1p"], a[1:], r[1:])[0]
    st = m.graph_states(G("n(u(p(e0,r0),p(e1,r1)))"), a, r)
    assert st.shape[0] == 1
    np.testing.assert_allclose(st[0], (1 / A + 1 / B) / 2, rtol=1e-15, atol=0)


def test_graph_double_negation_and_negated_answer():
    """BetaE: not(not(x)) restores x to fp64 rounding; a negated answer is the
    reciprocal of the 1p state."""
    w, m = tiny(O.BETAE)
    a = np.array([8], np.int32)
    r = np.array([2], np.int32)
    x = m.query_states(S["1p"], a, r)[0]
    nn = m.graph_states(G("n(n(p(e0,r0)))"), a, r)[0]
    np.testing.assert_allclose(nn, x, rtol=1e-15, atol=0)
    n1 = m.graph_states(G("n(p(e0,r0))"), a, r)[0]
    np.testing.assert_array_equal(n1, 1.0 / x)


@pytest.mark.parametrize("model", MODELS)
def test_graph_union_identities(model):
    """A or A scores as A; a three-way union is the max of three 1p rows;
    union is symmetric."""
    w, m = tiny(model)
    a = np.array([[3, 3, 9], [30, 30, 0]], np.int32)
    r = np.array([[1, 1, 4], [0, 0, 2]], np.int32)
    one = m.scores(S["1p"], a[:, :1], r[:, :1])
    np.testing.assert_array_equal(m.graph_scores(G("u(p(e0,r0),p(e1,r1))"), a[:, :2], r[:, :2]), one)
    three = m.graph_scores(G("u(p(e0,r0),p(e1,r1),p(e2,r2))"), a, r)
    rows = [m.scores(S["1p"], a[:, j:j + 1], r[:, j:j + 1]) for j in range(3)]
    np.testing.assert_array_equal(three, np.maximum(np.maximum(rows[0], rows[1]), rows[2]))
    swapped = m.graph_scores(G("u(p(e1,r1),p(e0,r0),p(e2,r2))"), a, r)
    np.testing.assert_array_equal(swapped, three)


def test_graph_projection_distributes_over_union():
    """(A or B).r2 equals A.r2 or B.r2 (Eq. 1), which is how the up structure
    is written in the oracle's formulas; checked here for a deeper chain."""
    w, m = tiny(O.Q2B)
    rng = np.random.default_rng(5)
    a = rng.integers(0, w.n_entities, (4, 2)).astype(np.int32)
    r = rng.integers(0, w.n_relations, (4, 4)).astype(np.int32)
    got = m.graph_scores(G("p(p(u(p(e0,r0),p(e1,r1)),r2),r3)"), a, r)
    left = m.scores(S["3p"], a[:, :1], r[:, [0, 2, 3]])
    right = m.scores(S["3p"], a[:, 1:], r[:, [1, 2, 3]])
    np.testing.assert_array_equal(got, np.maximum(left, right))


def test_graph_info_and_rejections():
    w, m = tiny(O.BETAE)
    assert m.graph_info(G("i(p(p(e0,r0),r1),n(p(e1,r2)))")) == (2, 3, 1)
    assert m.graph_info(G("i(u(p(e0,r0),p(e1,r1)),u(p(e2,r2),p(e3,r3)))")) == (4, 4, 4)
    bad = [
        np.array([[1, 0, 1, -1, -1, -1], [0, 0, -1, -1, -1, -1]]),          # input is a later node
        np.array([[0, 0, -1, -1, -1, -1], [2, -1, 0, -1, -1, -1]]),         # intersection of one input
        np.array([[0, 0, -1, -1, -1, -1], [7, 0, 0, -1, -1, -1]]),          # unknown op
        np.array([[0, 0, -1, -1, -1, -1], [1, 0, 0, -1, 0, -1]]),           # input after an unused slot
    ]
    for g in bad:
        with pytest.raises(ValueError):
            m.graph_info(g)
    # five two-term unions intersected: 32 terms, above the oracle's limit
    big = "i(" + ",".join(f"u(p(e{2*j},r{2*j}),p(e{2*j+1},r{2*j+1}))" for j in range(4)) + ")"
    big = f"i({big},u(p(e8,r8),p(e9,r9)))"
    with pytest.raises(ValueError):
        m.graph_info(G(big))
    _, mg = tiny(O.GQE)
    with pytest.raises(ValueError):
        mg.graph_info(G("n(p(e0,r0))"))
