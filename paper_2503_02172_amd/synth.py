"""Seeded synthetic inputs for the five benchmark workloads.

This module draws parameters and queries only. It performs none of the
method's arithmetic (no projection, intersection, negation or scoring), so
both the HIP path and the CPU oracle can take their inputs from it without
sharing any computation.

The paper measures on FB15K-237, FB15K and NELL with trained models
(Experiments, Datasets & Tasks). Neither the data nor the weights are
available, so seeded random tables of the same shapes stand in for them:
14,505 entities x 474 relations (FB15K-237's shape) and 63,361 entities x
400 relations (NELL's shape), embedding dimension 400.

Every array is drawn from ``numpy.random.Generator(PCG64(seed))`` in the
order written below, so a workload is fully determined by its name.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

# Structure ids follow the column order of the paper's Table 1.
STRUCTURES: List[str] = [
    "1p", "2p", "3p", "2i", "3i", "pi", "ip", "2u", "up",
    "2in", "3in", "inp", "pin", "pni",
]
STRUCTURE_ID: Dict[str, int] = {n: i for i, n in enumerate(STRUCTURES)}

# (number of anchor entities, number of relations) per structure. This is
# input bookkeeping only: how many ids a query of each shape carries.
ARITY: Dict[str, tuple] = {
    "1p": (1, 1), "2p": (1, 2), "3p": (1, 3), "2i": (2, 2), "3i": (3, 3),
    "pi": (2, 3), "ip": (2, 3), "2u": (2, 2), "up": (2, 3),
    "2in": (2, 2), "3in": (3, 3), "inp": (2, 3), "pin": (2, 3), "pni": (2, 3),
}

MODEL_GQE, MODEL_Q2B, MODEL_BETAE, MODEL_CONE, MODEL_LOGICE = 0, 1, 2, 3, 4
MODEL_NAMES = {MODEL_GQE: "gqe", MODEL_Q2B: "q2b", MODEL_BETAE: "betae", MODEL_CONE: "cone",
               MODEL_LOGICE: "logice"}
# LogicE intersection t-norms
TNORM_PRODUCT, TNORM_MIN, TNORM_LUKASIEWICZ = 0, 1, 2
TNORM_NAMES = {TNORM_PRODUCT: "product", TNORM_MIN: "min", TNORM_LUKASIEWICZ: "lukasiewicz"}
# models with a negation operator: they run all 14 structures
NEGATION_MODELS = (MODEL_BETAE, MODEL_CONE, MODEL_LOGICE)


def glorot(rng: np.random.Generator, out_f: int, in_f: int) -> np.ndarray:
    """Weight [out x in] ~ U(+-sqrt(6/(in+out)))."""
    lim = np.sqrt(6.0 / (in_f + out_f))
    return rng.uniform(-lim, lim, size=(out_f, in_f)).astype(np.float32)


def bias(rng: np.random.Generator, out_f: int, in_f: int) -> np.ndarray:
    """Bias [out] ~ U(+-1/sqrt(in))."""
    lim = 1.0 / np.sqrt(in_f)
    return rng.uniform(-lim, lim, size=(out_f,)).astype(np.float32)


def bf16_rne(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest even).

    Returns the bf16 bit patterns as uint16. NaN inputs do not occur here.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = (u + 0x7FFF + lsb) >> 16
    return r.astype(np.uint16)


def bf16_decode(h: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float32 values."""
    return (h.astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class QueryBatch:
    """One call's worth of queries.

    ``structure`` is a structure name for a single-structure call, or None for
    a mixed batch, where ``structure_ids`` holds one id per query and
    ``anchors``/``relations`` are [B x 3] padded with -1.
    """
    structure: Optional[str]
    anchors: np.ndarray          # int32 [B x nA] or [B x 3]
    relations: np.ndarray        # int32 [B x nR] or [B x 3]
    structure_ids: Optional[np.ndarray] = None  # int32 [B], mixed only

    @property
    def batch(self) -> int:
        return int(self.anchors.shape[0])


@dataclasses.dataclass
class Workload:
    name: str
    model: int
    n_entities: int
    n_relations: int
    dim: int
    gamma: float
    k: int
    rtol: float
    params: Dict[str, np.ndarray]      # float32 arrays (entity table may also have a bf16 copy)
    batches: List[QueryBatch]
    center_reg: float = 0.02
    entity_bf16: Optional[np.ndarray] = None   # uint16 [N x 2d] when the table is stored as bf16
    extra_models: Dict[str, dict] = dataclasses.field(default_factory=dict)
    tnorm: int = TNORM_PRODUCT                 # LogicE intersection t-norm


def _draw_single(rng, structure: str, n: int, n_ent: int, n_rel: int) -> QueryBatch:
    na, nr = ARITY[structure]
    anchors = rng.integers(0, n_ent, size=(n, na), dtype=np.int64).astype(np.int32)
    rels = rng.integers(0, n_rel, size=(n, nr), dtype=np.int64).astype(np.int32)
    return QueryBatch(structure, anchors, rels)


def _draw_mixed(rng, structures: List[str], n: int, n_ent: int, n_rel: int) -> QueryBatch:
    sid = np.array([STRUCTURE_ID[s] for s in structures], dtype=np.int32)
    pick = rng.integers(0, len(sid), size=n, dtype=np.int64)
    ids = sid[pick]
    anchors = rng.integers(0, n_ent, size=(n, 3), dtype=np.int64).astype(np.int32)
    rels = rng.integers(0, n_rel, size=(n, 3), dtype=np.int64).astype(np.int32)
    for q in range(n):
        na, nr = ARITY[STRUCTURES[ids[q]]]
        anchors[q, na:] = -1
        rels[q, nr:] = -1
    return QueryBatch(None, anchors, rels, ids.astype(np.int32))


def _q2b_params(rng, n_ent, n_rel, d, gamma) -> Dict[str, np.ndarray]:
    s = gamma / d
    p = {}
    p["entity"] = rng.uniform(-s, s, size=(n_ent, d)).astype(np.float32)
    p["relation.center"] = rng.uniform(-s, s, size=(n_rel, d)).astype(np.float32)
    # Offsets enter as raw values that the model passes through softplus.
    # The raw values are drawn so that the offsets themselves are uniform in
    # [gamma/(100 d), gamma/d]: comparable to the spread of the entity points,
    # so that some entities fall inside a box and some outside.
    u = rng.uniform(s / 100.0, s, size=(n_rel, d))
    p["relation.offset_raw"] = np.log(np.expm1(u)).astype(np.float32)
    for grp in ("inter.center", "inter.offset"):
        p[grp + ".w1"] = glorot(rng, d, d)
        p[grp + ".b1"] = bias(rng, d, d)
        p[grp + ".w2"] = glorot(rng, d, d)
        p[grp + ".b2"] = bias(rng, d, d)
    return p


def _betae_params(rng, n_ent, n_rel, d) -> Dict[str, np.ndarray]:
    p = {}
    p["entity.alpha_beta"] = np.maximum(
        1.0 + rng.uniform(-1.0, 1.0, size=(n_ent, 2 * d)), 0.05).astype(np.float32)
    p["relation"] = rng.uniform(-0.5, 0.5, size=(n_rel, 2 * d)).astype(np.float32)
    h = 4 * d  # 1600 at d = 400
    p["proj.w1"] = glorot(rng, h, 2 * d)
    p["proj.b1"] = bias(rng, h, 2 * d)
    p["proj.w2"] = glorot(rng, h, h)
    p["proj.b2"] = bias(rng, h, h)
    p["proj.w3"] = glorot(rng, 2 * d, h)
    p["proj.b3"] = bias(rng, 2 * d, h)
    p["inter.w1"] = glorot(rng, 2 * d, 2 * d)
    p["inter.b1"] = bias(rng, 2 * d, 2 * d)
    p["inter.w2"] = glorot(rng, d, 2 * d)
    p["inter.b2"] = bias(rng, d, 2 * d)
    return p


def _cone_params(rng, n_ent, n_rel, d, gamma) -> Dict[str, np.ndarray]:
    """ConE: entity axes uniform on the circle; relation axes uniform and
    relation half-apertures uniform in [0, pi] (both enter the projection
    input additively); MLP weights per Glorot; the distance scale of the
    model's score, 0.5 (gamma + 2) / d."""
    p = {}
    p["entity.axis"] = rng.uniform(-np.pi, np.pi, size=(n_ent, d)).astype(np.float32)
    rel_axis = rng.uniform(-np.pi, np.pi, size=(n_rel, d))
    rel_arg = rng.uniform(0.0, np.pi, size=(n_rel, d))
    p["relation"] = np.concatenate([rel_axis, rel_arg], axis=1).astype(np.float32)
    h = 4 * d
    p["proj.w1"] = glorot(rng, h, 2 * d)
    p["proj.b1"] = bias(rng, h, 2 * d)
    p["proj.w2"] = glorot(rng, h, h)
    p["proj.b2"] = bias(rng, h, h)
    p["proj.w3"] = glorot(rng, 2 * d, h)
    p["proj.b3"] = bias(rng, 2 * d, h)
    for grp in ("inter.axis", "inter.arg"):
        p[grp + ".w1"] = glorot(rng, d, 2 * d)
        p[grp + ".b1"] = bias(rng, d, 2 * d)
        p[grp + ".w2"] = glorot(rng, d, d)
        p[grp + ".b2"] = bias(rng, d, d)
    p["modulus"] = np.array([0.5 * (gamma + 2.0) / d], np.float32)
    return p


def _logice_params(rng, n_ent, n_rel, d) -> Dict[str, np.ndarray]:
    """LogicE: entity bounds l ~ U(0, 1), u = l + U(0, 1) (1 - l); relation
    vectors ~ U(-1, 1) (concatenated to the projection input); MLP weights
    per Glorot (the first layer takes 3d inputs)."""
    p = {}
    lo = rng.uniform(0.0, 1.0, size=(n_ent, d))
    hi = lo + rng.uniform(0.0, 1.0, size=(n_ent, d)) * (1.0 - lo)
    p["entity.bounds"] = np.concatenate([lo, hi], axis=1).astype(np.float32)
    p["relation"] = rng.uniform(-1.0, 1.0, size=(n_rel, d)).astype(np.float32)
    h = 4 * d
    p["proj.w1"] = glorot(rng, h, 3 * d)
    p["proj.b1"] = bias(rng, h, 3 * d)
    p["proj.w2"] = glorot(rng, h, h)
    p["proj.b2"] = bias(rng, h, h)
    p["proj.w3"] = glorot(rng, 2 * d, h)
    p["proj.b3"] = bias(rng, 2 * d, h)
    return p


EPFO = ["1p", "2p", "3p", "2i", "3i", "pi", "ip", "2u", "up"]


def make_workload(name: str) -> Workload:
    """Build one of the named workloads: C1..C5, and "cone" / "logice"."""
    if name == "C1":
        rng = np.random.Generator(np.random.PCG64(20250301))
        N, R, d = 1000, 20, 32
        p = {}
        p["entity"] = rng.uniform(-0.5, 0.5, size=(N, d)).astype(np.float32)
        p["relation"] = rng.uniform(-0.5, 0.5, size=(R, d)).astype(np.float32)
        p["inter.w1"] = glorot(rng, d, d)
        p["inter.b1"] = bias(rng, d, d)
        p["inter.w2"] = glorot(rng, d, d)
        p["inter.b2"] = bias(rng, d, d)
        batches = [_draw_single(rng, "1p", 16, N, R), _draw_single(rng, "2i", 16, N, R)]
        return Workload("C1", MODEL_GQE, N, R, d, 12.0, 10, 1e-4, p, batches)
    if name == "C2":
        rng = np.random.Generator(np.random.PCG64(20250302))
        N, R, d, g = 14505, 474, 400, 24.0
        p = _q2b_params(rng, N, R, d, g)
        batches = [_draw_single(rng, s, 512, N, R) for s in EPFO]
        return Workload("C2", MODEL_Q2B, N, R, d, g, 100, 1e-4, p, batches)
    if name == "C3":
        rng = np.random.Generator(np.random.PCG64(20250303))
        N, R, d = 14505, 474, 400
        p = _betae_params(rng, N, R, d)
        batches = [_draw_single(rng, s, 512, N, R)
                   for s in ["1p", "2in", "3in", "inp", "pin", "pni"]]
        return Workload("C3", MODEL_BETAE, N, R, d, 60.0, 100, 1e-4, p, batches)
    if name in ("C4", "C4-gqe", "C4-q2b"):
        rng = np.random.Generator(np.random.PCG64(20250304))
        N, R, d, g = 63361, 400, 400, 24.0
        p = _q2b_params(rng, N, R, d, g)
        batches = [_draw_mixed(rng, ["3p", "ip", "pi", "up", "3i"], 1024, N, R)]
        # GQE at the same shape reads the same point table, relation vectors
        # and center-attention weights.
        gqe = {"entity": p["entity"], "relation": p["relation.center"],
               "inter.w1": p["inter.center.w1"], "inter.b1": p["inter.center.b1"],
               "inter.w2": p["inter.center.w2"], "inter.b2": p["inter.center.b2"]}
        if name == "C4-gqe":
            return Workload("C4-gqe", MODEL_GQE, N, R, d, g, 100, 1e-4, gqe, batches)
        w = Workload("C4-q2b" if name == "C4-q2b" else "C4", MODEL_Q2B, N, R, d, g, 100, 1e-4, p, batches)
        w.extra_models["gqe"] = gqe
        return w
    if name == "C5":
        rng = np.random.Generator(np.random.PCG64(20250305))
        N, R, d = 63361, 400, 400
        p = _betae_params(rng, N, R, d)
        batches = [_draw_mixed(rng, STRUCTURES, 2048, N, R)]
        w = Workload("C5", MODEL_BETAE, N, R, d, 60.0, 100, 2e-3, p, batches)
        w.entity_bf16 = bf16_rne(p["entity.alpha_beta"])
        return w
    if name == "cone":
        # ConE at FB15K-237's shape, every structure
        rng = np.random.Generator(np.random.PCG64(20250306))
        N, R, d, g = 14505, 474, 400, 30.0
        p = _cone_params(rng, N, R, d, g)
        batches = [_draw_single(rng, s, 256, N, R) for s in STRUCTURES]
        return Workload("cone", MODEL_CONE, N, R, d, g, 100, 1e-4, p, batches)
    if name == "logice":
        # LogicE at FB15K-237's shape, every structure, product t-norm
        rng = np.random.Generator(np.random.PCG64(20250307))
        N, R, d, g = 14505, 474, 400, 1.0
        p = _logice_params(rng, N, R, d)
        batches = [_draw_single(rng, s, 512, N, R) for s in STRUCTURES]
        return Workload("logice", MODEL_LOGICE, N, R, d, g, 100, 1e-4, p, batches, tnorm=TNORM_PRODUCT)
    raise ValueError(f"unknown workload {name!r}")


def make_tiny(model: int, n_ent: int = 37, n_rel: int = 5, dim: int = 8, seed: int = 7,
              gamma: Optional[float] = None, tnorm: int = TNORM_PRODUCT) -> Workload:
    """A small workload of the given model with odd sizes (tile tails)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if model == MODEL_GQE:
        g = 12.0 if gamma is None else gamma
        p = {"entity": rng.uniform(-0.5, 0.5, size=(n_ent, dim)).astype(np.float32),
             "relation": rng.uniform(-0.5, 0.5, size=(n_rel, dim)).astype(np.float32),
             "inter.w1": glorot(rng, dim, dim), "inter.b1": bias(rng, dim, dim),
             "inter.w2": glorot(rng, dim, dim), "inter.b2": bias(rng, dim, dim)}
        return Workload("tiny-gqe", model, n_ent, n_rel, dim, g, 5, 1e-4, p, [])
    if model == MODEL_Q2B:
        g = 24.0 if gamma is None else gamma
        p = _q2b_params(rng, n_ent, n_rel, dim, g)
        return Workload("tiny-q2b", model, n_ent, n_rel, dim, g, 5, 1e-4, p, [])
    if model == MODEL_CONE:
        g = 30.0 if gamma is None else gamma
        p = _cone_params(rng, n_ent, n_rel, dim, g)
        return Workload("tiny-cone", model, n_ent, n_rel, dim, g, 5, 1e-4, p, [])
    if model == MODEL_LOGICE:
        g = 1.0 if gamma is None else gamma
        p = _logice_params(rng, n_ent, n_rel, dim)
        return Workload("tiny-logice", model, n_ent, n_rel, dim, g, 5, 1e-4, p, [], tnorm=tnorm)
    g = 60.0 if gamma is None else gamma
    p = _betae_params(rng, n_ent, n_rel, dim)
    return Workload("tiny-betae", model, n_ent, n_rel, dim, g, 5, 1e-4, p, [])


def draw_queries(structure: str, n: int, n_ent: int, n_rel: int, seed: int) -> QueryBatch:
    rng = np.random.Generator(np.random.PCG64(seed))
    return _draw_single(rng, structure, n, n_ent, n_rel)


def draw_mixed(structures: List[str], n: int, n_ent: int, n_rel: int, seed: int) -> QueryBatch:
    rng = np.random.Generator(np.random.PCG64(seed))
    return _draw_mixed(rng, structures, n, n_ent, n_rel)


def draw_answers(B: int, N: int, seed: int, max_len: int = 32, hard_share: float = 0.6,
                 special: Optional[Dict[int, int]] = None):
    """Synthetic answer sets for the ranking metrics (the datasets' answer
    sets are not available): query q gets n_q distinct entity ids, n_q
    uniform in [1, max_len] (special: {q: n_q} overrides, n_q may be 0), each
    marked hard with probability hard_share. Returns CSR (offsets [B+1],
    ids, hard) as int32 arrays."""
    rng = np.random.Generator(np.random.PCG64(seed))
    sizes = rng.integers(1, max_len + 1, size=B)
    for q, n in (special or {}).items():
        sizes[q] = n
    off = np.zeros(B + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    ids = np.empty(int(off[-1]), np.int32)
    for q in range(B):
        ids[off[q]:off[q + 1]] = rng.choice(N, size=int(sizes[q]), replace=False)
    hard = (rng.random(ids.shape[0]) < hard_share).astype(np.int32)
    return off.astype(np.int32), ids, hard


# ---------------------------------------------------------------------------
# Query structures as computation graphs
# ---------------------------------------------------------------------------
# A structure is a graph of anchor, projection, intersection, union and
# negation nodes (the paper's Eq. 2). Text form:
#   e<k>  anchor slot k        p(<x>,r<k>)  projection of x by relation slot k
#   i(<x>,<y>[,...])  intersection of 2-4      u(<x>,<y>[,...])  union of 2-4
#   n(<x>)  negation
# Node records: int32 [n x 6] = (op, slot, in0, in1, in2, in3), every node
# after its inputs, the answer last, unused inputs -1. This is an interface
# format shared by the library and the oracle, each of which reads it with
# code of its own; nothing here evaluates a graph.

OP_ANCHOR, OP_PROJECT, OP_AND, OP_OR, OP_NOT = 0, 1, 2, 3, 4

STRUCTURE_TEXT: Dict[str, str] = {
    "1p": "p(e0,r0)", "2p": "p(p(e0,r0),r1)", "3p": "p(p(p(e0,r0),r1),r2)",
    "2i": "i(p(e0,r0),p(e1,r1))", "3i": "i(p(e0,r0),p(e1,r1),p(e2,r2))",
    "pi": "i(p(p(e0,r0),r1),p(e1,r2))", "ip": "p(i(p(e0,r0),p(e1,r1)),r2)",
    "2u": "u(p(e0,r0),p(e1,r1))", "up": "p(u(p(e0,r0),p(e1,r1)),r2)",
    "2in": "i(p(e0,r0),n(p(e1,r1)))", "3in": "i(p(e0,r0),p(e1,r1),n(p(e2,r2)))",
    "inp": "p(i(p(e0,r0),n(p(e1,r1))),r2)", "pin": "i(p(p(e0,r0),r1),n(p(e1,r2)))",
    "pni": "i(n(p(p(e0,r0),r1)),p(e1,r2))",
}


def graph_nodes(text: str) -> np.ndarray:
    """Node records [n x 6] of a structure's text form."""
    s = text.replace(" ", "")
    nodes: List[List[int]] = []
    pos = 0

    def num() -> int:
        nonlocal pos
        j = pos
        while pos < len(s) and s[pos].isdigit():
            pos += 1
        if j == pos:
            raise ValueError(f"slot number expected at {j} in {text!r}")
        return int(s[j:pos])

    def eat(c: str):
        nonlocal pos
        if pos >= len(s) or s[pos] != c:
            raise ValueError(f"{c!r} expected at {pos} in {text!r}")
        pos += 1

    def node(op: int, slot: int, ins: List[int]) -> int:
        nodes.append([op, slot] + ins + [-1] * (4 - len(ins)))
        return len(nodes) - 1

    def expr() -> int:
        nonlocal pos
        c = s[pos] if pos < len(s) else ""
        pos += 1
        if c == "e":
            return node(OP_ANCHOR, num(), [])
        if c == "p":
            eat("(")
            x = expr()
            eat(",")
            eat("r")
            k = num()
            eat(")")
            return node(OP_PROJECT, k, [x])
        if c == "n":
            eat("(")
            x = expr()
            eat(")")
            return node(OP_NOT, -1, [x])
        if c in "iu":
            eat("(")
            ins = [expr()]
            while pos < len(s) and s[pos] == ",":
                pos += 1
                ins.append(expr())
            eat(")")
            if not 2 <= len(ins) <= 4:
                raise ValueError(f"2 to 4 subqueries expected in {text!r}")
            return node(OP_AND if c == "i" else OP_OR, -1, ins)
        raise ValueError(f"unexpected {c!r} at {pos - 1} in {text!r}")

    expr()
    if pos != len(s):
        raise ValueError(f"trailing text in {text!r}")
    return np.asarray(nodes, np.int32).reshape(-1, 6)


def graph_text(nodes: np.ndarray) -> str:
    """Text form of node records (the inverse of graph_nodes)."""
    g = np.asarray(nodes).reshape(-1, 6)

    def rec(i: int) -> str:
        op, slot = int(g[i, 0]), int(g[i, 1])
        ins = [int(v) for v in g[i, 2:] if v >= 0]
        if op == OP_ANCHOR:
            return f"e{slot}"
        if op == OP_PROJECT:
            return f"p({rec(ins[0])},r{slot})"
        if op == OP_NOT:
            return f"n({rec(ins[0])})"
        return ("i(" if op == OP_AND else "u(") + ",".join(rec(j) for j in ins) + ")"

    return rec(g.shape[0] - 1)


def graph_arity(nodes: np.ndarray) -> tuple:
    """(anchor slots, relation slots) a query of this structure carries."""
    g = np.asarray(nodes).reshape(-1, 6)
    na = int(g[g[:, 0] == OP_ANCHOR, 1].max()) + 1
    nr = int(g[g[:, 0] == OP_PROJECT, 1].max()) + 1
    return na, nr


def draw_graph_queries(nodes: np.ndarray, n: int, n_ent: int, n_rel: int, seed: int) -> QueryBatch:
    """n queries of one graph structure: anchors [n x A] and relations [n x R]
    drawn i.i.d. uniform (the recipe of the built-in structures)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    na, nr = graph_arity(nodes)
    a = rng.integers(0, n_ent, size=(n, na), dtype=np.int64).astype(np.int32)
    r = rng.integers(0, n_rel, size=(n, nr), dtype=np.int64).astype(np.int32)
    return QueryBatch(np.full(n, -1, np.int32), a, r)


def random_structure(seed: int, negation: bool, max_depth: int = 4, max_slots: int = 8,
                     max_terms: int = 4) -> str:
    """A seeded random structure in text form. Anchors only feed projections;
    intersections and unions take 2-3 subqueries; negation appears only if
    `negation`; every node has at most `max_terms` conjunctive terms in
    disjunctive normal form (union distributing over intersection and
    projection, the negation of a union being one intersection); at most
    `max_slots` anchor and relation slots. Draws are retried until a graph
    meets these limits."""
    rng = np.random.Generator(np.random.PCG64(seed))
    for _ in range(1000):
        ctr = {"a": 0, "r": 0}
        ok = [True]

        def gen(depth: int):
            kinds = ["leaf", "p", "i", "u"] + (["n"] if negation else [])
            w = np.array([3.0, 3.0, 2.0, 1.0] + ([1.5] if negation else []))
            if depth == 0:
                kind = "leaf"
            else:
                kind = kinds[int(rng.choice(len(kinds), p=w / w.sum()))]
            if kind == "leaf":
                a, r = ctr["a"], ctr["r"]
                ctr["a"] += 1
                ctr["r"] += 1
                return f"p(e{a},r{r})", 1
            if kind == "p":
                x, t = gen(depth - 1)
                r = ctr["r"]
                ctr["r"] += 1
                return f"p({x},r{r})", t
            if kind == "n":
                x, t = gen(depth - 1)
                if t > max_terms:
                    ok[0] = False
                return f"n({x})", 1
            k = int(rng.integers(2, 4))
            subs = [gen(depth - 1) for _ in range(k)]
            t = int(np.prod([s[1] for s in subs])) if kind == "i" else int(sum(s[1] for s in subs))
            if t > max_terms:
                ok[0] = False
            return f"{kind}(" + ",".join(s[0] for s in subs) + ")", t

        text, terms = gen(max_depth)
        if ok[0] and terms <= max_terms and ctr["a"] <= max_slots and ctr["r"] <= max_slots:
            return text
    raise RuntimeError("no structure within the limits")
