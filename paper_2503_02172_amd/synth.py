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

MODEL_GQE, MODEL_Q2B, MODEL_BETAE = 0, 1, 2
MODEL_NAMES = {MODEL_GQE: "gqe", MODEL_Q2B: "q2b", MODEL_BETAE: "betae"}


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


EPFO = ["1p", "2p", "3p", "2i", "3i", "pi", "ip", "2u", "up"]


def make_workload(name: str) -> Workload:
    """Build one of the five named workloads (C1..C5)."""
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
    raise ValueError(f"unknown workload {name!r}")


def make_tiny(model: int, n_ent: int = 37, n_rel: int = 5, dim: int = 8, seed: int = 7,
              gamma: Optional[float] = None) -> Workload:
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
