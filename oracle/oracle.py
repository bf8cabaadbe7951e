"""ctypes wrapper for the CPU oracle (liboracle.so).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg. The product path never imports it.

The oracle evaluates every operator node by node in double precision; see
kgq_oracle.c for the definitions it follows.
"""

from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

GQE, Q2B, BETAE, CONE, LOGICE = 0, 1, 2, 3, 4
TNORM_PRODUCT, TNORM_MIN, TNORM_LUKASIEWICZ = 0, 1, 2

_fp = ctypes.POINTER(ctypes.c_float)


class _Model(ctypes.Structure):
    _fields_ = [
        ("model", ctypes.c_int32), ("dim", ctypes.c_int32),
        ("n_entities", ctypes.c_int64), ("n_relations", ctypes.c_int32), ("pad_", ctypes.c_int32),
        ("gamma", ctypes.c_double), ("center_reg", ctypes.c_double),
        ("entity", _fp), ("relation", _fp), ("offset_raw", _fp),
        ("att_w1", _fp), ("att_b1", _fp), ("att_w2", _fp), ("att_b2", _fp),
        ("off_w1", _fp), ("off_b1", _fp), ("off_w2", _fp), ("off_b2", _fp),
        ("proj_w1", _fp), ("proj_b1", _fp), ("proj_w2", _fp), ("proj_b2", _fp),
        ("proj_w3", _fp), ("proj_b3", _fp),
        ("tnorm", ctypes.c_int32), ("pad2_", ctypes.c_int32), ("modulus", ctypes.c_double),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b  # type: ignore
            _b.build()
        L = ctypes.CDLL(LIB_PATH)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        mp = ctypes.POINTER(_Model)
        for name in ("kgo_digamma", "kgo_lgamma", "kgo_softplus"):
            getattr(L, name).restype = ctypes.c_double
            getattr(L, name).argtypes = [ctypes.c_double]
        L.kgo_lnbeta.restype = ctypes.c_double
        L.kgo_lnbeta.argtypes = [ctypes.c_double] * 2
        L.kgo_kl_beta.restype = ctypes.c_double
        L.kgo_kl_beta.argtypes = [ctypes.c_double] * 4
        L.kgo_state_width.restype = ctypes.c_int
        L.kgo_state_width.argtypes = [mp]
        L.kgo_anchor.restype = None
        L.kgo_anchor.argtypes = [mp, ctypes.c_int64, dp]
        L.kgo_project.restype = None
        L.kgo_project.argtypes = [mp, dp, ctypes.c_int32, dp]
        L.kgo_negate.restype = None
        L.kgo_negate.argtypes = [mp, dp, dp]
        L.kgo_intersect.restype = None
        L.kgo_intersect.argtypes = [mp, ctypes.c_int, ctypes.POINTER(dp), dp]
        L.kgo_score.restype = ctypes.c_double
        L.kgo_score.argtypes = [mp, dp, ctypes.c_int64]
        L.kgo_arity.restype = ctypes.c_int
        L.kgo_arity.argtypes = [ctypes.c_int, ip, ip]
        L.kgo_query_states.restype = ctypes.c_int
        L.kgo_query_states.argtypes = [mp, ctypes.c_int, ip, ip, dp]
        L.kgo_scores.restype = ctypes.c_int
        L.kgo_scores.argtypes = [mp, ctypes.c_int32, ip, ip, ctypes.c_int32, ip, ctypes.c_int32,
                                 dp, dp, ctypes.c_int]
        L.kgo_last_margin.restype = ctypes.c_double
        L.kgo_last_margin.argtypes = []
        L.kgo_graph_check.restype = ctypes.c_int
        L.kgo_graph_check.argtypes = [mp, ip, ctypes.c_int, ip, ip, ip]
        L.kgo_graph_states.restype = ctypes.c_int
        L.kgo_graph_states.argtypes = [mp, ip, ctypes.c_int, ip, ip, dp]
        L.kgo_graph_scores.restype = ctypes.c_int
        L.kgo_graph_scores.argtypes = [mp, ip, ctypes.c_int, ctypes.c_int32, ip, ctypes.c_int32, ip,
                                       ctypes.c_int32, dp, dp, ctypes.c_int]
        L.kgo_topk.restype = ctypes.c_int
        L.kgo_topk.argtypes = [dp, ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ip, dp,
                               ctypes.c_int]
        fp = ctypes.POINTER(ctypes.c_float)
        L.kgo_rank_answers.restype = ctypes.c_int
        L.kgo_rank_answers.argtypes = [fp, ctypes.c_int32, ctypes.c_int64, ip, ip, ip, ip, dp, ctypes.c_int]
        L.kgo_max_threads.restype = ctypes.c_int
        L.kgo_max_threads.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def _f32(a: Optional[np.ndarray]):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a):
    if a is None:
        return ctypes.cast(None, _fp)
    return a.ctypes.data_as(_fp)


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ip(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


class Model:
    """One model's parameters, held as float32 arrays for the oracle.

    ``params`` uses the library's parameter names: ``entity``, ``relation``
    (GQE) / ``relation.center`` + ``relation.offset_raw`` (Q2B);
    ``inter.w1`` ... (GQE, BetaE) / ``inter.center.*`` + ``inter.offset.*``
    (Q2B); ``entity.alpha_beta``, ``relation``, ``proj.*`` (BetaE).
    """

    def __init__(self, model: int, params: Dict[str, np.ndarray], gamma: float,
                 center_reg: float = 0.02, entity_override: Optional[np.ndarray] = None,
                 tnorm: int = TNORM_PRODUCT):
        self.model = model
        keep = {}
        modulus = 0.0
        if model == CONE:
            keep["entity"] = _f32(params["entity.axis"] if entity_override is None else entity_override)
            keep["relation"] = _f32(params["relation"])
            for k in ("w1", "b1", "w2", "b2"):
                keep["att_" + k] = _f32(params["inter.axis." + k])
                keep["off_" + k] = _f32(params["inter.arg." + k])
            for k in ("w1", "b1", "w2", "b2", "w3", "b3"):
                keep["proj_" + k] = _f32(params["proj." + k])
            modulus = float(np.asarray(params["modulus"], np.float32).reshape(-1)[0])
            dim = keep["entity"].shape[1]
        elif model == LOGICE:
            keep["entity"] = _f32(params["entity.bounds"] if entity_override is None else entity_override)
            keep["relation"] = _f32(params["relation"])
            for k in ("w1", "b1", "w2", "b2", "w3", "b3"):
                keep["proj_" + k] = _f32(params["proj." + k])
            dim = keep["entity"].shape[1] // 2
        elif model == BETAE:
            ent = params["entity.alpha_beta"] if entity_override is None else entity_override
            keep["entity"] = _f32(ent)
            keep["relation"] = _f32(params["relation"])
            for k in ("w1", "b1", "w2", "b2"):
                keep["att_" + k] = _f32(params["inter." + k])
            for k in ("w1", "b1", "w2", "b2", "w3", "b3"):
                keep["proj_" + k] = _f32(params["proj." + k])
            dim = keep["entity"].shape[1] // 2
        elif model == Q2B:
            keep["entity"] = _f32(params["entity"] if entity_override is None else entity_override)
            keep["relation"] = _f32(params["relation.center"])
            keep["offset_raw"] = _f32(params["relation.offset_raw"])
            for k in ("w1", "b1", "w2", "b2"):
                keep["att_" + k] = _f32(params["inter.center." + k])
                keep["off_" + k] = _f32(params["inter.offset." + k])
            dim = keep["entity"].shape[1]
        else:
            keep["entity"] = _f32(params["entity"] if entity_override is None else entity_override)
            keep["relation"] = _f32(params["relation"])
            for k in ("w1", "b1", "w2", "b2"):
                keep["att_" + k] = _f32(params["inter." + k])
            dim = keep["entity"].shape[1]
        self._keep = keep
        s = _Model()
        s.model = model
        s.dim = dim
        s.n_entities = keep["entity"].shape[0]
        s.n_relations = keep["relation"].shape[0]
        s.gamma = gamma
        s.center_reg = center_reg
        s.tnorm = tnorm
        s.modulus = modulus
        for name, _ in _Model._fields_:
            if name in keep:
                setattr(s, name, _ptr(keep[name]))
        self.s = s
        self.dim = dim
        self.n_entities = int(s.n_entities)
        self.width = dim if model == GQE else 2 * dim

    @property
    def ref(self):
        return ctypes.byref(self.s)

    # -- single operators -------------------------------------------------
    def anchor(self, e: int) -> np.ndarray:
        out = np.zeros(self.width, np.float64)
        lib().kgo_anchor(self.ref, e, _dp(out))
        return out

    def project(self, state: np.ndarray, r: int) -> np.ndarray:
        x = np.ascontiguousarray(state, np.float64)
        out = np.zeros(self.width, np.float64)
        lib().kgo_project(self.ref, _dp(x), r, _dp(out))
        return out

    def negate(self, state: np.ndarray) -> np.ndarray:
        x = np.ascontiguousarray(state, np.float64)
        out = np.zeros(self.width, np.float64)
        lib().kgo_negate(self.ref, _dp(x), _dp(out))
        return out

    def intersect(self, states: Sequence[np.ndarray]) -> np.ndarray:
        xs = [np.ascontiguousarray(s, np.float64) for s in states]
        arr = (ctypes.POINTER(ctypes.c_double) * len(xs))(*[_dp(x) for x in xs])
        out = np.zeros(self.width, np.float64)
        lib().kgo_intersect(self.ref, len(xs), arr, _dp(out))
        return out

    def score(self, state: np.ndarray, e: int) -> float:
        x = np.ascontiguousarray(state, np.float64)
        return float(lib().kgo_score(self.ref, _dp(x), e))

    def query_states(self, structure: int, anchors, rels) -> np.ndarray:
        a = np.ascontiguousarray(anchors, np.int32)
        r = np.ascontiguousarray(rels, np.int32)
        out = np.zeros(2 * self.width, np.float64)
        n = lib().kgo_query_states(self.ref, structure, _ip(a), _ip(r), _dp(out))
        if n < 0:
            raise ValueError("unsupported structure")
        return out[: n * self.width].reshape(n, self.width)

    @staticmethod
    def last_margin() -> float:
        """ConE: closest approach to a discontinuity of the operators in the
        query last evaluated by query_states / graph_states (inf if none)."""
        return float(lib().kgo_last_margin())

    # -- query computation graphs -------------------------------------------
    def graph_info(self, nodes) -> tuple:
        """(anchor slots, relation slots, answer terms) of a graph given as an
        int32 array [n_nodes x 6] (op, slot, in0..in3); ValueError if the
        oracle rejects it."""
        g = np.ascontiguousarray(nodes, np.int32).reshape(-1, 6)
        na, nr, nt = (ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32())
        rc = lib().kgo_graph_check(self.ref, _ip(g), g.shape[0], ctypes.byref(na), ctypes.byref(nr),
                                   ctypes.byref(nt))
        if rc != 0:
            raise ValueError("oracle rejected the graph")
        return na.value, nr.value, nt.value

    def graph_states(self, nodes, anchors, rels) -> np.ndarray:
        """Conjunctive terms [n_terms x width] of one query's answer."""
        g = np.ascontiguousarray(nodes, np.int32).reshape(-1, 6)
        _, _, nt = self.graph_info(g)
        a = np.ascontiguousarray(anchors, np.int32)
        r = np.ascontiguousarray(rels, np.int32)
        out = np.zeros(nt * self.width, np.float64)
        n = lib().kgo_graph_states(self.ref, _ip(g), g.shape[0], _ip(a), _ip(r), _dp(out))
        if n < 0:
            raise ValueError("oracle rejected the graph")
        return out[: n * self.width].reshape(n, self.width)

    def graph_scores(self, nodes, anchors: np.ndarray, rels: np.ndarray, nthreads: int = 0,
                     with_margin: bool = False):
        """[B x N] float64 scores of B queries sharing one graph (and, with
        with_margin, each query's ConE discontinuity margin [B])."""
        g = np.ascontiguousarray(nodes, np.int32).reshape(-1, 6)
        a = np.ascontiguousarray(anchors, np.int32)
        r = np.ascontiguousarray(rels, np.int32)
        if a.ndim == 1:
            a = a.reshape(-1, 1)
        if r.ndim == 1:
            r = r.reshape(-1, 1)
        B = a.shape[0]
        out = np.empty((B, self.n_entities), np.float64)
        mg = np.empty(B, np.float64)
        rc = lib().kgo_graph_scores(self.ref, _ip(g), g.shape[0], B, _ip(a), a.shape[1], _ip(r), r.shape[1],
                                    _dp(out), _dp(mg), nthreads)
        if rc != 0:
            raise ValueError("oracle rejected the graph or an id")
        return (out, mg) if with_margin else out

    # -- batched ------------------------------------------------------------
    def scores(self, structure_ids, anchors: np.ndarray, rels: np.ndarray,
               nthreads: int = 0, with_margin: bool = False):
        """[B x N] float64 scores. structure_ids: int or int array [B]. With
        with_margin, also each query's ConE discontinuity margin [B]."""
        a = np.ascontiguousarray(anchors, np.int32)
        r = np.ascontiguousarray(rels, np.int32)
        B = a.shape[0]
        if np.isscalar(structure_ids):
            sid = np.full(B, int(structure_ids), np.int32)
        else:
            sid = np.ascontiguousarray(structure_ids, np.int32)
        out = np.empty((B, self.n_entities), np.float64)
        mg = np.empty(B, np.float64)
        rc = lib().kgo_scores(self.ref, B, _ip(sid), _ip(a), a.shape[1], _ip(r), r.shape[1],
                              _dp(out), _dp(mg), nthreads)
        if rc != 0:
            raise ValueError("oracle rejected the batch (structure, arity or id out of range)")
        return (out, mg) if with_margin else out


def topk(scores: np.ndarray, k: int, nthreads: int = 0):
    s = np.ascontiguousarray(scores, np.float64)
    B, N = s.shape
    idx = np.empty((B, k), np.int32)
    val = np.empty((B, k), np.float64)
    rc = lib().kgo_topk(_dp(s), B, N, k, _ip(idx), _dp(val), nthreads)
    if rc != 0:
        raise ValueError("bad k")
    return idx, val


def rank_answers(scores: np.ndarray, offsets: np.ndarray, ids: np.ndarray, hard: Optional[np.ndarray] = None,
                 nthreads: int = 0):
    """Filtered ranks of each query's answers in its float32 score row, and
    per-query [MRR, Hits@1, Hits@3, Hits@10] over the hard answers (NaN for a
    query without hard answers). Answer lists are CSR: ids[offsets[q]:offsets[q+1]]."""
    s = np.ascontiguousarray(scores, np.float32)
    B, N = s.shape
    off = np.ascontiguousarray(offsets, np.int32)
    idv = np.ascontiguousarray(ids, np.int32)
    assert off.shape == (B + 1,) and off[0] == 0 and off[-1] == idv.shape[0]
    hv = None if hard is None else np.ascontiguousarray(hard, np.int32)
    rank = np.empty(idv.shape[0], np.int32)
    met = np.empty((B, 4), np.float64)
    rc = lib().kgo_rank_answers(s.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), B, N, _ip(off), _ip(idv),
                                _ip(hv) if hv is not None else None, _ip(rank), _dp(met), nthreads)
    if rc != 0:
        raise ValueError("bad answer lists")
    return rank, met


def digamma(x: float) -> float:
    return float(lib().kgo_digamma(x))


def lgamma(x: float) -> float:
    return float(lib().kgo_lgamma(x))


def lnbeta(a: float, b: float) -> float:
    return float(lib().kgo_lnbeta(a, b))


def kl_beta(a1: float, b1: float, a2: float, b2: float) -> float:
    return float(lib().kgo_kl_beta(a1, b1, a2, b2))


def softplus(x: float) -> float:
    return float(lib().kgo_softplus(x))


def max_threads(n: int = 0) -> int:
    return int(lib().kgo_max_threads(n))
