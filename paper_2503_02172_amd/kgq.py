"""ctypes binding of libkgq (include/kgq.h).

Argument marshalling only: every step of query execution runs in the HIP
library. PyTorch supplies device memory and the current stream. If the
library has not been built this module raises instead of falling back to
anything else.
"""

from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkgq.so")

GQE, Q2B, BETAE, CONE, LOGICE = 0, 1, 2, 3, 4
F32, BF16 = 0, 1
TNORM_PRODUCT, TNORM_MIN, TNORM_LUKASIEWICZ = 0, 1, 2
DENSE_AUTO, DENSE_FP32, DENSE_BF16X3 = 0, 1, 2
NUM_STRUCTURES = 14
MAX_K = 1024
PLAN_FIELDS = ["chains", "groups", "intersection_inputs", "level1", "level2", "level3", "post",
               "scored_rows", "union_pairs", "launches", "intersection_stages", "union_quads", "state_rows"]
INFO_FIELDS = ["anchors", "relations", "terms", "fused_ops", "intersection_stages", "launches", "max_batch",
               "negation"]
# Graph node ops (kgq_op) and the node record (kgq_node): op, slot, in[4].
OP_ANCHOR, OP_PROJECT, OP_AND, OP_OR, OP_NOT = 0, 1, 2, 3, 4
NODE_WORDS = 6
MAX_GRAPH_NODES = 64
STAGES = ["chain", "dense", "combine", "pack", "score", "topk"]

OK = 0
STATUS = {0: "OK", -1: "INVALID_ARG", -2: "OUT_OF_RANGE", -3: "NOT_LOADED", -4: "UNSUPPORTED",
          -5: "NO_DEVICE", -6: "OOM", -7: "DEVICE"}


class KgqError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


class Config(ctypes.Structure):
    _fields_ = [("model", ctypes.c_int32), ("dim", ctypes.c_int32), ("n_entities", ctypes.c_int64),
                ("n_relations", ctypes.c_int32), ("entity_dtype", ctypes.c_int32), ("gamma", ctypes.c_float),
                ("center_reg", ctypes.c_float), ("max_batch", ctypes.c_int32), ("device", ctypes.c_int32),
                ("concurrency", ctypes.c_int32), ("tnorm", ctypes.c_int32)]


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """Open libkgq.so (built in-tree by paper_2503_02172_amd/build.py)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run `python paper_2503_02172_amd/build.py` "
                          "(or __graft_entry__.build()) first")
    # PyTorch ships its own HIP runtime with the same SONAME as ROCm's. Loading
    # torch first makes libkgq bind to that one copy, so device pointers and
    # streams from torch are native to the runtime libkgq calls.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    i32p, i64p, dp = ctypes.POINTER(i32), ctypes.POINTER(i64), ctypes.POINTER(ctypes.c_double)
    sig = {
        "kgq_create": ([ctypes.POINTER(Config), ctypes.POINTER(vp)], i32),
        "kgq_load_params": ([vp, ctypes.c_char_p, vp, ctypes.c_size_t, i32, i32], i32),
        "kgq_structure_arity": ([i32, i32p, i32p], i32),
        "kgq_execute": ([vp, i32, i32, vp, vp, i32, vp, vp, vp, vp], i32),
        "kgq_execute_mixed": ([vp, i32, i32p, vp, vp, i32, vp, vp, vp, vp], i32),
        "kgq_execute_mixed_noalloc": ([vp, i32, i32p, vp, vp, i32, vp, vp, vp, vp], i32),
        "kgq_set_checked": ([vp, i32], i32),
        "kgq_set_dense_path": ([vp, i32], i32),
        "kgq_describe_plan": ([vp, i32, i32p, i32p], i32),
        "kgq_parse_structure": ([ctypes.c_char_p, i32p, i32, i32p], i32),
        "kgq_compile_structure": ([vp, i32p, i32, i32p], i32),
        "kgq_structure_info": ([vp, i32, i32p], i32),
        "kgq_memory": ([vp, i64p, i64p], i32),
        "kgq_rank_answers": ([vp, i32, vp, i64, vp, vp, vp, vp, vp, vp], i32),
        "kgq_dense": ([vp, vp, i32, i32, vp, vp, i32, i32, vp, vp], i32),
        "kgq_profile_enable": ([vp, i32], i32),
        "kgq_profile_read": ([vp, i32, dp, i64p], i32),
        "kgq_profile_reset": ([vp], i32),
        "kgq_profile_intervals": ([vp, i32, dp, i64, i64p], i32),
        "kgq_destroy": ([vp], i32),
        "kgq_status_string": ([i32], ctypes.c_char_p),
        "kgq_last_error": ([vp], ctypes.c_char_p),
        "kgq_create_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def arity(structure: int):
    a, r = ctypes.c_int32(), ctypes.c_int32()
    rc = lib().kgq_structure_arity(structure, ctypes.byref(a), ctypes.byref(r))
    if rc != OK:
        raise KgqError(rc, f"structure {structure}")
    return a.value, r.value


def parse_structure(text: str) -> np.ndarray:
    """Nodes [n x 6] int32 (op, slot, in0..in3) of a graph in the library's
    text form, e.g. "p(i(p(e0,r0),p(e1,r1)),r2)"; raises KgqError on a
    syntax error."""
    buf = np.zeros((MAX_GRAPH_NODES, NODE_WORDS), np.int32)
    n = ctypes.c_int32()
    rc = lib().kgq_parse_structure(text.encode(), buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                   MAX_GRAPH_NODES, ctypes.byref(n))
    if rc != OK:
        raise KgqError(rc, f"cannot parse {text!r}")
    return buf[: n.value].copy()


def _ptr(t) -> int:
    """Address of a torch tensor or numpy array (None -> 0)."""
    if t is None:
        return 0
    if hasattr(t, "data_ptr"):
        return int(t.data_ptr())
    return int(t.ctypes.data)


def _stream(stream) -> int:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


class Engine:
    """One kgq handle: a model's parameters on one GPU plus scratch space."""

    def __init__(self, model: int, n_entities: int, n_relations: int, dim: int, gamma: float,
                 max_batch: int, center_reg: float = 0.02, entity_dtype: int = F32, device: int = 0,
                 concurrency: int = 1, tnorm: int = TNORM_PRODUCT):
        self.cfg = Config(model, dim, n_entities, n_relations, entity_dtype, gamma, center_reg,
                          max_batch, device, concurrency, tnorm)
        h = ctypes.c_void_p()
        rc = lib().kgq_create(ctypes.byref(self.cfg), ctypes.byref(h))
        if rc != OK:
            raise KgqError(rc, lib().kgq_create_error().decode())
        self.h = h
        self.model, self.n_entities, self.dim = model, n_entities, dim
        self.device = device

    # -- lifecycle ------------------------------------------------------------
    def close(self):
        if getattr(self, "h", None):
            lib().kgq_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def _check(self, rc: int):
        if rc != OK:
            raise KgqError(rc, lib().kgq_last_error(self.h).decode())

    # -- parameters -----------------------------------------------------------
    def load(self, name: str, arr, dtype: int = F32):
        """Load one parameter from a numpy array (host) or a torch tensor."""
        if hasattr(arr, "data_ptr"):
            t = arr.contiguous()
            self._check(lib().kgq_load_params(self.h, name.encode(), t.data_ptr(),
                                              t.numel() * t.element_size(), dtype, int(t.is_cuda)))
            return
        a = np.ascontiguousarray(arr)
        self._check(lib().kgq_load_params(self.h, name.encode(), a.ctypes.data, a.nbytes, dtype, 0))

    def load_all(self, params: Dict[str, np.ndarray], entity_bf16: Optional[np.ndarray] = None):
        for name, arr in params.items():
            if entity_bf16 is not None and name.startswith("entity"):
                self.load(name, np.ascontiguousarray(entity_bf16, np.uint16), BF16)
            else:
                self.load(name, np.ascontiguousarray(arr, np.float32), F32)

    def set_checked(self, on: bool):
        self._check(lib().kgq_set_checked(self.h, int(bool(on))))

    def set_dense_path(self, path: int):
        """DENSE_AUTO, DENSE_FP32 or DENSE_BF16X3 (which matrix cores the
        dense layers run on)."""
        self._check(lib().kgq_set_dense_path(self.h, int(path)))

    # -- execution ------------------------------------------------------------
    def execute_into(self, structure: int, batch: int, anchors, relations, k: int,
                     out_scores=None, out_idx=None, out_score=None, stream=None):
        """Enqueue one single-structure batch with caller-owned outputs."""
        self._check(lib().kgq_execute(self.h, structure, batch, _ptr(anchors), _ptr(relations), k,
                                      _ptr(out_scores), _ptr(out_idx), _ptr(out_score),
                                      _stream(stream)))

    def execute_mixed_into(self, structure_ids: np.ndarray, anchors, relations, k: int,
                           out_scores=None, out_idx=None, out_score=None, stream=None):
        sid = np.ascontiguousarray(structure_ids, np.int32)
        self._check(lib().kgq_execute_mixed(self.h, sid.shape[0],
                                            sid.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                            _ptr(anchors), _ptr(relations), k, _ptr(out_scores),
                                            _ptr(out_idx), _ptr(out_score), _stream(stream)))

    def execute_mixed_noalloc_into(self, structure_ids: np.ndarray, anchors, relations, k: int,
                                   out_scores=None, out_idx=None, out_score=None, stream=None):
        """kgq_execute_mixed_noalloc: as execute_mixed_into, with the call's
        device scratch in the library's static array (no allocation)."""
        sid = np.ascontiguousarray(structure_ids, np.int32)
        self._check(lib().kgq_execute_mixed_noalloc(self.h, sid.shape[0],
                                                    sid.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                                    _ptr(anchors), _ptr(relations), k, _ptr(out_scores),
                                                    _ptr(out_idx), _ptr(out_score), _stream(stream)))

    def execute(self, structure, anchors, relations, k: Optional[int] = None, scores: bool = False,
                stream=None):
        """Run a batch and return torch tensors.

        structure: an id (all queries alike; anchors [B x nA], relations
        [B x nR]) or a host int array [B] (mixed; anchors/relations [B x 3]
        padded with -1). Returns dict(scores=[B x N] or None, idx, score).
        stream: a torch stream or a raw hipStream_t (int); None = the current
        stream. The device copies of anchors and relations and the outputs
        are allocated on that stream, so the caching allocator cannot hand
        their memory to other work before the library's kernels on it are
        done with them.
        """
        import torch
        dev = torch.device("cuda", self.device)
        if stream is None:
            ts = torch.cuda.current_stream(dev)
        elif isinstance(stream, int):
            ts = torch.cuda.ExternalStream(stream, device=dev)
        else:
            ts = stream
        with torch.cuda.stream(ts):
            a = torch.as_tensor(anchors, dtype=torch.int32, device=dev).contiguous()
            r = torch.as_tensor(relations, dtype=torch.int32, device=dev).contiguous()
            B = a.shape[0]
            out_s = torch.empty((B, self.n_entities), dtype=torch.float32, device=dev) if scores else None
            out_i = out_v = None
            if k is not None:
                out_i = torch.empty((B, k), dtype=torch.int32, device=dev)
                out_v = torch.empty((B, k), dtype=torch.float32, device=dev)
            kk = k if k is not None else 0
            if np.ndim(structure) == 0:
                self.execute_into(int(structure), B, a, r, kk, out_s, out_i, out_v, ts)
            else:
                self.execute_mixed_into(np.asarray(structure), a, r, kk, out_s, out_i, out_v, ts)
        # Inputs that were already device tensors on another stream: their
        # memory must also outlive the kernels on ts.
        for t, src in ((a, anchors), (r, relations)):
            if t is src or (hasattr(src, "data_ptr") and t.data_ptr() == src.data_ptr()):
                t.record_stream(ts)
        return {"scores": out_s, "idx": out_i, "score": out_v}

    def compile(self, structure) -> int:
        """Compile a structure (text form or nodes [n x 6]) into a new
        structure id of this handle."""
        nodes = parse_structure(structure) if isinstance(structure, str) else structure
        g = np.ascontiguousarray(nodes, np.int32).reshape(-1, NODE_WORDS)
        sid = ctypes.c_int32()
        self._check(lib().kgq_compile_structure(self.h, g.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                                g.shape[0], ctypes.byref(sid)))
        return sid.value

    def structure_info(self, structure_id: int) -> Dict[str, int]:
        info = (ctypes.c_int32 * len(INFO_FIELDS))()
        self._check(lib().kgq_structure_info(self.h, int(structure_id), info))
        return dict(zip(INFO_FIELDS, list(info)))

    def describe_plan(self, structure_ids: Sequence[int]) -> Dict[str, int]:
        sid = np.ascontiguousarray(structure_ids, np.int32)
        counts = (ctypes.c_int32 * len(PLAN_FIELDS))()
        self._check(lib().kgq_describe_plan(self.h, sid.shape[0],
                                            sid.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), counts))
        return dict(zip(PLAN_FIELDS, list(counts)))

    def rank_answers(self, scores, offsets, ids, hard=None, metrics: bool = True, stream=None):
        """Filtered ranks of each query's answers (CSR: ids[offsets[q]:offsets[q+1]])
        in its score row, and per-query [MRR, Hits@1, Hits@3, Hits@10] over
        the hard answers (torch tensors on the device; scores [B x ld] float32,
        offsets [B+1] / ids / hard int32). Returns (ranks int32, metrics
        float64 [B x 4] or None), enqueued on the current stream."""
        import torch
        if scores.dtype != torch.float32 or scores.dim() != 2 or scores.stride(1) != 1:
            raise TypeError("rank_answers: scores must be a float32 [B x ld] tensor with unit column stride")
        for name, t in (("offsets", offsets), ("ids", ids), ("hard", hard)):
            if t is not None and (t.dtype != torch.int32 or not t.is_contiguous() or not t.is_cuda):
                raise TypeError(f"rank_answers: {name} must be a contiguous int32 CUDA tensor")
        B = scores.shape[0]
        if offsets.numel() != B + 1:
            raise ValueError("rank_answers: offsets must have B + 1 entries")
        ranks = torch.empty(ids.numel(), dtype=torch.int32, device=scores.device)
        met = torch.empty((B, 4), dtype=torch.float64, device=scores.device) if metrics else None
        self._check(lib().kgq_rank_answers(self.h, B, _ptr(scores), scores.stride(0), _ptr(offsets), _ptr(ids),
                                           _ptr(hard), _ptr(ranks), _ptr(met), _stream(stream)))
        return ranks, met

    def memory(self) -> Dict[str, int]:
        """Device bytes held by the handle: parameters and derived tables,
        and the execute scratch (sized by max_batch and concurrency)."""
        pb, sb = ctypes.c_int64(0), ctypes.c_int64(0)
        self._check(lib().kgq_memory(self.h, ctypes.byref(pb), ctypes.byref(sb)))
        return {"param_bytes": pb.value, "scratch_bytes": sb.value}

    def dense(self, x, w, b=None, act: int = 0, out=None, stream=None):
        """y = act(x @ w.T + b) with the library's MFMA kernel (torch tensors)."""
        import torch
        for name, t in (("x", x), ("w", w), ("b", b), ("out", out)):
            if t is not None and (t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous()):
                raise TypeError(f"dense: {name} must be a contiguous float32 CUDA tensor")
        M, K = x.shape
        N = w.shape[0]
        if w.shape[1] != K or (b is not None and b.numel() != N):
            raise ValueError("dense: shapes do not match")
        y = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=x.device)
        if y.shape != (M, N):
            raise ValueError("dense: out has the wrong shape")
        self._check(lib().kgq_dense(self.h, _ptr(x), M, K, _ptr(w), _ptr(b), N, act, _ptr(y),
                                    _stream(stream)))
        return y

    # -- profiling ------------------------------------------------------------
    def profile(self, stages=None):
        """Time the given stages (names or ids; None = off, "all" = every stage)."""
        if stages is None:
            mask = 0
        elif stages == "all":
            mask = (1 << len(STAGES)) - 1
        else:
            mask = 0
            for s_ in stages:
                mask |= 1 << (STAGES.index(s_) if isinstance(s_, str) else int(s_))
        self._check(lib().kgq_profile_enable(self.h, mask))

    def profile_reset(self):
        self._check(lib().kgq_profile_reset(self.h))

    def profile_intervals(self, stage: str) -> np.ndarray:
        """[n x 2] start/end (ms) of every timed launch of a stage since the last reset."""
        i = STAGES.index(stage)
        n = ctypes.c_int64()
        self._check(lib().kgq_profile_intervals(self.h, i, None, 0, ctypes.byref(n)))
        out = np.zeros(2 * max(n.value, 1), np.float64)
        self._check(lib().kgq_profile_intervals(self.h, i, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                                n.value, ctypes.byref(n)))
        return out[: 2 * n.value].reshape(n.value, 2)

    def profile_read(self) -> Dict[str, tuple]:
        out = {}
        for i, name in enumerate(STAGES):
            ms, n = ctypes.c_double(), ctypes.c_int64()
            self._check(lib().kgq_profile_read(self.h, i, ctypes.byref(ms), ctypes.byref(n)))
            out[name] = (ms.value, n.value)
        return out


def engine_for(workload, max_batch: Optional[int] = None, device: int = 0, model: Optional[int] = None,
               params: Optional[Dict[str, np.ndarray]] = None, concurrency: int = 1) -> Engine:
    """Create an Engine for a synthetic workload and load its parameters."""
    m = workload.model if model is None else model
    p = workload.params if params is None else params
    bmax = max_batch or max(b.batch for b in workload.batches)
    bf16 = workload.entity_bf16 if (m == BETAE and workload.entity_bf16 is not None) else None
    eng = Engine(m, workload.n_entities, workload.n_relations, workload.dim, workload.gamma, bmax,
                 workload.center_reg, BF16 if bf16 is not None else F32, device, concurrency,
                 getattr(workload, "tnorm", TNORM_PRODUCT))
    eng.load_all(p, entity_bf16=bf16)
    return eng
