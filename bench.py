"""Benchmark: batched query answering (score every entity + top-k) on one MI355X.

One step = one pass of the whole hot path over one batch of the headline
workload, the largest that runs on one GPU: BetaE at 63,361 entities x 400
relations, d = 400, entity table stored as bf16, 2,048 queries drawn
uniformly over all 14 structures, executed as one mixed-structure call (the
plan lowering groups the operators of every structure, one scorer launch
covers every scored row), every query scored against all entities, top-100.
Inputs are resident in HBM before the timed region starts. --workload picks
another of the eight workloads; --per-structure issues one execute call per
structure batch instead, spread round-robin over --streams streams.

Prints one JSON line. `value` is queries/s over the timed steps.
`roofline` describes the dominant kernel (the entity scorer): the
algorithmic operations of one launch divided by the launch's average
duration (HIP events around each launch on the stream it runs on), against
the chip's published peak for the units it runs on (for BetaE the bf16
matrix cores at six bf16 products per FP32-accurate product, or the FP32
matrix cores with --matrix-path fp32; FP32 vector units for the others).
`cpu_baseline` times the CPU oracle on a bounded sample of the same workload,
on every host thread and on one. `others` reports the other workloads
(throughput and scorer fraction).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# Scorer rooflines.
# BetaE scores on the matrix cores; each (row, entity, dimension) triple is 2
# multiply-adds (alpha * U + beta * V), 4 flops. By default the contraction
# runs on the bf16 matrix cores with each FP32 operand split exactly into
# three bf16 parts and six part products kept (FP32 accuracy), so its ceiling
# is the published dense bf16 MFMA peak, 2.5 PFLOP/s, over 6: 416.7 TFLOP/s of
# FP32-accurate flops. On the FP32 matrix cores (--matrix-path fp32) it is the
# published dense FP32 MFMA peak, 157.3 TFLOP/s; that fraction is reported
# beside the other as `frac_of_fp32_mfma_peak`.
# GQE and Query2Box score on the vector units. Each sub / add / min of the
# scorer is one flop and one lane-operation (the library is compiled without
# packed FP32 instructions, so an instruction does one operation per lane).
# Two peaks are reported for them:
#   flops against the published FP32 vector peak, 157.3 TFLOP/s (which counts
#   a packed FMA, 4 flops per lane per clock: 256 CUs x 64 lanes x 4 x 2.4 GHz);
#   lane-operations against what one non-packed instruction stream can issue,
#   256 CUs x 4 SIMDs x 32 lanes per clock x 2.4 GHz = 78.64e12 per second
#   (a wave64 instruction takes 2 cycles on a 32-lane SIMD).
# The headline fraction of a VALU scorer is the flop one; the lane-operation
# fraction is reported beside it as `frac_of_issue_peak`.
PEAK_VALU_OPS = 256 * 4 * 32 * 2.4e9
PEAK_VALU_F32 = 157.3e12
PEAK_MFMA_F32 = 157.3e12
PEAK_MFMA_BF16 = 2.5e15
BF16X3_PRODUCTS = 6
HBM_PEAK = 8.0e12
# algorithmic flops per (query row, entity, scored coordinate) triple, the
# peak they are counted against, and its unit. ConE's sector distance is 10
# VALU instructions per triple, 3 of them fused multiply-adds (13 flops);
# LogicE's triple is one of its 2d bound coordinates scored by GQE's L1 form.
OPS_PER_TRIPLE = {0: 2, 1: 4, 2: 4, 3: 13, 4: 2}
# VALU lane-operations per triple (instructions per lane), for the issue-rate fraction
LANE_OPS_PER_TRIPLE = {0: 2, 1: 4, 3: 10, 4: 2}
SCORER_PEAK = {0: (PEAK_VALU_F32, "alu", "TFLOP/s"), 1: (PEAK_VALU_F32, "alu", "TFLOP/s"),
               2: (PEAK_MFMA_F32, "mfma", "TFLOP/s"), 3: (PEAK_VALU_F32, "alu", "TFLOP/s"),
               4: (PEAK_VALU_F32, "alu", "TFLOP/s")}
K_TOP = 100


def scorer_peak(model: int, matrix_path: str):
    """(peak, bound, unit, basis) of a model's scorer on the given matrix path."""
    if model == 2 and matrix_path != "fp32":
        return (PEAK_MFMA_BF16 / BF16X3_PRODUCTS, "mfma", "TFLOP/s",
                "dense bf16 MFMA peak 2.5 PFLOP/s / 6 bf16 products per FP32-accurate product")
    peak, bound, unit = SCORER_PEAK[model]
    basis = "dense FP32 MFMA peak" if model == 2 else "FP32 vector peak (packed FMA, 4 flops per lane per clock)"
    return peak, bound, unit, basis

WORKLOAD_DESC = {
    "C1": "GQE, 1,000 entities x 20 relations, d=32, fp32; 16 x 1p + 16 x 2i; top-10",
    "C2": "Query2Box, 14,505 entities x 474 relations, d=400, fp32; 512 queries per structure over "
          "1p,2p,3p,2i,3i,pi,ip,2u,up (4,608 queries); top-100",
    "C3": "BetaE, 14,505 entities x 474 relations, d=400, fp32; 512 queries per structure over "
          "1p,2in,3in,inp,pin,pni; top-100",
    "C4-q2b": "Query2Box, 63,361 entities x 400 relations, d=400, fp32; 1,024 mixed 3p/ip/pi/up/3i; top-100",
    "C4-gqe": "GQE, 63,361 entities x 400 relations, d=400, fp32; 1,024 mixed 3p/ip/pi/up/3i; top-100",
    "C5": "BetaE, 63,361 entities x 400 relations, d=400, bf16 entity table; 2,048 mixed over all 14 "
          "structures; top-100",
    "cone": "ConE, 14,505 entities x 474 relations, d=400, fp32; 256 queries per structure over all 14 "
            "structures (3,584 queries); top-100",
    "logice": "LogicE (product t-norm), 14,505 entities x 474 relations, d=400, fp32; 512 queries per structure "
              "over all 14 structures (7,168 queries); top-100",
}


# Oracle sample per workload (queries per batch on all threads, on one
# thread), sized for about 10 s and 6 s of CPU work on a 16-thread host.
# The one-thread leg is one pass: BetaE's per-entity function values are
# computed once per pass and shared by the pass's queries, so a pass of very
# few queries would mostly time that table.
CPU_SAMPLE = {"C1": (16, 16), "C2": (128, 32), "C3": (64, 32), "C4-q2b": (128, 16), "C4-gqe": (128, 16),
              "C5": (256, 32), "cone": (16, 2), "logice": (64, 8)}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Prepared:
    """A workload on the device: engine, resident inputs and outputs.

    merge: execute all of the workload's batches as one mixed-structure call
    (anchors/relations padded to 3 columns with -1, queries kept in batch
    order); otherwise one call per batch, round-robin over n_streams streams.
    """

    def __init__(self, name: str, n_streams: int = 1, merge: bool = True, inflight: int = 1,
                 matrix_path: str = "auto"):
        import torch
        from paper_2503_02172_amd import kgq, synth

        self.name = name
        w = synth.make_workload(name)
        self.w = w
        model = w.model
        params = w.params
        if name == "C4-gqe":
            model = kgq.GQE
        self.model = model
        groups = []
        for b in w.batches:
            if b.structure:
                groups.append((synth.STRUCTURE_ID[b.structure], b.batch, b.anchors, b.relations))
            else:
                groups.append((np.asarray(b.structure_ids, np.int32), b.batch, b.anchors, b.relations))
        if merge and len(groups) > 1:
            ids, A, R = [], [], []
            for sid, n, a, r in groups:
                pa = np.full((n, 3), -1, np.int32)
                pr = np.full((n, 3), -1, np.int32)
                pa[:, :a.shape[1]] = a
                pr[:, :r.shape[1]] = r
                ids.append(np.full(n, sid, np.int32) if np.ndim(sid) == 0 else sid)
                A.append(pa)
                R.append(pr)
            ids = np.concatenate(ids)
            groups = [(ids, ids.shape[0], np.concatenate(A), np.concatenate(R))]
        n_streams = min(n_streams, len(groups))
        # steps in flight: with one call per step, consecutive steps go to
        # `inflight` streams in turn, each with a scratch lane and outputs of
        # its own, so one step's small kernels overlap another's scorer
        self.inflight = max(1, inflight) if len(groups) == 1 else 1
        if self.inflight > 1:
            n_streams = self.inflight
        self.eng = kgq.engine_for(w, max_batch=max(g[1] for g in groups), model=model, params=params,
                                  concurrency=n_streams)
        self.matrix_path = matrix_path
        self.eng.set_dense_path(kgq.DENSE_FP32 if matrix_path == "fp32" else kgq.DENSE_AUTO)
        self.streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(n_streams - 1)]
        dev = torch.device("cuda", 0)
        self.calls = []
        for sid, n, a, r in groups:
            a = torch.as_tensor(a, dtype=torch.int32, device=dev).contiguous()
            r = torch.as_tensor(r, dtype=torch.int32, device=dev).contiguous()
            idx = torch.empty((n, w.k), dtype=torch.int32, device=dev)
            val = torch.empty((n, w.k), dtype=torch.float32, device=dev)
            self.calls.append((sid, n, a, r, idx, val))
        # outputs of the other in-flight steps
        self.outs = [(c[4], c[5]) for c in self.calls[:1]]
        for _ in range(self.inflight - 1):
            n = self.calls[0][1]
            self.outs.append((torch.empty((n, w.k), dtype=torch.int32, device=dev),
                              torch.empty((n, w.k), dtype=torch.float32, device=dev)))
        self.n_steps = 0
        self.n_queries = sum(c[1] for c in self.calls)
        # scored rows (union queries score two rows) -> triples per step
        rows = 0
        for c in self.calls:
            ids = np.full(c[1], c[0]) if np.ndim(c[0]) == 0 else c[0]
            rows += self.eng.describe_plan(ids)["scored_rows"]
        self.rows = rows
        # scored coordinates per entity: LogicE scores its 2d bounds
        self.width = 2 * w.dim if model == kgq.LOGICE else w.dim
        self.triples = rows * w.n_entities * self.width
        torch.cuda.synchronize()

    def step(self, n_streams=None):
        """Enqueue one step: the workload's execute calls, round-robin over the
        streams (independent batches, so calls on different streams overlap)."""
        S = len(self.streams) if n_streams is None else n_streams
        if self.inflight > 1:
            j = self.n_steps % S
            self.n_steps += 1
            sid, B, a, r, _, _ = self.calls[0]
            idx, val = self.outs[j]
            self.eng.execute_mixed_into(sid, a, r, self.w.k, None, idx, val, self.streams[j])
            return
        for i, (sid, B, a, r, idx, val) in enumerate(self.calls):
            st = self.streams[i % S]
            if np.ndim(sid) == 0:
                self.eng.execute_into(int(sid), B, a, r, self.w.k, None, idx, val, st)
            else:
                self.eng.execute_mixed_into(sid, a, r, self.w.k, None, idx, val, st)


def scorer_derivation(p: "Prepared") -> str:
    """How the scorer's algorithmic work per launch is counted."""
    w = p.w
    per = OPS_PER_TRIPLE[p.model]
    what = {0: "sub, add of |.| (GQE L1 distance)",
            1: "sub, add of |.|, min, add (Query2Box box distance, regrouped exactly)",
            2: "2 multiply-adds alpha_q*U_e + beta_q*V_e (BetaE KL, regrouped exactly)",
            3: "mul, fma, mul, fma, mul, fma, max, add, min, add: half-angle sine and cosine of the angle "
               "difference, outside and inside distance (ConE sector distance, regrouped exactly)",
            4: "sub, add of |.| over each of the 2d bound coordinates (LogicE L1 distance)"}[p.model]
    return (f"{per} flops per (scored row, entity, coordinate) triple [{what}] x {p.rows} scored rows x "
            f"{w.n_entities} entities x {p.width} coordinates = {per * p.triples:.4g} flops per launch")


def union_ms(iv: np.ndarray) -> float:
    """Length of the union of [start, end] intervals (ms)."""
    if len(iv) == 0:
        return 0.0
    iv = iv[np.argsort(iv[:, 0])]
    total, cs, ce = 0.0, iv[0, 0], iv[0, 1]
    for a, b in iv[1:]:
        if a > ce:
            total += ce - cs
            cs, ce = a, b
        else:
            ce = max(ce, b)
    return total + ce - cs


def time_steps(p: Prepared, steps: int, warmup: int, profile_score: bool, serial: bool = False):
    """Time `steps` steps. With profile_score, HIP events bracket every scorer
    launch on its stream; returns (seconds, scorer intervals [n x 2] ms).
    serial: one stream, one step at a time (no steps in flight)."""
    import torch
    ns = 1 if serial else None
    for _ in range(warmup):
        p.step(ns)
    torch.cuda.synchronize()
    if profile_score:
        p.eng.profile_reset()
        p.eng.profile(["score"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        p.step(ns)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    iv = None
    if profile_score:
        iv = p.eng.profile_intervals("score")
        p.eng.profile(None)
    return dt, iv


def stage_breakdown(p: Prepared, reps: int = 3):
    """Per-stage device time of one step, from a separate pass on one stream
    with every stage instrumented (so the stages do not overlap)."""
    import torch
    p.eng.profile_reset()
    p.eng.profile("all")
    for _ in range(reps):
        p.step(n_streams=1)
    torch.cuda.synchronize()
    r = p.eng.profile_read()
    p.eng.profile(None)
    p.eng.profile_reset()
    return {k: round(v[0] / reps, 4) for k, v in r.items()}


# Sources each scorer kernel is compiled from (the kernel file and the headers
# it includes); a traffic record is valid only while all of them are unchanged.
SCORER_SOURCES = {0: ["k_score.hip", "kgq_internal.hpp"], 1: ["k_score.hip", "kgq_internal.hpp"],
                  2: ["k_score_kl.hip", "mfma_tile.hpp", "kgq_internal.hpp"]}


def sources_sha256(files) -> str:
    h = hashlib.sha256()
    for f in files:
        h.update(open(os.path.join(ROOT, "paper_2503_02172_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def traffic_for(model: int, name: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current scorer sources (else (None, None)): FETCH_SIZE and
    WRITE_SIZE scaled by a plain copy kernel's readings, and the fetch counted
    by read-request size (plus WRITE_SIZE)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None, None
    try:
        rec = json.load(open(path)).get(name)
    except Exception:
        return None, None
    if not rec:
        return None, None
    files = SCORER_SOURCES[model]
    if rec.get("kernel_sources") != files or rec.get("sources_sha256") != sources_sha256(files):
        return None, None
    return rec.get("bytes_per_launch"), rec.get("bytes_per_launch_by_request_size")


def batch_sweep(name: str, sizes, reps: int):
    """Per-query time and device memory against batch size, per structure
    (the paper's batch-size study, Experiments RQ2), on the tables of one
    workload. One engine per batch size (max_batch = B): its memory is the
    handle's whole device footprint (parameters + scratch; execute allocates
    nothing). Prints one JSON line per batch size."""
    import torch
    from paper_2503_02172_amd import kgq, synth

    w = synth.make_workload(name)
    structures = list(synth.STRUCTURES) if w.model == kgq.BETAE else list(synth.STRUCTURES[:9])
    dev = torch.device("cuda", 0)
    for B in sizes:
        eng = kgq.engine_for(w, max_batch=B)
        mem = eng.memory()
        per_q = {}
        for si, st in enumerate(structures):
            qb = synth.draw_queries(st, B, w.n_entities, w.n_relations, seed=1000 + si)
            a = torch.as_tensor(qb.anchors, dtype=torch.int32, device=dev).contiguous()
            r = torch.as_tensor(qb.relations, dtype=torch.int32, device=dev).contiguous()
            idx = torch.empty((B, w.k), dtype=torch.int32, device=dev)
            val = torch.empty((B, w.k), dtype=torch.float32, device=dev)
            sid = synth.STRUCTURE_ID[st]
            for _ in range(3):
                eng.execute_into(sid, B, a, r, w.k, None, idx, val)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(reps):
                eng.execute_into(sid, B, a, r, w.k, None, idx, val)
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t0) / reps
            per_q[st] = round(dt / B * 1e3, 6)
        print(json.dumps({"sweep": name, "batch": B, "ms_per_query": per_q,
                          "device_bytes": mem["param_bytes"] + mem["scratch_bytes"],
                          "param_bytes": mem["param_bytes"], "scratch_bytes": mem["scratch_bytes"]}), flush=True)
        log(f"[sweep] {name} B={B}: memory {(mem['param_bytes'] + mem['scratch_bytes']) / 2**20:.1f} MiB, "
            f"ms/query {per_q}")
        eng.close()
        del eng
        torch.cuda.empty_cache()


def rank_bench(p: Prepared, reps: int = 20):
    """Filtered ranking metrics (kgq_rank_answers) over the workload's whole
    score matrix, with synthetic answer sets of 1..32 answers per query: mean
    launch time (HIP events on the stream) and the bytes it must move (the
    score matrix read once, answer lists read, ranks and metrics written)
    against the HBM peak."""
    import torch
    from paper_2503_02172_amd import synth

    w = p.w
    sid, B, a, r, idx, val = p.calls[0]
    if len(p.calls) != 1 or np.ndim(sid) == 0:
        return None
    dev = torch.device("cuda", 0)
    scores = torch.empty((B, w.n_entities), dtype=torch.float32, device=dev)
    p.eng.execute_mixed_into(sid, a, r, w.k, scores, idx, val)
    off, ids, hard = synth.draw_answers(B, w.n_entities, seed=77, max_len=32)
    to, ti, th = (torch.as_tensor(x, device=dev) for x in (off, ids, hard))
    for _ in range(3):
        p.eng.rank_answers(scores, to, ti, th)
    st = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for e0, e1 in ev:
        e0.record(st)
        p.eng.rank_answers(scores, to, ti, th)
        e1.record(st)
    torch.cuda.synchronize()
    ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    nbytes = B * w.n_entities * 4 + (B + 1) * 4 + ids.size * (4 + 4 + 4) + B * 4 * 8
    return {"kernel": "k_rank_stream (lists of up to 32 answers) + k_rank_answers (the rest)", "queries": B, "answers": int(ids.size), "avg_launch_ms": round(ms, 5),
            "bytes_per_launch": nbytes, "achieved_GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "frac_of_hbm_peak": round(nbytes / (ms * 1e-3) / HBM_PEAK, 4),
            "queries_per_s": round(B / (ms * 1e-3), 1)}


def _oracle_pass(m, w, n_queries: int):
    """The oracle on the first n_queries of every batch of the workload (a
    uniform sample: each batch's queries are drawn i.i.d.); returns the
    number of queries evaluated."""
    from oracle import oracle as O
    from paper_2503_02172_amd import synth

    nq = 0
    for b in w.batches:
        n = min(n_queries, b.batch)
        sid = synth.STRUCTURE_ID[b.structure] if b.structure else b.structure_ids[:n]
        sc = m.scores(sid, b.anchors[:n], b.relations[:n])
        O.topk(sc, w.k)
        nq += n
    return nq


def cpu_baseline(name: str, n_queries: int, n_queries_1t: int, min_seconds: float = 10.0,
                 min_seconds_1t: float = 0.0):
    """The CPU oracle (fp64, node by node, full scoring + top-k) on a bounded
    sample of the workload: the first n_queries of each batch, in whole passes
    repeated until min_seconds have elapsed, on every host thread; then the
    first n_queries_1t of each batch on one thread (one pass by default)."""
    from oracle import oracle as O
    from paper_2503_02172_amd import synth

    w = synth.make_workload(name)
    ent = synth.bf16_decode(w.entity_bf16) if w.entity_bf16 is not None else None
    m = O.Model(w.model, w.params, w.gamma, entity_override=ent)
    total = sum(b.batch for b in w.batches)

    def timed(nq_per_batch, threads, min_s):
        used = O.max_threads(threads)
        nq, passes, t0 = 0, 0, time.perf_counter()
        while True:
            nq += _oracle_pass(m, w, nq_per_batch)
            passes += 1
            if time.perf_counter() - t0 >= min_s:
                break
        dt = time.perf_counter() - t0
        return nq, passes, dt, used

    # all threads OpenMP gives the process (OMP_NUM_THREADS where it is set)
    all_threads = O.max_threads(0)
    nq, passes, dt, threads = timed(n_queries, all_threads, min_seconds)
    nq1, passes1, dt1, _ = timed(n_queries_1t, 1, min_seconds_1t)
    O.max_threads(all_threads)
    per_batch = f"{min(n_queries, w.batches[0].batch)} per batch" if len(w.batches) > 1 else "first"
    return {"value": round(nq / dt, 3), "unit": "queries/s", "cores": threads, "kind": "oracle",
            "sample": f"{nq // passes} of the workload's {total} queries ({per_batch}) x {passes} passes on "
                      f"{threads} threads: fp64 node-by-node evaluation, full scoring of all {w.n_entities} "
                      f"entities + top-{w.k}" + (" (entity table decoded from bf16)" if ent is not None else ""),
            "seconds": round(dt, 3),
            "entity_scores_per_s": round(nq / dt * w.n_entities, 1),
            "single_thread": {"value": round(nq1 / dt1, 3), "unit": "queries/s", "cores": 1,
                              "sample": f"{nq1 // passes1} queries x {passes1} passes on 1 thread",
                              "seconds": round(dt1, 3)}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="C5")
    ap.add_argument("--no-others", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-other-mode", action="store_true",
                    help="skip the second timing of the headline workload in the other in-flight mode (so that "
                         "a kernel trace of the run holds only headline-mode launches)")
    ap.add_argument("--cpu-queries", type=int, default=None,
                    help="oracle sample: queries per batch on all host threads (default: sized per workload)")
    ap.add_argument("--per-structure", action="store_true",
                    help="one execute call per structure batch instead of one mixed call per step")
    ap.add_argument("--streams", type=int, default=2,
                    help="with --per-structure: streams the independent calls are spread over")
    ap.add_argument("--inflight", type=int, default=1,
                    help="steps in flight in the headline timed region: 1 (default) times one step at a "
                         "time; 2 or more alternate consecutive steps over that many streams (one scratch lane "
                         "and output buffer each), so that one step's small kernels overlap another's scorer. "
                         "The other mode is timed after the headline and reported beside it")
    ap.add_argument("--matrix-path", choices=["auto", "fp32"], default="auto",
                    help="dense contractions (MLP layers, BetaE scorer) on the bf16 matrix cores with the exact "
                         "three-part split where it pays (auto, the library default) or on the FP32 matrix "
                         "cores only (fp32)")
    ap.add_argument("--sweep", default=None, metavar="SIZES",
                    help="instead of the benchmark: per-query time and device memory against batch size, per "
                         "structure, on --workload's tables (comma-separated batch sizes, e.g. 1,16,256,1024)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.sweep:
        batch_sweep(args.workload, [int(x) for x in args.sweep.split(",")], max(args.steps, 1))
        return

    log(f"[bench] preparing {args.workload}")
    merge = not args.per_structure
    # The engine always has two scratch lanes and two output buffers, so the
    # same prepared workload can be timed one step at a time and with two
    # steps in flight.
    p = Prepared(args.workload, args.streams, merge, max(2, args.inflight), args.matrix_path)
    headline_serial = args.inflight == 1
    n_streams = 1 if headline_serial else len(p.streams)
    log(f"[bench] warmup {args.warmup}, timing {args.steps} steps: {len(p.calls)} execute call(s) per "
        f"step on {n_streams} stream(s), {1 if headline_serial else p.inflight} step(s) in flight")
    dt, iv = time_steps(p, args.steps, args.warmup, profile_score=True, serial=headline_serial)
    ms_step = dt / args.steps * 1e3
    qps = p.n_queries * args.steps / dt
    busy = union_ms(iv)                         # time with a scorer launch in flight
    n_launch = len(iv)
    avg_launch_ms = float(np.mean(iv[:, 1] - iv[:, 0])) if n_launch else 0.0
    total_ops = OPS_PER_TRIPLE[p.model] * p.triples * args.steps
    ops_per_launch = total_ops / max(n_launch, 1)
    achieved = ops_per_launch / (avg_launch_ms * 1e-3) if avg_launch_ms > 0 else 0.0
    achieved_busy = total_ops / (busy * 1e-3) if busy > 0 else 0.0
    traffic, traffic_req = traffic_for(p.model, f"score:{args.workload}")
    peak, bound, unit, basis = scorer_peak(p.model, args.matrix_path)
    in_flight_now = 1 if headline_serial else p.inflight
    roofline = {"bound": bound, "kernel": "k_score (entity scorer)" if p.model != 2 else "k_score_kl (entity scorer)",
                "achieved": round(achieved / 1e12, 3), "peak": round(peak / 1e12, 2),
                "unit": unit, "frac": round(achieved / peak, 4), "peak_basis": basis, "traffic": traffic,
                "traffic_by_request_size": traffic_req,
                "ops_per_launch": ops_per_launch, "avg_launch_ms": round(avg_launch_ms, 5),
                "launches": n_launch, "scorer_busy_ms": round(busy, 4),
                "frac_over_busy_time": round(achieved_busy / peak, 4),
                "timing": f"HIP events around every scorer launch on its stream over the timed steps "
                          f"({in_flight_now} step(s) in flight); achieved = algorithmic ops per launch / average "
                          f"launch duration"}
    roofline["derivation"] = scorer_derivation(p)
    if p.model == 2:
        roofline["matrix_path"] = args.matrix_path
        roofline["frac_of_fp32_mfma_peak"] = round(achieved / PEAK_MFMA_F32, 4)
    if p.model != 2 and avg_launch_ms > 0:
        # lane-operations of one launch against the non-packed issue rate
        lane_ops_per_launch = LANE_OPS_PER_TRIPLE[p.model] * p.triples * args.steps / max(n_launch, 1)
        roofline["frac_of_issue_peak"] = round(lane_ops_per_launch / (avg_launch_ms * 1e-3) / PEAK_VALU_OPS, 4)
    log(f"[bench] {args.workload}: {ms_step:.3f} ms/step, {qps:.0f} q/s, scorer busy {busy:.2f} ms over "
        f"{n_launch} launches ({avg_launch_ms:.4f} ms each), {roofline['frac']*100:.1f}% of the {bound} peak")
    # The other mode, reported beside the headline: with two steps in flight
    # one step's small kernels and launch gaps overlap the other's scorer,
    # which raises the step rate; the scorer then shares the compute units,
    # so its launch interval stretches and no longer measures the kernel.
    other_name = "two_steps_in_flight" if headline_serial else "one_step_at_a_time"
    other_mode = None
    if not args.no_other_mode:
        d2, iv2 = time_steps(p, args.steps, 2, profile_score=True, serial=not headline_serial)
        avg2 = float(np.mean(iv2[:, 1] - iv2[:, 0])) if len(iv2) else 0.0
        other_mode = {"ms_per_step": round(d2 / args.steps * 1e3, 4),
                      "queries_per_s": round(p.n_queries * args.steps / d2, 2),
                      "scorer_launch_ms": round(avg2, 5),
                      "scorer_frac": round(ops_per_launch / (avg2 * 1e-3) / peak, 4) if avg2 > 0 else None}
        log(f"[bench] {other_name.replace('_', ' ')}: {other_mode['ms_per_step']:.3f} ms/step, "
            f"{other_mode['queries_per_s']:.0f} q/s, scorer {avg2:.4f} ms per launch")
    stages = stage_breakdown(p)
    log(f"[bench] stage ms per step (one stream, instrumented): {stages}")
    rank = rank_bench(p)
    if rank:
        log(f"[bench] ranking metrics over the score matrix: {rank['avg_launch_ms']} ms, "
            f"{rank['achieved_GBps']} GB/s ({rank['frac_of_hbm_peak'] * 100:.1f}% of HBM peak)")

    others = {}
    if not args.no_others:
        for name in ["C1", "C2", "C3", "C4-q2b", "C4-gqe", "C5", "cone", "logice"]:
            if name == args.workload:
                continue
            log(f"[bench] other workload {name}")
            q = Prepared(name, args.streams, merge, max(2, args.inflight), args.matrix_path)
            steps = max(3, min(args.steps, 30))
            # one step at a time (the scorer's launch interval measures the
            # kernel alone), then two steps in flight
            d1, iv2 = time_steps(q, steps, 2, profile_score=True, serial=True)
            d2, _ = time_steps(q, steps, 2, profile_score=False)
            ops = OPS_PER_TRIPLE[q.model] * q.triples * steps
            b2 = union_ms(iv2)
            avg2 = float(np.mean(iv2[:, 1] - iv2[:, 0])) if len(iv2) else 0.0
            others[name] = {"workload": WORKLOAD_DESC[name], "queries_per_s": round(q.n_queries * steps / d1, 1),
                            "ms_per_step": round(d1 / steps * 1e3, 4),
                            "queries_per_s_two_in_flight": round(q.n_queries * steps / d2, 1),
                            "ms_per_step_two_in_flight": round(d2 / steps * 1e3, 4),
                            "entity_scores_per_s": round(q.n_queries * q.w.n_entities * steps / d1, 1),
                            "scorer_busy_ms_per_step": round(b2 / steps, 5),
                            "scorer_launch_ms": round(avg2, 5),
                            "scorer_bound": scorer_peak(q.model, args.matrix_path)[1],
                            "scorer_frac": round(ops / len(iv2) / (avg2 * 1e-3)
                                                 / scorer_peak(q.model, args.matrix_path)[0], 4)
                            if avg2 > 0 else None,
                            "scorer_frac_of_fp32_mfma_peak": round(ops / len(iv2) / (avg2 * 1e-3) / PEAK_MFMA_F32, 4)
                            if avg2 > 0 and q.model == 2 else None,
                            "scorer_frac_of_issue_peak": round(LANE_OPS_PER_TRIPLE[q.model] * q.triples * steps
                                                               / len(iv2) / (avg2 * 1e-3) / PEAK_VALU_OPS, 4)
                            if avg2 > 0 and q.model != 2 else None,
                            "stage_ms": stage_breakdown(q, reps=2)}
            log(f"[bench]   {name}: {others[name]['queries_per_s']} q/s, scorer frac "
                f"{others[name]['scorer_frac']} of the {others[name]['scorer_bound']} peak")
            q.eng.close()
            del q
            torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu:
        log("[bench] CPU oracle baseline")
        nq, nq1 = CPU_SAMPLE.get(args.workload, (64, 4))
        cpu = cpu_baseline(args.workload, args.cpu_queries or nq, nq1)
        log(f"[bench]   oracle {cpu['value']:.1f} q/s on {cpu['cores']} threads ({cpu['seconds']} s), "
            f"{cpu['single_thread']['value']:.2f} q/s on 1 thread ({cpu['single_thread']['seconds']} s)")

    out = {
        "metric": "queries/sec (score all entities + top-k) and achieved VALU/HBM roofline %",
        "value": round(qps, 2),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "arithmetic": ("dense contractions (BetaE scorer, MLP layers) on the bf16 matrix cores: "
                       "each FP32 operand split exactly into three bf16 parts, six part products accumulated in FP32 "
                       "(FP32 error class); the rest FP32"
                       if args.matrix_path == "auto" else "FP32 throughout (FP32 matrix cores and vector units)"),
        "data": "synthetic (seeded random tables and queries of the workload's shapes)",
        "config": {"workload": WORKLOAD_DESC[args.workload], "name": args.workload,
                   "queries_per_step": p.n_queries, "scored_rows_per_step": p.rows, "k": p.w.k,
                   "execute_calls_per_step": len(p.calls), "streams": n_streams,
                   "steps_in_flight": in_flight_now},
        "entity_scores_per_s": round(qps * p.w.n_entities, 1),
        "roofline": roofline,
        other_name: other_mode,
        "stage_ms_per_step": stages,
        "ranking_metrics": rank,
        "cpu_baseline": cpu,
        "others": others,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
