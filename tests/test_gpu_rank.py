"""GPU parity of the filtered ranking metrics (kgq_rank_answers) against the
oracle: ranks bit-exact, MRR / Hits@k equal (both sum in double precision in
answer-list order). The score matrices are seeded synthetic values with many
exact ties (the ranking must agree on every tie); one test ranks the scores
of a real execute against its own top-k."""


import numpy as np
import pytest

from oracle import oracle as O
from paper_2503_02172_amd import synth

pytestmark = pytest.mark.gpu


def _engine(N: int, max_batch: int = 8):
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(O.GQE, n_ent=N, n_rel=3, dim=8, seed=2)
    return kgq.engine_for(w, max_batch=max_batch)


def _scores(B: int, N: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    s = (rng.integers(-300, 300, size=(B, N)) / 16.0).astype(np.float32)    # many exact ties
    s[0] = 0.5                                                             # an all-equal row
    if B > 2:
        s[2, ::2] = -0.0                                                   # -0 and +0 rank equal
        s[2, 1::2] = 0.0
    return s


def _check(eng, s: np.ndarray, off, ids, hard, ld_pad: int = 0):
    import torch
    B, N = s.shape
    dev = torch.device("cuda", 0)
    buf = np.zeros((B, N + ld_pad), np.float32)
    buf[:, :N] = s
    if ld_pad:
        buf[:, N:] = 1e30                                                  # outside the row: must be ignored
    ts = torch.as_tensor(buf, device=dev)
    to = torch.as_tensor(off, device=dev)
    ti = torch.as_tensor(ids, device=dev)
    th = None if hard is None else torch.as_tensor(hard, device=dev)
    ranks, met = eng.rank_answers(ts, to, ti, th)
    torch.cuda.synchronize()
    r_ref, m_ref = O.rank_answers(s, off, ids, hard)
    np.testing.assert_array_equal(ranks.cpu().numpy(), r_ref)
    m = met.cpu().numpy()
    assert np.array_equal(np.isnan(m), np.isnan(m_ref))
    ok = ~np.isnan(m_ref)
    np.testing.assert_array_equal(m[ok], m_ref[ok])


@pytest.mark.parametrize("N", [37, 1000, 14505])
def test_gpu_ranks_match_oracle(N):
    B = 24
    eng = _engine(N, max_batch=B)
    s = _scores(B, N, seed=N)
    # list sizes up to 64, plus: an empty list, one of length 1, one with
    # every entity (small N) or the maximum length, one with no hard answer
    big = min(N, 1024)
    off, ids, hard = synth.draw_answers(B, N, seed=N + 1, max_len=min(64, N), special={3: 0, 4: 1, 5: big})
    hard[off[6]:off[7]] = 0
    _check(eng, s, off, ids, hard)
    _check(eng, s, off, ids, None)                                          # every answer hard
    _check(eng, s, off, ids, hard, ld_pad=7)                                # a row stride above N


def test_gpu_ranks_at_the_63361_entity_shape():
    B, N = 6, 63361
    eng = _engine(N, max_batch=B)
    s = _scores(B, N, seed=9)
    off, ids, hard = synth.draw_answers(B, N, seed=10, max_len=300, special={1: 1024})
    _check(eng, s, off, ids, hard)


@pytest.mark.parametrize("B,N", [(2304, 14505), (520, 63361)], ids=["2304x14505", "520x63361"])
def test_gpu_ranks_at_batch_scale(B, N):
    """Batches large enough for the streaming kernel's wide forms: one
    wavefront per query (two queries a workgroup) on 14,505-entity rows, and
    rows of 63,361 split over four wavefronts; lists of every length up to 64
    (the streaming kernel takes up to 32, the workgroup kernel the rest)."""
    eng = _engine(N, max_batch=8)
    s = _scores(B, N, seed=B + N)
    off, ids, hard = synth.draw_answers(B, N, seed=B + N + 1, max_len=64, special={7: 0, 8: 1, 9: 32, 10: 33})
    _check(eng, s, off, ids, hard)


def test_gpu_ranks_agree_with_the_topk_order():
    """On the scores of a real execute: the top-k entries taken as answers are
    each preceded only by answers (rank 1); the k-th entry alone is preceded by
    the k - 1 entries above it (rank k)."""
    import torch
    from paper_2503_02172_amd import kgq
    w = synth.make_tiny(O.Q2B, n_ent=600, n_rel=5, dim=16, seed=11)
    eng = kgq.engine_for(w, max_batch=8)
    q = synth.draw_queries("2i", 8, 600, 5, seed=12)
    out = eng.execute(synth.STRUCTURE_ID["2i"], q.anchors, q.relations, k=20, scores=True)
    top = out["idx"].cpu().numpy()
    dev = torch.device("cuda", 0)
    lists = [top[b, :10].tolist() for b in range(8)] + [[int(top[b, 19])] for b in range(8)]
    off = np.zeros(17, np.int32)
    off[1:] = np.cumsum([len(l) for l in lists])
    ids = np.array([e for l in lists for e in l], np.int32)
    scores = torch.cat([out["scores"], out["scores"]], 0).contiguous()
    ranks, met = eng.rank_answers(scores, torch.as_tensor(off, device=dev), torch.as_tensor(ids, device=dev))
    torch.cuda.synchronize()
    r = ranks.cpu().numpy()
    assert (r[:80] == 1).all()
    assert (r[80:] == 20).all()
    m = met.cpu().numpy()
    assert (m[:8] == 1.0).all()
    assert np.allclose(m[8:, 0], 1 / 20) and (m[8:, 1:] == 0).all()


def test_gpu_rank_answers_checked_errors():
    import torch
    from paper_2503_02172_amd import kgq
    N = 100
    eng = _engine(N, max_batch=4)
    eng.set_checked(True)
    dev = torch.device("cuda", 0)
    s = torch.zeros((2, N), dtype=torch.float32, device=dev)
    off = torch.tensor([0, 1, 2], dtype=torch.int32, device=dev)
    with pytest.raises(kgq.KgqError) as e:
        eng.rank_answers(s, off, torch.tensor([5, N], dtype=torch.int32, device=dev))
    assert e.value.status == -2                                             # OUT_OF_RANGE
    long_off = torch.tensor([0, 1025, 1026], dtype=torch.int32, device=dev)
    long_ids = torch.as_tensor(np.arange(1026) % N, dtype=torch.int32, device=dev)
    with pytest.raises(kgq.KgqError) as e:
        eng.rank_answers(s, long_off, long_ids)
    assert e.value.status == -1                                             # INVALID_ARG
    ranks, met = eng.rank_answers(s, off, torch.tensor([5, 7], dtype=torch.int32, device=dev))
    torch.cuda.synchronize()
    # all scores equal: ties go by index, so entity 5 follows entities 0..4 and
    # entity 7 follows 0..6
    assert ranks.cpu().tolist() == [6, 8] and float(met[0, 0]) == 1 / 6
