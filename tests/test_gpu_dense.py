"""GPU parity of dense_ip_topk (exact inner-product top-k over an fp16 store) against the oracle.

The call has three regimes, each covered here:
  * the store is no larger than the exact sample (every row is scored and selected directly);
  * the filter path: rows past the sample are kept only when they beat the sample's k-th score;
  * the exact fallback: a query whose candidate list overflows is queued on the device and its
    k-th key found by a radix select over rescans of the store, then its top-k collected; the
    call stays asynchronous (it is captured and replayed in a HIP graph here).
Top-k lists are checked with the rules of tests/topk_check.py at tolerance 2e-3 (fp16 products
are exact in fp32, so scores differ from the oracle only by the fp32 summation order).
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2505_04846_amd as hpr
import synth
from topk_check import check_topk

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
REL = 2e-3
SAMPLE_ROWS = 131072  # rows scored exactly before the filtered scan (k <= 4096)


def _f16(t):
    return oracle.decode_fp16(t.detach().cpu().contiguous().view(torch.int16).numpy())


def _rows(n, dim, seed):
    g = torch.Generator().manual_seed(seed)
    return synth.unit_rows(n, dim, g, "cpu", torch.float16)


def _check_structure(s, i, n, k):
    assert s.shape[1] == k and i.shape[1] == k
    assert np.all((i >= 0) & (i < n))
    for q in range(s.shape[0]):
        assert np.unique(i[q]).size == k
        a, b = s[q, :-1], s[q, 1:]
        assert np.all((a > b) | ((a == b) & (i[q, :-1] < i[q, 1:])))


@pytest.mark.parametrize("nq,n,dim,k", [
    (1, 1, 8, 1),          # smallest shapes
    (37, 5000, 200, 10),   # K tail (200 = 6 chunks of 32 + 8), ragged query and row tiles
    (300, 2048, 4096, 100),
    (5, 1000, 8192, 1000),  # largest dim; k = n
    (3, 777, 24, 777),
    (64, 3000, 128, 10),   # the widest narrow (64-query) tile
    (65, 3000, 136, 10),   # the narrowest wide (256-query) tile
])
def test_dense_topk_whole_store_sampled(nq, n, dim, k):
    Q, X = _rows(nq, dim, 1 + n), _rows(n, dim, 2 + n)
    s, i = hpr.dense_ip_topk(Q.to(DEV), X.to(DEV), k)
    s, i = s.cpu().numpy(), i.cpu().numpy()
    O = oracle.dense_scores(_f16(Q), _f16(X))
    for q in range(nq):
        check_topk(s[q], i[q], O[q], k, rel=REL)


def test_dense_topk_filter_path_matches_oracle():
    nq, n, dim, k = 300, 200_000, 96, 50
    assert n > SAMPLE_ROWS
    Q, X = _rows(nq, dim, 11), _rows(n, dim, 12)
    s, i = hpr.dense_ip_topk(Q.to(DEV), X.to(DEV), k)
    s, i = s.cpu().numpy(), i.cpu().numpy()
    _check_structure(s, i, n, k)
    Xh = _f16(X)
    Qh = _f16(Q)
    # every returned score against the oracle's score of the same row
    for q in range(nq):
        o = Xh[i[q]] @ Qh[q]
        err = np.abs(s[q] - o)
        assert np.all(err <= REL * np.maximum(np.abs(o), 1e-3)), f"query {q}"
    # full oracle rows for the tile edges and a seeded sample of queries
    rng = np.random.default_rng(0)
    pick = sorted(set([0, 1, 255, 256, 299]) | set(rng.choice(nq, 11, replace=False).tolist()))
    O = oracle.dense_scores(Qh[pick], Xh)
    for r, q in enumerate(pick):
        res = check_topk(s[q], i[q], O[r], k, rel=REL)
        assert res["exact"] or res["exception_used"]


def test_dense_topk_filter_path_few_queries():
    # at most 64 queries take the narrow tile in the sample and in the filtered scan
    nq, n, dim, k = 17, 400_000, 256, 100
    Q, X = _rows(nq, dim, 13), _rows(n, dim, 14)
    s, i = hpr.dense_ip_topk(Q.to(DEV), X.to(DEV), k)
    s, i = s.cpu().numpy(), i.cpu().numpy()
    _check_structure(s, i, n, k)
    O = oracle.dense_scores(_f16(Q), _f16(X))
    for q in range(nq):
        check_topk(s[q], i[q], O[q], k, rel=REL)


def test_dense_topk_overflowing_lists_take_the_exact_fallback():
    nq, n, dim, k = 40, 150_000, 64, 20
    Q, X = _rows(nq, dim, 21), _rows(n, dim, 22)
    a0 = SAMPLE_ROWS + 100
    a1 = SAMPLE_ROWS + 5000
    X[a0:a0 + 3000] = Q[0]   # 3000 bit-identical rows equal to query 0, past the sample
    X[a1:a1 + 2000] = Q[1]
    Qd, Xd = Q.to(DEV), X.to(DEV)
    s, i = hpr.dense_ip_topk(Qd, Xd, k)
    s2, i2 = hpr.dense_ip_topk(Qd, Xd, k)
    assert torch.equal(s, s2) and torch.equal(i, i2)
    s, i = s.cpu().numpy(), i.cpu().numpy()
    _check_structure(s, i, n, k)
    # the copies tie exactly and outrank every other row: the lowest k indices win
    assert i[0].tolist() == list(range(a0, a0 + k))
    assert i[1].tolist() == list(range(a1, a1 + k))
    assert np.all(s[0] == s[0, 0]) and np.all(s[1] == s[1, 0])
    Qh, Xh = _f16(Q), _f16(X)
    O = oracle.dense_scores(Qh[:4], Xh)
    assert abs(s[0, 0] - O[0, a0]) <= REL * abs(O[0, a0])
    for q in range(2, 4):
        check_topk(s[q], i[q], O[q], k, rel=REL)


def _overflowing_store(nq, n, dim, copies, seed):
    # queries near a common direction u; `copies` bit-identical rows equal to u past the sample
    # outscore every random row for every query, so every candidate list overflows
    g = torch.Generator().manual_seed(seed)
    u = synth.unit_rows(1, dim, g, "cpu", torch.float32)
    noise = torch.randn((nq, dim), generator=g)
    Q = synth._normalise(u + 0.1 * noise / dim ** 0.5).to(torch.float16)
    X = _rows(n, dim, seed + 1)
    a0 = SAMPLE_ROWS + 777
    X[a0:a0 + copies] = u.to(torch.float16)
    return Q, X, a0


def test_dense_topk_every_list_overflows():
    # 70 queries: the scan takes the wide tile, the fallback two 64-query tiles
    nq, n, dim, k = 70, 140_000, 64, 100
    Q, X, a0 = _overflowing_store(nq, n, dim, 2500, 41)
    s, i = hpr.dense_ip_topk(Q.to(DEV), X.to(DEV), k)
    s, i = s.cpu().numpy(), i.cpu().numpy()
    _check_structure(s, i, n, k)
    for q in range(nq):
        assert i[q].tolist() == list(range(a0, a0 + k)), f"query {q}"
        assert np.all(s[q] == s[q, 0])
    Qh, Xh = _f16(Q), _f16(X)
    O = oracle.dense_scores(Qh[[0, 63, 64, 69]], Xh)
    for r, q in enumerate((0, 63, 64, 69)):
        check_topk(s[q], i[q], O[r], k, rel=REL)


def test_dense_topk_replays_in_a_hip_graph_with_overflow():
    # the whole call, the device-decided fallback included, is captured once and replayed with
    # eager work and synchronisation in between; every replay reproduces the eager result
    nq, n, dim, k = 40, 150_000, 64, 20
    Q, X = _rows(nq, dim, 21), _rows(n, dim, 22)
    a0 = SAMPLE_ROWS + 100
    X[a0:a0 + 3000] = Q[0]
    Qd, Xd = Q.to(DEV), X.to(DEV)
    ref_s, ref_i = hpr.dense_ip_topk(Qd, Xd, k)
    ws = hpr.dense_workspace(Qd, Xd, k)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        hpr.dense_ip_topk(Qd, Xd, k, ws=ws)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gs, gi = hpr.dense_ip_topk(Qd, Xd, k, ws=ws)
    for rep in range(3):
        gs.fill_(float("nan"))
        gi.fill_(-1)
        g.replay()
        hpr.dense_ip_topk(Qd[:3].contiguous(), Xd, 5)   # unrelated eager work
        torch.cuda.synchronize()
        assert torch.equal(gs, ref_s) and torch.equal(gi, ref_i), f"replay {rep}"
    assert gi[0].tolist() == list(range(a0, a0 + k))


def test_dense_topk_planted_rows_rank_first():
    w = synth.dense_retrieval(seed=0, device=DEV, nq=512, n=300_000, dim=512, k=10, n_planted=200)
    s, i = hpr.dense_ip_topk(w["Q"], w["X"], w["k"])
    pq, pr = w["planted_q"].cpu().numpy(), w["planted_row"].cpu().numpy()
    s, i = s.cpu().numpy(), i.cpu().numpy()
    assert np.array_equal(i[pq, 0], pr)
    assert np.all(np.abs(s[pq, 0] - w["cosine"]) < 3e-3)
    Qh = _f16(w["Q"][torch.as_tensor(pq[:8])])
    Xh = _f16(w["X"][torch.as_tensor(pr[:8])])
    o = np.sum(Qh * Xh, axis=1)
    assert np.all(np.abs(s[pq[:8], 0] - o) <= REL * np.abs(o))


def test_dense_topk_workspace_and_errors():
    Q, X = _rows(4, 64, 31).to(DEV), _rows(100, 64, 32).to(DEV)
    with pytest.raises(hpr.HprError) as e:
        hpr.dense_ip_topk(Q, X, 101)
    assert e.value.status_name == "HPR_ERR_INVALID_ARG"
    with pytest.raises(hpr.HprError) as e:
        hpr.dense_ip_topk(Q[:, :60].contiguous(), X[:, :60].contiguous(), 5)
    assert e.value.status_name == "HPR_ERR_UNSUPPORTED_SHAPE"
    ws = hpr.dense_workspace(Q, X, 5)
    s1, i1 = hpr.dense_ip_topk(Q, X, 5, ws=ws)
    s2, i2 = hpr.dense_ip_topk(Q, X, 5, ws=ws)
    assert torch.equal(s1, s2) and torch.equal(i1, i2)
