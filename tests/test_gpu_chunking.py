"""GPU parity of semantic_chunk and retrieval_metrics against the fp64 oracle, through the C ABI.

semantic_chunk: cosines within 2e-5 absolute (fp32 sums of exact fp16 products; the oracle is
fp64 on the same fp16 values), NaN exactly where the oracle's is.  The boundary decisions are
integers decided by floating point: each must equal the oracle's wherever the oracle's cosine is
more than 2e-5 from the threshold; inside that band either decision is valid, and the segment ids
must then be the exact prefix count of the GPU's own decisions.  retrieval_metrics: ranks bit-exact,
P@k and MRR@k within 1e-12.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2505_04846_amd as hpr
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
BAND = 2e-5
GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "chunking_metrics.json")))


def _f16(t):
    return oracle.decode_fp16(t.detach().cpu().contiguous().view(torch.int16).numpy())


def _check(E, off, thr, cos_g, seg_g, nseg_g):
    Eh = _f16(E)
    cos_o, seg_o, nseg_o = oracle.semantic_segments(Eh, None if off is None else off.numpy(), thr)
    nan_o = np.isnan(cos_o)
    assert np.array_equal(np.isnan(cos_g), nan_o), "NaN positions differ"
    assert np.all(np.abs(cos_g[~nan_o] - cos_o[~nan_o]) <= BAND), \
        f"worst cosine error {np.max(np.abs(cos_g[~nan_o] - cos_o[~nan_o])):.3g}"
    with np.errstate(invalid="ignore"):
        b_g = ~(cos_g > np.float32(thr))
        b_o = ~(cos_o > thr)
    clear = nan_o | (np.abs(cos_o - thr) > BAND)
    assert np.array_equal(b_g[clear], b_o[clear]), "boundary decisions differ outside the band"
    assert np.array_equal(seg_g, np.cumsum(b_g.astype(np.int64)) - 1), "ids are not the prefix count"
    assert nseg_g == int(b_g.sum())
    if clear.all():
        assert np.array_equal(seg_g, seg_o) and nseg_g == nseg_o
    return cos_o, seg_o


def _run(E, off, thr):
    r = hpr.semantic_chunk(E.to(DEV), None if off is None else off.to(DEV), thr, return_cos=True)
    return (r["cos"].cpu().numpy().astype(np.float64), r["seg"].cpu().numpy().astype(np.int64),
            int(r["n_segments"].item()))


@pytest.mark.parametrize("ex", GOLDEN["chunking"], ids=lambda e: e["name"])
def test_chunking_golden_examples(ex):
    # the 2-D fixtures embedded in dim 8 (zeros elsewhere), in fp16
    if "vectors" in ex:
        V = np.array(ex["vectors"], dtype=np.float64)
    else:
        a = np.radians(np.array(ex["angles_deg"], dtype=np.float64))
        r = np.array(ex["norms"], dtype=np.float64)
        V = np.stack([r * np.cos(a), r * np.sin(a)], axis=1)
    E = torch.zeros((V.shape[0], 8), dtype=torch.float16)
    E[:, :2] = torch.from_numpy(V).to(torch.float16)
    off = None if ex["paper_off"] is None else torch.tensor(ex["paper_off"], dtype=torch.int64)
    thr = ex["threshold"] if "threshold" in ex else math.cos(math.radians(ex["threshold_deg"]))
    cos_g, seg_g, n_g = _run(E, off, thr)
    _check(E, off, thr, cos_g, seg_g, n_g)
    assert seg_g.tolist() == ex["segments"] and n_g == ex["n_segments"]


@pytest.mark.parametrize("n_papers,dim,thr,with_off", [
    (1, 8, 0.5, False),
    (3, 64, 0.5, True),
    (40, 520, 0.6, True),      # dim not a power of two
    (60, 4096, 0.5, True),     # the largest dim
    (25, 128, -2.0, True),     # everything joins: one segment per non-empty paper
    (25, 128, 2.0, True),      # nothing joins: one segment per sentence
    (30, 256, 0.5, False),     # one paper across many wave ranges
])
def test_chunking_random_papers(n_papers, dim, thr, with_off):
    w = synth.sentence_stream(seed=n_papers, n_papers=n_papers, len_min=0 if n_papers > 1 else 1,
                              len_max=300, dim=dim)
    off = w["paper_off"] if with_off else None
    cos_g, seg_g, n_g = _run(w["E"], off, thr)
    _check(w["E"], off, thr, cos_g, seg_g, n_g)


def test_chunking_paper_starts_on_range_edges():
    # papers starting exactly at, just before and just after the 128-sentence wave ranges, and
    # runs of empty papers
    dim = 32
    g = torch.Generator().manual_seed(3)
    n = 1000
    E = synth.unit_rows(n, dim, g, "cpu", torch.float16)
    E[1::2] = E[0::2][: E[1::2].shape[0]]  # consecutive pairs identical: cosine 1
    off = torch.tensor([0, 127, 128, 128, 128, 129, 255, 256, 384, 511, 640, 1000, 1000],
                       dtype=torch.int64)
    for thr in (0.9, -2.0):
        cos_g, seg_g, n_g = _run(E, off, thr)
        _check(E, off, thr, cos_g, seg_g, n_g)


def test_chunking_zero_vectors_and_single_sentence():
    E = torch.zeros((5, 16), dtype=torch.float16)
    E[0, 0] = 1.0
    E[3, 1] = 2.0
    E[4, 1] = 1.0
    cos_g, seg_g, n_g = _run(E, None, 0.5)
    _check(E, None, 0.5, cos_g, seg_g, n_g)
    assert seg_g.tolist() == [0, 1, 2, 3, 3]
    cos_g, seg_g, n_g = _run(E[:1].contiguous(), None, 0.5)
    assert seg_g.tolist() == [0] and n_g == 1 and math.isnan(cos_g[0])


def test_chunking_is_deterministic_and_graph_replayable():
    w = synth.sentence_stream(seed=9, n_papers=20, dim=256)
    E, off = w["E"].to(DEV), w["paper_off"].to(DEV)
    ws = hpr.semantic_chunk_workspace(E)
    ref = hpr.semantic_chunk(E, off, 0.5, return_cos=True)
    out = {"seg": torch.empty_like(ref["seg"]), "n_segments": torch.empty_like(ref["n_segments"]),
           "cos": torch.empty_like(ref["cos"])}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        hpr.semantic_chunk(E, off, 0.5, return_cos=True, ws=ws, out=out)
    torch.cuda.current_stream().wait_stream(side)
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr):
        hpr.semantic_chunk(E, off, 0.5, return_cos=True, ws=ws, out=out)
    for rep in range(3):
        for key in out:
            out[key].fill_(-7)
        gr.replay()
        torch.cuda.synchronize()
        for key in out:  # bit patterns (the cosines hold NaNs)
            a, b = out[key], ref[key]
            if a.dtype == torch.float32:
                a, b = a.view(torch.int32), b.view(torch.int32)
            assert torch.equal(a, b), f"replay {rep}: {key}"


@pytest.mark.parametrize("ex", GOLDEN["metrics"], ids=lambda e: e["name"])
def test_metrics_golden_examples(ex):
    idx = torch.tensor(ex["topk_idx"], dtype=torch.int64, device=DEV)
    pos = torch.tensor(ex["positive"], dtype=torch.int64, device=DEV)
    r = hpr.retrieval_metrics(idx, pos, ex["k"])
    m = r["metrics"].cpu().numpy()
    assert r["ranks"].cpu().tolist() == ex["ranks"]
    assert abs(m[0] - ex["p_at_k"][0] / ex["p_at_k"][1]) < 1e-15
    assert abs(m[1] - ex["mrr_at_k"][0] / ex["mrr_at_k"][1]) < 1e-15


@pytest.mark.parametrize("nq,ld,k", [(1, 1, 1), (3000, 100, 10), (5000, 1000, 1000)])
def test_metrics_random(nq, ld, k):
    g = torch.Generator().manual_seed(nq + k)
    idx = torch.stack([torch.randperm(5 * ld, generator=g)[:ld] for _ in range(nq)])
    # positives: a third at a random rank within ld, the rest absent
    pos = torch.full((nq,), 10 * ld, dtype=torch.int64)
    sel = torch.arange(nq) % 3 == 0
    j = torch.randint(0, ld, (nq,), generator=g)
    pos[sel] = idx[torch.arange(nq), j][sel]
    r = hpr.retrieval_metrics(idx.to(DEV), pos.to(DEV), k)
    p, mrr, ranks = oracle.retrieval_metrics(idx.numpy(), pos.numpy(), k)
    assert np.array_equal(r["ranks"].cpu().numpy(), ranks)
    m = r["metrics"].cpu().numpy()
    assert abs(m[0] - p) < 1e-12 and abs(m[1] - mrr) < 1e-12


def test_metrics_of_dense_retrieval_with_planted_pairs():
    # end to end: the planted near-duplicate of each planted query is retrieved first
    w = synth.dense_retrieval(seed=1, device=DEV, nq=300, n=200_000, dim=256, k=10, n_planted=100)
    s, i = hpr.dense_ip_topk(w["Q"], w["X"], w["k"])
    pq, pr = w["planted_q"], w["planted_row"]
    r = hpr.retrieval_metrics(i[pq].contiguous(), pr.contiguous(), 10)
    m = r["metrics"].cpu().numpy()
    assert m[1] == 1.0 and abs(m[0] - 0.1) < 1e-15
    assert torch.all(r["ranks"] == 1)
