"""CPU checks of the seeded input generators (synth/): determinism, rounding to the storage
dtype, and the shapes and value distributions the workloads are specified with (lengths,
clones, planted near-duplicates, hard negatives, sentence topics).  Small sizes of every
generator; the statistics are checked with margins of several standard errors."""

import math

import numpy as np
import torch

import oracle
import synth


def _f(t):
    return t.detach().to(torch.float64)


def _cos(a, b):
    return (a * b).sum(-1) / (a.norm(dim=-1) * b.norm(dim=-1))


def test_generators_are_deterministic_per_seed():
    cases = [
        lambda s: synth.tiny_maxsim(seed=s, n_docs=16),
        lambda s: synth.coltrast_step(seed=s, nq=4, n_neg=3, ld=64),
        lambda s: synth.li_retrieval(seed=s, nq=4, n_docs=50),
        lambda s: synth.li_large(seed=s, nq=4, n_docs=50),
        lambda s: synth.dense_retrieval(seed=s, nq=8, n=300, dim=64, n_planted=4),
        lambda s: synth.sentence_stream(seed=s, n_papers=5, len_min=0, len_max=40, dim=64),
    ]
    for make in cases:
        a, b, c = make(3), make(3), make(4)
        keys = [k for k, v in a.items() if torch.is_tensor(v)]
        assert keys
        for k in keys:
            assert torch.equal(a[k], b[k]), k
        assert any(not torch.equal(a[k], c[k]) for k in keys if a[k].shape == c[k].shape)


def test_unit_rows_are_rounded_unit_vectors():
    g = torch.Generator().manual_seed(0)
    for dtype, ulp in ((torch.bfloat16, 2.0 ** -8), (torch.float16, 2.0 ** -11)):
        x = synth.unit_rows(2000, 128, g, "cpu", dtype)
        assert x.dtype == dtype
        n = _f(x).norm(dim=1)
        # each component is within half an ulp of its fp32 value: the norm within sqrt(dim) of it
        assert torch.all((n - 1).abs() <= math.sqrt(128) * ulp)
        assert (n - 1).abs().mean() < 4 * ulp


def test_fp16_store_keeps_subnormals():
    w = synth.dense_retrieval(seed=0, nq=4, n=2000, dim=4096, n_planted=2)
    bits = w["X"].view(torch.int16).numpy().astype(np.uint16)
    sub = ((bits & 0x7C00) == 0) & ((bits & 0x03FF) != 0)
    assert sub.mean() > 1e-3                       # components below 2^-14 stay subnormal
    vals = oracle.decode_fp16(bits[sub])
    assert np.all(np.abs(vals) < 2.0 ** -14) and np.all(vals != 0)


def test_li_retrieval_lengths_are_uniform():
    w = synth.li_retrieval(seed=0, nq=2, n_docs=20000)
    lens = (w["off"][1:] - w["off"][:-1]).numpy()
    assert lens.min() == 32 and lens.max() == 384
    assert abs(lens.mean() - 208.0) < 3.0            # 102 / sqrt(20000) = 0.72 standard error
    assert np.unique(lens).size == 353


def test_li_large_lengths_and_clones():
    n_docs = 20000
    w = synth.li_large(seed=0, nq=2, n_docs=n_docs)
    off, D = w["off"], w["D"]
    lens = (off[1:] - off[:-1]).numpy()
    assert lens.min() >= 16 and lens.max() <= 512
    assert abs(np.median(lens) - 200) <= 6
    assert abs((lens == 512).mean() - 0.031) < 0.006  # P(z > ln(512 / 200) / 0.5) = 3.1 %
    assert abs(lens.mean() - 223) < 4
    clones, src = w["clones"], w["clone_src"]
    assert clones.numel() == n_docs // 10
    assert not bool(torch.isin(src, clones).any())
    assert torch.equal(torch.as_tensor(lens)[clones], torch.as_tensor(lens)[src])
    for c, s in list(zip(clones.tolist(), src.tolist()))[:50]:
        a, b = _f(D[off[c]:off[c + 1]]), _f(D[off[s]:off[s + 1]])
        cs = _cos(a, b)
        assert cs.min() > 0.998, (c, s, float(cs.min()))   # sigma 0.002 per unit component


def test_dense_planted_rows_have_the_stated_cosine():
    w = synth.dense_retrieval(seed=0, nq=64, n=5000, dim=512, n_planted=40)
    pq, pr = w["planted_q"], w["planted_row"]
    assert pq.unique().numel() == 40 and pr.unique().numel() == 40
    cs = _cos(_f(w["X"][pr]), _f(w["Q"][pq]))
    assert torch.all((cs - 0.95).abs() < 2e-3)
    # the other rows are unrelated to those queries
    rest = torch.ones(w["X"].shape[0], dtype=torch.bool)
    rest[pr] = False
    others = _cos(_f(w["X"][rest][:500]), _f(w["Q"][pq[0]])[None])
    assert others.abs().max() < 0.3


def test_coltrast_step_positives_and_hard_negatives():
    nq, lq, n_neg, ld = 6, 32, 7, 256
    w = synth.coltrast_step(seed=0, nq=nq, lq=lq, n_neg=n_neg, ld=ld)
    Q, D, off, pos = _f(w["Q"]), _f(w["D"]), w["off"], w["pos"]
    assert torch.equal(pos, torch.arange(0, nq * (n_neg + 1), n_neg + 1, dtype=torch.int32))
    assert torch.equal(off, torch.arange(0, (nq * (n_neg + 1) + 1) * ld, ld))
    for h in range(n_neg + 1):
        sigma = 0.3 + 0.05 * h
        want = 1.0 / math.sqrt(1.0 + sigma * sigma)  # cos(q_raw, q_raw + sigma eps), dim large
        best = []
        for q in range(nq):
            d = q * (n_neg + 1) + h
            best.append((Q[q] @ D[off[d]:off[d + 1]].T).max(dim=1).values)
        best = torch.cat(best)
        assert abs(float(best.mean()) - want) < 0.02, (h, float(best.mean()), want)
    # a query's tokens against another query's documents: only the random maximum (~0.25)
    other = (Q[0] @ D[off[8]:off[9]].T).max(dim=1).values.mean()
    assert float(other) < 0.45


def test_sentence_stream_topics_and_lengths():
    w = synth.sentence_stream(seed=0, n_papers=60, len_min=5, len_max=120, dim=1024)
    E, off = _f(w["E"]), w["paper_off"]
    lens = (off[1:] - off[:-1]).numpy()
    assert lens.min() >= 5 and lens.max() <= 120
    c = _cos(E[1:], E[:-1]).numpy()
    first = np.zeros(E.shape[0], dtype=bool)
    first[off[:-1].numpy()] = True
    inner = c[~first[1:]]
    same = inner[inner > 0.5]
    assert abs(same.mean() - 1.0 / 1.25) < 0.02     # one topic: cos ~ 1 / (1 + 0.5^2)
    switch = (inner < 0.5).mean()
    assert abs(switch - 1.0 / 8.0) < 0.03           # a topic change every 8 sentences on average
    assert np.abs(inner[inner < 0.5]).max() < 0.2   # new topic: about orthogonal
