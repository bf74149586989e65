"""Pins of the oracle's semantic chunking (Sec. 3.2.2) and retrieval metrics (Sec. 4.2).

The hand-worked fixtures in tests/golden/chunking_metrics.json fix the cosine of each
consecutive pair (2-D vectors at known angles), the strict "above" rule, forced boundaries at
paper starts (an empty paper included), NaN cosines of zero vectors, and P@k / MRR@k as exact
fractions.  Invariants add scale invariance, the two threshold extremes, the monotone structure
of segment ids, and MRR >= P@k.  An off-by-one pairing, a >= instead of >, a missed paper start
or a wrong average fails at least one of them.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "chunking_metrics.json")))


def _vectors(ex):
    if "vectors" in ex:
        return np.array(ex["vectors"], dtype=np.float64)
    a = np.radians(np.array(ex["angles_deg"], dtype=np.float64))
    r = np.array(ex["norms"], dtype=np.float64)
    return np.stack([r * np.cos(a), r * np.sin(a)], axis=1)


@pytest.mark.parametrize("ex", GOLDEN["chunking"], ids=lambda e: e["name"])
def test_chunking_golden(ex):
    E = _vectors(ex)
    thr = ex["threshold"] if "threshold" in ex else math.cos(math.radians(ex["threshold_deg"]))
    cos, seg, n = oracle.semantic_segments(E, ex["paper_off"], thr)
    want_cos = ex.get("cos") or [None if c is None else math.cos(math.radians(c))
                                 for c in ex["cos_deg"]]
    for t, w in enumerate(want_cos):
        if w is None:
            assert math.isnan(cos[t]), t
        else:
            assert abs(cos[t] - w) < 1e-12, (t, cos[t], w)
    assert seg.tolist() == ex["segments"]
    assert n == ex["n_segments"]


@pytest.mark.parametrize("ex", GOLDEN["metrics"], ids=lambda e: e["name"])
def test_metrics_golden(ex):
    p, mrr, ranks = oracle.retrieval_metrics(ex["topk_idx"], ex["positive"], ex["k"])
    assert ranks.tolist() == ex["ranks"]
    assert abs(p - ex["p_at_k"][0] / ex["p_at_k"][1]) < 1e-15
    assert abs(mrr - ex["mrr_at_k"][0] / ex["mrr_at_k"][1]) < 1e-15


def _random_papers(rng, n_papers, dim, topic_len=5):
    lens = rng.integers(0, 12, n_papers)
    off = np.concatenate([[0], np.cumsum(lens)])
    n = int(off[-1])
    topics = rng.standard_normal((n // topic_len + 2, dim))
    E = topics[np.arange(n) // topic_len] + 0.3 * rng.standard_normal((n, dim))
    return E, off


def test_chunking_invariants():
    rng = np.random.default_rng(5)
    E, off = _random_papers(rng, 40, 16)
    n = E.shape[0]
    cos, seg, ns = oracle.semantic_segments(E, off, 0.5)
    # scaling sentences by positive factors changes nothing
    c = rng.uniform(0.1, 10.0, n)[:, None]
    cos2, seg2, ns2 = oracle.semantic_segments(E * c, off, 0.5)
    assert np.allclose(np.nan_to_num(cos2), np.nan_to_num(cos), atol=1e-12)
    assert np.array_equal(seg2, seg) and ns2 == ns
    # ids start at 0, never decrease, grow by at most one, and count the segments
    assert seg[0] == 0 and np.all(np.diff(seg) >= 0) and np.all(np.diff(seg) <= 1)
    assert seg[-1] + 1 == ns
    # every paper start opens a segment
    first = oracle.paper_starts(n, off)
    assert np.all(np.diff(seg)[first[1:]] == 1)
    # threshold below -1: one segment per non-empty paper; at or above 1: one per sentence
    _, _, lo = oracle.semantic_segments(E, off, -1.5)
    assert lo == int(np.sum(np.diff(off) > 0))
    _, seg_hi, hi = oracle.semantic_segments(E, off, 1.5)
    assert hi == n and np.array_equal(seg_hi, np.arange(n))
    # a looser threshold never adds boundaries
    _, _, ns_lo = oracle.semantic_segments(E, off, 0.2)
    assert ns_lo <= ns


def test_metrics_closed_forms():
    rng = np.random.default_rng(6)
    nq, k = 50, 10
    idx = np.stack([rng.permutation(1000)[:k] for _ in range(nq)])
    # the positive ranked first everywhere: MRR = 1, P@k = 1/k
    p, mrr, _ = oracle.retrieval_metrics(idx, idx[:, 0], k)
    assert p == 1.0 / k and mrr == 1.0
    # never retrieved: both zero
    p, mrr, r = oracle.retrieval_metrics(idx, np.full(nq, 5000), k)
    assert p == 0.0 and mrr == 0.0 and np.all(r == 0)
    # a random position j: MRR = mean 1 / (j + 1) >= P@k
    j = rng.integers(0, k, nq)
    p, mrr, r = oracle.retrieval_metrics(idx, idx[np.arange(nq), j], k)
    assert np.array_equal(r, j + 1)
    assert abs(mrr - np.mean(1.0 / (j + 1))) < 1e-15 and mrr >= p
