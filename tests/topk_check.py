"""Verification of a GPU top-k list against oracle scores of every candidate.

With floating-point scores several answers can be right: the GPU computes scores in fp32 from
bf16/fp16 products, the oracle in fp64, and documents whose scores lie within the tolerance of
the k-th score may legitimately swap places.  This module therefore verifies what is unique
and that the rest is valid, at tolerance T(x) = rel * max(|x|, 1e-3):

  1. indices are distinct and in range; the list is sorted by (GPU score desc, index asc);
  2. every returned score is within T of the oracle score of the same index;
  3. every candidate whose oracle score exceeds the oracle k-th score t by more than T(t) is
     returned, and every returned candidate has oracle score >= t - T(t);
  4. if the oracle's k-th and (k+1)-th scores differ by more than T, the returned set equals the
     oracle's top-k set exactly;
  5. no clear inversion: for positions a < b, oracle(a) >= oracle(b) - T.

It returns per-query diagnostics (exact ordered match, whether rule 4's exception was used).
"""

import numpy as np


def tol(x, rel):
    return rel * np.maximum(np.abs(x), 1e-3)


def check_topk(gpu_scores, gpu_idx, oracle_row_scores, k, rel=2e-3):
    """gpu_scores/gpu_idx: [k] arrays for one query; oracle_row_scores: fp64 [n] for that query."""
    gs = np.asarray(gpu_scores, dtype=np.float64)
    gi = np.asarray(gpu_idx, dtype=np.int64)
    o = np.asarray(oracle_row_scores, dtype=np.float64)
    n = o.size
    assert gs.shape == (k,) and gi.shape == (k,)
    # 1
    assert np.all((gi >= 0) & (gi < n)), "index out of range"
    assert np.unique(gi).size == k, "duplicate indices"
    for a in range(k - 1):
        assert gs[a] > gs[a + 1] or (gs[a] == gs[a + 1] and gi[a] < gi[a + 1]), \
            f"not sorted at position {a}: ({gs[a]}, {gi[a]}) then ({gs[a+1]}, {gi[a+1]})"
    # 2
    og = o[gi]
    bad = np.abs(gs - og) > tol(og, rel)
    assert not bad.any(), f"returned score off at positions {np.nonzero(bad)[0][:5]}"
    # oracle order
    order = np.lexsort((np.arange(n), -o))
    t = o[order[k - 1]]
    # 3
    must = np.nonzero(o > t + tol(t, rel))[0]
    missing = np.setdiff1d(must, gi)
    assert missing.size == 0, f"clearly-in documents missing: {missing[:5]}"
    assert np.all(og >= t - tol(t, rel)), "a returned document is clearly below the k-th score"
    # 4
    exception_used = False
    if k < n:
        t_next = o[order[k]]
        if t - t_next > tol(t, rel):
            assert set(gi.tolist()) == set(order[:k].tolist()), "top-k set differs"
        else:
            exception_used = True
    else:
        assert set(gi.tolist()) == set(range(n))
    # 5
    for a in range(k):
        later = og[a + 1:]
        assert np.all(og[a] >= later - tol(later, rel)), f"inversion after position {a}"
    exact = bool(np.array_equal(gi, order[:k]))
    return {"exact": exact, "exception_used": exception_used}
