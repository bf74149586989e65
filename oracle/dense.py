"""Single-vector (pooled-embedding) retrieval scores and exact top-k, fp64 (test infrastructure only).

At query time the paper ranks chunks by the cosine similarity between the pooled question
embedding and each pooled chunk embedding, and returns the IDs of the nearest neighbours
(Sec. 3.2.1 paragraph "Similarity metric"; Sec. 4.2 "ColTrast Retrieval Evaluation"; Sec. 2.3).
For L2-normalised embeddings the cosine is the inner product, which is what is computed here:

    s[q, n] = < Q[q, :], X[n, :] >

Ranking is by (score descending, row index ascending).
"""

import numpy as np

from .maxsim import rank_topk


def dense_scores(Q, X):
    """Inner products of every query row with every store row: float64 [nq, n]."""
    Q = np.asarray(Q, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    return Q @ X.T


def dense_topk(Q, X, k):
    """Exact top-k store rows per query: (scores float64 [nq, k], idx int64 [nq, k])."""
    return rank_topk(dense_scores(Q, X), k)
