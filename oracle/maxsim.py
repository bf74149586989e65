"""Late-interaction (MaxSim) similarity and exact top-k ranking, fp64 (test infrastructure only).

Definitions followed
  * Late interaction, the ColBERT mechanism the paper builds ColTrast on (Sec. 2.2, "Neural
    Information Retrieval and Metric Learning"; Sec. 3.2.1 paragraph "Similarity metric" and
    Fig. 3B): every query token is compared with every token of the document chunk, each query
    token keeps its best-matching (largest inner product) document token, and the per-token
    maxima are summed over the query tokens:

        S[q, d] = sum_i  max_{j in doc d}  < Q[q, i, :], D[j, :] >

    The similarity is the raw inner product; for L2-normalised tokens it is the cosine.
  * Retrieval returns the IDs of the nearest neighbours of a query in the chunk store (Sec. 2.3,
    "Retrieval-Augmented Generation"); documents are ranked by score, and equal scores are ranked
    by the lower document index.

Documents are stored CSR: the tokens of document d are rows offsets[d] .. offsets[d+1]-1 of D.
"""

import numpy as np


def _check_csr(D, offsets):
    off = np.asarray(offsets, dtype=np.int64)
    if off.ndim != 1 or off.size < 1 or off[0] != 0 or off[-1] != D.shape[0]:
        raise ValueError("offsets must start at 0 and end at the number of token rows")
    if np.any(np.diff(off) < 1):
        raise ValueError("every document needs at least one token and offsets must increase")
    return off


def _doc_similarities(Q, D, off, d):
    """<Q[q, i], D[j]> for every query token (q, i) and every token j of document d: [nq, lq, Ld]."""
    nq, lq, dim = Q.shape
    Dd = D[off[d]:off[d + 1]]                        # [Ld, dim]
    sim = Q.reshape(nq * lq, dim) @ Dd.T             # plain matrix product, float64
    return sim.reshape(nq, lq, Dd.shape[0])


def maxsim_scores(Q, D, offsets):
    """MaxSim scores S[q, d] (float64 [nq, n_docs]).

    Q: float64 [nq, lq, dim] query token embeddings.
    D: float64 [n_tok, dim] document token embeddings, CSR by `offsets` (int64 [n_docs + 1]).
    For each document: the full query-token x document-token inner-product table, its maximum
    over the document's tokens, then the sum over the query tokens (Sec. 2.2, Fig. 3B).
    """
    Q = np.asarray(Q, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    off = _check_csr(D, offsets)
    n_docs = off.size - 1
    S = np.empty((Q.shape[0], n_docs), dtype=np.float64)
    for d in range(n_docs):
        sim = _doc_similarities(Q, D, off, d)        # [nq, lq, Ld]
        per_token_max = sim.max(axis=2)              # [nq, lq]
        S[:, d] = per_token_max.sum(axis=1)
    return S


def maxsim_argmax(Q, D, offsets):
    """Index (within its document) of the document token attaining each query token's maximum.

    Returns (S, A): S as in `maxsim_scores`; A int64 [nq, lq, n_docs] with A[q, i, d] = the
    LOWEST local token index j (0 <= j < Ld) attaining max_j <Q[q, i], D[off[d] + j]>.  The
    lowest index is the reading taken here for ties (the paper does not discuss them); it decides
    which document token receives the subgradient of the max.
    """
    Q = np.asarray(Q, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    off = _check_csr(D, offsets)
    nq, lq, _ = Q.shape
    n_docs = off.size - 1
    S = np.empty((nq, n_docs), dtype=np.float64)
    A = np.empty((nq, lq, n_docs), dtype=np.int64)
    for d in range(n_docs):
        sim = _doc_similarities(Q, D, off, d)
        A[:, :, d] = np.argmax(sim, axis=2)          # numpy returns the first (lowest) maximiser
        S[:, d] = sim.max(axis=2).sum(axis=1)
    return S, A


def rank_topk(S, k):
    """Exact top-k of each row of S by (score descending, index ascending).

    Returns (scores float64 [nq, k], idx int64 [nq, k]).  A stable ordering on the key
    (-score, index) is a full sort of each row; the first k entries are the k nearest neighbours
    in the order a retriever returns them (Sec. 2.3).
    """
    S = np.asarray(S, dtype=np.float64)
    nq, n = S.shape
    if not 1 <= k <= n:
        raise ValueError("k must satisfy 1 <= k <= number of candidates")
    out_s = np.empty((nq, k), dtype=np.float64)
    out_i = np.empty((nq, k), dtype=np.int64)
    idx = np.arange(n, dtype=np.int64)
    for q in range(nq):
        # -0.0 and +0.0 are the same score: the negation below maps both to 0.0 for lexsort,
        # whose comparisons treat them as equal.
        order = np.lexsort((idx, -S[q]))             # primary key: -score; secondary: index
        out_i[q] = order[:k]
        out_s[q] = S[q, order[:k]]
    return out_s, out_i
