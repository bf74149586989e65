"""Semantic chunking boundaries and retrieval metrics, fp64 (test infrastructure only).

Semantic chunking (Sec. 3.2.2, "ColTrast Finetuning Dataset"): the sentences of a paper are
encoded and walked in order; a segment keeps growing while the cosine similarity of each
sentence with the one before it stays above a fixed threshold.  Readings taken here where the
paper is silent:
  * "above" is strict: sentence t joins the segment of sentence t - 1 iff cos > threshold;
  * segments never cross papers: the first sentence of every paper opens a segment;
  * a sentence of zero norm has an undefined cosine (NaN), which is not above any threshold,
    so it opens a segment (and so does the sentence after it);
  * segments are numbered 0, 1, ... in sentence order over the whole input.

Steps, in order:
  1. cos[t] = <E[t-1], E[t]> / (|E[t-1]| |E[t]|) for every t that is not the first sentence of
     its paper (NaN for first sentences);
  2. boundary[t] = t is first in its paper, or not (cos[t] > threshold);
  3. seg[t] = (number of boundaries at or before t) - 1.

Retrieval metrics (Sec. 4.2, "ColTrast Retrieval Evaluation"), one positive document per query:
  * P@k = N_rel / N_ret with N_ret = k, N_rel = 1 if the positive is among the k retrieved and 0
    otherwise, averaged over the queries (reading: the paper states P for one ranking);
  * MRR@k = (1 / N_q) sum_q 1 / rank_q, a term being 0 when the positive is ranked beyond k.
"""

import numpy as np


def paper_starts(n, paper_off):
    """Boolean [n]: sentence t is the first sentence of its paper (None: one paper)."""
    first = np.zeros(n, dtype=bool)
    if n == 0:
        return first
    if paper_off is None:
        first[0] = True
        return first
    off = np.asarray(paper_off, dtype=np.int64)
    starts = off[:-1][off[:-1] < off[1:]]  # papers with at least one sentence
    first[starts] = True
    return first


def chunk_cosines(E, paper_off=None):
    """Step 1: float64 [n], NaN at the first sentence of every paper."""
    E = np.asarray(E, dtype=np.float64)
    n = E.shape[0]
    cos = np.full(n, np.nan)
    first = paper_starts(n, paper_off)
    for t in range(1, n):
        if first[t]:
            continue
        a, b = E[t - 1], E[t]
        na, nb = np.sqrt(np.dot(a, a)), np.sqrt(np.dot(b, b))
        with np.errstate(invalid="ignore", divide="ignore"):
            cos[t] = np.dot(a, b) / (na * nb)
    return cos


def semantic_segments(E, paper_off, threshold):
    """Steps 1-3: (cos float64 [n], seg int64 [n], n_segments)."""
    E = np.asarray(E, dtype=np.float64)
    n = E.shape[0]
    cos = chunk_cosines(E, paper_off)
    first = paper_starts(n, paper_off)
    with np.errstate(invalid="ignore"):
        joins = cos > threshold  # NaN compares false
    boundary = first | ~joins
    seg = np.cumsum(boundary.astype(np.int64)) - 1
    return cos, seg, int(boundary.sum())


def retrieval_ranks(topk_idx, positive):
    """1-based rank of each query's positive among its retrieved indices, 0 when absent."""
    idx = np.asarray(topk_idx, dtype=np.int64)
    pos = np.asarray(positive, dtype=np.int64)
    ranks = np.zeros(idx.shape[0], dtype=np.int64)
    for q in range(idx.shape[0]):
        hit = np.nonzero(idx[q] == pos[q])[0]
        if hit.size:
            ranks[q] = int(hit[0]) + 1
    return ranks


def retrieval_metrics(topk_idx, positive, k):
    """(P@k, MRR@k, ranks) over the first k retrieved indices of every query."""
    idx = np.asarray(topk_idx, dtype=np.int64)[:, :k]
    ranks = retrieval_ranks(idx, positive)
    nq = idx.shape[0]
    found = ranks > 0
    p_at_k = float(np.sum(found) / k / nq)
    mrr = float(np.sum(np.where(found, 1.0 / np.maximum(ranks, 1), 0.0)) / nq)
    return p_at_k, mrr, ranks
