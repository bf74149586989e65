"""Candidate screening for top-k parity at full workload sizes (test infrastructure only).

At the full sizes the fp64 CPU oracle cannot score a whole store for one query in reasonable
time (500,000 to 10,000,000 documents).  A parity check there works in two steps:

  1. Screen.  Plain torch scores one query against every document on the GPU in float64: the
     bf16 / fp16 inputs are widened exactly, their products are exact in float64, and the sums
     carry a relative error of at most n * 2^-53 (n <= 4096 terms), i.e. well below 1e-9 for
     unit-norm tokens.  This shares no code with the HIP library and is used only to choose
     candidates.
  2. Check.  The oracle scores the M screened candidates (plus every index the GPU returned)
     one by one.  If the best screened score outside the candidate set, plus the screening error
     bound, lies below the oracle's k-th candidate score minus the parity tolerance, no document
     outside the set can belong to the top-k or to its tolerance band; the candidate set then
     decides the top-k exactly, and the ordinary top-k rules apply to it.
"""

import numpy as np
import torch

SCREEN_ABS_ERR = 1e-9  # bound on |float64 screen - exact| for the unit-norm workloads here


def maxsim_row_f64(Qq, D, off, chunk_tokens=1 << 22):
    """float64 MaxSim scores of one query (Qq bf16 [lq, dim], on the GPU) against every document
    of the CSR store (D bf16 [n_tok, dim], off int64 [n_docs + 1]): [n_docs] on the GPU."""
    dev = D.device
    n_docs = off.numel() - 1
    n_tok = D.shape[0]
    lens = off[1:] - off[:-1]
    doc_of_tok = torch.repeat_interleave(torch.arange(n_docs, device=dev), lens)
    q = Qq.to(torch.float64)
    best = torch.full((n_docs, q.shape[0]), float("-inf"), dtype=torch.float64, device=dev)
    for t0 in range(0, n_tok, chunk_tokens):
        t1 = min(n_tok, t0 + chunk_tokens)
        sims = D[t0:t1].to(torch.float64) @ q.T           # [chunk, lq]
        best.index_reduce_(0, doc_of_tok[t0:t1], sims, "amax", include_self=True)
    return best.sum(dim=1)


def dense_row_f64(q, X, chunk_rows=1 << 17):
    """float64 inner products of one query (fp16 [dim]) with every row of X (fp16 [n, dim])."""
    q64 = q.to(torch.float64)
    out = torch.empty(X.shape[0], dtype=torch.float64, device=X.device)
    for r0 in range(0, X.shape[0], chunk_rows):
        r1 = min(X.shape[0], r0 + chunk_rows)
        out[r0:r1] = X[r0:r1].to(torch.float64) @ q64
    return out


def candidates(screen_row, gpu_idx, m):
    """The m best screened indices (ties by lower index) plus the GPU's returned indices, and the
    best screened score outside that set (-inf when the set is everything)."""
    s = screen_row
    n = s.numel()
    m = min(m, n)
    order = torch.argsort(-s, stable=True)  # descending, lower index first among ties
    cand = torch.unique(torch.cat([order[:m], torch.as_tensor(gpu_idx, device=s.device)]))
    mask = torch.ones(n, dtype=torch.bool, device=s.device)
    mask[cand] = False
    outside = float(s[mask].max()) if bool(mask.any()) else float("-inf")
    return cand.cpu().numpy(), outside


def virtual_row(n, cand, oracle_scores, floor):
    """An n-entry oracle row holding the oracle's scores at `cand` and `floor` elsewhere (every
    non-candidate is proven to lie below the k-th score minus the tolerance, and `floor` is below
    all of them), for the top-k rules of tests/topk_check.py."""
    row = np.full(n, floor, dtype=np.float64)
    row[cand] = oracle_scores
    return row
