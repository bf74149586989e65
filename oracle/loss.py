"""ColTrast late-interaction loss L_LI and its gradients, fp64 (test infrastructure only).

The paper trains its encoder with L = (L_LI + L_C) / 2 (Sec. 3.2.1, paragraph "Embedding
performance: loss function").  L_LI is the MaxSim loss of ColBERT: a softmax cross-entropy over
MaxSim scores, applied to the local rank's batch only.  Readings taken here where the paper is
silent:
  * every query of the batch is scored against every document of the batch (in-batch InfoNCE);
    query q's positive is document pos[q], every other document is a negative;
  * the logits are s * S[q, d] with a caller-given scale s (the inverse temperature);
  * the loss is the mean over the queries of the batch.

Steps, in order:
  1. S[q, d] and the argmax table A[q, i, d] (lowest maximising token) from `maxsim_argmax`;
  2. logits l = s * S;
  3. LSE_q = M_q + log sum_d exp(l[q, d] - M_q) with M_q = max_d l[q, d];
  4. loss = (1/B) sum_q (LSE_q - l[q, pos[q]]);
  5. G[q, d] = dloss/dS[q, d] = (s/B) * (exp(l[q, d] - LSE_q) - [d == pos[q]]); for the positive,
     exp(l - LSE) - 1 is evaluated as minus the sum of the other documents' probabilities (the
     probabilities sum to one, so this is the same number): when the positive's probability is
     within ~1e-13 of 1, as at a logit scale of 50, 1 - p rounds to 0 in float64 while the sum of
     the others keeps every digit;
  6. dQ[q, i, :] = sum_d G[q, d] * D[off[d] + A[q, i, d], :]           (chain rule through the max);
  7. dD[j, :]    = sum over (q, i, d) with off[d] + A[q, i, d] == j of G[q, d] * Q[q, i, :].
"""

import numpy as np

from .maxsim import maxsim_argmax


def coltrast_li_loss(Q, D, offsets, pos, logit_scale):
    """Returns dict(loss, S, G, dQ, dD, A), all float64 except A (int64 local token indices)."""
    Q = np.asarray(Q, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    off = np.asarray(offsets, dtype=np.int64)
    pos = np.asarray(pos, dtype=np.int64)
    s = float(logit_scale)
    nq, lq, dim = Q.shape
    n_docs = off.size - 1
    if pos.shape != (nq,) or np.any(pos < 0) or np.any(pos >= n_docs):
        raise ValueError("pos must hold one in-range positive document per query")

    # 1-2
    S, A = maxsim_argmax(Q, D, off)
    logits = s * S

    # 3
    M = logits.max(axis=1)
    lse = M + np.log(np.exp(logits - M[:, None]).sum(axis=1))

    # 4
    rows = np.arange(nq)
    loss = (lse - logits[rows, pos]).sum() / nq

    # 5
    G = np.exp(logits - lse[:, None])
    for q in range(nq):
        G[q, pos[q]] = -np.delete(G[q], pos[q]).sum()   # p_pos - 1 = -(sum of the others)
    G *= s / nq

    # 6: for each (q, d), every query token i picks up G[q, d] times its maximising doc token
    dQ = np.zeros_like(Q)
    for q in range(nq):
        for d in range(n_docs):
            dQ[q] += G[q, d] * D[off[d] + A[q, :, d]]          # [lq, dim] gathered rows

    # 7: the transpose: each maximising doc token picks up G[q, d] times the query token.
    # np.add.at accumulates repeated row indices (two query tokens sharing one maximiser).
    dD = np.zeros_like(D)
    for q in range(nq):
        for d in range(n_docs):
            np.add.at(dD, off[d] + A[q, :, d], G[q, d] * Q[q])

    return {"loss": loss, "S": S, "G": G, "dQ": dQ, "dD": dD, "A": A}
