"""ColTrast's pooled contrastive loss L_C and the total loss L = (L_LI + L_C) / 2, fp64 (test
infrastructure only).

The paper trains its encoder with L = (L_LI + L_C) / 2 (Sec. 3.2.1, paragraph "Embedding
performance: loss function"): L_LI is the MaxSim loss (oracle/loss.py) and L_C the contrastive
loss of SimCSE computed on pooled embeddings, each local query compared with min(N, W) gathered
samples.  It ranks by the cosine of pooled embeddings (same section, "Similarity metric").
Readings taken here where the paper is silent:
  * pooling is the mean of a sequence's token embeddings (queries over their lq tokens,
    documents over their CSR rows);
  * the similarity is the cosine of the pooled embeddings, divided by a temperature tau;
  * on one GPU the gathered set is the local batch: every in-batch document is compared (the
    paper's "ND" variant, no all-gather), with the same positives as L_LI;
  * the loss is the mean over the queries.

Steps, in order:
  1. P_q = mean_i Q[q, i, :];  P_d = mean_{j in d} D[j, :];
  2. U = P / |P| (rows);  C[q, d] = <U_q, U_d> / tau;
  3. L_C = (1/B) sum_q (logsumexp_d C[q, d] - C[q, pos[q]]);
  4. dL_C/dC = (1/B) (softmax_d C[q, :] - onehot(pos[q])), the positive's entry taken as minus the sum
     of the other probabilities (the same number, without cancellation in float64);
  5. dL_C/dU_q = (1/tau) sum_d dC[q, d] U_d;  dL_C/dU_d = (1/tau) sum_q dC[q, d] U_q;
  6. dL_C/dP = (dU - U <U, dU>) / |P|   (the normalisation's Jacobian);
  7. dL_C/dQ[q, i] = dL_C/dP_q / lq;  dL_C/dD[j] = dL_C/dP_d / L_d for every token j of d.
"""

import numpy as np

from .loss import coltrast_li_loss


def pooled_means(Q, D, offsets):
    """Mean-pooled query and document embeddings: (P_q [nq, dim], P_d [n_docs, dim])."""
    Q = np.asarray(Q, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    off = np.asarray(offsets, dtype=np.int64)
    Pq = Q.mean(axis=1)
    Pd = np.stack([D[off[d]:off[d + 1]].mean(axis=0) for d in range(off.size - 1)])
    return Pq, Pd


def contrastive_loss(Q, D, offsets, pos, tau):
    """Returns dict(loss, C, dC, dQ, dD) in float64 (C: the cosine logits over tau)."""
    Q = np.asarray(Q, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    off = np.asarray(offsets, dtype=np.int64)
    pos = np.asarray(pos, dtype=np.int64)
    nq, lq, _ = Q.shape
    n_docs = off.size - 1
    if pos.shape != (nq,) or np.any(pos < 0) or np.any(pos >= n_docs):
        raise ValueError("pos must hold one in-range positive document per query")

    # 1-2
    Pq, Pd = pooled_means(Q, D, off)
    nPq = np.linalg.norm(Pq, axis=1)
    nPd = np.linalg.norm(Pd, axis=1)
    Uq = Pq / nPq[:, None]
    Ud = Pd / nPd[:, None]
    C = (Uq @ Ud.T) / tau

    # 3
    M = C.max(axis=1)
    lse = M + np.log(np.exp(C - M[:, None]).sum(axis=1))
    rows = np.arange(nq)
    loss = (lse - C[rows, pos]).sum() / nq

    # 4 (the positive's softmax - 1 as minus the other probabilities: the same number, without
    # the cancellation of 1 - p in float64 when p is within ~1e-13 of 1)
    dC = np.exp(C - lse[:, None])
    for q in range(nq):
        dC[q, pos[q]] = -np.delete(dC[q], pos[q]).sum()
    dC /= nq

    # 5-6
    dUq = (dC @ Ud) / tau
    dUd = (dC.T @ Uq) / tau
    dPq = (dUq - Uq * np.sum(Uq * dUq, axis=1, keepdims=True)) / nPq[:, None]
    dPd = (dUd - Ud * np.sum(Ud * dUd, axis=1, keepdims=True)) / nPd[:, None]

    # 7
    dQ = np.repeat(dPq[:, None, :] / lq, lq, axis=1)
    dD = np.zeros_like(D)
    for d in range(n_docs):
        dD[off[d]:off[d + 1]] = dPd[d] / (off[d + 1] - off[d])
    return {"loss": loss, "C": C, "dC": dC, "dQ": dQ, "dD": dD}


def coltrast_total_loss(Q, D, offsets, pos, logit_scale, tau):
    """L = (L_LI + L_C) / 2 and its gradients.  Returns dict(loss, loss_li, loss_c, dQ, dD)."""
    li = coltrast_li_loss(Q, D, offsets, pos, logit_scale)
    c = contrastive_loss(Q, D, offsets, pos, tau)
    return {
        "loss": (li["loss"] + c["loss"]) / 2.0,
        "loss_li": li["loss"],
        "loss_c": c["loss"],
        "dQ": (li["dQ"] + c["dQ"]) / 2.0,
        "dD": (li["dD"] + c["dD"]) / 2.0,
    }
