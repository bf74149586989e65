"""Per-row verification of the loss gradients dQ and dD against the oracle's.

The gradient of the MaxSim score reaches one document token per (query token, document): the
token attaining the maximum (lowest index on ties).  The GPU decides that maximum on fp32 dot
products (and on argmax keys that drop the 4 low mantissa bits), the oracle on fp64 ones; when
two tokens of a document come within 1e-5 of each other for a query token (a "near-tie"), both
choices are valid and the subgradient may legitimately go to either.  Such a choice moves
G[q, d] * Q[q, i] from one dD row to another and changes the dQ row of (q, i) by
G[q, d] * (D[j'] - D[j]).  Rather than excusing whole rows, the verification widens each row's bound
by exactly what those alternative choices can move:

  allow_dQ[q, i] = sum over near-ties (q, i, d) of |G[q, d]| * max_{j' in window} |D[j'] - D[j]|
  allow_dD[j']   = sum over near-ties (q, i, d) whose window holds j' of |G[q, d]| * |Q[q, i]|

(j the oracle's token, the window the tokens within 1e-5 of the maximum).  A near-tie in a
document of tiny softmax weight thus widens the bound by a tiny amount.  A second allowance covers rows whose terms cancel (conditioning_allowance).  Each row is a sum
of weighted rows -- dQ[q, i] = sum_d G[q, d] D[token], dD[j] = sum over the entries that selected
j of G[q, d] Q[q, i] -- and the GPU forms G in fp32 from its own fp32 scores.  When two documents
hold the same selected token with opposite weights (the positive and a negative that copies the
query's token), the row is far smaller than its terms, and 2e-3 of its norm lies below what the
fp32 inputs of the sum resolve.  Forward error analysis bounds what the GPU can legitimately
differ by: a weight's relative error is at most tau_q = 4 |scale| max_d |dS[q, d]| + 2^-20 (the
logits' deviation enters the term's own logit and the log-sum-exp; doubled for margin; the floor
covers fp32 rounding of the logits and of exp), and an fp32 sum of n products adds at most
(n + 1) 2^-24 of the sum of their magnitudes:

  cond_dQ[q, i] = (tau_q + (n_docs + 1) 2^-24) * sum_d |G[q, d]| * ||D[token of (q, i, d)]||
  cond_dD[j]    = sum over entries e = (q, i) selecting j of (tau_q + (c_j + 1) 2^-24)
                  * |G[q, d]| * ||Q[q, i]||          (c_j: the number of entries selecting j)

with dS the GPU's scores minus the oracle's.  For a well-conditioned row this is ~1e-6 of its
norm, far inside the 2e-3, so it excuses nothing there; a dropped or misplaced term of weight w
still fails whenever w exceeds 2e-3 of the row plus that bound.  Every row must then satisfy

  * oracle row exactly zero and no allowance (no term reaches the row: an unselected token, or
    weights that are all exactly zero): the GPU row is exactly zero.  With terms, an exact zero
    in the oracle can be fp64 absorption (a term of 1e-35 added to two cancelling terms of 1, in
    that order, is lost), so such a row falls under the next rule;
  * oracle row norm <= 1e-30 (terms that underflow fp32, e.g. softmax weights of exp(-190) at a
    logit scale of 50): the GPU row norm is <= 1e-30 + allowances;
  * otherwise ||gpu_row - oracle_row|| <= 2e-3 * ||oracle_row|| + allowances.
"""

import numpy as np

NEAR_TIE = 1e-5
UNDERFLOW = 1e-30
U32 = 2.0 ** -24


def near_tie_allowance(Q, D, offsets, G, eps=NEAR_TIE):
    """Per-row allowances of dQ and dD for argmax near-ties.

    Q float64 [nq, lq, dim], D float64 [n_tok, dim] (exact values of the bf16 inputs), offsets
    int64 [n_docs + 1], G float64 [nq, n_docs] (dL/dS of the loss being checked).  Returns
    (allow_dq [nq, lq], allow_dd [n_tok], entries), entries being the number of (q, i, d) whose
    two best tokens lie within eps.
    """
    Q = np.asarray(Q, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    off = np.asarray(offsets, dtype=np.int64)
    nq, lq, dim = Q.shape
    Qf = Q.reshape(nq * lq, dim)
    qn = np.linalg.norm(Qf, axis=1)
    allow_dq = np.zeros(nq * lq)
    allow_dd = np.zeros(D.shape[0])
    entries = 0
    for d in range(off.size - 1):
        a, b = int(off[d]), int(off[d + 1])
        if b - a < 2:
            continue
        sim = Qf @ D[a:b].T                               # [nq*lq, Ld]
        top = sim.max(axis=1, keepdims=True)
        within = sim >= top - eps                         # the maximum and its near-ties
        for e in np.flatnonzero(within.sum(axis=1) >= 2):
            entries += 1
            w = np.abs(G[e // lq, d])
            toks = np.flatnonzero(within[e])              # toks[0] is the oracle's (lowest)
            move = np.linalg.norm(D[a + toks] - D[a + toks[0]], axis=1).max()
            allow_dq[e] += w * move
            allow_dd[a + toks] += w * qn[e]
    return allow_dq.reshape(nq, lq), allow_dd, entries


def conditioning_allowance(Q, D, offsets, G, A, dS, scale):
    """Per-row allowances of dQ and dD for cancellation among their terms (module docstring).

    Q float64 [nq, lq, dim], D float64 [n_tok, dim], offsets int64 [n_docs + 1], G float64
    [nq, n_docs] (the oracle's dL/dS), A int64 [nq, lq, n_docs] (the oracle's argmax, local
    token indices), dS [nq, n_docs] (GPU scores minus oracle scores), scale the logit scale.
    Returns (cond_dq [nq, lq], cond_dd [n_tok]).
    """
    Q = np.asarray(Q, dtype=np.float64)
    D = np.asarray(D, dtype=np.float64)
    G = np.abs(np.asarray(G, dtype=np.float64))
    off = np.asarray(offsets, dtype=np.int64)
    nq, lq, _ = Q.shape
    n_docs = off.size - 1
    tau = 4.0 * abs(scale) * np.max(np.abs(np.asarray(dS, dtype=np.float64)), axis=1) + 2.0 ** -20
    rows = off[:-1][None, None, :] + np.asarray(A, dtype=np.int64)      # [nq, lq, n_docs]
    dn = np.linalg.norm(D, axis=1)
    qn = np.linalg.norm(Q, axis=2)                                      # [nq, lq]
    cond_dq = (tau[:, None] + (n_docs + 1) * U32) * np.sum(G[:, None, :] * dn[rows], axis=2)
    cnt = np.bincount(rows.ravel(), minlength=D.shape[0])
    w = G[:, None, :] * qn[:, :, None]                                  # |G[q, d]| ||Q[q, i]||
    per = (tau[:, None, None] + (cnt[rows] + 1) * U32) * w
    cond_dd = np.zeros(D.shape[0])
    np.add.at(cond_dd, rows.ravel(), per.ravel())
    return cond_dq, cond_dd


def check_rows(g, o, allow, what, rel=2e-3, cond=None):
    """Per-row check of a gradient (rows on the last axis) against the oracle's.

    allow: per-row near-tie allowance (the leading axes), from near_tie_allowance; cond: optional
    per-row conditioning allowance, from conditioning_allowance.  Returns the fraction of rows
    that carry a non-zero near-tie allowance.
    """
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    gr = g.reshape(-1, g.shape[-1])
    orr = o.reshape(-1, o.shape[-1])
    nt = np.asarray(allow, dtype=np.float64).reshape(-1)
    assert nt.size == gr.shape[0]
    al = nt if cond is None else nt + np.asarray(cond, dtype=np.float64).reshape(-1)
    assert al.size == gr.shape[0]
    on = np.linalg.norm(orr, axis=1)
    err = np.linalg.norm(gr - orr, axis=1)
    zero = ~np.any(orr != 0, axis=1) & (al == 0)
    nz = np.any(gr[zero] != 0, axis=1)
    assert not nz.any(), f"{what}: {int(nz.sum())} rows non-zero where the oracle's are zero"
    tiny = ~zero & (on <= UNDERFLOW)
    gn = np.linalg.norm(gr, axis=1)
    assert np.all(gn[tiny] <= UNDERFLOW + al[tiny]), \
        f"{what}: a row of norm <= 1e-30 in the oracle is larger on the GPU"
    big = on > UNDERFLOW
    lim = rel * on + al
    bad = big & (err > lim)
    if bad.any():
        r = np.flatnonzero(bad)
        worst = r[np.argmax(err[r] / lim[r])]
        raise AssertionError(f"{what}: {r.size} of {int(big.sum())} rows outside rel L2 {rel} "
                             f"(+ allowances); worst row {worst}: error "
                             f"{err[worst]:.3g}, oracle norm {on[worst]:.3g}, allowance "
                             f"{al[worst]:.3g}")
    return float((nt > 0).mean())
