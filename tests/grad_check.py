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
document of tiny softmax weight thus widens the bound by a tiny amount.  Every row must then
satisfy

  * oracle row exactly zero and no allowance: the GPU row is exactly zero;
  * oracle row norm <= 1e-30 (terms that underflow fp32, e.g. softmax weights of exp(-190) at a
    logit scale of 50): the GPU row norm is <= 1e-30 + allowance;
  * otherwise ||gpu_row - oracle_row|| <= 2e-3 * ||oracle_row|| + allowance.
"""

import numpy as np

NEAR_TIE = 1e-5
UNDERFLOW = 1e-30


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


def check_rows(g, o, allow, what, rel=2e-3):
    """Per-row check of a gradient (rows on the last axis) against the oracle's.

    allow: per-row allowance (the leading axes), from near_tie_allowance.  Returns the fraction
    of rows that carry a non-zero allowance.
    """
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    gr = g.reshape(-1, g.shape[-1])
    orr = o.reshape(-1, o.shape[-1])
    al = np.asarray(allow, dtype=np.float64).reshape(-1)
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
                             f"(+ near-tie allowance); worst row {worst}: error "
                             f"{err[worst]:.3g}, oracle norm {on[worst]:.3g}, allowance "
                             f"{al[worst]:.3g}")
    return float((al > 0).mean())
