"""Pins of the fp64 oracle's pooled contrastive loss L_C and the total ColTrast loss.

Each pin comes from outside the oracle's own formula (so a dropped term, a sign error, a wrong
normalisation or a transposed operand fails at least one):
  * central finite differences of L_C and of the total loss, for every coordinate of Q and D;
  * closed forms: documents whose pooled embeddings all point the same way give ln(n_docs) and
    dL/dC = (1/B)(1/n - onehot); a hand-built two-document case in 2-D, whose cosines are the
    cosines of known angles, gives the softplus of their difference over tau;
  * the tau -> infinity limit (every logit equal);
  * invariants: scaling a document's or a query's tokens by c > 0, permuting a document's tokens
    or appending its mean token leave L_C unchanged; L_C depends on each pooled vector only
    through its direction, so sum_j D[j] . dD[j] = 0 per document and sum_i Q[q,i] . dQ[q,i] = 0
    per query (Euler's theorem for degree-0 functions); sum_d dL/dC[q, d] = 0.
"""

import itertools
import math

import numpy as np

import oracle


def _csr(rng, lens, dim):
    off = np.zeros(len(lens) + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    return rng.standard_normal((int(off[-1]), dim)), off


def test_contrastive_gradients_match_central_finite_differences():
    rng = np.random.default_rng(31)
    dim, lq = 4, 3
    D, off = _csr(rng, [3, 2, 4, 1], dim)
    Q = rng.standard_normal((3, lq, dim))
    pos = [2, 0, 3]
    tau = 0.3
    r = oracle.contrastive_loss(Q, D, off, pos, tau)
    h = 1e-6

    def loss_at(Qx, Dx):
        return oracle.contrastive_loss(Qx, Dx, off, pos, tau)["loss"]

    for idx in itertools.product(range(3), range(lq), range(dim)):
        Qp, Qm = Q.copy(), Q.copy()
        Qp[idx] += h
        Qm[idx] -= h
        fd = (loss_at(Qp, D) - loss_at(Qm, D)) / (2 * h)
        assert abs(fd - r["dQ"][idx]) <= 1e-6 * max(1.0, abs(fd)), idx
    for idx in itertools.product(range(D.shape[0]), range(dim)):
        Dp, Dm = D.copy(), D.copy()
        Dp[idx] += h
        Dm[idx] -= h
        fd = (loss_at(Q, Dp) - loss_at(Q, Dm)) / (2 * h)
        assert abs(fd - r["dD"][idx]) <= 1e-6 * max(1.0, abs(fd)), idx


def test_total_loss_gradients_match_central_finite_differences():
    rng = np.random.default_rng(32)
    dim, lq = 5, 2
    D, off = _csr(rng, [4, 3, 5], dim)
    Q = rng.standard_normal((2, lq, dim))
    pos = [1, 2]
    s, tau = 1.3, 0.4
    # stay away from MaxSim argmax switches (the L_LI half is piecewise smooth)
    for d in range(3):
        sim = np.einsum("qik,jk->qij", Q, D[off[d]:off[d + 1]])
        top2 = np.sort(sim, axis=2)[:, :, -2:]
        assert np.all(top2[:, :, 1] - top2[:, :, 0] > 1e-3)
    r = oracle.coltrast_total_loss(Q, D, off, pos, s, tau)
    h = 1e-6

    def loss_at(Qx, Dx):
        return oracle.coltrast_total_loss(Qx, Dx, off, pos, s, tau)["loss"]

    for idx in itertools.product(range(2), range(lq), range(dim)):
        Qp, Qm = Q.copy(), Q.copy()
        Qp[idx] += h
        Qm[idx] -= h
        fd = (loss_at(Qp, D) - loss_at(Qm, D)) / (2 * h)
        assert abs(fd - r["dQ"][idx]) <= 1e-6 * max(1.0, abs(fd)), idx
    for idx in itertools.product(range(D.shape[0]), range(dim)):
        Dp, Dm = D.copy(), D.copy()
        Dp[idx] += h
        Dm[idx] -= h
        fd = (loss_at(Q, Dp) - loss_at(Q, Dm)) / (2 * h)
        assert abs(fd - r["dD"][idx]) <= 1e-6 * max(1.0, abs(fd)), idx
    # the halves are the separately pinned losses
    assert abs(r["loss_li"] - oracle.coltrast_li_loss(Q, D, off, pos, s)["loss"]) < 1e-15
    assert abs(r["loss"] - (r["loss_li"] + r["loss_c"]) / 2) < 1e-15


def test_contrastive_equal_directions_give_log_n():
    # every document's tokens are positive multiples of one vector: all cosines are equal
    rng = np.random.default_rng(33)
    dim, n = 6, 5
    v = rng.standard_normal(dim)
    lens = [2, 1, 3, 2, 4]
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    D = np.concatenate([np.outer(rng.uniform(0.5, 2.0, L), v) for L in lens])
    Q = rng.standard_normal((3, 4, dim))
    pos = [0, 4, 2]
    r = oracle.contrastive_loss(Q, D, off, pos, 0.05)
    assert abs(r["loss"] - math.log(n)) < 1e-12
    want = np.full((3, n), 1.0 / n)
    want[np.arange(3), pos] -= 1.0
    assert np.allclose(r["dC"], want / 3, atol=1e-14)


def test_contrastive_two_documents_is_softplus_of_cosine_gap():
    # 2-D: the query pools to (1, 0); the positive to (cos a, sin a) times 2, the negative to
    # (cos b, sin b) times 0.5 (each as the mean of two tokens); cosines are cos a and cos b
    a, b, tau = 0.4, 1.1, 0.2
    Q = np.array([[[1.5, 0.3], [0.5, -0.3]]])             # mean (1, 0)
    pos_pool = 2.0 * np.array([math.cos(a), math.sin(a)])
    neg_pool = 0.5 * np.array([math.cos(b), math.sin(b)])
    dev = np.array([0.25, -0.5])
    D = np.stack([pos_pool + dev, pos_pool - dev, neg_pool - dev, neg_pool + dev])
    off = np.array([0, 2, 4])
    r = oracle.contrastive_loss(Q, D, off, [0], tau)
    want = math.log1p(math.exp((math.cos(b) - math.cos(a)) / tau))
    assert abs(r["loss"] - want) < 1e-13


def test_contrastive_large_temperature_limit():
    rng = np.random.default_rng(34)
    D, off = _csr(rng, [3, 3, 2, 5], 7)
    Q = rng.standard_normal((2, 3, 7))
    r = oracle.contrastive_loss(Q, D, off, [1, 3], 1e9)
    assert abs(r["loss"] - math.log(4)) < 1e-8


def test_contrastive_invariants():
    rng = np.random.default_rng(35)
    dim = 6
    D, off = _csr(rng, [4, 2, 5], dim)
    Q = rng.standard_normal((2, 3, dim))
    pos = [2, 1]
    tau = 0.1
    r = oracle.contrastive_loss(Q, D, off, pos, tau)
    # scaling one document's tokens, and one query's tokens, by c > 0
    D2 = D.copy()
    D2[off[1]:off[2]] *= 3.7
    Q2 = Q.copy()
    Q2[0] *= 0.2
    assert abs(oracle.contrastive_loss(Q2, D2, off, pos, tau)["loss"] - r["loss"]) < 1e-12
    # permuting a document's tokens
    D3 = D.copy()
    D3[off[2]:off[3]] = D[off[2]:off[3]][::-1]
    assert abs(oracle.contrastive_loss(Q, D3, off, pos, tau)["loss"] - r["loss"]) < 1e-12
    # appending the document's own mean token leaves its mean unchanged
    m0 = D[off[0]:off[1]].mean(axis=0)
    D4 = np.concatenate([D[:off[1]], m0[None], D[off[1]:]])
    off4 = off.copy()
    off4[1:] += 1
    assert abs(oracle.contrastive_loss(Q, D4, off4, pos, tau)["loss"] - r["loss"]) < 1e-12
    # Euler: the loss is of degree 0 in each document's and each query's tokens
    for d in range(3):
        sl = slice(off[d], off[d + 1])
        assert abs(np.sum(D[sl] * r["dD"][sl])) < 1e-12
    for q in range(2):
        assert abs(np.sum(Q[q] * r["dQ"][q])) < 1e-12
    assert np.allclose(r["dC"].sum(axis=1), 0.0, atol=1e-15)
