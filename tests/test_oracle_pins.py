"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Kinds of pin used (each function has several, so a dropped term, a sign error, a wrong index or a
transposed operand fails at least one):
  * hand-worked examples (tests/golden/hand_examples.json), derived from the definitions by hand;
  * brute force on tiny inputs by a different computation: the MaxSim score is the maximum, over
    every assignment of one document token to each query token, of the summed inner products;
  * special cases with closed forms (Lq = 1, Ld = 1, document made of the query's own unit
    tokens, all-equal scores, B = 1 with two documents = pairwise softplus);
  * invariants (token permutation / duplication, appending tokens, shift invariance of the loss,
    sum of G over documents = 0);
  * central finite differences of the loss for dQ and dD;
  * ranking by repeated extraction of the best remaining (score, lowest index).
"""

import itertools
import math

import numpy as np
import pytest

import oracle


def _ns(**kw):
    env = {"ln": math.log, "exp": math.exp}
    env.update(kw)
    return env


def _rand_unit(rng, n, dim):
    x = rng.standard_normal((n, dim))
    return x / np.linalg.norm(x, axis=1, keepdims=True)


def _rand_csr(rng, lens, dim):
    off = np.zeros(len(lens) + 1, dtype=np.int64)
    off[1:] = np.cumsum(lens)
    return rng.standard_normal((int(off[-1]), dim)), off


# ---------------------------------------------------------------- decoding

def test_decode_bf16_exact_values():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x8000, 0x4049, 0x3C00, 0x7F7F, 0x0001], np.uint16)
    v = oracle.decode_bf16(bits)
    assert v[0] == 1.0 and v[1] == -1.0 and v[2] == 0.0 and v[3] == 0.0
    assert math.copysign(1.0, v[3]) == -1.0
    assert v[4] == 3.140625                       # 0x4049 = 0 10000000 1001001 -> 1.5703125 * 2
    assert v[5] == 2.0 ** -7                      # 0x3C00 = exponent 120, mantissa 0
    assert v[6] == (2 - 2.0 ** -7) * 2.0 ** 127   # largest finite bf16
    assert v[7] == 2.0 ** -133                    # smallest bf16 subnormal


def test_decode_fp16_exact_values():
    bits = np.array([0x3C00, 0xC000, 0x0001, 0x03FF, 0x7BFF, 0x3555], np.uint16)
    v = oracle.decode_fp16(bits)
    assert v[0] == 1.0 and v[1] == -2.0
    assert v[2] == 2.0 ** -24                     # smallest subnormal
    assert v[3] == 1023 * 2.0 ** -24              # largest subnormal
    assert v[4] == 65504.0
    assert v[5] == (1 + 0x155 / 1024) * 2.0 ** -2


# ---------------------------------------------------------------- MaxSim

def test_maxsim_hand_example(golden):
    g = golden["maxsim"]
    Q, D, off = np.array(g["Q"], float), np.array(g["D"], float), np.array(g["offsets"])
    S, A = oracle.maxsim_argmax(Q, D, off)
    assert np.array_equal(S, np.array(g["S"], float))
    assert np.array_equal(A, np.array(g["argmax"]))
    assert np.array_equal(oracle.maxsim_scores(Q, D, off), S)


def test_maxsim_argmax_tie_takes_lowest_index(golden):
    g = golden["argmax_tie"]
    S, A = oracle.maxsim_argmax(np.array(g["Q"], float), np.array(g["D"], float), g["offsets"])
    assert np.array_equal(S, np.array(g["S"], float))
    assert np.array_equal(A, np.array(g["argmax"]))


@pytest.mark.parametrize("lq,lens,dim", [(1, [1, 4], 3), (2, [3, 1, 2], 4), (3, [3, 2], 2),
                                         (3, [4, 4, 1], 5)])
def test_maxsim_equals_best_assignment_brute_force(lq, lens, dim):
    # max over all maps f: query token -> doc token of sum_i <q_i, d_f(i)>; a different
    # computation from per-token maxima (they agree because the terms are independent).
    rng = np.random.default_rng(11 + lq + dim)
    Q = rng.standard_normal((2, lq, dim))
    D, off = _rand_csr(rng, lens, dim)
    S = oracle.maxsim_scores(Q, D, off)
    for q in range(2):
        for d in range(len(lens)):
            toks = D[off[d]:off[d + 1]]
            best = -math.inf
            for f in itertools.product(range(len(toks)), repeat=lq):
                tot = math.fsum(math.fsum(Q[q, i, c] * toks[f[i], c] for c in range(dim))
                                for i in range(lq))
                best = max(best, tot)
            assert abs(S[q, d] - best) <= 1e-12 * max(1.0, abs(best))


def test_maxsim_lq1_is_top1_dense_inner_product():
    rng = np.random.default_rng(3)
    dim = 16
    lens = [5, 1, 9, 3]
    D, off = _rand_csr(rng, lens, dim)
    Q = rng.standard_normal((3, 1, dim))
    S = oracle.maxsim_scores(Q, D, off)
    for d in range(len(lens)):
        top_s, _ = oracle.dense_topk(Q[:, 0, :], D[off[d]:off[d + 1]], 1)
        assert np.allclose(S[:, d], top_s[:, 0], rtol=0, atol=1e-13)


def test_maxsim_ld1_is_inner_product_with_summed_query():
    rng = np.random.default_rng(4)
    dim, lq = 8, 5
    D = rng.standard_normal((6, dim))
    off = np.arange(7)
    Q = rng.standard_normal((2, lq, dim))
    S = oracle.maxsim_scores(Q, D, off)
    for q in range(2):
        qsum = [math.fsum(Q[q, i, c] for i in range(lq)) for c in range(dim)]
        for d in range(6):
            want = math.fsum(qsum[c] * D[d, c] for c in range(dim))
            assert abs(S[q, d] - want) < 1e-12


def test_maxsim_doc_of_own_unit_tokens_scores_lq():
    # Cauchy-Schwarz: with unit doc tokens, <q_i, d_j> <= 1 = <q_i, q_i>, so each query token's
    # maximum is 1 and S = Lq exactly (up to fp64 rounding of the norms).
    rng = np.random.default_rng(5)
    dim, lq = 32, 7
    Q = _rand_unit(rng, lq, dim)[None]
    extra = _rand_unit(rng, 20, dim)
    toks = np.concatenate([extra[:9], Q[0][::-1], extra[9:]])
    S, A = oracle.maxsim_argmax(Q, toks, [0, len(toks)])
    assert abs(S[0, 0] - lq) < 1e-12
    assert list(A[0, :, 0]) == [9 + (lq - 1 - i) for i in range(lq)]


def test_maxsim_invariances_and_bounds():
    rng = np.random.default_rng(6)
    dim, lq = 12, 4
    Q = rng.standard_normal((3, lq, dim))
    toks = rng.standard_normal((10, dim))
    base = oracle.maxsim_scores(Q, toks, [0, 10])
    perm = rng.permutation(10)
    assert np.array_equal(oracle.maxsim_scores(Q, toks[perm], [0, 10]), base)  # exact
    dup = np.concatenate([toks, toks[[2, 7, 7]]])
    assert np.array_equal(oracle.maxsim_scores(Q, dup, [0, 13]), base)
    more = np.concatenate([toks, rng.standard_normal((3, dim))])
    assert np.all(oracle.maxsim_scores(Q, more, [0, 13]) >= base)
    bound = np.linalg.norm(Q, axis=2).sum(axis=1) * np.linalg.norm(toks, axis=1).max()
    assert np.all(np.abs(base[:, 0]) <= bound + 1e-12)


def test_maxsim_docs_are_independent_of_neighbours():
    rng = np.random.default_rng(7)
    Q = rng.standard_normal((2, 3, 6))
    D, off = _rand_csr(rng, [4, 2, 5], 6)
    S = oracle.maxsim_scores(Q, D, off)
    for d in range(3):
        alone = oracle.maxsim_scores(Q, D[off[d]:off[d + 1]], [0, off[d + 1] - off[d]])
        assert np.array_equal(alone[:, 0], S[:, d])


def test_maxsim_rejects_empty_doc():
    with pytest.raises(ValueError):
        oracle.maxsim_scores(np.zeros((1, 1, 2)), np.zeros((2, 2)), [0, 2, 2])


# ---------------------------------------------------------------- top-k

def _extract_topk(row, k):
    # repeated extraction of the best remaining entry: larger score first, then lower index
    remaining = list(range(len(row)))
    out = []
    for _ in range(k):
        best = remaining[0]
        for j in remaining[1:]:
            if row[j] > row[best]:
                best = j
        out.append(best)
        remaining.remove(best)
    return out


def test_topk_hand_example(golden):
    g = golden["maxsim"]
    S = np.array(g["S"], float)
    s2, i2 = oracle.rank_topk(S, 2)
    assert i2.tolist() == g["top2_idx"] and s2.tolist() == g["top2_scores"]
    _, i3 = oracle.rank_topk(S, 3)
    assert i3.tolist() == g["top3_idx"]


@pytest.mark.parametrize("n,k", [(1, 1), (7, 3), (40, 40), (100, 10)])
def test_topk_matches_repeated_extraction_with_ties(n, k):
    rng = np.random.default_rng(n + k)
    S = rng.integers(-3, 4, size=(4, n)).astype(float)     # many exact ties
    S[0, :] = 0.0
    S[1, ::2] = -0.0                                        # -0 ties +0
    vals, idx = oracle.rank_topk(S, k)
    for q in range(4):
        want = _extract_topk(S[q], k)
        assert idx[q].tolist() == want
        assert vals[q].tolist() == [S[q, j] for j in want]


def test_topk_full_k_is_a_sorted_permutation():
    rng = np.random.default_rng(9)
    S = rng.standard_normal((3, 50))
    vals, idx = oracle.rank_topk(S, 50)
    for q in range(3):
        assert sorted(idx[q].tolist()) == list(range(50))
        assert np.all(np.diff(vals[q]) <= 0)


# ---------------------------------------------------------------- L_LI loss

def _expected_from_exprs(g):
    loss = eval(g["loss"]["loss_expr"], _ns())
    G = [eval(e, _ns()) for e in g["loss"]["G_expr"]]
    env = _ns(G0=G[0], G1=G[1], G2=G[2])
    dQ = np.array([[[eval(e, env) for e in row] for row in q] for q in g["loss"]["dQ_expr"]])
    dD = np.array([[eval(e, env) for e in row] for row in g["loss"]["dD_expr"]])
    return loss, np.array(G), dQ, dD


def test_loss_hand_example(golden):
    g = golden["maxsim"]
    r = oracle.coltrast_li_loss(np.array(g["Q"], float), np.array(g["D"], float), g["offsets"],
                                golden["loss"]["pos"], golden["loss"]["logit_scale"])
    loss, G, dQ, dD = _expected_from_exprs(golden)
    assert abs(r["loss"] - loss) < 1e-15
    assert np.allclose(r["G"][0], G, rtol=0, atol=1e-15)
    assert np.allclose(r["dQ"], dQ, rtol=0, atol=1e-15)
    assert np.allclose(r["dD"], dD, rtol=0, atol=1e-15)


def test_loss_pairwise_is_softplus(golden):
    g = golden["pairwise"]
    r = oracle.coltrast_li_loss(np.array(g["Q"], float), np.array(g["D"], float), g["offsets"],
                                g["pos"], g["logit_scale"])
    assert np.array_equal(r["S"], np.array(g["S"], float))
    assert abs(r["loss"] - eval(g["loss_expr"], _ns())) < 1e-15


def test_loss_all_equal_scores_is_log_n():
    # every doc holds the same tokens -> all scores equal -> loss = ln n, G = (s/B)(1/n - onehot)
    rng = np.random.default_rng(12)
    dim, lq, n, B, s = 8, 3, 5, 2, 3.0
    toks = rng.standard_normal((4, dim))
    D = np.concatenate([toks] * n)
    off = np.arange(0, 4 * n + 1, 4)
    Q = rng.standard_normal((B, lq, dim))
    pos = [1, 4]
    r = oracle.coltrast_li_loss(Q, D, off, pos, s)
    assert abs(r["loss"] - math.log(n)) < 1e-13
    G = np.full((B, n), (s / B) / n)
    G[0, 1] -= s / B
    G[1, 4] -= s / B
    assert np.allclose(r["G"], G, rtol=0, atol=1e-14)


def test_loss_invariants():
    rng = np.random.default_rng(13)
    dim, lq = 6, 3
    D, off = _rand_csr(rng, [3, 5, 2, 4], dim)
    Q = rng.standard_normal((3, lq, dim))
    pos = [2, 0, 3]
    r = oracle.coltrast_li_loss(Q, D, off, pos, 2.5)
    assert np.allclose(r["G"].sum(axis=1), 0.0, atol=1e-14)
    assert np.all(r["G"][np.arange(3), pos] < 0)
    # s -> 0: every doc equally likely, loss -> ln n
    r0 = oracle.coltrast_li_loss(Q, D, off, pos, 1e-9)
    assert abs(r0["loss"] - math.log(4)) < 1e-8
    # shift invariance per query: add a dimension in which every doc token holds 1 and only
    # query 0's tokens hold c; S[0, :] rises by lq * c for every doc and the loss is unchanged.
    c = 0.75
    Qs = np.concatenate([Q, np.zeros((3, lq, 1))], axis=2)
    Qs[0, :, -1] = c
    Ds = np.concatenate([D, np.ones((D.shape[0], 1))], axis=1)
    rs = oracle.coltrast_li_loss(Qs, Ds, off, pos, 2.5)
    assert np.allclose(rs["S"][0], r["S"][0] + lq * c, atol=1e-13)
    assert abs(rs["loss"] - r["loss"]) < 1e-13


def test_loss_gradients_match_central_finite_differences():
    rng = np.random.default_rng(14)
    dim, lq = 5, 3
    D, off = _rand_csr(rng, [4, 3, 5], dim)
    Q = rng.standard_normal((2, lq, dim))
    pos = [1, 2]
    s = 1.7
    r = oracle.coltrast_li_loss(Q, D, off, pos, s)
    h = 1e-6

    def loss_at(Qx, Dx):
        return oracle.coltrast_li_loss(Qx, Dx, off, pos, s)["loss"]

    # stay away from argmax switches: every query-token maximum must beat the runner-up by > 1e-3
    for d in range(3):
        sim = np.einsum("qik,jk->qij", Q, D[off[d]:off[d + 1]])
        top2 = np.sort(sim, axis=2)[:, :, -2:]
        assert np.all(top2[:, :, 1] - top2[:, :, 0] > 1e-3)
    for idx in itertools.product(range(2), range(lq), range(dim)):
        Qp, Qm = Q.copy(), Q.copy()
        Qp[idx] += h
        Qm[idx] -= h
        fd = (loss_at(Qp, D) - loss_at(Qm, D)) / (2 * h)
        assert abs(fd - r["dQ"][idx]) <= 1e-6 * max(1.0, abs(fd))
    for idx in itertools.product(range(D.shape[0]), range(dim)):
        Dp, Dm = D.copy(), D.copy()
        Dp[idx] += h
        Dm[idx] -= h
        fd = (loss_at(Q, Dp) - loss_at(Q, Dm)) / (2 * h)
        assert abs(fd - r["dD"][idx]) <= 1e-6 * max(1.0, abs(fd))


def test_loss_rejects_bad_positive():
    with pytest.raises(ValueError):
        oracle.coltrast_li_loss(np.zeros((1, 1, 2)), np.ones((2, 2)), [0, 1, 2], [2], 1.0)


# ---------------------------------------------------------------- dense retrieval

def test_dense_planted_cosine_and_rank1():
    rng = np.random.default_rng(15)
    dim, n = 64, 500
    X = _rand_unit(rng, n, dim)
    Q = _rand_unit(rng, 4, dim)
    rows = [17, 3, 499, 250]
    for p, row in enumerate(rows):
        g = rng.standard_normal(dim)
        g -= (g @ Q[p]) * Q[p]
        u = g / np.linalg.norm(g)
        X[row] = 0.95 * Q[p] + math.sqrt(1 - 0.95 ** 2) * u
    vals, idx = oracle.dense_topk(Q, X, 5)
    assert idx[:, 0].tolist() == rows
    assert np.allclose(vals[:, 0], 0.95, atol=1e-12)


def test_dense_orthonormal_basis_scores():
    dim = 6
    X = np.eye(dim)[[4, 0, 5, 1, 3, 2]]
    Q = np.array([[1.0, -2.0, 3.0, -4.0, 5.0, -6.0]])
    s = oracle.dense_scores(Q, X)
    assert s[0].tolist() == [5.0, 1.0, -6.0, -2.0, -4.0, 3.0]
    vals, idx = oracle.dense_topk(Q, X, 3)
    assert idx[0].tolist() == [0, 5, 1] and vals[0].tolist() == [5.0, 3.0, 1.0]


def test_dense_duplicate_rows_rank_lower_index_first():
    rng = np.random.default_rng(16)
    X = _rand_unit(rng, 30, 8)
    X[20] = X[7]
    Q = X[[7]].copy()
    vals, idx = oracle.dense_topk(Q, X, 2)
    assert idx[0].tolist() == [7, 20] and vals[0, 0] == vals[0, 1]
