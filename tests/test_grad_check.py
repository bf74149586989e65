"""CPU checks of the per-row gradient verification (tests/grad_check.py): it must accept the oracle's
own gradients, the alternative a near-tie allows and the rounding a cancelling row cannot resolve,
and reject planted mistakes (a scaled row in a document of small softmax weight, a dropped row,
a row moved without a tie), also when the conditioning allowance is in force."""

import numpy as np
import pytest

import oracle
from grad_check import check_rows, conditioning_allowance, near_tie_allowance


def _unit(x):
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _case(seed=0, nq=3, lq=4, lens=(6, 9, 5, 7), dim=16, scale=2.0):
    g = np.random.default_rng(seed)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    Q = _unit(g.standard_normal((nq, lq, dim)))
    D = _unit(g.standard_normal((int(off[-1]), dim)))
    pos = np.arange(nq) % len(lens)
    return Q, D, off, pos, oracle.coltrast_li_loss(Q, D, off, pos, scale)


def test_oracle_gradients_pass_with_no_allowance():
    Q, D, off, pos, o = _case()
    aq, ad, n = near_tie_allowance(Q, D, off, o["G"])
    assert n == 0 and not aq.any() and not ad.any()
    assert check_rows(o["dQ"], o["dQ"], aq, "dQ") == 0.0
    assert check_rows(o["dD"], o["dD"], ad, "dD") == 0.0


def test_planted_error_in_a_low_weight_document_is_caught():
    # the document with the smallest softmax weight: scaling one of its selected rows by 1 %
    # is far below 2e-3 of the whole tensor's norm but not of the row's
    Q, D, off, pos, o = _case(scale=12.0)
    aq, ad, _ = near_tie_allowance(Q, D, off, o["G"])
    w = np.abs(o["G"]).sum(axis=0)
    d = int(np.argmin(w))
    rows = np.flatnonzero(np.any(o["dD"][off[d]:off[d + 1]] != 0, axis=1)) + off[d]
    bad = o["dD"].copy()
    bad[rows[0]] *= 1.01
    assert np.linalg.norm(bad - o["dD"]) < 2e-3 * np.linalg.norm(o["dD"])
    with pytest.raises(AssertionError):
        check_rows(bad, o["dD"], ad, "dD")


def test_dropped_and_moved_rows_are_caught():
    Q, D, off, pos, o = _case(seed=1)
    aq, ad, _ = near_tie_allowance(Q, D, off, o["G"])
    sel = np.flatnonzero(np.any(o["dD"] != 0, axis=1))
    dropped = o["dD"].copy()
    dropped[sel[0]] = 0.0
    with pytest.raises(AssertionError):
        check_rows(dropped, o["dD"], ad, "dD")
    free = np.flatnonzero(~np.any(o["dD"] != 0, axis=1))
    moved = o["dD"].copy()
    moved[free[0]] = moved[sel[0]]
    moved[sel[0]] = 0.0
    with pytest.raises(AssertionError):
        check_rows(moved, o["dD"], ad, "dD")
    wrong_q = o["dQ"].copy()
    wrong_q[0, 0] = -wrong_q[0, 0]
    with pytest.raises(AssertionError):
        check_rows(wrong_q, o["dQ"], aq, "dQ")


def test_tie_alternative_is_accepted_only_with_its_allowance():
    # document 0 holds two bit-identical copies (rows 1 and 4) of a token that is query token
    # 0's maximum: the oracle sends the gradient to row 1; a GPU may send it to row 4
    Q, D, off, pos, _ = _case(seed=2, nq=1, lq=2, lens=(6, 5), dim=8)
    D = D.copy()
    D[1] = _unit(Q[0, 0] + 0.01 * np.arange(8))
    D[4] = D[1]
    o = oracle.coltrast_li_loss(Q, D, off, pos, 2.0)
    assert o["A"][0, 0, 0] == 1
    aq, ad, n = near_tie_allowance(Q, D, off, o["G"])
    assert n >= 1 and ad[1] > 0 and ad[4] > 0
    alt = o["dD"].copy()
    part = o["G"][0, 0] * Q[0, 0]
    alt[1] -= part
    alt[4] += part
    check_rows(alt, o["dD"], ad, "dD")                 # the alternative choice is valid
    check_rows(o["dQ"], o["dQ"], aq, "dQ")             # equal tokens: dQ does not move
    with pytest.raises(AssertionError):
        check_rows(alt, o["dD"], np.zeros_like(ad), "dD")


def _cancelling_case():
    # query 0's token 0 is copied into its positive (document 0) and into document 1, and the
    # large logit scale puts almost all the softmax weight on those two: dQ[0, 0] is the sum of
    # two nearly opposite terms on the same vector
    g = np.random.default_rng(7)
    off = np.array([0, 6, 12, 18], dtype=np.int64)
    Q = _unit(g.standard_normal((1, 3, 16)))
    D = _unit(g.standard_normal((18, 16)))
    D[2] = Q[0, 0]
    D[9] = Q[0, 0]
    D[3], D[10] = Q[0, 1], Q[0, 1]
    D[4], D[11] = Q[0, 2], Q[0, 2]
    pos = np.array([0])
    return Q, D, off, pos, 12.0, oracle.coltrast_li_loss(Q, D, off, pos, 12.0)


def test_cancelling_row_needs_and_gets_the_conditioning_allowance():
    Q, D, off, pos, scale, o = _cancelling_case()
    q_row = o["dQ"][0, 0]
    terms = np.abs(o["G"][0]).sum()
    assert np.linalg.norm(q_row) < 1e-3 * terms          # the row is far smaller than its terms
    # what a GPU may legitimately return: the weight of document 1 off by 1e-7 relative (its
    # scores within 1e-8 of the oracle's), which moves the row by 1e-7 of that term
    dS = np.full_like(o["S"], 1e-8)
    alt = o["dQ"].copy()
    alt[0, 0] += 1e-7 * o["G"][0, 1] * D[9]
    aq, ad, _ = near_tie_allowance(Q, D, off, o["G"])
    cq, cd = conditioning_allowance(Q, D, off, o["G"], o["A"], dS, scale)
    if np.linalg.norm(1e-7 * o["G"][0, 1] * D[9]) > 2e-3 * np.linalg.norm(q_row):
        with pytest.raises(AssertionError):
            check_rows(alt, o["dQ"], aq, "dQ")
    check_rows(alt, o["dQ"], aq, "dQ", cond=cq)
    check_rows(o["dD"], o["dD"], ad, "dD", cond=cd)


def test_conditioning_allowance_excuses_no_real_mistake():
    Q, D, off, pos, o = _case(seed=3, scale=2.0)
    dS = np.full_like(o["S"], 1e-6)   # GPU scores 1e-6 off: tau = 4 * 2 * 1e-6 + 2^-20
    aq, ad, _ = near_tie_allowance(Q, D, off, o["G"])
    cq, cd = conditioning_allowance(Q, D, off, o["G"], o["A"], dS, 2.0)
    qn = np.linalg.norm(o["dQ"], axis=2)
    assert np.all(cq <= 1e-4 * np.abs(o["G"]).sum(axis=1)[:, None] * 1.01)
    assert np.median(cq / qn) < 1e-3
    # a dropped selected dD row and a sign flip in dQ still fail with both allowances
    sel = np.flatnonzero(np.any(o["dD"] != 0, axis=1))
    j = sel[np.argmax(np.linalg.norm(o["dD"][sel], axis=1))]
    dropped = o["dD"].copy()
    dropped[j] = 0.0
    with pytest.raises(AssertionError):
        check_rows(dropped, o["dD"], ad, "dD", cond=cd)
    wrong_q = o["dQ"].copy()
    e = np.unravel_index(np.argmax(qn), qn.shape)
    wrong_q[e] = -wrong_q[e]
    with pytest.raises(AssertionError):
        check_rows(wrong_q, o["dQ"], aq, "dQ", cond=cq)
