"""CPU checks of the per-row gradient verification (tests/grad_check.py): it must accept the oracle's
own gradients and the alternative a near-tie allows, and reject planted mistakes (a scaled
row in a document of small softmax weight, a dropped row, a row moved without a tie)."""

import numpy as np
import pytest

import oracle
from grad_check import check_rows, near_tie_allowance


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
