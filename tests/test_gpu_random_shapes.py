"""GPU parity on seeded random shapes: every compute entry point against the oracle.

The other GPU tests pick their shapes by hand (tile edges, ragged tails, limits).  Here each
entry point also runs a fixed list of configurations drawn from a seeded generator -- query
counts, query lengths, feature dimensions (every multiple of 8 in range), document counts and
length mixes, k, logit scales, paper layouts and thresholds -- with some documents holding
copies of query tokens, so that maxima are attained exactly and ties occur.  Each configuration
is printed before its call, so a failure names it.  The bars are those of the hand-picked tests:
scores within 2e-3 and a tight 1e-4 (bf16 and fp16 products are exact in fp32), top-k lists by
the rules of tests/topk_check.py, gradients per row (tests/grad_check.py, with its allowance for
rows whose terms cancel), chunking decisions exact away from the threshold.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2505_04846_amd as hpr
import synth
from grad_check import check_rows, conditioning_allowance, near_tie_allowance
from topk_check import check_topk

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
REL = 2e-3


def _bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy()


def _close(g, o, rel, what):
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    err = np.abs(g - o)
    lim = rel * np.maximum(np.abs(o), 1e-3)
    assert np.all(err <= lim), f"{what}: worst {(err / lim).max():.3g}x the bound at rel {rel}"


def _store(rng, nq, lq, dim, n_docs, max_len, plant):
    """Queries [nq, lq, dim] and a CSR store (bf16); with `plant`, about a fifth of the documents
    hold exact copies of some query tokens at random positions."""
    g = torch.Generator().manual_seed(int(rng.integers(1 << 30)))
    lens = torch.as_tensor(rng.integers(1, max_len + 1, n_docs), dtype=torch.int64)
    off = synth.csr_offsets(lens)
    Q = synth.unit_rows(nq * lq, dim, g, "cpu", torch.bfloat16)
    D = synth.unit_rows(int(off[-1]), dim, g, "cpu", torch.bfloat16)
    if plant:
        for d in np.flatnonzero(rng.random(n_docs) < 0.2):
            a, b = int(off[d]), int(off[d + 1])
            m = int(rng.integers(1, b - a + 1))
            D[a + rng.choice(b - a, m, replace=False)] = Q[rng.integers(0, nq * lq, m)]
    return Q.reshape(nq, lq, dim), D, off


def _dim(rng, hi):
    return 8 * int(rng.integers(1, hi // 8 + 1))


def _tight_scores(S, O, A, Qo, Do, off, what):
    """The tight 1e-4 on MaxSim scores where a score is not a near-cancellation of its
    per-token maxima (their magnitudes summing to at most ten times the score): single-token
    documents can sum maxima of both signs to about zero, below fp32 resolution."""
    m = np.abs(np.einsum("qik,qidk->qid", Qo, Do[np.asarray(off)[:-1][None, None, :] + A]))
    well = m.sum(axis=1) <= 10.0 * np.maximum(np.abs(O), 1e-3)
    _close(S[well], O[well], 1e-4, what)


def test_maxsim_score_random_shapes():
    rng = np.random.default_rng(101)
    for c in range(20):
        dim = _dim(rng, 256)
        lq = int(rng.integers(1, (128 if dim <= 128 else 64) + 1))
        nq = int(rng.integers(1, 41))
        n_docs = int(rng.integers(1, 101))
        max_len = int(rng.integers(1, 121))
        print(f"config {c}: nq={nq} lq={lq} dim={dim} n_docs={n_docs} max_len={max_len}",
              flush=True)
        Q, D, off = _store(rng, nq, lq, dim, n_docs, max_len, plant=c % 2 == 0)
        S = hpr.maxsim_score(Q.to(DEV), D.to(DEV), off.to(DEV)).cpu().numpy()
        Qo, Do = oracle.decode_bf16(_bits(Q)), oracle.decode_bf16(_bits(D))
        O, A = oracle.maxsim_argmax(Qo, Do, off.numpy())
        _close(S, O, REL, f"config {c}")
        _tight_scores(S, O, A, Qo, Do, off.numpy(), f"config {c} (tight)")


def test_maxsim_score_dim128_many_query_slots():
    # dim 128 with more than 256 query slots: the score kernel's variant that stages its tiles
    # straight into LDS, four per stage (ragged documents end at every row of a tile and at any
    # tile of a stage)
    rng = np.random.default_rng(707)
    for c in range(8):
        lq = int(rng.integers(1, 129))
        lqp = (lq + 31) // 32 * 32
        nq = int(rng.integers(256 // lqp + 1, 257 // lqp + 40))
        n_docs = int(rng.integers(1, 301))
        max_len = int(rng.integers(1, 200))
        print(f"config {c}: nq={nq} lq={lq} dim=128 n_docs={n_docs} max_len={max_len}",
              flush=True)
        Q, D, off = _store(rng, nq, lq, 128, n_docs, max_len, plant=c % 2 == 0)
        S = hpr.maxsim_score(Q.to(DEV), D.to(DEV), off.to(DEV)).cpu().numpy()
        Qo, Do = oracle.decode_bf16(_bits(Q)), oracle.decode_bf16(_bits(D))
        O, A = oracle.maxsim_argmax(Qo, Do, off.numpy())
        _close(S, O, REL, f"config {c}")
        _tight_scores(S, O, A, Qo, Do, off.numpy(), f"config {c} (tight)")


def test_maxsim_topk_random_shapes():
    rng = np.random.default_rng(202)
    for c in range(10):
        long_rows = c >= 8  # rows long enough for the streaming select
        dim = _dim(rng, 32 if long_rows else 128)
        lq = int(rng.integers(1, 33))
        nq = int(rng.integers(1, 9))
        n_docs = int(rng.integers(9_000, 40_001)) if long_rows else int(rng.integers(1, 3001))
        k = int(rng.integers(1, min(n_docs, 1024) + 1))
        print(f"config {c}: nq={nq} lq={lq} dim={dim} n_docs={n_docs} k={k}", flush=True)
        Q, D, off = _store(rng, nq, lq, dim, n_docs, 4 if long_rows else 24, plant=True)
        s, i = hpr.maxsim_topk(Q.to(DEV), D.to(DEV), off.to(DEV), k)
        s, i = s.cpu().numpy(), i.cpu().numpy()
        O = oracle.maxsim_scores(oracle.decode_bf16(_bits(Q)), oracle.decode_bf16(_bits(D)),
                                 off.numpy())
        for q in range(nq):
            check_topk(s[q], i[q], O[q], k, rel=REL)
            check_topk(s[q], i[q], O[q], k, rel=1e-5)


def test_loss_random_shapes():
    rng = np.random.default_rng(303)
    for c in range(10):
        dim = _dim(rng, 256)
        lq = int(rng.integers(1, (64 if dim <= 128 else 32) + 1))
        nq = int(rng.integers(1, 17))
        n_docs = int(rng.integers(1, 41))
        scale = float(np.exp(rng.uniform(np.log(0.3), np.log(30.0))))
        print(f"config {c}: nq={nq} lq={lq} dim={dim} n_docs={n_docs} scale={scale:.3f}",
              flush=True)
        Q, D, off = _store(rng, nq, lq, dim, n_docs, 200, plant=True)
        pos = torch.as_tensor(rng.integers(0, n_docs, nq), dtype=torch.int32)
        r = hpr.coltrast_loss_fwd_bwd(Q.to(DEV), D.to(DEV), off.to(DEV), pos.to(DEV), scale,
                                      return_scores=True)
        Qo, Do = oracle.decode_bf16(_bits(Q)), oracle.decode_bf16(_bits(D))
        o = oracle.coltrast_li_loss(Qo, Do, off.numpy(), pos.numpy(), scale)
        S = r["scores"].cpu().numpy()
        _close(S, o["S"], REL, f"config {c} scores")
        _tight_scores(S, o["S"], o["A"], Qo, Do, off.numpy(), f"config {c} scores (tight)")
        _close(r["loss"].cpu().numpy()[0], o["loss"], REL, f"config {c} loss")
        aq, ad, _ = near_tie_allowance(Qo, Do, off.numpy(), o["G"])
        # copies of a query's token in its positive and in a negative make rows whose terms
        # cancel: their bound includes what fp32 weights and sums cannot resolve
        cq, cd = conditioning_allowance(Qo, Do, off.numpy(), o["G"], o["A"], S - o["S"], scale)
        check_rows(r["dq"].cpu().numpy(), o["dQ"], aq, f"config {c} dQ", cond=cq)
        check_rows(r["dd"].cpu().numpy(), o["dD"], ad, f"config {c} dD", cond=cd)


def test_total_loss_random_shapes():
    rng = np.random.default_rng(606)
    for c in range(8):
        dim = _dim(rng, 256)
        lq = int(rng.integers(1, (64 if dim <= 128 else 32) + 1))
        nq = int(rng.integers(1, 17))
        n_docs = int(rng.integers(1, 41))
        scale = float(np.exp(rng.uniform(np.log(0.3), np.log(30.0))))
        tau = float(np.exp(rng.uniform(np.log(0.02), np.log(1.0))))
        print(f"config {c}: nq={nq} lq={lq} dim={dim} n_docs={n_docs} scale={scale:.3f} "
              f"tau={tau:.3f}", flush=True)
        Q, D, off = _store(rng, nq, lq, dim, n_docs, 200, plant=True)
        pos = torch.as_tensor(rng.integers(0, n_docs, nq), dtype=torch.int32)
        args = (Q.to(DEV), D.to(DEV), off.to(DEV), pos.to(DEV), scale)
        r = hpr.coltrast_total_loss_fwd_bwd(*args, tau)
        S = hpr.coltrast_loss_fwd_bwd(*args, return_scores=True)["scores"].cpu().numpy()
        Qo, Do = oracle.decode_bf16(_bits(Q)), oracle.decode_bf16(_bits(D))
        o = oracle.coltrast_total_loss(Qo, Do, off.numpy(), pos.numpy(), scale, tau)
        li = oracle.coltrast_li_loss(Qo, Do, off.numpy(), pos.numpy(), scale)
        got = r["loss"].cpu().numpy()
        for j, key in enumerate(("loss", "loss_li", "loss_c")):
            _close(got[j], o[key], REL, f"config {c} {key}")
        # the L_LI half carries weights G / 2
        aq, ad, _ = near_tie_allowance(Qo, Do, off.numpy(), 0.5 * li["G"])
        cq, cd = conditioning_allowance(Qo, Do, off.numpy(), 0.5 * li["G"], li["A"], S - li["S"],
                                        scale)
        check_rows(r["dq"].cpu().numpy(), o["dQ"], aq, f"config {c} dQ", cond=cq)
        check_rows(r["dd"].cpu().numpy(), o["dD"], ad, f"config {c} dD", cond=cd)


def test_dense_topk_random_shapes():
    rng = np.random.default_rng(404)
    for c in range(8):
        big = c % 3 == 2  # past the exact sample: the filtered scan and its merge
        dim = _dim(rng, 64 if big else 1024)
        n = int(rng.integers(131_073, 250_001)) if big else int(rng.integers(1, 20_001))
        nq = int(rng.integers(1, 65 if big else 301))
        k = int(rng.integers(1, min(n, 1024) + 1))
        print(f"config {c}: nq={nq} n={n} dim={dim} k={k}", flush=True)
        g = torch.Generator().manual_seed(int(rng.integers(1 << 30)))
        Q = synth.unit_rows(nq, dim, g, "cpu", torch.float16)
        X = synth.unit_rows(n, dim, g, "cpu", torch.float16)
        s, i = hpr.dense_ip_topk(Q.to(DEV), X.to(DEV), k)
        s, i = s.cpu().numpy(), i.cpu().numpy()
        O = oracle.dense_scores(oracle.decode_fp16(_bits(Q)), oracle.decode_fp16(_bits(X)))
        for q in range(nq):
            check_topk(s[q], i[q], O[q], k, rel=REL)
        del O


def test_semantic_chunk_random_shapes():
    rng = np.random.default_rng(505)
    band = 2e-5
    for c in range(8):
        dim = _dim(rng, 2048)
        n_papers = int(rng.integers(1, 41))
        thr = float(rng.uniform(-0.2, 0.95))
        print(f"config {c}: n_papers={n_papers} dim={dim} threshold={thr:.4f}", flush=True)
        w = synth.sentence_stream(seed=int(rng.integers(1 << 30)), n_papers=n_papers,
                                  len_min=0 if n_papers > 1 else 1, len_max=300, dim=dim)
        E, off = w["E"], w["paper_off"]
        r = hpr.semantic_chunk(E.to(DEV), off.to(DEV), thr, return_cos=True)
        cos_g = r["cos"].cpu().numpy().astype(np.float64)
        seg_g = r["seg"].cpu().numpy().astype(np.int64)
        cos_o, seg_o, n_o = oracle.semantic_segments(oracle.decode_fp16(_bits(E)), off.numpy(),
                                                     thr)
        nan_o = np.isnan(cos_o)
        assert np.array_equal(np.isnan(cos_g), nan_o), f"config {c}: NaN positions"
        assert np.all(np.abs(cos_g[~nan_o] - cos_o[~nan_o]) <= band), f"config {c}: cosines"
        with np.errstate(invalid="ignore"):
            b_g = ~(cos_g > np.float32(thr))
            b_o = ~(cos_o > thr)
        clear = nan_o | (np.abs(cos_o - thr) > band)
        assert np.array_equal(b_g[clear], b_o[clear]), f"config {c}: decisions"
        assert np.array_equal(seg_g, np.cumsum(b_g.astype(np.int64)) - 1), f"config {c}: ids"
        assert int(r["n_segments"].item()) == int(b_g.sum())
        if clear.all():
            assert np.array_equal(seg_g, seg_o) and int(r["n_segments"].item()) == n_o
