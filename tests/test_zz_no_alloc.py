"""maxsim_score_noalloc (the entry point that allocates nothing; its scratch is a static device
array of the library) against maxsim_score through the C ABI: bit-identical scores on two calls
in a row, the second on a smaller input, and both within the score tolerance of the oracle."""

import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2505_04846_amd as hpr
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _bf(t):
    return oracle.decode_bf16(t.detach().cpu().contiguous().view(torch.int16).numpy())


def _inputs(seed, nq, lq, n_docs, ld_max, dim):
    g = torch.Generator().manual_seed(seed)
    lens = torch.randint(1, ld_max + 1, (n_docs,), generator=g)
    off = synth.csr_offsets(lens)
    Q = synth.unit_rows(nq * lq, dim, g, "cpu", torch.bfloat16).reshape(nq, lq, dim)
    D = synth.unit_rows(int(off[-1]), dim, g, "cpu", torch.bfloat16)
    return Q, D, off


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _call_both(Q, D, off):
    """(noalloc scores, maxsim_score scores), both through the C ABI on the current stream."""
    L = hpr.lib()
    Qd, Dd, od = Q.to(DEV), D.to(DEV), off.to(DEV)
    nq, lq, dim = Q.shape
    n_docs, n_tok = off.numel() - 1, D.shape[0]
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    a = torch.full((nq, n_docs), float("nan"), dtype=torch.float32, device=DEV)
    b = torch.full((nq, n_docs), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.empty(max(1, L.maxsim_score_workspace_size(nq, lq, n_docs, n_tok, dim)),
                     dtype=torch.uint8, device=DEV)
    torch.cuda.synchronize()
    st = L.maxsim_score_noalloc(_p(Qd), nq, lq, _p(Dd), _p(od), n_docs, n_tok, dim, _p(a), s)
    assert st == 0, L.hpr_last_error()
    st = L.maxsim_score(_p(Qd), nq, lq, _p(Dd), _p(od), n_docs, n_tok, dim, _p(b), _p(ws),
                        ws.numel(), s)
    assert st == 0, L.hpr_last_error()
    torch.cuda.synchronize()
    return a.cpu(), b.cpu()


def test_noalloc_matches_maxsim_score_on_two_calls_in_a_row():
    # first call: 3,000 documents (many ranges in the static table); second: a smaller store
    # whose table is shorter, so stale entries of the first call must not be read
    for seed, shape in ((1, (6, 32, 3000, 300, 128)), (2, (3, 20, 40, 90, 64))):
        Q, D, off = _inputs(seed, *shape)
        a, b = _call_both(Q, D, off)
        assert torch.equal(a, b), f"seed {seed}: noalloc scores differ from maxsim_score's"
        o = oracle.maxsim_scores(_bf(Q), _bf(D), off.numpy())
        err = np.abs(a.numpy().astype(np.float64) - o)
        assert np.all(err <= 1e-4 * np.maximum(np.abs(o), 1e-3)), f"seed {seed}: vs oracle"


def test_noalloc_rejects_bad_arguments_without_launching():
    L = hpr.lib()
    Q, D, off = _inputs(3, 2, 8, 5, 10, 64)
    Qd, Dd, od = Q.to(DEV), D.to(DEV), off.to(DEV)
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = torch.empty((2, 5), dtype=torch.float32, device=DEV)
    assert L.maxsim_score_noalloc(_p(Qd), 2, 8, _p(Dd), _p(od), 5, D.shape[0], 64,
                                  ctypes.c_void_p(0), s) == 1
    assert L.maxsim_score_noalloc(_p(Qd), 2, 8, _p(Dd), _p(od), 5, D.shape[0], 12, _p(out), s) == 4
