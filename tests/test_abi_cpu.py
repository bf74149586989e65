"""CPU-only checks of the C ABI: the built library loads, exports every entry point declared in
include/hiperrag.h, and rejects bad arguments on the host before touching a device."""

import ctypes
import os
import re

import pytest

import paper_2505_04846_amd as hpr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hiperrag.h")

FAKE = ctypes.c_void_p(0x10000)       # non-NULL, 16-byte aligned, never dereferenced on the host
FAKE_ODD = ctypes.c_void_p(0x10008)   # misaligned
NULL = ctypes.c_void_p(0)
BIG = 1 << 40


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w]*\s*\*?\s+\*?([A-Za-z_]\w*)\s*\(", text, re.M)
    return sorted(set(names))


def test_library_exports_every_declared_function():
    names = _declared_functions()
    assert "maxsim_score" in names and "dense_ip_topk" in names and "hpr_last_error" in names
    lib = hpr.lib()
    for n in names:
        assert hasattr(lib, n), f"{n} declared in hiperrag.h but not exported"
    assert set(hpr._SIGNATURES) == set(names)


def test_abi_version_and_status_strings():
    lib = hpr.lib()
    assert lib.hpr_abi_version() == 1
    assert lib.hpr_status_string(0) == b"HPR_OK"
    assert lib.hpr_status_string(5) == b"HPR_ERR_WORKSPACE_TOO_SMALL"
    for code, name in hpr.STATUS_NAMES.items():
        assert lib.hpr_status_string(code).decode() == name


def _score(**kw):
    a = dict(q=FAKE, nq=2, lq=32, d=FAKE, off=FAKE, n_docs=4, n_tok=64, dim=128, scores=FAKE,
             ws=FAKE, ws_bytes=BIG, stream=NULL)
    a.update(kw)
    lib = hpr.lib()
    return lib.maxsim_score(a["q"], a["nq"], a["lq"], a["d"], a["off"], a["n_docs"], a["n_tok"],
                            a["dim"], a["scores"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(q=NULL), 1), (dict(d=NULL), 1), (dict(off=NULL), 1), (dict(scores=NULL), 1),
    (dict(ws=NULL), 1), (dict(nq=0), 1), (dict(lq=0), 1), (dict(n_docs=0), 1),
    (dict(n_tok=3), 1), (dict(dim=0), 1), (dict(dim=12), 4), (dict(dim=264), 4), (dict(dim=4), 4),
    (dict(lq=129, dim=64), 4), (dict(lq=129), 4), (dict(lq=65, dim=256), 4), (dict(q=FAKE_ODD), 1), (dict(ws_bytes=0), 5),
])
def test_maxsim_score_rejects(kw, status):
    assert _score(**kw) == status
    assert hpr.lib().hpr_last_error()  # a message is set


@pytest.mark.parametrize("kw,status", [
    (dict(q=NULL), 1), (dict(d=NULL), 1), (dict(off=NULL), 1), (dict(scores=NULL), 1),
    (dict(nq=0), 1), (dict(n_tok=3), 1), (dict(dim=12), 4), (dict(lq=129), 4),
    (dict(q=FAKE_ODD), 1),
])
def test_maxsim_score_noalloc_rejects(kw, status):
    a = dict(q=FAKE, nq=2, lq=32, d=FAKE, off=FAKE, n_docs=4, n_tok=64, dim=128, scores=FAKE)
    a.update(kw)
    assert hpr.lib().maxsim_score_noalloc(a["q"], a["nq"], a["lq"], a["d"], a["off"], a["n_docs"],
                                          a["n_tok"], a["dim"], a["scores"], NULL) == status
    assert hpr.lib().hpr_last_error()


def _topk(k, n_docs=10, ws_bytes=BIG):
    return hpr.lib().maxsim_topk(FAKE, 2, 8, FAKE, FAKE, n_docs, 100, 64, k, FAKE, FAKE, FAKE,
                                 ws_bytes, NULL)


def test_maxsim_topk_rejects_bad_k_and_small_workspace():
    assert _topk(0) == 1
    assert _topk(11) == 1
    assert _topk(1025, n_docs=5000) == 1
    assert _topk(5, ws_bytes=16) == 5


def _loss(**kw):
    a = dict(q=FAKE, nq=4, lq=32, d=FAKE, off=FAKE, n_docs=8, n_tok=256, dim=128, pos=FAKE,
             scale=50.0, loss=FAKE, dq=FAKE, dd=FAKE, scores=NULL, ws=FAKE, ws_bytes=BIG)
    a.update(kw)
    return hpr.lib().coltrast_loss_fwd_bwd(a["q"], a["nq"], a["lq"], a["d"], a["off"], a["n_docs"],
                                           a["n_tok"], a["dim"], a["pos"], a["scale"], a["loss"],
                                           a["dq"], a["dd"], a["scores"], a["ws"], a["ws_bytes"],
                                           NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(pos=NULL), 1), (dict(loss=NULL), 1), (dict(scale=float("nan")), 1),
    (dict(scale=float("inf")), 1), (dict(nq=1024, lq=32), 4), (dict(dq=FAKE_ODD), 1),
    (dict(lq=65), 4), (dict(lq=33, dim=256), 4),
    (dict(ws_bytes=100), 5),
    # dD's LDS per workgroup (10 E + 4 nq + 10244 bytes) above a CU's 160 KiB
    (dict(nq=480, lq=32, n_docs=500, n_tok=16000), 4), (dict(nq=4096, lq=4, n_docs=500, n_tok=16000), 4),
])
def test_loss_rejects(kw, status):
    assert _loss(**kw) == status


def _total(**kw):
    a = dict(q=FAKE, nq=4, lq=32, d=FAKE, off=FAKE, n_docs=8, n_tok=256, dim=128, pos=FAKE,
             scale=50.0, tau=0.05, loss=FAKE, dq=FAKE, dd=FAKE, ws=FAKE, ws_bytes=BIG)
    a.update(kw)
    return hpr.lib().coltrast_total_loss_fwd_bwd(
        a["q"], a["nq"], a["lq"], a["d"], a["off"], a["n_docs"], a["n_tok"], a["dim"], a["pos"],
        a["scale"], a["tau"], a["loss"], a["dq"], a["dd"], a["ws"], a["ws_bytes"], NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(pos=NULL), 1), (dict(loss=NULL), 1), (dict(ws=NULL), 1), (dict(q=NULL), 1),
    (dict(scale=float("nan")), 1), (dict(tau=0.0), 1), (dict(tau=-0.05), 1),
    (dict(tau=float("nan")), 1), (dict(tau=float("inf")), 1), (dict(tau=1e-40), 1),
    (dict(nq=1024, lq=32), 4), (dict(dd=FAKE_ODD), 1), (dict(lq=65), 4), (dict(dim=12), 4),
    (dict(ws_bytes=100), 5), (dict(nq=512, lq=32, n_docs=500, n_tok=16000), 4),
])
def test_total_loss_rejects(kw, status):
    assert _total(**kw) == status
    assert hpr.lib().hpr_last_error()


def test_total_loss_workspace_holds_the_li_workspace():
    lib = hpr.lib()
    li = lib.coltrast_loss_workspace_size(64, 32, 512, 131072, 128)
    tot = lib.coltrast_total_loss_workspace_size(64, 32, 512, 131072, 128)
    # plus pooled rows, norms, dL_C/dc, terms and the gradient parts
    extra = 4 * (2 * 64 * 128 + 2 * 512 * 128 + 2 * 64 + 512 + 64 * 512)
    assert tot >= li + extra and tot % 256 == 0
    assert _total(ws_bytes=tot - 1, nq=64, n_docs=512, n_tok=131072) == 5
    assert lib.coltrast_total_loss_workspace_size(0, 32, 512, 131072, 128) == 0


def _chunk(**kw):
    a = dict(emb=FAKE, n=1000, dim=4096, off=NULL, n_papers=0, thr=0.5, cos=NULL, seg=FAKE,
             nseg=FAKE, ws=FAKE, ws_bytes=BIG)
    a.update(kw)
    return hpr.lib().semantic_chunk(a["emb"], a["n"], a["dim"], a["off"], a["n_papers"], a["thr"],
                                    a["cos"], a["seg"], a["nseg"], a["ws"], a["ws_bytes"], NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(emb=NULL), 1), (dict(seg=NULL), 1), (dict(nseg=NULL), 1), (dict(ws=NULL), 1),
    (dict(n=0), 1), (dict(n=1 << 31), 1), (dict(dim=12), 4), (dict(dim=4104), 4), (dict(dim=0), 4),
    (dict(thr=float("nan")), 1), (dict(off=FAKE, n_papers=0), 1), (dict(emb=FAKE_ODD), 1),
    (dict(ws_bytes=16), 5),
])
def test_semantic_chunk_rejects(kw, status):
    assert _chunk(**kw) == status
    assert hpr.lib().hpr_last_error()


def test_semantic_chunk_workspace():
    lib = hpr.lib()
    n = 2_000_000
    w = lib.semantic_chunk_workspace_size(n, 4096)
    ranges = (n + 127) // 128
    assert w >= 4 * ranges + 8 * ranges + 4 * n and w % 256 == 0
    assert lib.semantic_chunk_workspace_size(0, 4096) == 0
    assert _chunk(n=n, ws_bytes=w - 1) == 5


def test_retrieval_metrics_rejects():
    lib = hpr.lib()
    f = lib.retrieval_metrics
    assert f(NULL, 4, 10, 10, FAKE, NULL, FAKE, NULL) == 1
    assert f(FAKE, 4, 10, 10, NULL, NULL, FAKE, NULL) == 1
    assert f(FAKE, 4, 10, 10, FAKE, NULL, NULL, NULL) == 1
    assert f(FAKE, 0, 10, 10, FAKE, NULL, FAKE, NULL) == 1
    assert f(FAKE, 4, 10, 11, FAKE, NULL, FAKE, NULL) == 1
    assert f(FAKE, 4, 10, 0, FAKE, NULL, FAKE, NULL) == 1


def test_calibration_rejects_bad_arguments():
    lib = hpr.lib()
    flops = ctypes.c_double(0)
    assert lib.hpr_mfma_calibration(0, 0, FAKE, ctypes.byref(flops), NULL) == 1
    assert lib.hpr_mfma_calibration(10, 2, FAKE, ctypes.byref(flops), NULL) == 1
    assert lib.hpr_mfma_calibration(10, -1, FAKE, ctypes.byref(flops), NULL) == 1
    assert lib.hpr_mfma_calibration(10, 1, NULL, ctypes.byref(flops), NULL) == 1
    assert lib.hpr_mfma_calibration(10, 0, FAKE, None, NULL) == 1
    assert lib.hpr_read_calibration(NULL, 1024, FAKE, NULL) == 1
    assert lib.hpr_read_calibration(FAKE, 1000, FAKE, NULL) == 1
    assert lib.hpr_read_calibration(FAKE_ODD, 1024, FAKE, NULL) == 1
    assert lib.hpr_read_calibration(FAKE, 1024, NULL, NULL) == 1


def test_workspace_sizes_are_consistent():
    lib = hpr.lib()
    s1 = lib.maxsim_score_workspace_size(64, 32, 512, 131072, 128)
    s2 = lib.maxsim_topk_workspace_size(64, 32, 512, 131072, 128, 10)
    s3 = lib.coltrast_loss_workspace_size(64, 32, 512, 131072, 128)
    assert 0 < s1 < s2 < s3
    assert s2 >= 64 * 512 * 4 and s3 >= 2 * 64 * 512 * 4 + 512 * 64 * 32 * 2
    for s in (s1, s2, s3):
        assert s % 256 == 0
    assert lib.maxsim_score_workspace_size(64, 32, 0, 0, 128) == 0


def test_csr_validate_and_scale_reject_null():
    lib = hpr.lib()
    bad = ctypes.c_int64(0)
    assert lib.hpr_csr_validate(NULL, 4, 10, FAKE, NULL, ctypes.byref(bad)) == 1
    assert lib.hpr_csr_validate(FAKE, 0, 10, FAKE, NULL, ctypes.byref(bad)) == 1
    assert lib.hpr_scale_f32(NULL, 4, FAKE, NULL) == 1
    assert lib.hpr_scale_f32(FAKE, -1, FAKE, NULL) == 1


def test_binding_refuses_cpu_tensors():
    import torch
    Q = torch.zeros((1, 1, 8), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        hpr.maxsim_score(Q, torch.zeros((1, 8), dtype=torch.bfloat16),
                         torch.tensor([0, 1], dtype=torch.int64))
