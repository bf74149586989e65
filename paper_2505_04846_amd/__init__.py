"""Python binding of libhiperrag.so: MI355X MaxSim scoring, InfoNCE and exact top-k.

Argument marshalling only.  Every computation runs in the HIP kernels of the shared library;
torch provides device memory (outputs and workspaces) and the current stream.  There is no
fallback: if the library is not built, or a call fails, an exception is raised.

    maxsim_score(Q, D, off)                       -> scores fp32 [nq, n_docs]
    maxsim_score_noalloc(Q, D, off)               -> the same, with no device allocation
    maxsim_topk(Q, D, off, k)                     -> (scores fp32 [nq, k], idx int64 [nq, k])
    coltrast_loss_fwd_bwd(Q, D, off, pos, scale)  -> dict(loss, dq, dd, scores)
    coltrast_loss(Q, D, off, pos, scale)          -> loss with autograd to Q and D
    coltrast_total_loss_fwd_bwd(Q, D, off, pos, scale, tau)
                                                  -> dict(loss [3]: L, L_LI, L_C; dq, dd)
    coltrast_total_loss(Q, D, off, pos, scale, tau) -> L with autograd to Q and D
    dense_ip_topk(Q, X, k)                        -> (scores fp32 [nq, k], idx int64 [nq, k])
    semantic_chunk(E, paper_off, threshold)       -> dict(seg int32 [n], n_segments, cos)
    retrieval_metrics(idx, positive, k)           -> dict(p_at_k, mrr_at_k, ranks) on the device
    csr_validate(off, n_tok)                      -> (status name, first bad document or -1)

Q and D are bf16 CUDA tensors ([nq, lq, dim] and [n_tok, dim]); off is int64 [n_docs + 1];
pos is int32 [nq]; Q and X of dense_ip_topk are fp16 [nq, dim] and [n, dim].  A valid CSR is a
precondition of the MaxSim calls (the library never reads the offsets on the host); with the
environment variable HPR_VALIDATE=1 every MaxSim call first checks it with csr_validate (one
synchronisation) and raises HprError on an invalid one.
"""

import ctypes
import os

import torch

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG_DIR, "libhiperrag.so")

STATUS_NAMES = {
    0: "HPR_OK",
    1: "HPR_ERR_INVALID_ARG",
    2: "HPR_ERR_BAD_CSR",
    3: "HPR_ERR_EMPTY_DOC",
    4: "HPR_ERR_UNSUPPORTED_SHAPE",
    5: "HPR_ERR_WORKSPACE_TOO_SMALL",
    6: "HPR_ERR_CAPACITY",
    7: "HPR_ERR_HIP",
}


class HprError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.status_name = STATUS_NAMES.get(status, str(status))


_lib = None

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_F32 = ctypes.c_float

_SIGNATURES = {
    "maxsim_score": (_I32, [_P, _I32, _I32, _P, _P, _I64, _I64, _I32, _P, _P, _SZ, _P]),
    "maxsim_score_noalloc": (_I32, [_P, _I32, _I32, _P, _P, _I64, _I64, _I32, _P, _P]),
    "maxsim_topk": (_I32, [_P, _I32, _I32, _P, _P, _I64, _I64, _I32, _I32, _P, _P, _P, _SZ, _P]),
    "coltrast_loss_fwd_bwd": (_I32, [_P, _I32, _I32, _P, _P, _I64, _I64, _I32, _P, _F32,
                                     _P, _P, _P, _P, _P, _SZ, _P]),
    "coltrast_total_loss_fwd_bwd": (_I32, [_P, _I32, _I32, _P, _P, _I64, _I64, _I32, _P, _F32,
                                           _F32, _P, _P, _P, _P, _SZ, _P]),
    "dense_ip_topk": (_I32, [_P, _I32, _P, _I64, _I32, _I32, _P, _P, _P, _SZ, _P]),
    "maxsim_score_workspace_size": (_SZ, [_I32, _I32, _I64, _I64, _I32]),
    "maxsim_topk_workspace_size": (_SZ, [_I32, _I32, _I64, _I64, _I32, _I32]),
    "coltrast_loss_workspace_size": (_SZ, [_I32, _I32, _I64, _I64, _I32]),
    "coltrast_total_loss_workspace_size": (_SZ, [_I32, _I32, _I64, _I64, _I32]),
    "dense_ip_topk_workspace_size": (_SZ, [_I32, _I64, _I32, _I32]),
    "semantic_chunk": (_I32, [_P, _I64, _I32, _P, _I64, _F32, _P, _P, _P, _P, _SZ, _P]),
    "semantic_chunk_workspace_size": (_SZ, [_I64, _I32]),
    "retrieval_metrics": (_I32, [_P, _I32, _I32, _I32, _P, _P, _P, _P]),
    "hpr_mfma_calibration": (_I32, [_I64, _I32, _P, ctypes.POINTER(ctypes.c_double), _P]),
    "hpr_read_calibration": (_I32, [_P, _I64, _P, _P]),
    "hpr_csr_validate": (_I32, [_P, _I64, _I64, _P, _P, _P]),
    "hpr_scale_f32": (_I32, [_P, _I64, _P, _P]),
    "hpr_kernel_timing": (_I32, [_I32]),
    "hpr_kernel_timing_read": (_I32, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_int64)]),
    "hpr_status_string": (ctypes.c_char_p, [_I32]),
    "hpr_last_error": (ctypes.c_char_p, []),
    "hpr_abi_version": (_I32, []),
}


def lib():
    """The loaded shared library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2505_04846_amd.build` "
                "(there is no fallback implementation)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(status):
    if status != 0:
        raise HprError(status, lib().hpr_last_error().decode())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _need(t, name, dtype, ndim, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got {t.dim()}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _workspace(nbytes, device):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _maxsim_inputs(Q, D, off):
    _need(Q, "Q", torch.bfloat16, 3)
    dev = Q.device
    _need(D, "D", torch.bfloat16, 2, dev)
    _need(off, "off", torch.int64, 1, dev)
    nq, lq, dim = Q.shape
    if D.shape[1] != dim:
        raise ValueError(f"D has dim {D.shape[1]}, Q has {dim}")
    if os.environ.get("HPR_VALIDATE") == "1":  # debugging aid: checks the CSR, synchronising
        status, doc = csr_validate(off, D.shape[0])
        if status != "HPR_OK":
            raise HprError({v: k for k, v in STATUS_NAMES.items()}[status],
                           f"invalid CSR offsets (first bad document {doc})")
    return dev, nq, lq, dim, off.numel() - 1, D.shape[0]


def maxsim_score(Q, D, off, ws=None):
    dev, nq, lq, dim, n_docs, n_tok = _maxsim_inputs(Q, D, off)
    L = lib()
    need = L.maxsim_score_workspace_size(nq, lq, n_docs, n_tok, dim)
    ws = ws if ws is not None and ws.numel() >= need else _workspace(need, dev)
    scores = torch.empty((nq, n_docs), dtype=torch.float32, device=dev)
    with torch.cuda.device(dev):
        _check(L.maxsim_score(_ptr(Q), nq, lq, _ptr(D), _ptr(off), n_docs, n_tok, dim,
                              _ptr(scores), _ptr(ws), ws.numel(), _stream(dev)))
    return scores


def maxsim_score_noalloc(Q, D, off, out=None):
    """maxsim_score through the entry point that allocates no device memory (its scratch is a
    static array of the library); `out` may be a preallocated fp32 [nq, n_docs] tensor."""
    dev, nq, lq, dim, n_docs, n_tok = _maxsim_inputs(Q, D, off)
    scores = out if out is not None else torch.empty((nq, n_docs), dtype=torch.float32,
                                                     device=dev)
    _need(scores, "out", torch.float32, 2, dev)
    if tuple(scores.shape) != (nq, n_docs):
        raise ValueError(f"out must be [{nq}, {n_docs}]")
    with torch.cuda.device(dev):
        _check(lib().maxsim_score_noalloc(_ptr(Q), nq, lq, _ptr(D), _ptr(off), n_docs, n_tok, dim,
                                          _ptr(scores), _stream(dev)))
    return scores


def maxsim_topk(Q, D, off, k, ws=None):
    dev, nq, lq, dim, n_docs, n_tok = _maxsim_inputs(Q, D, off)
    L = lib()
    need = L.maxsim_topk_workspace_size(nq, lq, n_docs, n_tok, dim, k)
    ws = ws if ws is not None and ws.numel() >= need else _workspace(need, dev)
    out_s = torch.empty((nq, k), dtype=torch.float32, device=dev)
    out_i = torch.empty((nq, k), dtype=torch.int64, device=dev)
    with torch.cuda.device(dev):
        _check(L.maxsim_topk(_ptr(Q), nq, lq, _ptr(D), _ptr(off), n_docs, n_tok, dim, int(k),
                             _ptr(out_s), _ptr(out_i), _ptr(ws), ws.numel(), _stream(dev)))
    return out_s, out_i


def coltrast_workspace(Q, D, off):
    dev, nq, lq, dim, n_docs, n_tok = _maxsim_inputs(Q, D, off)
    return _workspace(lib().coltrast_loss_workspace_size(nq, lq, n_docs, n_tok, dim), dev)


def coltrast_loss_fwd_bwd(Q, D, off, pos, logit_scale, need_dq=True, need_dd=True,
                          return_scores=False, ws=None, out=None):
    """Loss (fp32 [1]), dQ (fp32 like Q or None), dD (fp32 like D or None), scores or None.

    `out` may hold preallocated outputs {"loss", "dq", "dd", "scores"} (reused as given).
    """
    dev, nq, lq, dim, n_docs, n_tok = _maxsim_inputs(Q, D, off)
    _need(pos, "pos", torch.int32, 1, dev)
    if pos.numel() != nq:
        raise ValueError("pos must hold one positive per query")
    L = lib()
    need = L.coltrast_loss_workspace_size(nq, lq, n_docs, n_tok, dim)
    ws = ws if ws is not None and ws.numel() >= need else _workspace(need, dev)
    out = {} if out is None else out
    loss = out.get("loss")
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=dev)
    dq = out.get("dq") if need_dq else None
    if need_dq and dq is None:
        dq = torch.empty(Q.shape, dtype=torch.float32, device=dev)
    dd = out.get("dd") if need_dd else None
    if need_dd and dd is None:
        dd = torch.empty(D.shape, dtype=torch.float32, device=dev)
    scores = out.get("scores") if return_scores else None
    if return_scores and scores is None:
        scores = torch.empty((nq, n_docs), dtype=torch.float32, device=dev)
    with torch.cuda.device(dev):
        _check(L.coltrast_loss_fwd_bwd(_ptr(Q), nq, lq, _ptr(D), _ptr(off), n_docs, n_tok, dim,
                                       _ptr(pos), float(logit_scale), _ptr(loss), _ptr(dq),
                                       _ptr(dd), _ptr(scores), _ptr(ws), ws.numel(),
                                       _stream(dev)))
    return {"loss": loss, "dq": dq, "dd": dd, "scores": scores}


def coltrast_total_workspace(Q, D, off):
    dev, nq, lq, dim, n_docs, n_tok = _maxsim_inputs(Q, D, off)
    return _workspace(lib().coltrast_total_loss_workspace_size(nq, lq, n_docs, n_tok, dim), dev)


def coltrast_total_loss_fwd_bwd(Q, D, off, pos, logit_scale, temperature, need_dq=True,
                                need_dd=True, ws=None, out=None):
    """Loss (fp32 [3]: L, L_LI, L_C), dQ (fp32 like Q or None), dD (fp32 like D or None).

    `out` may hold preallocated outputs {"loss", "dq", "dd"} (reused as given).
    """
    dev, nq, lq, dim, n_docs, n_tok = _maxsim_inputs(Q, D, off)
    _need(pos, "pos", torch.int32, 1, dev)
    if pos.numel() != nq:
        raise ValueError("pos must hold one positive per query")
    L = lib()
    need = L.coltrast_total_loss_workspace_size(nq, lq, n_docs, n_tok, dim)
    ws = ws if ws is not None and ws.numel() >= need else _workspace(need, dev)
    out = {} if out is None else out
    loss = out.get("loss")
    if loss is None:
        loss = torch.empty(3, dtype=torch.float32, device=dev)
    dq = out.get("dq") if need_dq else None
    if need_dq and dq is None:
        dq = torch.empty(Q.shape, dtype=torch.float32, device=dev)
    dd = out.get("dd") if need_dd else None
    if need_dd and dd is None:
        dd = torch.empty(D.shape, dtype=torch.float32, device=dev)
    with torch.cuda.device(dev):
        _check(L.coltrast_total_loss_fwd_bwd(_ptr(Q), nq, lq, _ptr(D), _ptr(off), n_docs, n_tok,
                                             dim, _ptr(pos), float(logit_scale),
                                             float(temperature), _ptr(loss), _ptr(dq), _ptr(dd),
                                             _ptr(ws), ws.numel(), _stream(dev)))
    return {"loss": loss, "dq": dq, "dd": dd}


def scale_(x, scale):
    """x *= scale in place (x fp32 contiguous CUDA tensor, scale a 1-element fp32 CUDA tensor)."""
    with torch.cuda.device(x.device):
        _check(lib().hpr_scale_f32(_ptr(x), x.numel(), _ptr(scale), _stream(x.device)))
    return x


class _ColTrastLI(torch.autograd.Function):
    @staticmethod
    def forward(ctx, Q, D, off, pos, logit_scale):
        r = coltrast_loss_fwd_bwd(Q.detach(), D.detach(), off, pos, logit_scale,
                                  need_dq=ctx.needs_input_grad[0],
                                  need_dd=ctx.needs_input_grad[1])
        ctx.save_for_backward(*(t for t in (r["dq"], r["dd"]) if t is not None))
        ctx.has = (r["dq"] is not None, r["dd"] is not None)
        return r["loss"][0]

    @staticmethod
    def backward(ctx, grad_out):
        saved = list(ctx.saved_tensors)
        g = grad_out.reshape(1).to(torch.float32).contiguous()
        dq = saved.pop(0) if ctx.has[0] else None
        dd = saved.pop(0) if ctx.has[1] else None
        # scale copies: the saved gradients stay as the forward left them, so a second backward
        # over a retained graph scales them afresh
        dq = scale_(dq.clone(), g) if dq is not None else None
        dd = scale_(dd.clone(), g) if dd is not None else None
        return dq, dd, None, None, None


def coltrast_loss(Q, D, off, pos, logit_scale):
    """L_LI as a differentiable scalar (gradients reach Q and D)."""
    return _ColTrastLI.apply(Q, D, off, pos, float(logit_scale))


class _ColTrastTotal(torch.autograd.Function):
    @staticmethod
    def forward(ctx, Q, D, off, pos, logit_scale, temperature):
        r = coltrast_total_loss_fwd_bwd(Q.detach(), D.detach(), off, pos, logit_scale,
                                        temperature, need_dq=ctx.needs_input_grad[0],
                                        need_dd=ctx.needs_input_grad[1])
        ctx.save_for_backward(*(t for t in (r["dq"], r["dd"]) if t is not None))
        ctx.has = (r["dq"] is not None, r["dd"] is not None)
        return r["loss"][0]

    @staticmethod
    def backward(ctx, grad_out):
        dq, dd = _ColTrastLI.backward(ctx, grad_out)[:2]
        return dq, dd, None, None, None, None


def coltrast_total_loss(Q, D, off, pos, logit_scale, temperature):
    """The ColTrast loss (L_LI + L_C) / 2 as a differentiable scalar."""
    return _ColTrastTotal.apply(Q, D, off, pos, float(logit_scale), float(temperature))


def dense_ip_topk(Q, X, k, ws=None):
    _need(Q, "Q", torch.float16, 2)
    dev = Q.device
    _need(X, "X", torch.float16, 2, dev)
    nq, dim = Q.shape
    n = X.shape[0]
    if X.shape[1] != dim:
        raise ValueError(f"X has dim {X.shape[1]}, Q has {dim}")
    L = lib()
    need = L.dense_ip_topk_workspace_size(nq, n, dim, k)
    ws = ws if ws is not None and ws.numel() >= need else _workspace(need, dev)
    out_s = torch.empty((nq, k), dtype=torch.float32, device=dev)
    out_i = torch.empty((nq, k), dtype=torch.int64, device=dev)
    with torch.cuda.device(dev):
        _check(L.dense_ip_topk(_ptr(Q), nq, _ptr(X), n, dim, int(k), _ptr(out_s), _ptr(out_i),
                               _ptr(ws), ws.numel(), _stream(dev)))
    return out_s, out_i


def dense_workspace(Q, X, k):
    return _workspace(lib().dense_ip_topk_workspace_size(Q.shape[0], X.shape[0], Q.shape[1], k),
                      Q.device)


def semantic_chunk(E, paper_off, threshold, return_cos=False, ws=None, out=None):
    """Segment ids of fp16 sentence embeddings E [n, dim] (paper_off int64 [n_papers + 1] or
    None for one paper).  Returns dict(seg int32 [n], n_segments int64 [1], cos fp32 [n] or None),
    all on the device.  `out` may hold preallocated {"seg", "n_segments", "cos"}."""
    _need(E, "E", torch.float16, 2)
    dev = E.device
    n, dim = E.shape
    n_papers = 0
    if paper_off is not None:
        _need(paper_off, "paper_off", torch.int64, 1, dev)
        n_papers = paper_off.numel() - 1
    L = lib()
    need = L.semantic_chunk_workspace_size(n, dim)
    ws = ws if ws is not None and ws.numel() >= need else _workspace(need, dev)
    out = {} if out is None else out
    seg = out.get("seg")
    if seg is None:
        seg = torch.empty(n, dtype=torch.int32, device=dev)
    n_seg = out.get("n_segments")
    if n_seg is None:
        n_seg = torch.empty(1, dtype=torch.int64, device=dev)
    cos = out.get("cos") if return_cos else None
    if return_cos and cos is None:
        cos = torch.empty(n, dtype=torch.float32, device=dev)
    with torch.cuda.device(dev):
        _check(L.semantic_chunk(_ptr(E), n, dim, _ptr(paper_off), n_papers, float(threshold),
                                _ptr(cos), _ptr(seg), _ptr(n_seg), _ptr(ws), ws.numel(),
                                _stream(dev)))
    return {"seg": seg, "n_segments": n_seg, "cos": cos}


def semantic_chunk_workspace(E):
    return _workspace(lib().semantic_chunk_workspace_size(E.shape[0], E.shape[1]), E.device)


def retrieval_metrics(idx, positive, k=None):
    """P@k and MRR@k of index lists idx int64 [nq, ld] against positive int64 [nq].  Returns
    dict(metrics fp64 [2] = (P@k, MRR@k), ranks int32 [nq]) on the device."""
    _need(idx, "idx", torch.int64, 2)
    dev = idx.device
    _need(positive, "positive", torch.int64, 1, dev)
    nq, ld = idx.shape
    k = ld if k is None else int(k)
    if positive.numel() != nq:
        raise ValueError("positive must hold one index per query")
    metrics = torch.empty(2, dtype=torch.float64, device=dev)
    ranks = torch.empty(nq, dtype=torch.int32, device=dev)
    with torch.cuda.device(dev):
        _check(lib().retrieval_metrics(_ptr(idx), nq, ld, k, _ptr(positive), _ptr(ranks),
                                       _ptr(metrics), _stream(dev)))
    return {"metrics": metrics, "ranks": ranks}


def calibrate(device="cuda:0", mfma_iters=20000, read_bytes=16 << 30, reps=3):
    """Measured ceilings of this device: bf16 MFMA TFLOP/s on a fixed low-entropy operand
    pattern and on random embedding-sized operands, and the HBM read rate in GB/s; each the
    best of `reps` timed launches of the library's calibration kernels on the current stream."""
    dev = torch.device(device)
    L = lib()
    sink_f = torch.empty(4096, dtype=torch.float32, device=dev)
    sink_u = torch.empty(16384, dtype=torch.int32, device=dev)
    buf = torch.ones(read_bytes // 4, dtype=torch.float32, device=dev)
    flops = ctypes.c_double(0.0)
    best = [0.0, 0.0, 0.0]
    with torch.cuda.device(dev):
        s = _stream(dev)

        def timed(launch):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            launch()
            b.record()
            b.synchronize()
            return a.elapsed_time(b) * 1e-3

        for rep in range(reps + 1):  # the first of each is a warm-up
            for operands in (0, 1):
                t = timed(lambda: _check(L.hpr_mfma_calibration(
                    mfma_iters, operands, _ptr(sink_f), ctypes.byref(flops), s)))
                if rep:
                    best[operands] = max(best[operands], flops.value / t / 1e12)
            t = timed(lambda: _check(L.hpr_read_calibration(_ptr(buf), buf.numel() * 4,
                                                            _ptr(sink_u), s)))
            if rep:
                best[2] = max(best[2], buf.numel() * 4 / t / 1e9)
    del buf
    return tuple(best)


def kernel_timing(enable):
    """Turns per-kernel HIP-event timing inside the library on or off."""
    _check(lib().hpr_kernel_timing(1 if enable else 0))


def kernel_timing_read(name):
    """(total milliseconds, launches) recorded for kernel `name` since the last read."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib().hpr_kernel_timing_read(name.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def csr_validate(off, n_tok):
    """Checks CSR offsets on the device (synchronises).  Returns (status name, first bad doc)."""
    _need(off, "off", torch.int64, 1)
    ws = _workspace(16, off.device)
    bad = ctypes.c_int64(-1)
    with torch.cuda.device(off.device):
        st = lib().hpr_csr_validate(_ptr(off), off.numel() - 1, int(n_tok), _ptr(ws),
                                    _stream(off.device), ctypes.byref(bad))
    if st not in (0, 2, 3):
        _check(st)
    return STATUS_NAMES[st], bad.value
