"""Seeded synthetic inputs for the MaxSim / InfoNCE / top-k path.

This module is shared by the tests, the benchmark and the smoke check.  It holds input
generation only (random draws, L2 normalisation, rounding to the storage dtype, CSR layout) and
none of the method's arithmetic.  Everything is generated with torch on the requested device
from `torch.Generator`s seeded per stream, so a (seed, device) pair always yields the same
bits; CPU and GPU generators are different streams, so a workload is generated on one device and
copied where it is needed.

Streams (each its own generator, seeded with seed * 1000 + stream):
  1 query tokens, 2 document tokens, 3 document lengths, 4 positive/negative noise,
  5 positions and subsets, 6 clone noise, 7 planted orthogonal noise.

Workloads (sizes are the defaults; every generator takes smaller sizes for parity runs):
  tiny_maxsim      8 queries x 32 tokens, 256 docs x 64 tokens, dim 128, top-10
  coltrast_step    64 queries x 32 tokens; 512 docs x 256 tokens; doc 8q is query q's positive,
                   docs 8q+1..8q+7 its hard negatives; dim 128
  li_retrieval     1,024 queries x 32 tokens vs 500,000 docs, Ld uniform in [32, 384], top-100
  dense_retrieval  4,096 queries vs 10,000,000 rows, dim 4096, fp16, 1,000 planted rows at
                   cosine 0.95 to 1,000 distinct queries, top-100
  li_large         4,096 queries x 64 tokens vs 1,000,000 docs, Ld lognormal (median 200,
                   sigma 0.5) clipped to [16, 512], 10 % of docs noisy clones, top-1000
  sentence_stream  10,000 papers of 50..350 sentence embeddings (dim 4096, fp16) whose topic
                   changes after a geometric number of sentences (mean 8), for semantic chunking
"""

import math

import torch

__all__ = [
    "stream_gen",
    "unit_rows",
    "csr_offsets",
    "tiny_maxsim",
    "coltrast_step",
    "li_retrieval",
    "dense_retrieval",
    "li_large",
    "sentence_stream",
]

_CHUNK_ROWS = 1 << 22


def stream_gen(seed, stream, device):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000 + int(stream))
    return g


def _normalise(x):
    return x / torch.linalg.vector_norm(x, dim=-1, keepdim=True).clamp_min(1e-30)


def unit_rows(n, dim, gen, device, dtype, chunk_rows=_CHUNK_ROWS):
    """n rows of N(0, I) fp32 draws, each L2-normalised in fp32 and rounded (RNE) to `dtype`."""
    out = torch.empty((n, dim), dtype=dtype, device=device)
    for r0 in range(0, n, chunk_rows):
        r1 = min(n, r0 + chunk_rows)
        raw = torch.randn((r1 - r0, dim), generator=gen, device=device, dtype=torch.float32)
        out[r0:r1] = _normalise(raw).to(dtype)
    return out


def csr_offsets(lengths):
    lengths = lengths.to(torch.int64)
    off = torch.zeros(lengths.numel() + 1, dtype=torch.int64, device=lengths.device)
    off[1:] = torch.cumsum(lengths, 0)
    return off


def tiny_maxsim(seed=0, device="cpu", nq=8, lq=32, n_docs=256, ld=64, dim=128, k=10):
    """Uniform-length workload; also returns the fp32 tokens the bf16 ones were rounded from."""
    gq = stream_gen(seed, 1, device)
    gd = stream_gen(seed, 2, device)
    q32 = unit_rows(nq * lq, dim, gq, device, torch.float32).reshape(nq, lq, dim)
    d32 = unit_rows(n_docs * ld, dim, gd, device, torch.float32)
    off = torch.arange(0, (n_docs + 1) * ld, ld, dtype=torch.int64, device=device)
    return {
        "Q": q32.to(torch.bfloat16), "D": d32.to(torch.bfloat16), "off": off, "k": k,
        "Q_f32": q32, "D_f32": d32,
    }


def coltrast_step(seed=0, device="cpu", nq=64, lq=32, n_neg=7, ld=256, dim=128,
                  sigma0=0.3, sigma_step=0.05):
    """In-batch training batch: (1 positive + n_neg hard negatives) docs per query.

    Doc (n_neg+1)*q + h (h = 0 positive, h >= 1 hard negative) holds, in lq distinct random
    slots, normalise(q_raw[i] + sigma_h * eps) with sigma_h = sigma0 + sigma_step * h, where
    q_raw is the query's raw N(0, I) draw; its other slots hold fresh unit Gaussian tokens.
    """
    per_q = n_neg + 1
    n_docs = nq * per_q
    gq = stream_gen(seed, 1, device)
    gd = stream_gen(seed, 2, device)
    gn = stream_gen(seed, 4, device)
    gp = stream_gen(seed, 5, device)
    q_raw = torch.randn((nq, lq, dim), generator=gq, device=device, dtype=torch.float32)
    Q = _normalise(q_raw).to(torch.bfloat16)
    D = unit_rows(n_docs * ld, dim, gd, device, torch.bfloat16).reshape(n_docs, ld, dim)
    if lq > ld:
        raise ValueError("each doc needs room for the query's lq planted tokens")
    for q in range(nq):
        for h in range(per_q):
            d = q * per_q + h
            sigma = sigma0 + sigma_step * h
            slots = torch.randperm(ld, generator=gp, device=device)[:lq]
            eps = torch.randn((lq, dim), generator=gn, device=device, dtype=torch.float32)
            D[d, slots] = _normalise(q_raw[q] + sigma * eps).to(torch.bfloat16)
    off = torch.arange(0, (n_docs + 1) * ld, ld, dtype=torch.int64, device=device)
    pos = torch.arange(0, n_docs, per_q, dtype=torch.int32, device=device)
    return {"Q": Q, "D": D.reshape(n_docs * ld, dim), "off": off, "pos": pos}


def li_retrieval(seed=0, device="cpu", nq=1024, lq=32, n_docs=500_000, ld_min=32, ld_max=384,
                 dim=128, k=100):
    """Ragged CSR store, Ld = ld_min + floor(u * (ld_max - ld_min + 1))."""
    gq = stream_gen(seed, 1, device)
    gd = stream_gen(seed, 2, device)
    gl = stream_gen(seed, 3, device)
    u = torch.rand(n_docs, generator=gl, device=device, dtype=torch.float64)
    lengths = ld_min + torch.floor(u * (ld_max - ld_min + 1)).to(torch.int64)
    lengths.clamp_(ld_min, ld_max)
    off = csr_offsets(lengths)
    n_tok = int(off[-1].item())
    Q = unit_rows(nq * lq, dim, gq, device, torch.bfloat16).reshape(nq, lq, dim)
    D = unit_rows(n_tok, dim, gd, device, torch.bfloat16)
    return {"Q": Q, "D": D, "off": off, "k": k}


def dense_retrieval(seed=0, device="cpu", nq=4096, n=10_000_000, dim=4096, k=100,
                    n_planted=1000, cosine=0.95, chunk_rows=1 << 18):
    """fp16 pooled store with planted near-duplicates of queries.

    planted_q[p] and planted_row[p] (distinct queries, distinct rows) are paired:
    X[row] = cosine * qhat + sqrt(1 - cosine^2) * uhat, uhat a unit vector orthogonal to qhat,
    with qhat the query's fp16 value normalised; built in fp64 then rounded to fp16.
    """
    gq = stream_gen(seed, 1, device)
    gd = stream_gen(seed, 2, device)
    gp = stream_gen(seed, 5, device)
    go = stream_gen(seed, 7, device)
    Q = unit_rows(nq, dim, gq, device, torch.float16)
    X = unit_rows(n, dim, gd, device, torch.float16, chunk_rows=chunk_rows)
    n_planted = min(n_planted, nq, n)
    pq = torch.randperm(nq, generator=gp, device=device)[:n_planted]
    pr = torch.randperm(n, generator=gp, device=device)[:n_planted]
    qhat = _normalise(Q[pq].to(torch.float64))
    g = torch.randn((n_planted, dim), generator=go, device=device, dtype=torch.float64)
    g = g - (g * qhat).sum(-1, keepdim=True) * qhat
    uhat = _normalise(g)
    X[pr] = (cosine * qhat + math.sqrt(1.0 - cosine * cosine) * uhat).to(torch.float16)
    return {"Q": Q, "X": X, "k": k, "planted_q": pq, "planted_row": pr, "cosine": cosine}


def li_large(seed=0, device="cpu", nq=4096, lq=64, n_docs=1_000_000, median=200.0, sigma=0.5,
             ld_min=16, ld_max=512, clone_frac=0.10, clone_sigma=0.002, dim=128, k=1000):
    """Lognormal ragged store with noisy clones (near-ties).

    Ld = clip(round(exp(ln(median) + sigma * z)), ld_min, ld_max).  A random clone_frac of the
    docs are clones: each copies the length of a random non-clone source and holds
    normalise(src_token + clone_sigma * eps) for each source token (unit-vector space).
    """
    gq = stream_gen(seed, 1, device)
    gd = stream_gen(seed, 2, device)
    gl = stream_gen(seed, 3, device)
    gp = stream_gen(seed, 5, device)
    gc = stream_gen(seed, 6, device)
    z = torch.randn(n_docs, generator=gl, device=device, dtype=torch.float64)
    lengths = torch.round(torch.exp(math.log(median) + sigma * z)).to(torch.int64)
    lengths.clamp_(ld_min, ld_max)
    n_clones = int(round(clone_frac * n_docs)) if n_docs > 1 else 0
    perm = torch.randperm(n_docs, generator=gp, device=device)
    clones = perm[:n_clones]
    sources_pool = perm[n_clones:]
    src = sources_pool[torch.randint(0, sources_pool.numel(), (n_clones,), generator=gp,
                                     device=device)]
    lengths[clones] = lengths[src]
    off = csr_offsets(lengths)
    n_tok = int(off[-1].item())
    Q = unit_rows(nq * lq, dim, gq, device, torch.bfloat16).reshape(nq, lq, dim)
    D = unit_rows(n_tok, dim, gd, device, torch.bfloat16)
    if n_clones:
        cl_len = lengths[clones]
        # token row indices of every clone token and of its source token, in the same order
        within = torch.arange(int(cl_len.sum().item()), device=device, dtype=torch.int64)
        starts = torch.repeat_interleave(torch.cumsum(cl_len, 0) - cl_len, cl_len)
        within = within - starts
        dst_rows = torch.repeat_interleave(off[clones], cl_len) + within
        src_rows = torch.repeat_interleave(off[src], cl_len) + within
        for c0 in range(0, dst_rows.numel(), _CHUNK_ROWS):
            c1 = min(dst_rows.numel(), c0 + _CHUNK_ROWS)
            base = D[src_rows[c0:c1]].to(torch.float32)
            eps = torch.randn(base.shape, generator=gc, device=device, dtype=torch.float32)
            D[dst_rows[c0:c1]] = _normalise(base + clone_sigma * eps).to(torch.bfloat16)
    return {"Q": Q, "D": D, "off": off, "k": k, "clones": clones, "clone_src": src}


def sentence_stream(seed=0, device="cpu", n_papers=10_000, len_min=50, len_max=350, dim=4096,
                    topic_mean=8.0, sigma=0.5, chunk_rows=1 << 18):
    """Sentence embeddings of consecutive papers (fp16 [n, dim], paper offsets int64).

    Paper lengths are uniform in [len_min, len_max] (stream 3).  Within a paper the topic changes
    after a geometric number of sentences with mean topic_mean (stream 5); every topic is a fresh
    unit vector (stream 1), and a sentence is normalise(topic + sigma * g / sqrt(dim)) with g a
    standard normal draw (stream 2), rounded to fp16.  Consecutive sentences of one topic then
    have cosine ~ 1 / (1 + sigma^2) (0.8 at sigma = 0.5); of different topics ~ 0.
    """
    gl = stream_gen(seed, 3, device)
    gt = stream_gen(seed, 5, device)
    gu = stream_gen(seed, 1, device)
    gn = stream_gen(seed, 2, device)
    u = torch.rand(n_papers, generator=gl, device=device, dtype=torch.float64)
    lens = (len_min + torch.floor(u * (len_max - len_min + 1))).to(torch.int64)
    lens.clamp_(len_min, len_max)
    off = csr_offsets(lens)
    n = int(off[-1].item())
    # topic switch before sentence t (t not a paper start) with probability 1 / topic_mean
    switch = torch.rand(n, generator=gt, device=device) < (1.0 / topic_mean)
    starts = off[:-1]
    switch[starts[starts < n]] = True  # every non-empty paper opens with a new topic
    topic = torch.cumsum(switch.to(torch.int64), 0) - 1
    n_topics = int(topic[-1].item()) + 1
    E = torch.empty((n, dim), dtype=torch.float16, device=device)
    topics = torch.empty((0, dim), dtype=torch.float32, device=device)
    t_lo = 0
    for r0 in range(0, n, chunk_rows):
        r1 = min(n, r0 + chunk_rows)
        t_hi = int(topic[r1 - 1].item()) + 1
        if t_hi > t_lo:  # the topics this chunk introduces, drawn in topic order
            new = _normalise(torch.randn((t_hi - t_lo, dim), generator=gu, device=device,
                                         dtype=torch.float32))
            topics = torch.cat([topics[-1:], new]) if topics.numel() else new
            base = t_lo - (1 if topics.shape[0] > t_hi - t_lo else 0)
            t_lo = t_hi
        tv = topics[topic[r0:r1] - base]
        g = torch.randn((r1 - r0, dim), generator=gn, device=device, dtype=torch.float32)
        E[r0:r1] = _normalise(tv + (sigma / math.sqrt(dim)) * g).to(torch.float16)
    return {"E": E, "paper_off": off, "n_topics": n_topics, "threshold": 0.5}
