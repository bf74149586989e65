"""Plain fp64 CPU oracle for the ColTrast retrieval path (HiPerRAG, arXiv 2505.04846).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU-baseline leg of the
benchmark may import this package.  The product path (the HIP library and its Python binding)
never imports, calls or links anything here, and nothing here imports the product path.

Every function computes its result straight from the definition it cites, in float64, with no
blocking, fusion or reordering beyond what the definition states.  Inputs arrive as float64
arrays holding the exact real values of the bf16/fp16 bits the GPU reads (see `decode_bf16` and
`decode_fp16`).

Contents
  decode_bf16, decode_fp16     exact widening of 16-bit float bit patterns to float64
  maxsim_scores, maxsim_argmax late-interaction similarity (Sec. 2.2, Sec. 3.2.1, Fig. 3B)
  rank_topk                    exact top-k by (score desc, index asc) (Sec. 2.3 nearest neighbours)
  coltrast_li_loss             InfoNCE over MaxSim scores and its gradients (Sec. 3.2.1, L_LI)
  contrastive_loss             InfoNCE over cosines of mean-pooled embeddings (Sec. 3.2.1, L_C)
  coltrast_total_loss          L = (L_LI + L_C) / 2 and its gradients (Sec. 3.2.1)
  dense_scores, dense_topk     inner-product / cosine retrieval on pooled embeddings (Sec. 3.2.1,
                               Sec. 4.2)
  semantic_segments            semantic chunking boundaries by consecutive-sentence cosine
                               (Sec. 3.2.2)
  retrieval_metrics            P@k and MRR@k of a ranking with one positive per query (Sec. 4.2)

Every function here is pinned by the CPU tests (tests/test_oracle_*.py) against hand-worked
fixtures, closed forms, invariants, brute force on tiny inputs and finite differences.
"""

from .bits import decode_bf16, decode_fp16
from .maxsim import maxsim_scores, maxsim_argmax, rank_topk
from .loss import coltrast_li_loss
from .contrastive import contrastive_loss, coltrast_total_loss, pooled_means
from .dense import dense_scores, dense_topk
from .chunking import (chunk_cosines, semantic_segments, paper_starts, retrieval_ranks,
                       retrieval_metrics)

__all__ = [
    "decode_bf16",
    "decode_fp16",
    "maxsim_scores",
    "maxsim_argmax",
    "rank_topk",
    "coltrast_li_loss",
    "contrastive_loss",
    "coltrast_total_loss",
    "pooled_means",
    "dense_scores",
    "dense_topk",
    "chunk_cosines",
    "semantic_segments",
    "paper_starts",
    "retrieval_ranks",
    "retrieval_metrics",
]
