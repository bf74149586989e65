/*
 * hiperrag.h -- C ABI of the MI355X (gfx950) late-interaction scoring, InfoNCE and exact top-k
 * library.  It implements the data-parallel core of the ColTrast retrieval path of HiPerRAG
 * (arXiv 2505.04846).
 *
 * The operations (see each entry point for its defining passage in the paper):
 *   maxsim_score           late-interaction (MaxSim) scores of every query against every
 *                          document of a CSR token store.
 *   maxsim_topk            exact top-k documents per query under MaxSim.
 *   coltrast_loss_fwd_bwd  in-batch InfoNCE loss over MaxSim scores (the L_LI half of the
 *                          ColTrast loss) with its gradients.
 *   coltrast_total_loss_fwd_bwd
 *                          the whole ColTrast loss (L_LI + L_C) / 2, L_C being a contrastive
 *                          loss on the cosines of mean-pooled embeddings, with its gradients.
 *   dense_ip_topk          exact top-k rows of a pooled-embedding store by inner product
 *                          (= cosine for L2-normalised rows).
 *   semantic_chunk         segment ids of a stream of sentence embeddings cut where the cosine
 *                          of consecutive sentences is not above a threshold.
 *   retrieval_metrics      P@k and MRR@k of retrieved index lists against one positive per
 *                          query.
 *
 * Conventions shared by every entry point
 *   Pointers.  Every array argument is a DEVICE pointer on the current HIP device, owned by
 *     the caller, unless it is marked [host].  bf16 and fp16 values are passed as raw 16-bit
 *     patterns (uint16_t).  `stream` is a hipStream_t passed as void* (NULL = the default
 *     stream).
 *   Layouts.  Row-major and dense.  Queries Q are [nq, lq, dim]; the document store is CSR:
 *     tokens d_tok [n_tok, dim] and offsets d_off [n_docs + 1] (int64), the tokens of
 *     document d being rows d_off[d] .. d_off[d+1]-1.
 *   Asynchrony.  Every compute call only validates its arguments on the host (O(1), no device
 *     reads, no synchronisation) and enqueues kernels on `stream`; results are valid once the
 *     stream has reached that point.  Device faults surface at the caller's next
 *     synchronisation, as in HIP.
 *   Memory.  The library never allocates device memory.  Scratch space comes from the caller as
 *     a workspace `ws` of `ws_bytes` bytes (256-byte aligned), sized by the matching
 *     *_workspace_size() query.  A workspace may be reused by later calls on the same stream;
 *     concurrent calls need distinct workspaces.
 *   Preconditions not checked by the compute calls (checking them would need a device read and
 *     a synchronisation): the CSR offsets are valid (d_off[0] = 0, strictly increasing,
 *     d_off[n_docs] = n_tok, so every document has at least one token; hpr_csr_validate checks
 *     this) and every input value is finite.  Violating them gives unspecified results but no
 *     out-of-bounds access.
 *   Errors.  A status code is returned and no exception crosses the ABI; hpr_last_error()
 *     describes the last non-OK status of the calling thread.
 *   Alignment.  Every device pointer must be 16-byte aligned.
 *   Threads.  Entry points are reentrant.
 */
#ifndef HIPERRAG_H
#define HIPERRAG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t hpr_status;

#define HPR_OK 0
#define HPR_ERR_INVALID_ARG 1         /* NULL pointer, non-positive size, k out of range ...   */
#define HPR_ERR_BAD_CSR 2             /* hpr_csr_validate: offsets not a valid CSR             */
#define HPR_ERR_EMPTY_DOC 3           /* hpr_csr_validate: a document with no token            */
#define HPR_ERR_UNSUPPORTED_SHAPE 4   /* valid, but outside the limits this version supports   */
#define HPR_ERR_WORKSPACE_TOO_SMALL 5 /* ws_bytes below the *_workspace_size() value            */
#define HPR_ERR_CAPACITY 6            /* reserved: no entry point of this version returns it    */
#define HPR_ERR_HIP 7                 /* a HIP runtime call or kernel launch failed             */

#define HPR_ABI_VERSION 1

/* Shape limits of this version (HPR_ERR_UNSUPPORTED_SHAPE beyond them).
 *   MaxSim calls: dim % 8 == 0, 8 <= dim <= 256; lq <= 128 when dim <= 128, lq <= 64 when
 *     dim <= 256; coltrast_loss_fwd_bwd: lq <= 64 when dim <= 128, lq <= 32 when dim <= 256;
 *     n_tok < 2^31 (a store of 2^31 bf16 tokens of dim 128 would not fit one GPU's HBM).
 *   Top-k: 1 <= k <= min(n, 1024) (k outside that range is HPR_ERR_INVALID_ARG).
 *   coltrast_loss_fwd_bwd and coltrast_total_loss_fwd_bwd: the same lq limits, nq * lq <= 16384;
 *     with dd requested also 10 * nq * lq + 4 * nq (nq <= 4096; else 0) + 10244 <= 163840 (the
 *     dD kernel's LDS per workgroup against a CU's 160 KiB: nq * lq up to about 15,000); and
 *     every document has at most 65536 tokens (the latter is checked on the device: a
 *     longer document scores NaN, which makes the loss NaN).
 *   dense_ip_topk: dim % 8 == 0, 8 <= dim <= 8192; n < 2^31.
 *   semantic_chunk: dim % 8 == 0, 8 <= dim <= 4096; 1 <= n < 2^31.
 */

/* ---------------------------------------------------------------------------------------------
 * maxsim_score -- late-interaction (MaxSim) scores.
 *
 * Defined by the late-interaction mechanism (Sec. 2.2, and Sec. 3.2.1 with Fig. 3B): every query
 * token is compared with every token of the document, keeps its largest inner product, and the
 * per-token maxima are summed over the query tokens:
 *     scores[q * n_docs + d] = sum_{i < lq} max_{d_off[d] <= j < d_off[d+1]} <Q[q,i,:], D[j,:]>
 * Arithmetic: bf16 x bf16 products accumulated in fp32 (MFMA); max and sum in fp32; the sum
 * over i is taken in a fixed order, so results are bit-reproducible and do not depend on the
 * order of a document's tokens.
 *
 *   q      bf16 [nq, lq, dim]        query token embeddings
 *   d_tok  bf16 [n_tok, dim]         document token embeddings (CSR rows)
 *   d_off  int64 [n_docs + 1]        CSR offsets
 *   scores fp32 [nq, n_docs]         output, fully overwritten
 *   ws     workspace of maxsim_score_workspace_size(...) bytes
 * ------------------------------------------------------------------------------------------- */
hpr_status maxsim_score(const uint16_t* q, int32_t nq, int32_t lq,
                        const uint16_t* d_tok, const int64_t* d_off, int64_t n_docs,
                        int64_t n_tok, int32_t dim, float* scores,
                        void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------------
 * maxsim_score_noalloc -- maxsim_score for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid allocation): no workspace
 * argument, and no hipMalloc, hipFree or allocating library routine on any path.
 *
 * Same arguments, results (bit for bit) and kernels as maxsim_score, except that the scratch
 * (the document-range table, at most 65,536 ranges) lives in a static device array of
 * 65,537 int64 (512 KiB + 8 bytes) that each GPU the library runs on holds until the process
 * ends.  Every call on a GPU shares that GPU's array, so calls that overlap on one GPU (on
 * different streams or host threads) race and give unspecified scores; calls in order on one
 * stream are safe.  The array's address is looked up on the first call on each device.
 *
 *   Returns HPR_ERR_UNSUPPORTED_SHAPE if a shape would need more ranges than the array holds
 *   (the range count is capped at 65,536, so this does not happen for any accepted shape).
 * ------------------------------------------------------------------------------------------- */
hpr_status maxsim_score_noalloc(const uint16_t* q, int32_t nq, int32_t lq,
                                const uint16_t* d_tok, const int64_t* d_off, int64_t n_docs,
                                int64_t n_tok, int32_t dim, float* scores, void* stream);

/* ---------------------------------------------------------------------------------------------
 * maxsim_topk -- exact top-k documents of each query under MaxSim.
 *
 * Retrieval returns the IDs of a query's nearest neighbours in the chunk store (Sec. 2.3);
 * scored here with the late-interaction score of maxsim_score, over every document (exact, no
 * candidate pre-filter).  Results per query are sorted by score descending, equal scores by
 * lower document index first (-0.0 and +0.0 are equal).
 *
 *   out_scores fp32 [nq, k]; out_idx int64 [nq, k] (document indices in [0, n_docs)).
 *   ws     workspace of maxsim_topk_workspace_size(...) bytes (it holds the [nq, n_docs] fp32
 *          score matrix).
 * ------------------------------------------------------------------------------------------- */
hpr_status maxsim_topk(const uint16_t* q, int32_t nq, int32_t lq,
                       const uint16_t* d_tok, const int64_t* d_off, int64_t n_docs,
                       int64_t n_tok, int32_t dim, int32_t k,
                       float* out_scores, int64_t* out_idx,
                       void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------------
 * coltrast_loss_fwd_bwd -- in-batch InfoNCE over MaxSim scores, forward and backward.
 *
 * The ColTrast loss is L = (L_LI + L_C) / 2 with L_LI the MaxSim loss of ColBERT applied to the
 * local batch only (Sec. 3.2.1, "Embedding performance: loss function").  This call computes
 * L_LI as a softmax cross-entropy of every query against all n_docs documents of the batch:
 *     l[q,d]  = logit_scale * S[q,d]                       (S as in maxsim_score)
 *     loss    = (1/nq) sum_q ( log sum_d exp(l[q,d]) - l[q, pos_idx[q]] )
 *     G[q,d]  = (logit_scale/nq) * (softmax_d(l[q,:])[d] - [d == pos_idx[q]])
 *     dq[q,i,:] = sum_d G[q,d] * D[a(q,i,d), :]
 *     dd[j,:]   = sum over (q,i,d) with a(q,i,d) = j of G[q,d] * Q[q,i,:]
 * where a(q,i,d) is the lowest-index token of document d attaining query token (q,i)'s maximum.
 * Gradients are with respect to the bf16 inputs taken as real numbers.
 *
 *   pos_idx     int32 [nq], positives; an out-of-range entry makes *loss NaN (device check).
 *   logit_scale the inverse temperature s.
 *   loss        fp32 [1] output (stays on the device).
 *   dq          fp32 [nq, lq, dim] output, or NULL to skip it.
 *   dd          fp32 [n_tok, dim] output (every row written; rows no query token selects are 0),
 *               or NULL to skip it.
 *   scores      fp32 [nq, n_docs] optional copy of S, or NULL.
 *   The dd reduction is deterministic (fixed summation order): repeated calls give identical
 *   bits.
 * ------------------------------------------------------------------------------------------- */
hpr_status coltrast_loss_fwd_bwd(const uint16_t* q, int32_t nq, int32_t lq,
                                 const uint16_t* d_tok, const int64_t* d_off, int64_t n_docs,
                                 int64_t n_tok, int32_t dim,
                                 const int32_t* pos_idx, float logit_scale,
                                 float* loss, float* dq, float* dd, float* scores,
                                 void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------------
 * coltrast_total_loss_fwd_bwd -- the whole ColTrast loss L = (L_LI + L_C) / 2, forward and
 * backward.
 *
 * The paper trains its encoder on the mean of two losses (Sec. 3.2.1, "Embedding performance:
 * loss function"): L_LI, the MaxSim loss of coltrast_loss_fwd_bwd, and L_C, SimCSE's
 * contrastive loss applied to pooled embeddings and compared by cosine (same section,
 * "Similarity metric").  Pooling is the mean over a sequence's tokens, and L_C compares each
 * query with every in-batch document, with the positives of L_LI:
 *     P_q = (1/lq) sum_i Q[q,i,:];   P_d = (1/L_d) sum_{j in d} D[j,:]   (L_d: d's token count)
 *     c[q,d] = <P_q, P_d> / (|P_q| |P_d| temperature)
 *     L_C = (1/nq) sum_q ( log sum_d exp(c[q,d]) - c[q, pos_idx[q]] )
 * The gradients are those of L with respect to the bf16 inputs taken as real numbers: half the
 * gradients of coltrast_loss_fwd_bwd plus half those of L_C, the latter the same for every token
 * of a query (or of a document).  Arithmetic: pooled sums and cosines in fp32, in a fixed order;
 * repeated calls give identical bits.
 *
 *   pos_idx      int32 [nq] positives; an out-of-range entry makes all three losses NaN.
 *   logit_scale  the inverse temperature of L_LI (finite).
 *   temperature  the temperature of L_C (> 0, finite, with a finite fp32 inverse; 0.05 in
 *                SimCSE).
 *   loss         fp32 [3] output: (L, L_LI, L_C) (stays on the device).
 *   dq           fp32 [nq, lq, dim] output, or NULL to skip it.
 *   dd           fp32 [n_tok, dim] output (every row written), or NULL to skip it.
 *   ws           workspace of coltrast_total_loss_workspace_size(...) bytes.
 * A pooled embedding of zero norm (an all-zero query or document) gives NaN.
 * ------------------------------------------------------------------------------------------- */
hpr_status coltrast_total_loss_fwd_bwd(const uint16_t* q, int32_t nq, int32_t lq,
                                       const uint16_t* d_tok, const int64_t* d_off,
                                       int64_t n_docs, int64_t n_tok, int32_t dim,
                                       const int32_t* pos_idx, float logit_scale,
                                       float temperature, float* loss, float* dq, float* dd,
                                       void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------------
 * dense_ip_topk -- exact top-k rows of a pooled-embedding store by inner product.
 *
 * At query time the paper ranks chunks by the cosine between the pooled question embedding and
 * each pooled chunk embedding and returns the nearest neighbours' IDs (Sec. 3.2.1 "Similarity
 * metric"; Sec. 4.2; Sec. 2.3).  For L2-normalised rows the cosine is the inner product:
 *     s[q,n] = <Q[q,:], X[n,:]>  (fp16 x fp16 products, fp32 accumulation)
 * Results are sorted by score descending, equal scores by lower row index first.  Exact for any
 * input (no approximate index): the score matrix is never stored; rows past an exactly scored
 * sample are kept only when they beat the sample's k-th key, and a query whose candidate list
 * overflows the workspace's capacity (adversarial stores: thousands of rows above that key) is
 * finished on the device by a radix select over rescans of the store.  Like every call it is
 * asynchronous (no host synchronisation, no status decided on the device), so it can be
 * captured in a HIP graph; it never returns HPR_ERR_CAPACITY.
 *
 *   q   fp16 [nq, dim]; x fp16 [n, dim]; out_scores fp32 [nq, k]; out_idx int64 [nq, k].
 *   ws  workspace of dense_ip_topk_workspace_size(...) bytes.
 * ------------------------------------------------------------------------------------------- */
hpr_status dense_ip_topk(const uint16_t* q, int32_t nq, const uint16_t* x, int64_t n,
                         int32_t dim, int32_t k, float* out_scores, int64_t* out_idx,
                         void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------------
 * semantic_chunk -- semantic chunking boundaries.
 *
 * The paper chunks each paper's text by walking its encoded sentences in order and growing a
 * segment while the cosine similarity of consecutive sentences stays above a fixed threshold
 * (Sec. 3.2.2, "ColTrast Finetuning Dataset").  Here, for sentence t of the input:
 *     cos[t] = <E[t-1], E[t]> / (|E[t-1]| |E[t]|), NaN when t is the first sentence of its paper
 *     boundary[t] = not (cos[t] > threshold)          (strict; NaN opens a segment)
 *     seg[t] = (number of boundaries at or before t) - 1
 * so the first sentence of every paper, and every sentence after (and of) a zero vector, opens a
 * segment.  Arithmetic: fp16 x fp16 products accumulated in fp32 (v_dot2_f32_f16); the decision
 * compares the fp32 cosine with the fp32 threshold.
 *
 *   emb        fp16 [n, dim] sentence embeddings, papers concatenated in order.
 *   paper_off  int64 [n_papers + 1] paper offsets into the sentences (valid CSR: 0, ..., n;
 *              empty papers allowed), or NULL for a single paper.  Not checked on the device;
 *              invalid offsets give unspecified ids but no out-of-bounds access.
 *   threshold  any non-NaN value.
 *   cos_out    fp32 [n] output of the cosines, or NULL.
 *   seg_out    int32 [n] output: segment ids, 0, 1, ... in sentence order.
 *   n_segments int64 [1] output (device): the number of segments.
 *   ws         workspace of semantic_chunk_workspace_size(n, dim) bytes.
 * ------------------------------------------------------------------------------------------- */
hpr_status semantic_chunk(const uint16_t* emb, int64_t n, int32_t dim, const int64_t* paper_off,
                          int64_t n_papers, float threshold, float* cos_out, int32_t* seg_out,
                          int64_t* n_segments, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------------
 * retrieval_metrics -- P@k and MRR@k of retrieval results with one positive per query.
 *
 * The paper evaluates retrieval by precision P = N_rel / N_ret with N_ret = k, and by
 * MRR@k = (1/N_q) sum_q 1/rank_q, a term being zero when the positive is ranked beyond k
 * (Sec. 4.2, "ColTrast Retrieval Evaluation").  With one positive per query, N_rel is 1 when the
 * positive is among the first k retrieved indices; P@k is averaged over the queries.
 *
 *   topk_idx    int64 [nq, ld] retrieved indices per query, best first (e.g. maxsim_topk's or
 *               dense_ip_topk's out_idx with ld = their k); the first k of each row are used.
 *   positive    int64 [nq] the positive index of each query.
 *   ranks_out   int32 [nq] output: 1-based rank of the positive, 0 when not within k; or NULL.
 *   metrics_out fp64 [2] output (device): P@k, MRR@k (sums in fp64 in a fixed order).
 * No workspace.
 * ------------------------------------------------------------------------------------------- */
hpr_status retrieval_metrics(const int64_t* topk_idx, int32_t nq, int32_t ld, int32_t k,
                             const int64_t* positive, int32_t* ranks_out, double* metrics_out,
                             void* stream);

/* Workspace sizes in bytes for the calls above (0 is a valid size only when stated). */
size_t maxsim_score_workspace_size(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok,
                                   int32_t dim);
size_t maxsim_topk_workspace_size(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok,
                                  int32_t dim, int32_t k);
size_t coltrast_loss_workspace_size(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok,
                                    int32_t dim);
size_t coltrast_total_loss_workspace_size(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok,
                                          int32_t dim);
size_t dense_ip_topk_workspace_size(int32_t nq, int64_t n, int32_t dim, int32_t k);
size_t semantic_chunk_workspace_size(int64_t n, int32_t dim);

/* ---------------------------------------------------------------------------------------------
 * hpr_csr_validate -- checks a CSR offsets array on the device and SYNCHRONISES `stream`.
 *   Returns HPR_OK, HPR_ERR_BAD_CSR (d_off[0] != 0, d_off[n_docs] != n_tok, or a decrease) or
 *   HPR_ERR_EMPTY_DOC (two equal neighbours).  *h_first_bad_doc [host] receives the lowest
 *   offending document index, or -1.  ws needs 16 bytes.
 * ------------------------------------------------------------------------------------------- */
hpr_status hpr_csr_validate(const int64_t* d_off, int64_t n_docs, int64_t n_tok, void* ws,
                            void* stream, int64_t* h_first_bad_doc);

/* hpr_scale_f32 -- x[i] *= *scale for i < n (scale is a device scalar); used to apply an
 * upstream gradient to the gradients of the loss calls without a host round trip. */
hpr_status hpr_scale_f32(float* x, int64_t n, const float* scale, void* stream);

/* Calibration for benchmarks: what the device sustains, to report beside the published peaks.
 *   hpr_mfma_calibration  launches a kernel of 8 waves per CU, each running `iters` iterations
 *                         of four independent v_mfma_f32_32x32x16_bf16 on register operands (no
 *                         memory traffic); *flops [host] receives its FLOP count.  operands: 0 =
 *                         a fixed low-entropy bit pattern, 1 = random bf16 values of the size of
 *                         unit-vector components (the matrix cores' sustained rate depends on
 *                         the operands' bits; 1 is the ceiling for embeddings).  sink: device
 *                         fp32 [4096] scratch.  Time it on `stream` (or with
 *                         hpr_kernel_timing_read("mfma_calibration")).
 *   hpr_read_calibration  streams `bytes` (a positive multiple of 16) of device memory at `buf`
 *                         with 16-byte loads.  sink: device uint32 [16384] scratch.  Timing
 *                         name "read_calibration". */
hpr_status hpr_mfma_calibration(int64_t iters, int32_t operands, float* sink, double* flops,
                                void* stream);
hpr_status hpr_read_calibration(const void* buf, int64_t bytes, uint32_t* sink, void* stream);

/* Per-kernel timing for benchmarks.  While enabled, every kernel the library launches is
 * bracketed by two HIP events recorded on its launch stream.  hpr_kernel_timing_read
 * synchronises on the events recorded for kernel `name` ("partition", "maxsim",
 * "maxsim_argmax", "topk", "infonce", "pool", "contrastive", "grad_q", "grad_d",
 * "dense_sample", "dense_scan", "dense_merge", "dense_fallback", "semantic_chunk",
 * "retrieval_metrics",
 * "mfma_calibration", "read_calibration"), returns
 * the sum of their durations in milliseconds and the launch count, and forgets them. */
hpr_status hpr_kernel_timing(int32_t enable);
hpr_status hpr_kernel_timing_read(const char* name, double* total_ms, int64_t* launches);

const char* hpr_status_string(hpr_status s);
const char* hpr_last_error(void); /* thread-local description of the last non-OK status */
int32_t hpr_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HIPERRAG_H */
