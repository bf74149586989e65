// Internal launchers of the library's kernels (host side).  Every launcher enqueues on `stream`
// and returns the hipError_t of the launch; argument validation happens in abi.hip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hpr {

// Per-call scratch layout helpers --------------------------------------------------------------
constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// MaxSim work decomposition ---------------------------------------------------------------------
constexpr int kMaxRanges = 1 << 16;   // upper bound on document ranges (partition table size)

struct MaxsimPlan {
  int ks;          // k-steps of 16 (dim <= 16 * ks)
  int nb;          // 32-slot query blocks per wave
  int wpw;         // waves per workgroup
  int lqp;         // query slots per query (lq rounded up to 32)
  int qpw;         // queries per wave
  int n_qgroups;   // workgroups along the query axis
  int n_ranges;    // document ranges (workgroups along the document axis)
  bool persist;    // score kernel: one range per XCD, one launch of one resident round per pass
                   // of query groups
  int64_t grid;    // workgroups per launch
};

// Returns false when the shape is outside the supported limits.
bool maxsim_plan(int nq, int lq, int64_t n_docs, int64_t n_tok, int dim, bool argmax, int n_cu,
                 MaxsimPlan* plan);

// part[r], r = 0..R: first document of range r (token-balanced, documents never split), the
// range table of the score kernel.  Also zeroes ctrl[0 .. n_ctrl) (if ctrl is non-null).
hipError_t launch_partition(const int64_t* off, int64_t n_docs, int64_t n_tok, int n_ranges,
                            int64_t* part, int32_t* ctrl, int n_ctrl, hipStream_t stream);

// MaxSim scores (and, when amax != nullptr, the lowest-index argmax token per (q, i, d), stored
// as uint16 [n_docs, nq * lq]).  Without amax the kernel reads the range table `part` of
// launch_partition.  With amax it finds its ranges itself (part is not read), zeroes
// ctrl[0 .. n_ctrl) (the control words of the later kernels of the call; ctrl may be null), and
// scores a document longer than 65536 tokens as NaN.
// Launches per call of the score kernel (passes of a persistent plan; 1 otherwise); pass p
// of launch_maxsim scores query groups [p G / 8, (p + 1) G / 8) of a persistent plan.
int maxsim_passes(const MaxsimPlan& plan);
hipError_t launch_maxsim(const MaxsimPlan& plan, int pass, const uint16_t* q, int nq, int lq,
                         const uint16_t* d_tok, const int64_t* off, int64_t n_docs,
                         int64_t n_tok, int dim, const int64_t* part, float* scores,
                         uint16_t* amax, int32_t* ctrl, int n_ctrl, hipStream_t stream);

// CSR validation: writes the lowest offending (doc * 2 + is_empty) into *bad (uint64, ~0 = ok).
hipError_t launch_csr_validate(const int64_t* off, int64_t n_docs, int64_t n_tok,
                               unsigned long long* bad, hipStream_t stream);

// Exact top-k of each row of a [rows, n] fp32 matrix (row stride ld), sorted (score desc,
// index asc).
hipError_t launch_topk_rows(const float* scores, int64_t rows, int64_t n, int64_t ld, int k,
                            float* out_scores, int64_t* out_idx, hipStream_t stream);

// InfoNCE over a [nq, n_docs] score matrix: G (dloss/dS), the loss scalar and an optional copy
// of the scores.  ctrl[0] != 0 (raised earlier) or an out-of-range positive makes the loss NaN;
// ctrl[1] is a completion counter that must be 0 on entry (it is 0 again on exit); terms is
// scratch of nq floats.
// G is multiplied by gw (the loss's weight when it is one term of a weighted sum); *loss is the
// unweighted mean.
hipError_t launch_infonce(const float* S, int nq, int64_t n_docs, const int32_t* pos,
                          float scale, float gw, float* G, float* terms, float* loss,
                          float* scores_out, int32_t* ctrl, hipStream_t stream);

// dQ over `grad_q_ranges` document ranges; part holds grad_q_ranges(...) * nq * lq * dim
// floats of partial sums.  dqc (optional, [nq][dim]) is added to every token row of its query.
// With defer_sum the sum over the ranges is left to launch_grad_d (which must then be given
// part, dq and the same dqc).
int grad_q_ranges(int64_t n_docs, int64_t n_tok, int64_t E, int dim);
hipError_t launch_grad_q(const uint16_t* d_tok, const int64_t* off, int64_t n_docs, int64_t n_tok,
                         int dim, int nq, int lq, const uint16_t* amax, const float* G,
                         float* part, float* dq, bool defer_sum, const float* dqc,
                         hipStream_t stream);

// LDS bytes the dD kernel needs per workgroup in its smallest (256-thread) form for nq queries
// of lq tokens; a call whose value exceeds the CU's 160 KiB cannot run and is rejected on the
// host (nq * lq up to about 15,000).
constexpr int kMaxLdsBytes = 160 * 1024;
int grad_d_lds_bytes(int nq, int lq);

// dD; when dq_part is non-null it also finishes a deferred dQ (sums dq_part's ranges into dq,
// adding dqc); ddc (optional, [n_docs][dim]) is added to every token row of its document.
hipError_t launch_grad_d(const uint16_t* q, const int64_t* off, int64_t n_docs, int64_t n_tok,
                         int dim, int nq, int lq, const uint16_t* amax, const float* G, float* dd,
                         const float* dq_part, float* dq, const float* dqc, const float* ddc,
                         hipStream_t stream);

// Pooled contrastive loss (contrastive.hip).  launch_pool: the unit mean-pooled rows Uq
// [nq][dim], Ud [n_docs][dim] and the gradient scales 1 / (|P| L).  launch_contrastive: the loss
// term per query, dC = w_c dL_C/dc [nq][n_docs], the per-query and per-document gradient parts
// dqc [nq][dim] and ddc [n_docs][dim] (weighted by w_c), and loss[2] = L_C,
// loss[0] = w_li loss[1] + w_c loss[2] (loss[1] written earlier by launch_infonce).
// dim % 8 == 0, dim <= 256.
hipError_t launch_pool(const uint16_t* q, int nq, int lq, const uint16_t* d_tok,
                       const int64_t* off, int64_t n_docs, int64_t n_tok, int dim, float* Uq,
                       float* Ud, float* gsc_q, float* gsc_d, hipStream_t stream);
hipError_t launch_contrastive(const float* Uq, const float* gsc_q, const float* Ud,
                              const float* gsc_d, int nq, int64_t n_docs, int dim,
                              const int32_t* pos, float tau, float w_li, float w_c, float* dC,
                              float* terms, float* dqc, float* ddc, float* loss, int32_t* ctrl,
                              hipStream_t stream);

hipError_t launch_scale(float* x, int64_t n, const float* scale, hipStream_t stream);

// Dense inner-product top-k ----------------------------------------------------------------------
// Rows [0, S) are the exact sample; candidate lists hold `cap` entries per query.
struct DensePlan {
  int64_t S;
  int64_t cap;
};
inline DensePlan dense_plan(int64_t n, int k) {
  DensePlan p;
  const int64_t target = (int64_t)32 * k > 131072 ? (int64_t)32 * k : 131072;
  p.S = n < target ? n : target;
  if (p.S == n) {
    p.cap = 0;
  } else {
    const int64_t expect = ((int64_t)k * (n - p.S) + p.S - 1) / p.S;
    int64_t cap = 4 * expect + 256;
    cap = cap > 1024 ? cap : 1024;
    p.cap = (cap + 63) / 64 * 64;
  }
  return p;
}

// One GEMM launch of dense_ip_topk: the scores of queries q[0 .. nqa) (fp16 [nqa, dim])
// against rows [r0, r1) of x, consumed by the epilogue's mode:
//   0 store:     scores[q * ld + (r - r0)];
//   1 filter:    (score, row) appended to the candidate list of global query
//                g = qmap ? qmap[q] : q when its key is >= the bound (theta[g], tie[g]), i.e.
//                score > theta or (score == theta and row <= tie);
//   2 histogram: for every key >= the bound whose bits above byte `shift / 8` equal
//                prefix[g], bin (key >> shift) & 255 of hist[q] is incremented
//                (key = score key << 32 | ~row).
// With m_dev the launch is a persistent grid over the *m_dev queries (read on the device; qmap
// required; nqa unused), narrow tiles, filter or histogram mode.
struct DenseGemm {
  int mode;
  const uint16_t* q;
  int nqa;
  const int32_t* qmap;
  const int32_t* m_dev;
  const uint16_t* x;
  int64_t r0, r1;
  int dim;
  float* scores;
  int64_t ld;
  const float* theta;
  const int64_t* tie;
  int32_t* count;
  float* cand_s;
  uint32_t* cand_i;
  int64_t cap;
  uint32_t* hist;
  const unsigned long long* prefix;
  int shift;
};
hipError_t launch_dense_gemm(const DenseGemm& g, int n_cu, hipStream_t stream);
// theta[q] = ss[q, k-1], tie[q] = -1, count[q] = 0; *n_queued = 0.
hipError_t launch_dense_init(const float* ss, int nq, int k, float* theta, int64_t* tie,
                             int32_t* count, int32_t* n_queued, hipStream_t stream);
// Final top-k of (sample top-k) U (candidates) for queries 0 .. nq_grid (qsel null) or queued
// queries qsel[b], b < *m_dev (m_dev non-null).  With n_queued non-null, queries whose lists
// overflowed are appended to qlist_out (their bound raised, radix state reset).
hipError_t launch_dense_merge(const float* ss, const int64_t* si, int nq_grid, int k,
                              const int32_t* count, const float* cand_s, const uint32_t* cand_i,
                              int64_t cap, const int32_t* qsel, const int32_t* m_dev,
                              float* out_s, int64_t* out_i, float* theta, int64_t* tie,
                              int32_t* n_queued, int32_t* qlist_out, unsigned long long* prefix,
                              uint32_t* remaining, hipStream_t stream);
// The *m_dev queued queries' rows gathered into qc [m, dim]; their histograms zeroed.
hipError_t launch_dense_fallback_prep(const uint16_t* q, int dim, const int32_t* qlist,
                                      const int32_t* m_dev, uint16_t* qc, uint32_t* hist,
                                      int n_cu, hipStream_t stream);
// One byte (at `shift`) of the exact radix select of each queued query's k-th key; at shift 0
// the bound becomes that key and the list is emptied.
hipError_t launch_dense_radix(const int32_t* m_dev, const int32_t* qlist, int nq_grid, int shift,
                              const float* ss, const int64_t* si, int k, uint32_t* hist,
                              unsigned long long* prefix, uint32_t* remaining, float* theta,
                              int64_t* tie, int32_t* count, hipStream_t stream);

// Semantic chunking (chunking.hip): cos_out [n] (NaN at paper starts), seg [n] segment ids,
// *n_seg the segment count; cnt [chunk_ranges(n)] int32 and base [chunk_ranges(n)] int64 are
// scratch.  off (paper offsets, n_papers + 1 entries) may be null: one paper.  dim % 8 == 0,
// 8 <= dim <= kMaxChunkDim.
constexpr int kMaxChunkDim = 4096;
constexpr int kRowsPerWave = 128;  // sentences per wave range
int64_t chunk_ranges(int64_t n);
hipError_t launch_semantic_chunk(const uint16_t* E, int64_t n, int dim, const int64_t* off,
                                 int64_t n_papers, float thr, float* cos_out, int32_t* cnt,
                                 int64_t* base, int32_t* seg, int64_t* n_seg,
                                 hipStream_t stream);
// P@k and MRR@k (out[0], out[1], fp64) and the 1-based rank of each positive (ranks, may be
// null; 0 when absent) over the first k of the ld-strided index rows.
hipError_t launch_retrieval_metrics(const int64_t* idx, int nq, int64_t ld, int k,
                                    const int64_t* pos, int32_t* ranks, double* out,
                                    hipStream_t stream);

// Calibration (calibration.hip): a pure-MFMA kernel of mfma_calibration_waves(n_cu) waves, each
// running `iters` iterations of four v_mfma_f32_32x32x16_bf16 (sink: at least one float per
// 4-wave workgroup); a pure streaming read of `bytes` (a multiple of 16) with `blocks`
// workgroups (sink: one word per workgroup).
int64_t mfma_calibration_waves(int n_cu);
hipError_t launch_mfma_calibration(float* sink, int64_t iters, int n_cu, bool random_operands,
                                   hipStream_t stream);
hipError_t launch_read_calibration(const void* buf, int64_t bytes, uint32_t* sink, int blocks,
                                   hipStream_t stream);

}  // namespace hpr
