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
  int ks;          // k-steps of 32 (dim <= 32 * ks)
  int nb;          // 16-column query-slot blocks per wave
  int wpw;         // waves per workgroup
  int lqp;         // query slots per query (lq rounded up to 16)
  int qpw;         // queries per wave
  int n_qgroups;   // workgroups along the query axis
  int n_ranges;    // document ranges (workgroups along the document axis)
};

// Returns false when the shape is outside the supported limits.
bool maxsim_plan(int nq, int lq, int64_t n_docs, int64_t n_tok, int dim, bool argmax, int n_cu,
                 MaxsimPlan* plan);

// part[r], r = 0..R: first document of range r (token-balanced, documents never split).
// Also zeroes ctrl[0] and ctrl[1] (if ctrl is non-null): the error flag and the completion
// counter used by later kernels of the same call.
hipError_t launch_partition(const int64_t* off, int64_t n_docs, int64_t n_tok, int n_ranges,
                            int64_t* part, int32_t* ctrl, hipStream_t stream);

// MaxSim scores (and, when amax != nullptr, the lowest-index argmax token per (q, i, d), stored
// as uint16 [n_docs, nq * lq]; a document longer than 65536 tokens raises *flag).
hipError_t launch_maxsim(const MaxsimPlan& plan, const uint16_t* q, int nq, int lq,
                         const uint16_t* d_tok, const int64_t* off, int64_t n_docs,
                         int64_t n_tok, int dim, const int64_t* part, float* scores,
                         uint16_t* amax, int32_t* flag, hipStream_t stream);

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
hipError_t launch_infonce(const float* S, int nq, int64_t n_docs, const int32_t* pos,
                          float scale, float* G, float* terms, float* loss, float* scores_out,
                          int32_t* ctrl, hipStream_t stream);

hipError_t launch_grad_q(const uint16_t* d_tok, const int64_t* off, int64_t n_docs, int64_t n_tok,
                         int dim, int nq, int lq, const uint16_t* amax, const float* G, float* dq,
                         hipStream_t stream);

hipError_t launch_grad_d(const uint16_t* q, const int64_t* off, int64_t n_docs, int64_t n_tok,
                         int dim, int nq, int lq, const uint16_t* amax, const float* G, float* dd,
                         hipStream_t stream);

hipError_t launch_scale(float* x, int64_t n, const float* scale, hipStream_t stream);

}  // namespace hpr
