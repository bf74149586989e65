// C ABI of the library: host-side argument validation, workspace carving and kernel dispatch.
// Validation never touches the device, so every error path below runs without a GPU.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "hiperrag.h"
#include "kernels.h"

using namespace hpr;

namespace {

thread_local std::string g_last_error;

hpr_status fail(hpr_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

hpr_status hip_fail(hipError_t e, const char* where) {
  return fail(HPR_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int kMaxDevices = 64;
std::atomic<int> g_cu_count[kMaxDevices];

// Compute-unit count of the current device (cached per device).
hpr_status current_cu_count(int* n_cu) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev >= 0 && dev < kMaxDevices) {
    const int c = g_cu_count[dev].load(std::memory_order_relaxed);
    if (c > 0) {
      *n_cu = c;
      return HPR_OK;
    }
  }
  int c = 0;
  e = hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  if (dev >= 0 && dev < kMaxDevices) g_cu_count[dev].store(c, std::memory_order_relaxed);
  *n_cu = c;
  return HPR_OK;
}

// Scratch of maxsim_score_noalloc: the score kernel's document-range table (at most kMaxRanges
// ranges, kMaxRanges + 1 int64 entries: 512 KiB + 8 bytes), one copy per GPU, held until the
// process ends.  Host code never uses `scratch` itself as an address: each device's address is
// looked up once (hipGetSymbolAddress, with that device current) and kept in g_scratch_ptr.
constexpr size_t kScratchEntries = (size_t)kMaxRanges + 1;
static __device__ __align__(256) int64_t scratch[kScratchEntries];
std::mutex g_scratch_mu;
int64_t* g_scratch_ptr[kMaxDevices];

// Device address of the current device's `scratch` (looked up on the first call per device).
hpr_status scratch_address(int64_t** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "device %d beyond the %d devices the library tracks", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(HPR_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = static_cast<int64_t*>(p);
  }
  *out = g_scratch_ptr[dev];
  return HPR_OK;
}

// Optional per-kernel timing: when enabled, every launch made through `timed` is bracketed by
// two HIP events recorded on the launch stream; hpr_kernel_timing_read sums their durations.
std::atomic<int> g_timing_on{0};
std::mutex g_timing_mu;
std::map<std::string, std::vector<std::pair<hipEvent_t, hipEvent_t>>> g_timing;

template <class F>
hipError_t timed(const char* name, hipStream_t s, F&& launch) {
  if (!g_timing_on.load(std::memory_order_relaxed)) return launch();
  hipEvent_t a = nullptr, b = nullptr;
  if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return launch();
  (void)hipEventRecord(a, s);
  const hipError_t e = launch();
  (void)hipEventRecord(b, s);
  std::lock_guard<std::mutex> g(g_timing_mu);
  g_timing[name].emplace_back(a, b);
  return e;
}

// Shared checks of the MaxSim calls (query tensor + CSR store).
hpr_status check_maxsim_args(const uint16_t* q, int32_t nq, int32_t lq, const uint16_t* d_tok,
                             const int64_t* d_off, int64_t n_docs, int64_t n_tok, int32_t dim) {
  if (!q || !d_tok || !d_off) return fail(HPR_ERR_INVALID_ARG, "q, d_tok and d_off must be non-NULL");
  if (nq < 1 || lq < 1) return fail(HPR_ERR_INVALID_ARG, "nq (%d) and lq (%d) must be >= 1", nq, lq);
  if (n_docs < 1) return fail(HPR_ERR_INVALID_ARG, "n_docs (%lld) must be >= 1", (long long)n_docs);
  if (n_tok < n_docs)
    return fail(HPR_ERR_INVALID_ARG, "n_tok (%lld) < n_docs (%lld): every document needs a token",
                (long long)n_tok, (long long)n_docs);
  if (dim < 1) return fail(HPR_ERR_INVALID_ARG, "dim (%d) must be >= 1", dim);
  if (dim % 8 != 0 || dim < 8 || dim > 256)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "MaxSim needs dim %% 8 == 0 and 8 <= dim <= 256 (dim=%d)", dim);
  if ((int64_t)nq * n_docs > (int64_t(1) << 40))
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "nq * n_docs too large");
  if (n_tok >= (int64_t(1) << 31))
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "n_tok must be below 2^31 (got %lld)", (long long)n_tok);
  if (!aligned16(q) || !aligned16(d_tok) || !aligned16(d_off))
    return fail(HPR_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  return HPR_OK;
}

// Query-length limit of the MaxSim kernels (query slots a wave holds).
hpr_status check_lq(int32_t lq, int32_t dim, bool argmax) {
  const int lqp = (lq + 31) / 32 * 32;
  const int max_slots = argmax ? (dim <= 128 ? 64 : 32) : (dim <= 128 ? 128 : 64);
  if (lqp > max_slots)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "lq=%d exceeds the limit %d for dim=%d%s", lq,
                max_slots, dim, argmax ? " in the loss" : "");
  return HPR_OK;
}

// Control words of the loss call: the error flag and the InfoNCE completion counter (both
// zeroed by the MaxSim argmax kernel of the call).
constexpr int kLossCtrlWords = 2;

size_t part_bytes(int64_t n_docs) {
  const int64_t r = n_docs < kMaxRanges ? n_docs : kMaxRanges;
  return align_up((size_t)(r + 1) * sizeof(int64_t));
}

// Carves consecutive 256-byte aligned regions out of a workspace.
struct Carver {
  char* base;
  size_t used = 0;
  explicit Carver(void* ws) : base(static_cast<char*>(ws)) {}
  template <class T>
  T* take(size_t bytes) {
    T* p = reinterpret_cast<T*>(base + used);
    used += align_up(bytes);
    return p;
  }
};

// Score calls: `part` is the range table, of part_bytes bytes; after its n_ranges + 1 entries
// a persistent plan keeps its checkpoint counters (8 per pass) there when they fit.
hpr_status run_maxsim(const uint16_t* q, int32_t nq, int32_t lq, const uint16_t* d_tok,
                      const int64_t* d_off, int64_t n_docs, int64_t n_tok, int32_t dim,
                      float* scores, uint16_t* amax, int32_t* ctrl, int n_ctrl, int64_t* part,
                      size_t part_bytes_avail, hipStream_t stream) {
  int n_cu = 0;
  hpr_status st = current_cu_count(&n_cu);
  if (st != HPR_OK) return st;
  MaxsimPlan plan;
  if (!maxsim_plan(nq, lq, n_docs, n_tok, dim, amax != nullptr, n_cu, &plan))
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "no MaxSim plan for this shape");
  if (!amax && (size_t)(plan.n_ranges + 1) * sizeof(int64_t) > part_bytes_avail)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "%d document ranges exceed the range table",
                plan.n_ranges);
  if (!amax && plan.persist) {
    const size_t used = (size_t)(plan.n_ranges + 1) * sizeof(int64_t);
    const size_t words = (size_t)8 * maxsim_passes(plan);
    if (used + words * sizeof(int32_t) <= part_bytes_avail) {
      ctrl = reinterpret_cast<int32_t*>(part + plan.n_ranges + 1);
      n_ctrl = (int)words;
    }
  }
  hipError_t e = hipSuccess;
  if (!amax) {  // the argmax kernel finds its own ranges (one round of workgroups)
    e = timed("partition", stream, [&] {
      return launch_partition(d_off, n_docs, n_tok, plan.n_ranges, part, ctrl, n_ctrl, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "partition launch");
  }
  for (int pass = 0; pass < maxsim_passes(plan); ++pass) {
    e = timed(amax ? "maxsim_argmax" : "maxsim", stream, [&] {
      return launch_maxsim(plan, pass, q, nq, lq, d_tok, d_off, n_docs, n_tok, dim, part, scores,
                           amax, ctrl, n_ctrl, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "maxsim launch");
  }
  return HPR_OK;
}

// Workspace of the loss calls: S, G, the argmax table, control words, loss
// terms and dQ partial sums; with the contrastive half also the pooled rows and their norms,
// dL_C/dc, its terms and the per-query / per-document gradient parts.
size_t loss_ws_bytes(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok, int32_t dim,
                     bool contrastive) {
  if (nq < 1 || lq < 1 || n_docs < 1 || dim < 1) return 0;
  const size_t sd = align_up((size_t)nq * (size_t)n_docs * sizeof(float));
  const size_t am = align_up((size_t)n_docs * (size_t)nq * (size_t)lq * sizeof(uint16_t));
  const int64_t E = (int64_t)nq * lq;
  const size_t gq = align_up((size_t)grad_q_ranges(n_docs, n_tok, E, dim) * (size_t)E *
                             (size_t)dim * sizeof(float));
  size_t b = 2 * sd + am + align_up((size_t)kLossCtrlWords * sizeof(int32_t)) +
             align_up((size_t)nq * sizeof(float)) + gq;
  if (contrastive) {
    const size_t qd = align_up((size_t)nq * (size_t)dim * sizeof(float));
    const size_t dd = align_up((size_t)n_docs * (size_t)dim * sizeof(float));
    b += 2 * qd + 2 * dd + 2 * align_up((size_t)nq * sizeof(float)) +
         align_up((size_t)n_docs * sizeof(float)) + sd;
  }
  return b;
}

// Both loss calls.  tau > 0 adds the contrastive half: L = w L_LI + w L_C with w = 1/2, loss[0..2]
// = (L, L_LI, L_C); otherwise loss[0] = L_LI.
hpr_status run_loss(const uint16_t* q, int32_t nq, int32_t lq, const uint16_t* d_tok,
                    const int64_t* d_off, int64_t n_docs, int64_t n_tok, int32_t dim,
                    const int32_t* pos_idx, float logit_scale, float tau, float* loss, float* dq,
                    float* dd, float* scores, void* ws, size_t ws_bytes, void* stream) {
  const bool total = tau > 0.f;
  hpr_status st = check_maxsim_args(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim);
  if (st == HPR_OK) st = check_lq(lq, dim, true);
  if (st != HPR_OK) return st;
  if (!pos_idx || !loss || !ws) return fail(HPR_ERR_INVALID_ARG, "pos_idx, loss and ws must be non-NULL");
  if (!(logit_scale == logit_scale) || logit_scale > 3.0e38f || logit_scale < -3.0e38f)
    return fail(HPR_ERR_INVALID_ARG, "logit_scale must be finite");
  if ((int64_t)nq * lq > 16384)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "nq * lq = %lld exceeds 16384", (long long)nq * lq);
  if (dd && grad_d_lds_bytes(nq, lq) > kMaxLdsBytes)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE,
                "dD for nq=%d x lq=%d needs %d bytes of LDS per workgroup, above the CU's %d",
                nq, lq, grad_d_lds_bytes(nq, lq), kMaxLdsBytes);
  if ((dq && !aligned16(dq)) || (dd && !aligned16(dd)))
    return fail(HPR_ERR_INVALID_ARG, "gradient outputs must be 16-byte aligned");
  const size_t need = loss_ws_bytes(nq, lq, n_docs, n_tok, dim, total);
  if (ws_bytes < need)
    return fail(HPR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu < %zu bytes", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(ws);
  float* S = c.take<float>((size_t)nq * n_docs * sizeof(float));
  float* G = c.take<float>((size_t)nq * n_docs * sizeof(float));
  uint16_t* amax = c.take<uint16_t>((size_t)n_docs * nq * lq * sizeof(uint16_t));
  const int n_ctrl = kLossCtrlWords;
  int32_t* ctrl = c.take<int32_t>((size_t)n_ctrl * sizeof(int32_t));
  float* terms = c.take<float>((size_t)nq * sizeof(float));
  float* gq_part = c.take<float>((size_t)grad_q_ranges(n_docs, n_tok, (int64_t)nq * lq, dim) *
                                 (size_t)nq * lq * dim * sizeof(float));
  st = run_maxsim(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim, S, amax, ctrl, n_ctrl, nullptr, 0,
                  s);
  if (st != HPR_OK) return st;
  const float w = total ? 0.5f : 1.0f;
  hipError_t e = timed("infonce", s, [&] {
    return launch_infonce(S, nq, n_docs, pos_idx, logit_scale, w, G, terms, total ? loss + 1 : loss,
                          scores, ctrl, s);
  });
  if (e != hipSuccess) return hip_fail(e, "infonce launch");
  float* dqc = nullptr;
  float* ddc = nullptr;
  if (total) {
    float* Uq = c.take<float>((size_t)nq * dim * sizeof(float));
    float* Ud = c.take<float>((size_t)n_docs * dim * sizeof(float));
    float* gsc_q = c.take<float>((size_t)nq * sizeof(float));
    float* gsc_d = c.take<float>((size_t)n_docs * sizeof(float));
    float* dC = c.take<float>((size_t)nq * n_docs * sizeof(float));
    float* terms_c = c.take<float>((size_t)nq * sizeof(float));
    dqc = c.take<float>((size_t)nq * dim * sizeof(float));
    ddc = c.take<float>((size_t)n_docs * dim * sizeof(float));
    e = timed("pool", s, [&] {
      return launch_pool(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim, Uq, Ud, gsc_q, gsc_d, s);
    });
    if (e != hipSuccess) return hip_fail(e, "pooling launch");
    e = timed("contrastive", s, [&] {
      return launch_contrastive(Uq, gsc_q, Ud, gsc_d, nq, n_docs, dim, pos_idx, tau, w, w, dC,
                                terms_c, dqc, ddc, loss, ctrl, s);
    });
    if (e != hipSuccess) return hip_fail(e, "contrastive launch");
  }
  // With both gradients, the last step of dQ (the sum over its document ranges, plus the
  // contrastive part) rides in the dD launch, saving a kernel launch.
  const bool fold = dq && dd;
  if (dq) {
    e = timed("grad_q", s, [&] {
      return launch_grad_q(d_tok, d_off, n_docs, n_tok, dim, nq, lq, amax, G, gq_part, dq, fold,
                           dqc, s);
    });
    if (e != hipSuccess) return hip_fail(e, "dQ launch");
  }
  if (dd) {
    e = timed("grad_d", s, [&] {
      return launch_grad_d(q, d_off, n_docs, n_tok, dim, nq, lq, amax, G, dd,
                           fold ? gq_part : nullptr, dq, fold ? dqc : nullptr, ddc, s);
    });
    if (e != hipSuccess) return hip_fail(e, "dD launch");
  }
  return HPR_OK;
}

}  // namespace

extern "C" {

size_t maxsim_score_workspace_size(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok,
                                   int32_t dim) {
  (void)nq, (void)lq, (void)n_tok, (void)dim;
  return n_docs < 1 ? 0 : part_bytes(n_docs);
}

size_t maxsim_topk_workspace_size(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok,
                                  int32_t dim, int32_t k) {
  (void)lq, (void)n_tok, (void)dim, (void)k;
  if (nq < 1 || n_docs < 1) return 0;
  return align_up((size_t)nq * (size_t)n_docs * sizeof(float)) + part_bytes(n_docs);
}

size_t coltrast_loss_workspace_size(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok,
                                    int32_t dim) {
  return loss_ws_bytes(nq, lq, n_docs, n_tok, dim, false);
}

size_t coltrast_total_loss_workspace_size(int32_t nq, int32_t lq, int64_t n_docs, int64_t n_tok,
                                          int32_t dim) {
  return loss_ws_bytes(nq, lq, n_docs, n_tok, dim, true);
}

hpr_status maxsim_score(const uint16_t* q, int32_t nq, int32_t lq, const uint16_t* d_tok,
                        const int64_t* d_off, int64_t n_docs, int64_t n_tok, int32_t dim,
                        float* scores, void* ws, size_t ws_bytes, void* stream) {
  hpr_status st = check_maxsim_args(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim);
  if (st == HPR_OK) st = check_lq(lq, dim, false);
  if (st != HPR_OK) return st;
  if (!scores || !ws) return fail(HPR_ERR_INVALID_ARG, "scores and ws must be non-NULL");
  const size_t need = maxsim_score_workspace_size(nq, lq, n_docs, n_tok, dim);
  if (ws_bytes < need)
    return fail(HPR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu < %zu bytes", ws_bytes, need);
  Carver c(ws);
  int64_t* part = c.take<int64_t>(part_bytes(n_docs));
  return run_maxsim(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim, scores, nullptr, nullptr, 0,
                    part, part_bytes(n_docs), static_cast<hipStream_t>(stream));
}

hpr_status maxsim_score_noalloc(const uint16_t* q, int32_t nq, int32_t lq, const uint16_t* d_tok,
                                const int64_t* d_off, int64_t n_docs, int64_t n_tok, int32_t dim,
                                float* scores, void* stream) {
  hpr_status st = check_maxsim_args(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim);
  if (st == HPR_OK) st = check_lq(lq, dim, false);
  if (st != HPR_OK) return st;
  if (!scores) return fail(HPR_ERR_INVALID_ARG, "scores must be non-NULL");
  int n_cu = 0;
  st = current_cu_count(&n_cu);
  if (st != HPR_OK) return st;
  MaxsimPlan plan;
  if (!maxsim_plan(nq, lq, n_docs, n_tok, dim, false, n_cu, &plan))
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "no MaxSim plan for this shape");
  if ((size_t)plan.n_ranges + 1 > kScratchEntries)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "%d document ranges exceed the %zu-entry scratch",
                plan.n_ranges, kScratchEntries - 1);
  int64_t* part = nullptr;
  st = scratch_address(&part);
  if (st != HPR_OK) return st;
  // The same launches as maxsim_score (partition, then the score passes, the checkpoint
  // counters of a persistent plan after the range table), without the timing events.
  int32_t* sync = nullptr;
  int n_sync = 0;
  if (plan.persist && ((size_t)plan.n_ranges + 1) * sizeof(int64_t) +
                              (size_t)8 * maxsim_passes(plan) * sizeof(int32_t) <=
                          sizeof(scratch)) {
    sync = reinterpret_cast<int32_t*>(part + plan.n_ranges + 1);
    n_sync = 8 * maxsim_passes(plan);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_partition(d_off, n_docs, n_tok, plan.n_ranges, part, sync, n_sync, s);
  if (e != hipSuccess) return hip_fail(e, "partition launch");
  for (int pass = 0; pass < maxsim_passes(plan) && e == hipSuccess; ++pass)
    e = launch_maxsim(plan, pass, q, nq, lq, d_tok, d_off, n_docs, n_tok, dim, part, scores,
                      nullptr, sync, n_sync, s);
  return e == hipSuccess ? HPR_OK : hip_fail(e, "maxsim launch");
}

hpr_status maxsim_topk(const uint16_t* q, int32_t nq, int32_t lq, const uint16_t* d_tok,
                       const int64_t* d_off, int64_t n_docs, int64_t n_tok, int32_t dim,
                       int32_t k, float* out_scores, int64_t* out_idx, void* ws,
                       size_t ws_bytes, void* stream) {
  hpr_status st = check_maxsim_args(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim);
  if (st == HPR_OK) st = check_lq(lq, dim, false);
  if (st != HPR_OK) return st;
  if (!out_scores || !out_idx || !ws)
    return fail(HPR_ERR_INVALID_ARG, "out_scores, out_idx and ws must be non-NULL");
  if (k < 1 || k > 1024 || (int64_t)k > n_docs)
    return fail(HPR_ERR_INVALID_ARG, "k=%d must satisfy 1 <= k <= min(n_docs, 1024)", k);
  const size_t need = maxsim_topk_workspace_size(nq, lq, n_docs, n_tok, dim, k);
  if (ws_bytes < need)
    return fail(HPR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu < %zu bytes", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(ws);
  float* scores = c.take<float>((size_t)nq * n_docs * sizeof(float));
  int64_t* part = c.take<int64_t>(part_bytes(n_docs));
  st = run_maxsim(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim, scores, nullptr, nullptr, 0, part,
                  part_bytes(n_docs), s);
  if (st != HPR_OK) return st;
  hipError_t e = timed("topk", s, [&] {
    return launch_topk_rows(scores, nq, n_docs, n_docs, k, out_scores, out_idx, s);
  });
  if (e != hipSuccess) return hip_fail(e, "top-k launch");
  return HPR_OK;
}

hpr_status coltrast_loss_fwd_bwd(const uint16_t* q, int32_t nq, int32_t lq,
                                 const uint16_t* d_tok, const int64_t* d_off, int64_t n_docs,
                                 int64_t n_tok, int32_t dim, const int32_t* pos_idx,
                                 float logit_scale, float* loss, float* dq, float* dd,
                                 float* scores, void* ws, size_t ws_bytes, void* stream) {
  return run_loss(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim, pos_idx, logit_scale, 0.f, loss,
                  dq, dd, scores, ws, ws_bytes, stream);
}

hpr_status coltrast_total_loss_fwd_bwd(const uint16_t* q, int32_t nq, int32_t lq,
                                       const uint16_t* d_tok, const int64_t* d_off,
                                       int64_t n_docs, int64_t n_tok, int32_t dim,
                                       const int32_t* pos_idx, float logit_scale,
                                       float temperature, float* loss, float* dq, float* dd,
                                       void* ws, size_t ws_bytes, void* stream) {
  if (!(temperature > 0.f) || temperature > 3.0e38f || !(1.0f / temperature < 3.0e38f))
    return fail(HPR_ERR_INVALID_ARG, "temperature must be positive, finite, with finite inverse");
  return run_loss(q, nq, lq, d_tok, d_off, n_docs, n_tok, dim, pos_idx, logit_scale, temperature,
                  loss, dq, dd, nullptr, ws, ws_bytes, stream);
}

size_t semantic_chunk_workspace_size(int64_t n, int32_t dim) {
  (void)dim;
  if (n < 1) return 0;
  const int64_t R = chunk_ranges(n);
  return align_up((size_t)R * sizeof(int32_t)) + align_up((size_t)R * sizeof(int64_t)) +
         align_up((size_t)n * sizeof(float));
}

hpr_status semantic_chunk(const uint16_t* emb, int64_t n, int32_t dim, const int64_t* paper_off,
                          int64_t n_papers, float threshold, float* cos_out, int32_t* seg_out,
                          int64_t* n_segments, void* ws, size_t ws_bytes, void* stream) {
  if (!emb || !seg_out || !n_segments || !ws)
    return fail(HPR_ERR_INVALID_ARG, "emb, seg_out, n_segments and ws must be non-NULL");
  if (n < 1 || n >= (int64_t(1) << 31))
    return fail(HPR_ERR_INVALID_ARG, "n (%lld) must satisfy 1 <= n < 2^31", (long long)n);
  if (dim % 8 != 0 || dim < 8 || dim > kMaxChunkDim)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE,
                "semantic_chunk needs dim %% 8 == 0 and 8 <= dim <= %d (dim=%d)", kMaxChunkDim, dim);
  if (!(threshold == threshold))
    return fail(HPR_ERR_INVALID_ARG, "threshold must not be NaN");
  if (paper_off && n_papers < 1)
    return fail(HPR_ERR_INVALID_ARG, "n_papers (%lld) must be >= 1 with paper offsets",
                (long long)n_papers);
  if (!aligned16(emb)) return fail(HPR_ERR_INVALID_ARG, "emb must be 16-byte aligned");
  const size_t need = semantic_chunk_workspace_size(n, dim);
  if (ws_bytes < need)
    return fail(HPR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu < %zu bytes", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(ws);
  const int64_t R = chunk_ranges(n);
  int32_t* cnt = c.take<int32_t>((size_t)R * sizeof(int32_t));
  int64_t* base = c.take<int64_t>((size_t)R * sizeof(int64_t));
  float* cos_ws = c.take<float>((size_t)n * sizeof(float));
  hipError_t e = timed("semantic_chunk", s, [&] {
    return launch_semantic_chunk(emb, n, dim, paper_off, paper_off ? n_papers : 0, threshold,
                                 cos_out ? cos_out : cos_ws, cnt, base, seg_out, n_segments, s);
  });
  return e == hipSuccess ? HPR_OK : hip_fail(e, "semantic chunking launch");
}

hpr_status retrieval_metrics(const int64_t* topk_idx, int32_t nq, int32_t ld, int32_t k,
                             const int64_t* positive, int32_t* ranks_out, double* metrics_out,
                             void* stream) {
  if (!topk_idx || !positive || !metrics_out)
    return fail(HPR_ERR_INVALID_ARG, "topk_idx, positive and metrics_out must be non-NULL");
  if (nq < 1) return fail(HPR_ERR_INVALID_ARG, "nq (%d) must be >= 1", nq);
  if (k < 1 || k > ld)
    return fail(HPR_ERR_INVALID_ARG, "k=%d must satisfy 1 <= k <= ld (%d)", k, ld);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = timed("retrieval_metrics", s, [&] {
    return launch_retrieval_metrics(topk_idx, nq, ld, k, positive, ranks_out, metrics_out, s);
  });
  return e == hipSuccess ? HPR_OK : hip_fail(e, "retrieval metrics launch");
}

hpr_status hpr_mfma_calibration(int64_t iters, int32_t operands, float* sink, double* flops,
                                void* stream) {
  if (!sink || !flops) return fail(HPR_ERR_INVALID_ARG, "sink and flops must be non-NULL");
  if (operands != 0 && operands != 1)
    return fail(HPR_ERR_INVALID_ARG, "operands (%d) must be 0 or 1", operands);
  if (iters < 1 || iters > (int64_t(1) << 32))
    return fail(HPR_ERR_INVALID_ARG, "iters (%lld) must be in [1, 2^32]", (long long)iters);
  int n_cu = 0;
  hpr_status st = current_cu_count(&n_cu);
  if (st != HPR_OK) return st;
  *flops = (double)mfma_calibration_waves(n_cu) * (double)iters * 4.0 * 32768.0;
  hipError_t e = timed("mfma_calibration", static_cast<hipStream_t>(stream), [&] {
    return launch_mfma_calibration(sink, iters, n_cu, operands == 1,
                                   static_cast<hipStream_t>(stream));
  });
  return e == hipSuccess ? HPR_OK : hip_fail(e, "MFMA calibration launch");
}

hpr_status hpr_read_calibration(const void* buf, int64_t bytes, uint32_t* sink, void* stream) {
  if (!buf || !sink) return fail(HPR_ERR_INVALID_ARG, "buf and sink must be non-NULL");
  if (bytes < 16 || bytes % 16 != 0 || !aligned16(buf))
    return fail(HPR_ERR_INVALID_ARG, "bytes must be a positive multiple of 16, buf 16-byte aligned");
  int n_cu = 0;
  hpr_status st = current_cu_count(&n_cu);
  if (st != HPR_OK) return st;
  const int blocks = n_cu * 32 < 16384 ? n_cu * 32 : 16384;  // 8 waves per SIMD
  hipError_t e = timed("read_calibration", static_cast<hipStream_t>(stream), [&] {
    return launch_read_calibration(buf, bytes, sink, blocks, static_cast<hipStream_t>(stream));
  });
  return e == hipSuccess ? HPR_OK : hip_fail(e, "read calibration launch");
}

size_t dense_ip_topk_workspace_size(int32_t nq, int64_t n, int32_t dim, int32_t k) {
  if (nq < 1 || n < 1 || dim < 1 || k < 1) return 0;
  const DensePlan p = dense_plan(n, k);
  size_t b = align_up((size_t)nq * (size_t)p.S * sizeof(float));  // sample scores
  if (p.S == n) return b;
  b += align_up((size_t)nq * k * sizeof(float)) + align_up((size_t)nq * k * sizeof(int64_t));
  b += align_up((size_t)nq * sizeof(float)) + align_up((size_t)nq * sizeof(int64_t)) +
       align_up((size_t)nq * sizeof(int32_t));
  b += align_up((size_t)nq * (size_t)p.cap * sizeof(float)) +
       align_up((size_t)nq * (size_t)p.cap * sizeof(uint32_t));
  b += align_up(sizeof(int32_t)) + align_up((size_t)nq * sizeof(int32_t));   // queue
  b += align_up((size_t)nq * (size_t)dim * sizeof(uint16_t));                   // queued rows
  b += align_up((size_t)nq * 256 * sizeof(uint32_t)) +                          // radix select
       align_up((size_t)nq * sizeof(unsigned long long)) + align_up((size_t)nq * sizeof(uint32_t));
  return b;
}

hpr_status dense_ip_topk(const uint16_t* q, int32_t nq, const uint16_t* x, int64_t n,
                         int32_t dim, int32_t k, float* out_scores, int64_t* out_idx, void* ws,
                         size_t ws_bytes, void* stream) {
  if (!q || !x || !out_scores || !out_idx || !ws)
    return fail(HPR_ERR_INVALID_ARG, "q, x, out_scores, out_idx and ws must be non-NULL");
  if (nq < 1 || n < 1) return fail(HPR_ERR_INVALID_ARG, "nq (%d) and n (%lld) must be >= 1", nq,
                                   (long long)n);
  if (dim < 1) return fail(HPR_ERR_INVALID_ARG, "dim (%d) must be >= 1", dim);
  if (dim % 8 != 0 || dim < 8 || dim > 8192)
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "dense_ip_topk needs dim %% 8 == 0 and 8 <= dim <= 8192 (dim=%d)", dim);
  if (n >= (int64_t(1) << 31))
    return fail(HPR_ERR_UNSUPPORTED_SHAPE, "n must be below 2^31 (got %lld)", (long long)n);
  if (k < 1 || k > 1024 || (int64_t)k > n)
    return fail(HPR_ERR_INVALID_ARG, "k=%d must satisfy 1 <= k <= min(n, 1024)", k);
  if (!aligned16(q) || !aligned16(x) || !aligned16(out_scores) || !aligned16(out_idx))
    return fail(HPR_ERR_INVALID_ARG, "device pointers must be 16-byte aligned");
  const size_t need = dense_ip_topk_workspace_size(nq, n, dim, k);
  if (ws_bytes < need)
    return fail(HPR_ERR_WORKSPACE_TOO_SMALL, "workspace %zu < %zu bytes", ws_bytes, need);
  int n_cu = 0;
  hpr_status st = current_cu_count(&n_cu);
  if (st != HPR_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const DensePlan p = dense_plan(n, k);
  Carver c(ws);
  float* sample = c.take<float>((size_t)nq * (size_t)p.S * sizeof(float));
  DenseGemm g = {};
  g.mode = 0;
  g.q = q;
  g.nqa = nq;
  g.x = x;
  g.r0 = 0;
  g.r1 = p.S;
  g.dim = dim;
  g.scores = sample;
  g.ld = p.S;
  hipError_t e = timed("dense_sample", s, [&] { return launch_dense_gemm(g, n_cu, s); });
  if (e != hipSuccess) return hip_fail(e, "dense sample launch");
  if (p.S == n) {  // the sample is the whole store
    e = timed("topk", s, [&] {
      return launch_topk_rows(sample, nq, n, n, k, out_scores, out_idx, s);
    });
    return e == hipSuccess ? HPR_OK : hip_fail(e, "top-k launch");
  }
  float* ss = c.take<float>((size_t)nq * k * sizeof(float));
  int64_t* si = c.take<int64_t>((size_t)nq * k * sizeof(int64_t));
  float* theta = c.take<float>((size_t)nq * sizeof(float));
  int64_t* tie = c.take<int64_t>((size_t)nq * sizeof(int64_t));
  int32_t* count = c.take<int32_t>((size_t)nq * sizeof(int32_t));
  float* cand_s = c.take<float>((size_t)nq * (size_t)p.cap * sizeof(float));
  uint32_t* cand_i = c.take<uint32_t>((size_t)nq * (size_t)p.cap * sizeof(uint32_t));
  int32_t* n_queued = c.take<int32_t>(sizeof(int32_t));
  int32_t* qlist = c.take<int32_t>((size_t)nq * sizeof(int32_t));
  uint16_t* qc = c.take<uint16_t>((size_t)nq * dim * sizeof(uint16_t));
  uint32_t* hist = c.take<uint32_t>((size_t)nq * 256 * sizeof(uint32_t));
  unsigned long long* prefix = c.take<unsigned long long>((size_t)nq * sizeof(unsigned long long));
  uint32_t* remaining = c.take<uint32_t>((size_t)nq * sizeof(uint32_t));

  e = timed("topk", s, [&] { return launch_topk_rows(sample, nq, p.S, p.S, k, ss, si, s); });
  if (e != hipSuccess) return hip_fail(e, "top-k launch");
  e = launch_dense_init(ss, nq, k, theta, tie, count, n_queued, s);
  if (e != hipSuccess) return hip_fail(e, "dense init launch");
  g.mode = 1;
  g.r0 = p.S;
  g.r1 = n;
  g.scores = nullptr;
  g.ld = 0;
  g.theta = theta;
  g.tie = tie;
  g.count = count;
  g.cand_s = cand_s;
  g.cand_i = cand_i;
  g.cap = p.cap;
  e = timed("dense_scan", s, [&] { return launch_dense_gemm(g, n_cu, s); });
  if (e != hipSuccess) return hip_fail(e, "dense scan launch");
  e = timed("dense_merge", s, [&] {
    return launch_dense_merge(ss, si, nq, k, count, cand_s, cand_i, p.cap, nullptr, nullptr,
                              out_scores, out_idx, theta, tie, n_queued, qlist, prefix, remaining,
                              s);
  });
  if (e != hipSuccess) return hip_fail(e, "dense merge launch");
  // Exact fallback for the queued queries (their lists overflowed): every launch below reads
  // the queue length on the device and does nothing when it is 0.  A radix select over the
  // rescanned keys (8 bytes, most significant first) finds each queued query's k-th key;
  // one more rescan collects the keys at or above it (at most k) and the merge rewrites the
  // query's output.
  e = launch_dense_fallback_prep(q, dim, qlist, n_queued, qc, hist, n_cu, s);
  if (e != hipSuccess) return hip_fail(e, "dense fallback launch");
  DenseGemm f = g;
  f.q = qc;
  f.qmap = qlist;
  f.m_dev = n_queued;
  f.hist = hist;
  f.prefix = prefix;
  for (int shift = 56; shift >= 0; shift -= 8) {
    f.mode = 2;
    f.shift = shift;
    e = timed("dense_fallback", s, [&] { return launch_dense_gemm(f, n_cu, s); });
    if (e == hipSuccess)
      e = launch_dense_radix(n_queued, qlist, nq, shift, ss, si, k, hist, prefix, remaining,
                             theta, tie, count, s);
    if (e != hipSuccess) return hip_fail(e, "dense fallback launch");
  }
  f.mode = 1;
  e = timed("dense_fallback", s, [&] { return launch_dense_gemm(f, n_cu, s); });
  if (e == hipSuccess)
    e = launch_dense_merge(ss, si, nq, k, count, cand_s, cand_i, p.cap, qlist, n_queued,
                           out_scores, out_idx, theta, tie, nullptr, nullptr, nullptr, nullptr,
                           s);
  return e == hipSuccess ? HPR_OK : hip_fail(e, "dense fallback launch");
}

hpr_status hpr_csr_validate(const int64_t* d_off, int64_t n_docs, int64_t n_tok, void* ws,
                            void* stream, int64_t* h_first_bad_doc) {
  if (!d_off || !ws || !h_first_bad_doc)
    return fail(HPR_ERR_INVALID_ARG, "d_off, ws and h_first_bad_doc must be non-NULL");
  if (n_docs < 1 || n_tok < 0)
    return fail(HPR_ERR_INVALID_ARG, "n_docs must be >= 1 and n_tok >= 0");
  *h_first_bad_doc = -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned long long* bad = static_cast<unsigned long long*>(ws);
  hipError_t e = launch_csr_validate(d_off, n_docs, n_tok, bad, s);
  if (e != hipSuccess) return hip_fail(e, "csr validate launch");
  unsigned long long h = 0;
  e = hipMemcpyAsync(&h, bad, sizeof(h), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(e, "csr validate copy");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "csr validate sync");
  if (h == ~0ull) return HPR_OK;
  *h_first_bad_doc = (int64_t)(h >> 1);
  if (h & 1ull)
    return fail(HPR_ERR_EMPTY_DOC, "document %lld has no token", (long long)(h >> 1));
  return fail(HPR_ERR_BAD_CSR, "offsets invalid at document %lld", (long long)(h >> 1));
}

hpr_status hpr_scale_f32(float* x, int64_t n, const float* scale, void* stream) {
  if (!x || !scale) return fail(HPR_ERR_INVALID_ARG, "x and scale must be non-NULL");
  if (n < 0) return fail(HPR_ERR_INVALID_ARG, "n must be >= 0");
  if (n == 0) return HPR_OK;
  hipError_t e = launch_scale(x, n, scale, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "scale launch");
  return HPR_OK;
}

hpr_status hpr_kernel_timing(int32_t enable) {
  g_timing_on.store(enable ? 1 : 0, std::memory_order_relaxed);
  return HPR_OK;
}

hpr_status hpr_kernel_timing_read(const char* name, double* total_ms, int64_t* launches) {
  if (!name || !total_ms || !launches)
    return fail(HPR_ERR_INVALID_ARG, "name, total_ms and launches must be non-NULL");
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
  {
    std::lock_guard<std::mutex> g(g_timing_mu);
    auto it = g_timing.find(name);
    if (it != g_timing.end()) ev.swap(it->second);
  }
  double tot = 0.0;
  hpr_status st = HPR_OK;
  for (auto& p : ev) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(p.second);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.first, p.second);
    if (e != hipSuccess && st == HPR_OK) st = hip_fail(e, "kernel timing");
    tot += ms;
    (void)hipEventDestroy(p.first);
    (void)hipEventDestroy(p.second);
  }
  *total_ms = tot;
  *launches = (int64_t)ev.size();
  return st;
}

const char* hpr_status_string(hpr_status s) {
  switch (s) {
    case HPR_OK: return "HPR_OK";
    case HPR_ERR_INVALID_ARG: return "HPR_ERR_INVALID_ARG";
    case HPR_ERR_BAD_CSR: return "HPR_ERR_BAD_CSR";
    case HPR_ERR_EMPTY_DOC: return "HPR_ERR_EMPTY_DOC";
    case HPR_ERR_UNSUPPORTED_SHAPE: return "HPR_ERR_UNSUPPORTED_SHAPE";
    case HPR_ERR_WORKSPACE_TOO_SMALL: return "HPR_ERR_WORKSPACE_TOO_SMALL";
    case HPR_ERR_CAPACITY: return "HPR_ERR_CAPACITY";
    case HPR_ERR_HIP: return "HPR_ERR_HIP";
    default: return "HPR_ERR_UNKNOWN";
  }
}

const char* hpr_last_error(void) { return g_last_error.c_str(); }

int32_t hpr_abi_version(void) { return HPR_ABI_VERSION; }

}  // extern "C"
