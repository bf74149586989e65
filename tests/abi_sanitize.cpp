// Host-only driver of the C ABI for a build whose host code carries AddressSanitizer and
// UndefinedBehaviorSanitizer: every entry point is called with arguments that its host-side
// validation must reject (NULL pointers, non-positive or oversized sizes, misaligned pointers,
// short workspaces), plus valid arguments, which on a machine without a GPU must come back as
// HPR_ERR_HIP from the first runtime call.  No pointer is ever dereferenced by the host code
// (the fake device pointers below are never touched).  Exits non-zero on an unexpected status;
// the sanitizers abort on any host memory or UB error.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include <hip/hip_runtime_api.h>

#include "hiperrag.h"

static int failures = 0;

static void expect(const char* what, hpr_status got, hpr_status want) {
  const char* msg = hpr_last_error();
  if (got != want) {
    std::fprintf(stderr, "FAIL %s: got %s, want %s (%s)\n", what, hpr_status_string(got),
                 hpr_status_string(want), msg ? msg : "");
    ++failures;
  } else if (got != HPR_OK && (!msg || !*msg)) {
    std::fprintf(stderr, "FAIL %s: no error message\n", what);
    ++failures;
  }
}

int main() {
  // The "valid arguments" calls below must not reach a device: with fake pointers a launch
  // would fault.  This driver is for machines without a GPU only.
  int n_dev = 0;
  if (hipGetDeviceCount(&n_dev) == hipSuccess && n_dev > 0) {
    std::printf("skipped: a GPU is visible\n");
    return 0;
  }
  const uint16_t* q = reinterpret_cast<const uint16_t*>(0x10000);
  const uint16_t* qodd = reinterpret_cast<const uint16_t*>(0x10008);
  const uint16_t* d = reinterpret_cast<const uint16_t*>(0x20000);
  const int64_t* off = reinterpret_cast<const int64_t*>(0x30000);
  const int32_t* pos = reinterpret_cast<const int32_t*>(0x40000);
  float* out = reinterpret_cast<float*>(0x50000);
  int64_t* idx = reinterpret_cast<int64_t*>(0x60000);
  void* ws = reinterpret_cast<void*>(0x70000);
  const size_t big = size_t(1) << 40;
  const hpr_status H = HPR_ERR_HIP;  // valid arguments, no device

  // maxsim_score / maxsim_score_noalloc / maxsim_topk
  expect("score null q", maxsim_score(nullptr, 2, 32, d, off, 4, 64, 128, out, ws, big, nullptr), 1);
  expect("score nq 0", maxsim_score(q, 0, 32, d, off, 4, 64, 128, out, ws, big, nullptr), 1);
  expect("score dim 12", maxsim_score(q, 2, 32, d, off, 4, 64, 12, out, ws, big, nullptr), 4);
  expect("score lq 129", maxsim_score(q, 2, 129, d, off, 4, 64, 128, out, ws, big, nullptr), 4);
  expect("score odd", maxsim_score(qodd, 2, 32, d, off, 4, 64, 128, out, ws, big, nullptr), 1);
  expect("score n_tok", maxsim_score(q, 2, 32, d, off, 4, 3, 128, out, ws, big, nullptr), 1);
  expect("score huge", maxsim_score(q, 2, 32, d, off, 4, int64_t(1) << 31, 128, out, ws, big,
                                    nullptr), 4);
  expect("score ws", maxsim_score(q, 2, 32, d, off, 4, 64, 128, out, ws, 0, nullptr), 5);
  expect("score ok", maxsim_score(q, 2, 32, d, off, 4, 64, 128, out, ws, big, nullptr), H);
  expect("noalloc null", maxsim_score_noalloc(q, 2, 32, d, off, 4, 64, 128, nullptr, nullptr), 1);
  expect("noalloc dim", maxsim_score_noalloc(q, 2, 32, d, off, 4, 64, 20, out, nullptr), 4);
  expect("noalloc ok", maxsim_score_noalloc(q, 2, 32, d, off, 4, 64, 128, out, nullptr), H);
  expect("topk k 0", maxsim_topk(q, 2, 8, d, off, 10, 100, 64, 0, out, idx, ws, big, nullptr), 1);
  expect("topk k > n", maxsim_topk(q, 2, 8, d, off, 10, 100, 64, 11, out, idx, ws, big, nullptr), 1);
  expect("topk k 1025", maxsim_topk(q, 2, 8, d, off, 5000, 9000, 64, 1025, out, idx, ws, big,
                                    nullptr), 1);
  expect("topk ws", maxsim_topk(q, 2, 8, d, off, 10, 100, 64, 5, out, idx, ws, 16, nullptr), 5);
  expect("topk ok", maxsim_topk(q, 2, 8, d, off, 10, 100, 64, 5, out, idx, ws, big, nullptr), H);

  // the two loss calls
  expect("loss null pos", coltrast_loss_fwd_bwd(q, 4, 32, d, off, 8, 256, 128, nullptr, 1.f, out,
                                                out, out, nullptr, ws, big, nullptr), 1);
  expect("loss nan scale", coltrast_loss_fwd_bwd(q, 4, 32, d, off, 8, 256, 128, pos, NAN, out,
                                                 out, out, nullptr, ws, big, nullptr), 1);
  expect("loss nq*lq", coltrast_loss_fwd_bwd(q, 1024, 32, d, off, 8, 256, 128, pos, 1.f, out,
                                             out, out, nullptr, ws, big, nullptr), 4);
  expect("loss lds", coltrast_loss_fwd_bwd(q, 480, 32, d, off, 500, 16000, 128, pos, 1.f, out,
                                           out, out, nullptr, ws, big, nullptr), 4);
  expect("loss ws", coltrast_loss_fwd_bwd(q, 4, 32, d, off, 8, 256, 128, pos, 1.f, out, out, out,
                                          nullptr, ws, 100, nullptr), 5);
  expect("loss ok", coltrast_loss_fwd_bwd(q, 4, 32, d, off, 8, 256, 128, pos, 1.f, out, out, out,
                                          nullptr, ws, big, nullptr), H);
  expect("total tau", coltrast_total_loss_fwd_bwd(q, 4, 32, d, off, 8, 256, 128, pos, 1.f, 0.f,
                                                  out, out, out, ws, big, nullptr), 1);
  expect("total tau tiny", coltrast_total_loss_fwd_bwd(q, 4, 32, d, off, 8, 256, 128, pos, 1.f,
                                                       1e-40f, out, out, out, ws, big, nullptr), 1);
  expect("total ok", coltrast_total_loss_fwd_bwd(q, 4, 32, d, off, 8, 256, 128, pos, 1.f, 0.05f,
                                                 out, out, out, ws, big, nullptr), H);
  for (int nq : {1, 7, 64, 512})
    if (coltrast_loss_workspace_size(nq, 32, 512, 131072, 128) == 0 ||
        coltrast_total_loss_workspace_size(nq, 32, 512, 131072, 128) <
            coltrast_loss_workspace_size(nq, 32, 512, 131072, 128)) {
      std::fprintf(stderr, "FAIL loss workspace sizes for nq=%d\n", nq);
      ++failures;
    }

  // dense_ip_topk
  expect("dense k", dense_ip_topk(q, 4, d, 100, 64, 101, out, idx, ws, big, nullptr), 1);
  expect("dense dim", dense_ip_topk(q, 4, d, 100, 60, 5, out, idx, ws, big, nullptr), 4);
  expect("dense n", dense_ip_topk(q, 4, d, int64_t(1) << 31, 64, 5, out, idx, ws, big, nullptr), 4);
  expect("dense ws", dense_ip_topk(q, 4, d, 200000, 64, 5, out, idx, ws, 64, nullptr), 5);
  expect("dense ok", dense_ip_topk(q, 4, d, 200000, 64, 5, out, idx, ws, big, nullptr), H);
  if (dense_ip_topk_workspace_size(4096, 10000000, 4096, 100) <
      dense_ip_topk_workspace_size(4096, 100000, 4096, 100)) {
    std::fprintf(stderr, "FAIL dense workspace sizes\n");
    ++failures;
  }

  // semantic_chunk, retrieval_metrics, helpers
  int32_t* seg = reinterpret_cast<int32_t*>(0x80000);
  int64_t* nseg = reinterpret_cast<int64_t*>(0x90000);
  expect("chunk nan", semantic_chunk(q, 100, 64, off, 3, NAN, nullptr, seg, nseg, ws, big, nullptr), 1);
  expect("chunk dim", semantic_chunk(q, 100, 4104, off, 3, 0.5f, nullptr, seg, nseg, ws, big, nullptr), 4);
  expect("chunk papers", semantic_chunk(q, 100, 64, off, 0, 0.5f, nullptr, seg, nseg, ws, big, nullptr), 1);
  expect("chunk ok", semantic_chunk(q, 100, 64, off, 3, 0.5f, nullptr, seg, nseg, ws, big, nullptr), H);
  double* met = reinterpret_cast<double*>(0xa0000);
  expect("metrics k", retrieval_metrics(idx, 4, 10, 11, idx, nullptr, met, nullptr), 1);
  expect("metrics ok", retrieval_metrics(idx, 4, 10, 10, idx, nullptr, met, nullptr), H);
  int64_t bad = 0;
  expect("csr null", hpr_csr_validate(nullptr, 4, 10, ws, nullptr, &bad), 1);
  expect("scale n", hpr_scale_f32(out, -1, out, nullptr), 1);
  expect("scale 0", hpr_scale_f32(out, 0, out, nullptr), HPR_OK);
  double total = 0;
  int64_t launches = 0;
  expect("timing read", hpr_kernel_timing_read("maxsim", &total, &launches), HPR_OK);
  expect("timing null", hpr_kernel_timing_read(nullptr, &total, &launches), 1);
  for (int s = -1; s <= 8; ++s)
    if (!hpr_status_string(s) || !*hpr_status_string(s)) ++failures;
  if (hpr_abi_version() != HPR_ABI_VERSION) ++failures;
  std::printf("%s: %d failures\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
