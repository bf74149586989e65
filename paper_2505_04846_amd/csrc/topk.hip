// Exact top-k of each row of an fp32 score matrix, ordered (score desc, index asc).
//
// One 1024-thread workgroup per row:
//   1. Radix select on order-preserving uint32 keys, 8 bits per pass from the most significant
//      byte: an LDS histogram of the next digit among the elements that match the prefix found
//      so far, then one wave scans the 256 bins from the top to find the bin holding the k-th
//      largest key.  After four passes the k-th largest key K is known exactly, together with
//      how many elements equal to K are needed (the rest of the k are strictly greater).
//   2. Gather: every element with key > K is kept; among elements with key == K the lowest
//      indices are kept, found with an in-order workgroup prefix count (ballot + popcount).
//   3. A bitonic network in LDS sorts the k (key, index) pairs into (key desc, index asc).
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxK = 1024;

__global__ __launch_bounds__(kThreads) void topk_rows_kernel(const float* __restrict__ S,
                                                             int64_t n, int64_t ld, int k,
                                                             float* out_s, int64_t* out_i) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t sk[kMaxK];
  __shared__ uint32_t si[kMaxK];
  __shared__ uint32_t wave_cnt[kWaves];
  __shared__ uint32_t sh_bin, sh_above, sh_gt;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const float* x = S + (int64_t)blockIdx.x * ld;

  // ---- 1. radix select
  uint32_t prefix = 0, pmask = 0;
  uint32_t remaining = (uint32_t)k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) hist[tid] = 0;
    if (tid == 0) {  // defaults, only kept if the counts cannot reach k (precondition k <= n)
      sh_bin = 0;
      sh_above = 0;
    }
    __syncthreads();
    for (int64_t i = tid; i < n; i += kThreads) {
      const uint32_t key = score_key(x[i]);
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      uint32_t c[4], tot = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = hist[255 - 4 * lane - j];
        tot += c[j];
      }
      uint32_t incl = tot;  // count of keys in bins >= 252 - 4*lane (this lane's lowest bin)
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
      const uint32_t excl = incl - tot;
      if (excl < remaining && remaining <= incl) {
        uint32_t acc = excl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (acc + c[j] >= remaining) {
            sh_bin = 255u - 4u * lane - j;
            sh_above = acc;
            break;
          }
          acc += c[j];
        }
      }
    }
    __syncthreads();
    prefix |= sh_bin << shift;
    pmask |= 255u << shift;
    remaining -= sh_above;
    __syncthreads();
  }
  const uint32_t K = prefix;
  const uint32_t need_eq = remaining;          // >= 1
  const uint32_t n_gt = (uint32_t)k - need_eq;  // elements strictly above K

  // ---- 2. gather
  if (tid == 0) sh_gt = 0;
  __syncthreads();
  uint32_t eq_base = 0;
  for (int64_t base = 0; base < n; base += kThreads) {
    const int64_t i = base + tid;
    bool gt = false, eq = false;
    uint32_t key = 0;
    if (i < n) {
      key = score_key(x[i]);
      gt = key > K;
      eq = key == K;
    }
    if (gt) {
      const uint32_t p = atomicAdd(&sh_gt, 1u);
      if (p < n_gt) {  // always true for finite inputs; keeps the stores in bounds regardless
        sk[p] = key;
        si[p] = (uint32_t)i;
      }
    }
    const unsigned long long m = __ballot(eq);
    if (lane == 0) wave_cnt[wave] = (uint32_t)__popcll(m);
    __syncthreads();
    const uint32_t gt_found = sh_gt;  // stable here: this chunk's atomics are done, the next
                                      // chunk's start after the barrier below
    uint32_t before = 0, chunk_total = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t cw = wave_cnt[w];
      before += w < wave ? cw : 0u;
      chunk_total += cw;
    }
    if (eq) {
      const uint32_t r = eq_base + before + (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
      if (r < need_eq) {
        sk[n_gt + r] = key;
        si[n_gt + r] = (uint32_t)i;
      }
    }
    eq_base += chunk_total;
    __syncthreads();
    if (eq_base >= need_eq && gt_found == n_gt) break;  // everything needed is collected
  }

  // ---- 3. sort the k pairs: (key desc, index asc)
  uint32_t P = 1;
  while (P < (uint32_t)k) P <<= 1;
  for (uint32_t i = k + tid; i < P; i += kThreads) {
    sk[i] = 0u;  // below every finite score's key
    si[i] = 0xffffffffu;
  }
  for (uint32_t size = 2; size <= P; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      for (uint32_t i = tid; i < P; i += kThreads) {
        const uint32_t j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;
          const uint32_t ki = sk[i], kj = sk[j], ii = si[i], ij = si[j];
          const bool j_first = kj > ki || (kj == ki && ij < ii);
          if (j_first == up) {
            sk[i] = kj;
            sk[j] = ki;
            si[i] = ij;
            si[j] = ii;
          }
        }
      }
    }
  }
  __syncthreads();
  for (int p = tid; p < k; p += kThreads) {
    out_s[(int64_t)blockIdx.x * k + p] = key_score(sk[p]);
    out_i[(int64_t)blockIdx.x * k + p] = (int64_t)si[p];
  }
}

}  // namespace

hipError_t launch_topk_rows(const float* scores, int64_t rows, int64_t n, int64_t ld, int k,
                            float* out_scores, int64_t* out_idx, hipStream_t stream) {
  if (k < 1 || k > kMaxK || rows < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(topk_rows_kernel, dim3((unsigned)rows), dim3(kThreads), 0, stream, scores,
                     n, ld, k, out_scores, out_idx);
  return hipGetLastError();
}

}  // namespace hpr
