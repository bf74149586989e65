// Semantic chunking boundaries over a stream of sentence embeddings, and P@k / MRR@k of a
// retrieval ranking.
//
// Chunking: a segment grows while the cosine of each sentence with the one before it (in the same
// paper) stays strictly above a threshold; the first sentence of every paper opens a segment.
//   chunk_scan_kernel   one wave per range of kRowsPerWave consecutive sentences: each row is
//                       read once (16-byte streaming loads, the next row in flight while the
//                       current one is reduced; the row before the range is read once more for
//                       its norm), its
//                       squared norm and its dot product with the previous row come from
//                       v_dot2_f32_f16 (exact fp16 products, fp32 sums) and two wave reductions;
//                       cos[t] = dot / sqrt(|prev|^2 |cur|^2), NaN at a paper's first sentence.
//                       The range's boundary count (cos not above the threshold, NaN included)
//                       goes to cnt[range].
//   chunk_offsets_kernel  one workgroup: exclusive scan of the range counts (fixed order), and
//                       the total, the number of segments.
//   chunk_ids_kernel    one wave per range: seg[t] = (boundaries at or before t) - 1 from the
//                       range's offset and a ballot prefix over the range's cosines.
// The three passes read the embeddings once (the HBM-bound part) and the cosines twice.
//
// Metrics: one workgroup finds each query's 1-based rank of its positive among the first k
// retrieved indices (0 when absent) and sums the hits and the reciprocal ranks in fp64 in a
// fixed order.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

constexpr int kChunkThreads = 256;
constexpr int kChunkWaves = kChunkThreads / kWave;
constexpr int kMaxCpl = kMaxChunkDim / 512;  // 16-byte chunks per lane at the largest dim

typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;

__device__ __forceinline__ float dot2_acc(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a), __builtin_bit_cast(f16x2, b), c,
                                false);
}

// Row t's chunks for this lane: chunk c = lane + 64 i (16 bytes each), zeros past `dim`.
__device__ __forceinline__ void load_row(const uint16_t* __restrict__ E, int64_t t, int dim,
                                         int lane, u32x4 (&v)[kMaxCpl]) {
  const uint16_t* row = E + t * dim;
#pragma unroll
  for (int i = 0; i < kMaxCpl; ++i) {
    const int c = lane + 64 * i;
    // streaming (non-temporal) loads: every row is read once (3.02 -> 2.53 ms at 2 M x 4096)
    v[i] = 8 * c < dim ? load16_stream(row + 8 * c) : u32x4{0u, 0u, 0u, 0u};
  }
}

__device__ __forceinline__ float row_dot(const u32x4 (&a)[kMaxCpl], const u32x4 (&b)[kMaxCpl]) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxCpl; ++i) {
    s = dot2_acc(a[i].x, b[i].x, s);
    s = dot2_acc(a[i].y, b[i].y, s);
    s = dot2_acc(a[i].z, b[i].z, s);
    s = dot2_acc(a[i].w, b[i].w, s);
  }
  return s;
}

// First index d in [0, n_papers] with off[d] > t (n_papers + 1 when none): the next paper start
// after t is off[d] (skipping empty papers, whose offsets repeat).
__device__ __forceinline__ int64_t next_start_index(const int64_t* off, int64_t n_papers,
                                                    int64_t t) {
  int64_t lo = 0, hi = n_papers + 1;
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if (off[mid] <= t)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(kChunkThreads) void chunk_scan_kernel(
    const uint16_t* __restrict__ E, int64_t n, int dim, const int64_t* __restrict__ off,
    int64_t n_papers, float thr, int64_t n_ranges, float* __restrict__ cos_out,
    int32_t* __restrict__ cnt) {
  const int lane = threadIdx.x & 63;
  const int64_t range = (int64_t)blockIdx.x * kChunkWaves + (threadIdx.x >> 6);
  if (range >= n_ranges) return;  // whole wave
  const int64_t t0 = range * kRowsPerWave;
  const int64_t t1 = t0 + kRowsPerWave < n ? t0 + kRowsPerWave : n;
  // paper starts: is t0 one, and the next start after t0 (uniform, scalar)
  bool t0_start;
  int64_t dnext;
  if (off) {
    dnext = next_start_index(off, n_papers, t0);
    t0_start = dnext > 0 && off[dnext - 1] == t0;  // off[dnext-1] <= t0 < off[dnext]
  } else {
    dnext = 0;
    t0_start = t0 == 0;
  }
  int64_t next_start = off ? (dnext <= n_papers ? off[dnext] : n) : n;
  u32x4 prev[kMaxCpl], cur[kMaxCpl], nxt[kMaxCpl];
  float pn = 0.f;  // |prev|^2
  if (!t0_start) {
    load_row(E, t0 - 1, dim, lane, prev);
    pn = wave_sum(row_dot(prev, prev));
  }
  load_row(E, t0, dim, lane, cur);
  int32_t boundaries = 0;
  for (int64_t t = t0; t < t1; ++t) {
    if (t + 1 < t1) load_row(E, t + 1, dim, lane, nxt);  // in flight during this row
    const float cn = wave_sum(row_dot(cur, cur));
    bool first = t == t0 ? t0_start : t == next_start;
    if (off && t == next_start) {  // advance past every paper starting at t
      while (dnext <= n_papers && off[dnext] <= t) ++dnext;
      next_start = dnext <= n_papers ? off[dnext] : n;
    }
    float c;
    if (first) {
      c = __builtin_nanf("");
    } else {
      const float d = wave_sum(row_dot(prev, cur));
      c = d / sqrtf(pn * cn);
    }
    if (lane == 0) cos_out[t] = c;
    boundaries += (c > thr) ? 0 : 1;
    pn = cn;
#pragma unroll
    for (int i = 0; i < kMaxCpl; ++i) {
      prev[i] = cur[i];
      cur[i] = nxt[i];
    }
  }
  if (lane == 0) cnt[range] = boundaries;
}

constexpr int kScanThreads = 1024;

// Exclusive scan of cnt[0 .. n_ranges) into base[], total into *n_seg: each thread sums a
// contiguous slice, a block scan orders the slices, then each thread writes its slice.
__global__ __launch_bounds__(kScanThreads) void chunk_offsets_kernel(const int32_t* __restrict__ cnt,
                                                                     int64_t n_ranges,
                                                                     int64_t* __restrict__ base,
                                                                     int64_t* __restrict__ n_seg) {
  __shared__ int64_t part[kScanThreads];
  const int tid = threadIdx.x;
  const int64_t per = (n_ranges + kScanThreads - 1) / kScanThreads;
  const int64_t a = tid * per, b = a + per < n_ranges ? a + per : n_ranges;
  int64_t s = 0;
  for (int64_t i = a; i < b; ++i) s += cnt[i];
  part[tid] = s;
  __syncthreads();
  for (int o = 1; o < kScanThreads; o <<= 1) {  // inclusive Hillis-Steele scan
    const int64_t v = tid >= o ? part[tid - o] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int64_t run = tid > 0 ? part[tid - 1] : 0;
  for (int64_t i = a; i < b; ++i) {
    base[i] = run;
    run += cnt[i];
  }
  if (tid == kScanThreads - 1) *n_seg = part[tid];
}

__global__ __launch_bounds__(kChunkThreads) void chunk_ids_kernel(const float* __restrict__ cos_in,
                                                                  int64_t n, float thr,
                                                                  int64_t n_ranges,
                                                                  const int64_t* __restrict__ base,
                                                                  int32_t* __restrict__ seg) {
  const int lane = threadIdx.x & 63;
  const int64_t range = (int64_t)blockIdx.x * kChunkWaves + (threadIdx.x >> 6);
  if (range >= n_ranges) return;
  const int64_t t0 = range * kRowsPerWave;
  const int64_t t1 = t0 + kRowsPerWave < n ? t0 + kRowsPerWave : n;
  int64_t run = base[range];
  const uint64_t le_mask = lane == 63 ? ~0ull : ((2ull << lane) - 1ull);
  for (int64_t t = t0; t < t1; t += 64) {
    const int64_t i = t + lane;
    const bool ok = i < t1;
    const bool bnd = ok && !(cos_in[i] > thr);
    const uint64_t m = __ballot(bnd);
    if (ok) seg[i] = (int32_t)(run + __popcll(m & le_mask) - 1);
    run += __popcll(m);
  }
}

constexpr int kMetricThreads = 1024;

__global__ __launch_bounds__(kMetricThreads) void metrics_kernel(
    const int64_t* __restrict__ idx, int nq, int64_t ld, int k, const int64_t* __restrict__ pos,
    int32_t* __restrict__ ranks, double* __restrict__ out) {
  __shared__ double sh_hit[kMetricThreads], sh_rr[kMetricThreads];
  const int tid = threadIdx.x;
  double hit = 0.0, rr = 0.0;
  for (int q = tid; q < nq; q += kMetricThreads) {  // fixed order per thread
    const int64_t p = pos[q];
    int r = 0;
    for (int j = 0; j < k; ++j)
      if (idx[(int64_t)q * ld + j] == p) {
        r = j + 1;
        break;
      }
    if (ranks) ranks[q] = r;
    if (r > 0) {
      hit += 1.0;
      rr += 1.0 / (double)r;
    }
  }
  sh_hit[tid] = hit;
  sh_rr[tid] = rr;
  __syncthreads();
  for (int o = kMetricThreads / 2; o > 0; o >>= 1) {  // fixed pairwise tree
    if (tid < o) {
      sh_hit[tid] += sh_hit[tid + o];
      sh_rr[tid] += sh_rr[tid + o];
    }
    __syncthreads();
  }
  if (tid == 0) {
    out[0] = sh_hit[0] / (double)k / (double)nq;
    out[1] = sh_rr[0] / (double)nq;
  }
}

}  // namespace

int64_t chunk_ranges(int64_t n) { return (n + kRowsPerWave - 1) / kRowsPerWave; }

hipError_t launch_semantic_chunk(const uint16_t* E, int64_t n, int dim, const int64_t* off,
                                 int64_t n_papers, float thr, float* cos_out, int32_t* cnt,
                                 int64_t* base, int32_t* seg, int64_t* n_seg,
                                 hipStream_t stream) {
  const int64_t R = chunk_ranges(n);
  const unsigned blocks = (unsigned)((R + kChunkWaves - 1) / kChunkWaves);
  hipLaunchKernelGGL(chunk_scan_kernel, dim3(blocks), dim3(kChunkThreads), 0, stream, E, n, dim,
                     off, n_papers, thr, R, cos_out, cnt);
  hipLaunchKernelGGL(chunk_offsets_kernel, dim3(1), dim3(kScanThreads), 0, stream, cnt, R, base,
                     n_seg);
  hipLaunchKernelGGL(chunk_ids_kernel, dim3(blocks), dim3(kChunkThreads), 0, stream, cos_out, n,
                     thr, R, base, seg);
  return hipGetLastError();
}

hipError_t launch_retrieval_metrics(const int64_t* idx, int nq, int64_t ld, int k,
                                    const int64_t* pos, int32_t* ranks, double* out,
                                    hipStream_t stream) {
  hipLaunchKernelGGL(metrics_kernel, dim3(1), dim3(kMetricThreads), 0, stream, idx, nq, ld, k,
                     pos, ranks, out);
  return hipGetLastError();
}

}  // namespace hpr
