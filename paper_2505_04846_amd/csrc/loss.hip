// In-batch InfoNCE over MaxSim scores (the L_LI half of the ColTrast loss) and its backward.
//
//   infonce_kernel  one workgroup: per query row the max logit, a log1p-form log-sum-exp, the
//                   loss term and G = dloss/dS; the batch mean is reduced in a fixed order.
//   grad_q_kernel   dQ[q,i,:] = sum_d G[q,d] * D[argmax token of (q,i,d)]: one wave per 4 query
//                   tokens of one query; 16 lanes per token, 8 columns per lane.
//   grad_d_kernel   dD: one workgroup per document.  The (q,i) entries are sorted by the token
//                   they selected (bitonic sort of (token << 14 | entry) keys in LDS), then each
//                   token row is summed over its entries in entry order, so the result is
//                   deterministic without atomics; rows nobody selected are written as zeros.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

constexpr int kRowThreads = 256;

// Deterministic 256-thread block reductions (fixed tree: wave butterfly, then waves in order).
__device__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

__device__ void block_argmax(float& M, int64_t& dM, float* redf, int64_t* redi) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float oM = __shfl_xor(M, m);
    const int64_t od = __shfl_xor(dM, m);
    if (oM > M || (oM == M && od < dM)) {
      M = oM;
      dM = od;
    }
  }
  __syncthreads();
  if (lane == 0) {
    redf[wave] = M;
    redi[wave] = dM;
  }
  __syncthreads();
  M = redf[0];
  dM = redi[0];
  for (int w = 1; w < kRowThreads / kWave; ++w)
    if (redf[w] > M || (redf[w] == M && redi[w] < dM)) {
      M = redf[w];
      dM = redi[w];
    }
}

// One workgroup per query row q: G[q, :] and the row's loss term; the last workgroup to finish
// reduces the terms in query order into the mean.  ctrl[0] = error flag raised by earlier
// kernels of the call, ctrl[1] = completion counter (both zeroed at the start of the call).
__global__ __launch_bounds__(kRowThreads) void infonce_kernel(const float* __restrict__ S, int nq,
                                                              int64_t n, const int32_t* pos,
                                                              float s, float* G, float* terms,
                                                              float* loss, float* scores_out,
                                                              int32_t* ctrl) {
  // No FMA contraction in this kernel: every logit must be the same rounded product s * S.
  // Contracted, M - s * S[pos] becomes fma(-s, S[pos], M), the rounding error of M's own
  // product (up to half an ulp of ~1e3 when s = 50) instead of exactly 0 when the positive
  // holds the maximum -- larger than the whole loss in that regime.
#pragma clang fp contract(off)
  __shared__ float redf[kRowThreads / kWave];
  __shared__ int64_t redi[kRowThreads / kWave];
  __shared__ int last;
  const int tid = threadIdx.x;
  const int q = blockIdx.x;
  const float* Sq = S + (int64_t)q * n;
  float* Gq = G + (int64_t)q * n;
  const float gscale = s / (float)nq;

  float M = -__builtin_huge_valf();
  int64_t dM = n;
  for (int64_t d = tid; d < n; d += kRowThreads) {
    const float l = (s * Sq[d]);
    if (l > M) {
      M = l;
      dM = d;
    }
  }
  block_argmax(M, dM, redf, redi);
  // log-sum-exp = M + log1p(sum over d != dM of exp(l - M)): keeps the loss accurate when one
  // logit dominates (the loss is then ~ the small sum, which log(1 + x) would lose).
  float so = 0.f;
  for (int64_t d = tid; d < n; d += kRowThreads)
    if (d != dM) so += expf((s * Sq[d]) - M);
  so = block_sum(so, redf);
  const float l1p = log1pf(so);
  const float lse = M + l1p;
  const int64_t p = pos[q];
  const bool bad = p < 0 || p >= n;
  float term = 0.f;
  if (bad) {
    for (int64_t d = tid; d < n; d += kRowThreads) Gq[d] = 0.f;
    if (tid == 0) atomicOr(&ctrl[0], 2);
  } else {
    term = (M - (s * Sq[p])) + l1p;
    // G[q,d] = (s/B) softmax; the positive gets -(s/B) * (sum of the other probabilities),
    // which equals (s/B) (p_pos - 1) without the cancellation of 1 - p_pos in fp32.
    float rest = 0.f;
    for (int64_t d = tid; d < n; d += kRowThreads) {
      const float sd = Sq[d];
      if (scores_out) scores_out[(int64_t)q * n + d] = sd;
      if (d != p) {
        const float e = expf((s * sd) - lse);
        Gq[d] = gscale * e;
        rest += e;
      }
    }
    rest = block_sum(rest, redf);
    if (tid == 0) Gq[p] = -gscale * rest;
  }
  if (tid == 0) {
    terms[q] = term;
    __threadfence();
    last = atomicAdd(&ctrl[1], 1) == nq - 1;
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  float acc = 0.f;  // fixed order: thread t sums queries t, t + 256, ...; then a fixed tree
  for (int qq = tid; qq < nq; qq += kRowThreads)
    acc += __hip_atomic_load(&terms[qq], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  acc = block_sum(acc, redf);
  if (tid == 0) {
    *loss = ctrl[0] != 0 ? __builtin_nanf("") : acc / (float)nq;
    ctrl[1] = 0;
  }
}

constexpr int kGqWaves = 16;
constexpr int kGqUnroll = 8;

// dQ: one workgroup per (query q, group of 4 query tokens); wave w sums a contiguous chunk of
// the documents, keeping kGqUnroll independent row gathers in flight; the 16 partial sums are
// then added in wave order (deterministic).  Lane: token (lane >> 4), 8 columns at
// 8 * ((lane & 15) + 16 cc).
template <int CPL>
__global__ __launch_bounds__(64 * kGqWaves) void grad_q_kernel(
    const uint16_t* __restrict__ D, const int64_t* __restrict__ off, int64_t n_docs,
    int64_t n_tok, int dim, int nq, int lq, const uint16_t* __restrict__ amax,
    const float* __restrict__ G, float* dq) {
  __shared__ float part[kGqWaves][4][128 * CPL];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int groups = (lq + 3) / 4;
  const int q = blockIdx.x / groups;
  const int i0 = (blockIdx.x - q * groups) * 4;
  const int sub = lane >> 4;
  const int i = i0 + sub;
  const bool active = i < lq;
  const int c = lane & 15;
  const int64_t E = (int64_t)nq * lq;
  const int64_t e = (int64_t)q * lq + (active ? i : 0);
  const int64_t last_tok = n_tok - 1;
  const int64_t chunk = (n_docs + kGqWaves - 1) / kGqWaves;
  const int64_t dbeg = wave * chunk;
  const int64_t dend = dbeg + chunk < n_docs ? dbeg + chunk : n_docs;

  float acc[CPL][8];
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc)
#pragma unroll
    for (int v = 0; v < 8; ++v) acc[cc][v] = 0.f;

  for (int64_t d0 = dbeg; d0 < dend; d0 += kGqUnroll) {
    float g[kGqUnroll];
    int64_t row[kGqUnroll];
#pragma unroll
    for (int u = 0; u < kGqUnroll; ++u) {
      const int64_t d = d0 + u;
      const bool ok = d < dend;
      g[u] = ok ? G[(int64_t)q * n_docs + d] : 0.f;
      int64_t base = ok ? off[d] : 0;
      base = base < 0 ? 0 : (base > last_tok ? last_tok : base);
      const int64_t r = base + (ok ? amax[d * E + e] : 0);
      row[u] = r > last_tok ? last_tok : r;
    }
    u32x4 w[kGqUnroll][CPL];
#pragma unroll
    for (int u = 0; u < kGqUnroll; ++u)
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int k = 8 * (c + 16 * cc);
        w[u][cc] = k < dim ? load16(D + row[u] * dim + k) : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
    for (int u = 0; u < kGqUnroll; ++u)
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        acc[cc][0] += g[u] * bf16_lo(w[u][cc].x);
        acc[cc][1] += g[u] * bf16_hi(w[u][cc].x);
        acc[cc][2] += g[u] * bf16_lo(w[u][cc].y);
        acc[cc][3] += g[u] * bf16_hi(w[u][cc].y);
        acc[cc][4] += g[u] * bf16_lo(w[u][cc].z);
        acc[cc][5] += g[u] * bf16_hi(w[u][cc].z);
        acc[cc][6] += g[u] * bf16_lo(w[u][cc].w);
        acc[cc][7] += g[u] * bf16_hi(w[u][cc].w);
      }
  }
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc)
#pragma unroll
    for (int v = 0; v < 8; ++v) part[wave][sub][8 * (c + 16 * cc) + v] = acc[cc][v];
  __syncthreads();
  for (int o = tid; o < 4 * 128 * CPL; o += 64 * kGqWaves) {
    const int t = o / (128 * CPL), k = o % (128 * CPL);
    if (i0 + t < lq && k < dim) {
      float v = 0.f;
#pragma unroll
      for (int w2 = 0; w2 < kGqWaves; ++w2) v += part[w2][t][k];
      dq[((int64_t)q * lq + i0 + t) * dim + k] = v;
    }
  }
}

constexpr int kGdThreads = 1024;
constexpr int kGdUnroll = 16;

// dD: one workgroup per document d.  Entry e = q * lq + i selected token a(e) = amax[d][e];
// keys (a(e) << 14 | e) are bitonic-sorted in LDS, so each token's entries are contiguous and
// in entry order.  Wave w owns a contiguous range of the document's token rows and walks the
// entries of those rows as one flat stream, kGdUnroll entries (independent Q-row gathers) at a
// time, flushing a row's sum when the next row starts and writing zeros for rows no entry
// selected.  Lane: 2 consecutive columns per 128-column block.
template <int CP>
__global__ __launch_bounds__(kGdThreads) void grad_d_kernel(
    const uint16_t* __restrict__ Q, const int64_t* __restrict__ off, int64_t n_docs,
    int64_t n_tok, int dim, int nq, int lq, uint64_t lq_magic,
    const uint16_t* __restrict__ amax, const float* __restrict__ G, float* dd, int P) {
  extern __shared__ uint32_t keys[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int kWaves = kGdThreads / kWave;
  const int64_t d = blockIdx.x;
  const int E = nq * lq;
  for (int e = tid; e < P; e += kGdThreads)
    keys[e] = e < E ? ((uint32_t)amax[d * E + e] << 14) | (uint32_t)e : 0xffffffffu;
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      for (int i = tid; i < P; i += kGdThreads) {
        const int j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;
          const uint32_t ki = keys[i], kj = keys[j];
          if ((ki > kj) == up) {
            keys[i] = kj;
            keys[j] = ki;
          }
        }
      }
    }
  }
  __syncthreads();

  const int64_t last_tok = n_tok - 1;
  int64_t lo_t = off[d], hi_t = off[d + 1];
  lo_t = lo_t < 0 ? 0 : (lo_t > last_tok ? last_tok : lo_t);
  hi_t = hi_t <= lo_t ? lo_t + 1 : (hi_t > n_tok ? n_tok : hi_t);
  const int64_t len = hi_t - lo_t;
  // this wave's rows [j0, j1)
  const int64_t rows_per = (len + kWaves - 1) / kWaves;
  const int64_t j0 = wave * rows_per < len ? wave * rows_per : len;
  const int64_t j1 = j0 + rows_per < len ? j0 + rows_per : len;
  if (j0 >= j1) return;
  auto lower = [&](int64_t j) {  // first sorted position whose token is >= j
    if (j >= 65536) return E;
    const uint32_t target = (uint32_t)j << 14;
    int lo = 0, hi = E;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (keys[mid] < target)
        lo = mid + 1;
      else
        hi = mid;
    }
    return lo;
  };
  const int p0 = lower(j0), p1 = lower(j1);

  float acc[CP][2];
  auto zero_acc = [&]() {
#pragma unroll
    for (int cc = 0; cc < CP; ++cc) acc[cc][0] = acc[cc][1] = 0.f;
  };
  auto write_row = [&](int64_t j) {
#pragma unroll
    for (int cc = 0; cc < CP; ++cc) {
      const int c = 2 * lane + 128 * cc;
      if (c < dim)
        *reinterpret_cast<float2*>(dd + (lo_t + j) * dim + c) = make_float2(acc[cc][0], acc[cc][1]);
    }
  };
  zero_acc();
  int64_t cur = j0;  // row being accumulated; rows < cur are written
  for (int p = p0; p < p1; p += kGdUnroll) {
    uint32_t kk[kGdUnroll];
    float g[kGdUnroll];
    uint32_t w[kGdUnroll][CP];
#pragma unroll
    for (int u = 0; u < kGdUnroll; ++u) {
      kk[u] = p + u < p1 ? keys[p + u] : 0xffffffffu;
      const uint32_t e = kk[u] & 0x3fffu;
      const uint32_t qq = (uint32_t)(((uint64_t)e * lq_magic) >> 32);
      g[u] = p + u < p1 ? G[(int64_t)qq * n_docs + d] : 0.f;
#pragma unroll
      for (int cc = 0; cc < CP; ++cc) {
        const int c = 2 * lane + 128 * cc;
        w[u][cc] = (p + u < p1 && c < dim)
                       ? *reinterpret_cast<const uint32_t*>(Q + (int64_t)e * dim + c)
                       : 0u;
      }
    }
#pragma unroll
    for (int u = 0; u < kGdUnroll; ++u) {
      if (p + u < p1) {
        const int64_t j = kk[u] >> 14;
        while (cur < j) {  // finish the current row, zero-fill rows nobody selected
          write_row(cur);
          zero_acc();
          ++cur;
        }
#pragma unroll
        for (int cc = 0; cc < CP; ++cc) {
          acc[cc][0] += g[u] * bf16_lo(w[u][cc]);
          acc[cc][1] += g[u] * bf16_hi(w[u][cc]);
        }
      }
    }
  }
  while (cur < j1) {
    write_row(cur);
    zero_acc();
    ++cur;
  }
}

__global__ void scale_kernel(float* x, int64_t n, const float* scale) {
  const float s = *scale;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    x[i] *= s;
}

}  // namespace

hipError_t launch_infonce(const float* S, int nq, int64_t n_docs, const int32_t* pos, float scale,
                          float* G, float* terms, float* loss, float* scores_out, int32_t* ctrl,
                          hipStream_t stream) {
  hipLaunchKernelGGL(infonce_kernel, dim3((unsigned)nq), dim3(kRowThreads), 0, stream, S, nq,
                     n_docs, pos, scale, G, terms, loss, scores_out, ctrl);
  return hipGetLastError();
}

hipError_t launch_grad_q(const uint16_t* d_tok, const int64_t* off, int64_t n_docs, int64_t n_tok,
                         int dim, int nq, int lq, const uint16_t* amax, const float* G, float* dq,
                         hipStream_t stream) {
  const unsigned blocks = (unsigned)((int64_t)nq * ((lq + 3) / 4));
  if (dim <= 128)
    hipLaunchKernelGGL(grad_q_kernel<1>, dim3(blocks), dim3(64 * kGqWaves), 0, stream, d_tok, off,
                       n_docs, n_tok, dim, nq, lq, amax, G, dq);
  else
    hipLaunchKernelGGL(grad_q_kernel<2>, dim3(blocks), dim3(64 * kGqWaves), 0, stream, d_tok, off,
                       n_docs, n_tok, dim, nq, lq, amax, G, dq);
  return hipGetLastError();
}

hipError_t launch_grad_d(const uint16_t* q, const int64_t* off, int64_t n_docs, int64_t n_tok,
                         int dim, int nq, int lq, const uint16_t* amax, const float* G, float* dd,
                         hipStream_t stream) {
  const int E = nq * lq;
  int P = 1;
  while (P < E) P <<= 1;
  const size_t lds = (size_t)P * sizeof(uint32_t);
  // floor(e / lq) = (e * ceil(2^32 / lq)) >> 32 for e < 2^14 and lq <= 128: the product
  // overshoots e / lq by less than e / 2^32 < 2^-18, below the 1 / lq gap to the next integer.
  const uint64_t magic = (0x100000000ull + (uint64_t)lq - 1) / (uint64_t)lq;
  if (dim <= 128)
    hipLaunchKernelGGL(grad_d_kernel<1>, dim3((unsigned)n_docs), dim3(kGdThreads), lds, stream,
                       q, off, n_docs, n_tok, dim, nq, lq, magic, amax, G, dd, P);
  else
    hipLaunchKernelGGL(grad_d_kernel<2>, dim3((unsigned)n_docs), dim3(kGdThreads), lds, stream,
                       q, off, n_docs, n_tok, dim, nq, lq, magic, amax, G, dd, P);
  return hipGetLastError();
}

hipError_t launch_scale(float* x, int64_t n, const float* scale, hipStream_t stream) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(scale_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, x, n, scale);
  return hipGetLastError();
}

}  // namespace hpr
