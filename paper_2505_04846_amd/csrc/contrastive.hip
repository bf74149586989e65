// ColTrast's pooled contrastive loss L_C (SimCSE-style InfoNCE on the cosines of mean-pooled
// embeddings) and its gradient, for the total loss L = (L_LI + L_C) / 2.
//
//   pool_kernel     one workgroup per document and per query: the mean P of its token rows
//                   (fp32, fixed summation order), written as the unit row U = P / |P|, with
//                   the gradient scale 1 / (|P| L) (L: the sequence's token count).  Reads the
//                   store once.
//   cl_rows_kernel  one workgroup per query: logits c[q, d] = <U_q, U_d> / tau, the row's
//                   log-sum-exp and loss term, w dL/dc (w: the loss weight), and the query side
//                   of the gradient, dL/dQ[q, i] = (dU_q - U_q <U_q, dU_q>) / (|P_q| lq) with
//                   dU_q = (1/tau) sum_d w dL/dc[q, d] U_d -- the same for every token i.
//   cl_docs_kernel  one workgroup per document: the document side, dL/dD[j] = (dU_d - U_d
//                   <U_d, dU_d>) / (|P_d| L_d) for every token j of d, with dU_d = (1/tau)
//                   sum_q w dL/dc[q, d] U_q; workgroup 0 also reduces the loss terms in query
//                   order and writes L_C and the total loss.
// The sums over documents (or queries) are split between row groups of threads, each thread
// owning four columns; the groups' partial sums are combined in group order, so every result
// is deterministic.  dim <= 256 (the ABI's limit) lets one thread own one column in the
// per-column epilogues.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

constexpr int kClThreads = 256;      // pooling and per-document workgroups
constexpr int kClRowThreads = 1024;  // per-query workgroups: more loads in flight per row
constexpr int kClRowLdsDocs = 8192;  // rows of up to this many documents are kept in LDS

// Block-wide reductions over NT threads (NT / 64 waves): wave reduction, then the wave
// results in wave order.  Every thread receives the result.
template <int NT>
__device__ float cl_block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = red[0];
#pragma unroll
  for (int i = 1; i < NT / kWave; ++i) t += red[i];
  __syncthreads();
  return t;
}

template <int NT>
__device__ float cl_block_max(float v, float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = red[0];
#pragma unroll
  for (int i = 1; i < NT / kWave; ++i) t = fmaxf(t, red[i]);
  __syncthreads();
  return t;
}

template <int NT>
__device__ int64_t cl_block_min(int64_t v, int64_t* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int o = 32; o > 0; o >>= 1) {
    const int64_t u = __shfl_xor(v, o);
    v = u < v ? u : v;
  }
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int64_t t = red[0];
#pragma unroll
  for (int i = 1; i < NT / kWave; ++i) t = red[i] < t ? red[i] : t;
  __syncthreads();
  return t;
}

// Block b < n_docs pools document b (rows off[b] .. off[b+1]-1, clamped into the store), block
// n_docs + q pools query q (rows q lq .. q lq + lq - 1 of Q).  Thread t sums chunk t % CH (8
// columns) over the rows r = t / CH, t / CH + RG, ... (RG = 256 / CH row groups); the groups'
// partial sums are added in group order.
__global__ __launch_bounds__(kClThreads) void pool_kernel(
    const uint16_t* __restrict__ Q, int nq, int lq, const uint16_t* __restrict__ D,
    const int64_t* __restrict__ off, int64_t n_docs, int64_t n_tok, int dim,
    float* __restrict__ Uq, float* __restrict__ Ud, float* __restrict__ gsc_q,
    float* __restrict__ gsc_d) {
  extern __shared__ float cl_part[];  // [RG][dim]
  __shared__ float red[kClThreads / kWave];
  const int tid = threadIdx.x;
  const int CH = dim / 8, RG = kClThreads / CH;
  const int64_t b = blockIdx.x;
  const uint16_t* src;
  int64_t rows;
  float* dst;
  float* gsc;
  if (b < n_docs) {
    const int64_t last_tok = n_tok - 1;
    int64_t lo = off[b], hi = off[b + 1];
    lo = lo < 0 ? 0 : (lo > last_tok ? last_tok : lo);
    hi = hi <= lo ? lo + 1 : (hi > n_tok ? n_tok : hi);
    src = D + lo * dim;
    rows = hi - lo;
    dst = Ud + b * dim;
    gsc = gsc_d + b;
  } else {
    const int64_t q = b - n_docs;
    src = Q + q * lq * dim;
    rows = lq;
    dst = Uq + q * dim;
    gsc = gsc_q + q;
  }
  const int c = tid % CH, g = tid / CH;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (g < RG) {
    constexpr int kU = 8;  // rows in flight per thread
    for (int64_t r0 = g; r0 < rows; r0 += kU * RG) {
      u32x4 v[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t r = r0 + (int64_t)u * RG;
        v[u] = r < rows ? load16(src + r * dim + 8 * c) : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        acc[0] += bf16_lo(v[u].x);
        acc[1] += bf16_hi(v[u].x);
        acc[2] += bf16_lo(v[u].y);
        acc[3] += bf16_hi(v[u].y);
        acc[4] += bf16_lo(v[u].z);
        acc[5] += bf16_hi(v[u].z);
        acc[6] += bf16_lo(v[u].w);
        acc[7] += bf16_hi(v[u].w);
      }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) cl_part[g * dim + 8 * c + k] = acc[k];
  }
  __syncthreads();
  float m = 0.f;  // column tid of the mean
  if (tid < dim) {
    float s = 0.f;
    for (int gg = 0; gg < RG; ++gg) s += cl_part[gg * dim + tid];
    m = s * (1.0f / (float)rows);
  }
  const float nrm = sqrtf(cl_block_sum<kClThreads>(m * m, red));
  if (tid < dim) dst[tid] = m / nrm;
  if (tid == 0) *gsc = 1.0f / (nrm * (float)rows);
}

// Column tid (tid < dim) of sum_r w[r] V[r, :] over r < n, V row-major [n][dim] fp32 with rows
// of stride dim, w[r] = wts[r * wstride]: thread (c4, g) of the NT sums four columns over the
// rows g, g + NG, ...; the NG groups are combined in group order through `part` ([NG][dim]).
template <int NT>
__device__ float cl_weighted_rows(const float* __restrict__ wts, int64_t wstride,
                                  const float* __restrict__ V, int64_t n, int dim, float* part) {
  const int tid = threadIdx.x;
  const int CW = dim / 4, NG = NT / CW;
  const int c4 = tid % CW, g = tid / CW;
  if (g < NG) {
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    constexpr int kU = 8;  // rows in flight per thread
    for (int64_t r0 = g; r0 < n; r0 += kU * NG) {
      f32x4 v[kU];
      float wv[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t r = r0 + (int64_t)u * NG;
        const bool ok = r < n;
        wv[u] = ok ? wts[r * wstride] : 0.f;
        v[u] = ok ? reinterpret_cast<const f32x4*>(V + r * dim)[c4] : f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) s += wv[u] * v[u];
    }
    *reinterpret_cast<f32x4*>(part + g * dim + 4 * c4) = s;
  }
  __syncthreads();
  float t = 0.f;
  if (tid < dim)
    for (int gg = 0; gg < NG; ++gg) t += part[gg * dim + tid];
  __syncthreads();  // part may be reused by the caller
  return t;
}

// One workgroup per query q.  dC (the weighted dL/dc) doubles as the row's logit scratch.
__global__ __launch_bounds__(kClRowThreads) void cl_rows_kernel(
    const float* __restrict__ Uq, const float* __restrict__ gsc_q, const float* __restrict__ Ud,
    int nq, int64_t n_docs, int dim, const int32_t* __restrict__ pos, float inv_tau, float w,
    float* __restrict__ dC, float* __restrict__ terms, float* __restrict__ dqc,
    int32_t* __restrict__ ctrl) {
  // LDS: u_q [dim], the column-group partials [NG][dim], then (when row_in_lds) the row
  extern __shared__ __attribute__((aligned(16))) float cl_sm[];
  __shared__ float red[kClRowThreads / kWave];
  __shared__ int64_t redi[kClRowThreads / kWave];
  const int tid = threadIdx.x;
  const int q = blockIdx.x;
  const int64_t p = pos[q];  // issued early: the loads below do not depend on each other
  const float gsc = gsc_q[q];
  float* uq = cl_sm;
  for (int k = tid; k < dim; k += kClRowThreads) uq[k] = Uq[(int64_t)q * dim + k];
  __syncthreads();
  // the row's logits, then its weighted dL/dc: in LDS when it fits (each pass over it is then
  // an LDS round trip, not an L2 one), copied to dC at the end
  float* const out_row = dC + (int64_t)q * n_docs;
  const bool row_in_lds = n_docs <= kClRowLdsDocs;
  float* row = row_in_lds ? cl_sm + (kClRowThreads / (dim / 4) + 1) * dim : out_row;
  // logits: a group of LPD lanes (LPD = dim / 4 rounded up to a power of two) takes one
  // document, each lane four columns of it (coalesced 16-byte loads), and the group's partial
  // dot products are added by butterfly shuffles inside the group
  const int n4 = dim / 4;
  int LPD = 1;
  while (LPD < n4) LPD <<= 1;
  const int lane = tid & 63, wave = tid >> 6;
  const int DPW = kWave / LPD;  // documents per wave and step
  const int c4 = lane % LPD, slot = lane / LPD;
  const bool col_ok = c4 < n4;
  const f32x4 u = col_ok ? reinterpret_cast<const f32x4*>(uq)[c4] : f32x4{0.f, 0.f, 0.f, 0.f};
  float M = -__builtin_huge_valf();
  constexpr int kU = 8;  // documents in flight per lane
  constexpr int kNW = kClRowThreads / kWave;
  for (int64_t d0 = (int64_t)wave * DPW; d0 < n_docs; d0 += (int64_t)kU * kNW * DPW) {
    f32x4 a[kU];
#pragma unroll
    for (int v = 0; v < kU; ++v) {
      const int64_t d = d0 + (int64_t)v * kNW * DPW + slot;
      a[v] = (col_ok && d < n_docs) ? reinterpret_cast<const f32x4*>(Ud + d * dim)[c4]
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int v = 0; v < kU; ++v) {
      float t = a[v].x * u.x;
      t += a[v].y * u.y;
      t += a[v].z * u.z;
      t += a[v].w * u.w;
      for (int m = 1; m < LPD; m <<= 1) t += __shfl_xor(t, m);
      const int64_t d = d0 + (int64_t)v * kNW * DPW + slot;
      if (c4 == 0 && d < n_docs) {
        const float cv = t * inv_tau;
        row[d] = cv;
        M = fmaxf(M, cv);
      }
    }
  }
  __syncthreads();  // row[] complete before other threads read it
  M = cl_block_max<kClRowThreads>(M, red);
  int64_t dM = n_docs;
  for (int64_t d = tid; d < n_docs; d += kClRowThreads)
    if (row[d] == M && d < dM) dM = d;
  dM = cl_block_min<kClRowThreads>(dM, redi);
  // log-sum-exp = M + log1p(sum over d != dM of exp(c - M)), accurate when one logit dominates
  float so = 0.f;
  for (int64_t d = tid; d < n_docs; d += kClRowThreads)
    if (d != dM) so += expf(row[d] - M);
  const float l1p = log1pf(cl_block_sum<kClRowThreads>(so, red));
  const float lse = M + l1p;
  const bool bad = p < 0 || p >= n_docs;
  if (tid == 0) {
    terms[q] = bad ? __builtin_nanf("") : (M - row[p]) + l1p;
    if (bad) atomicOr(&ctrl[0], 2);
  }
  __syncthreads();  // row[p] is read above before it is overwritten below
  // w dL/dc = (w/B)(softmax - onehot); the positive gets -(w/B) (sum of the other
  // probabilities), which avoids the cancellation in p_pos - 1
  const float gs = w / (float)nq;
  float rest = 0.f;
  for (int64_t d = tid; d < n_docs; d += kClRowThreads) {
    const float pr = bad ? 0.f : expf(row[d] - lse);
    if (d != p) {
      row[d] = gs * pr;
      rest += pr;
    }
  }
  rest = cl_block_sum<kClRowThreads>(rest, red);
  if (tid == 0 && !bad) row[p] = -gs * rest;
  __syncthreads();
  if (row_in_lds)
    for (int64_t d = tid; d < n_docs; d += kClRowThreads) out_row[d] = row[d];
  // dU_q = (1/tau) sum_d dC[q, d] U_d, then the projection off U_q
  const float dv = cl_weighted_rows<kClRowThreads>(row, 1, Ud, n_docs, dim, cl_sm + dim) * inv_tau;
  const float ud = cl_block_sum<kClRowThreads>(tid < dim ? uq[tid] * dv : 0.f, red);
  if (tid < dim) dqc[(int64_t)q * dim + tid] = (dv - uq[tid] * ud) * gsc;
}

// One workgroup per document d (workgroup 0 also finishes the loss).
__global__ __launch_bounds__(kClThreads) void cl_docs_kernel(
    const float* __restrict__ Uq, const float* __restrict__ Ud, const float* __restrict__ gsc_d,
    int nq, int64_t n_docs, int dim, float inv_tau, const float* __restrict__ dC,
    const float* __restrict__ terms, float w_li, float w_c, float* __restrict__ loss,
    float* __restrict__ ddc, const int32_t* __restrict__ ctrl) {
  extern __shared__ __attribute__((aligned(16))) float cl_sm[];  // [NG][dim]
  __shared__ float red[kClThreads / kWave];
  const int tid = threadIdx.x;
  const int64_t d = blockIdx.x;
  // dU_d = (1/tau) sum_q dC[q, d] U_q, then the projection off U_d
  const float dv = cl_weighted_rows<kClThreads>(dC + d, n_docs, Uq, nq, dim, cl_sm) * inv_tau;
  const float u = tid < dim ? Ud[d * dim + tid] : 0.f;
  const float dot = cl_block_sum<kClThreads>(u * dv, red);
  if (tid < dim) ddc[d * dim + tid] = (dv - u * dot) * gsc_d[d];
  if (d != 0) return;
  float acc = 0.f;  // fixed order: thread t sums queries t, t + 256, ...; then a fixed tree
  for (int qq = tid; qq < nq; qq += kClThreads) acc += terms[qq];
  acc = cl_block_sum<kClThreads>(acc, red);
  if (tid == 0) {
    const float lc = ctrl[0] != 0 ? __builtin_nanf("") : acc / (float)nq;
    loss[2] = lc;
    loss[0] = w_li * loss[1] + w_c * lc;
  }
}

}  // namespace

hipError_t launch_pool(const uint16_t* q, int nq, int lq, const uint16_t* d_tok,
                       const int64_t* off, int64_t n_docs, int64_t n_tok, int dim, float* Uq,
                       float* Ud, float* gsc_q, float* gsc_d, hipStream_t stream) {
  const int CH = dim / 8, RG = kClThreads / CH;
  const size_t lds = (size_t)RG * dim * sizeof(float);
  hipLaunchKernelGGL(pool_kernel, dim3((unsigned)(n_docs + nq)), dim3(kClThreads), lds, stream,
                     q, nq, lq, d_tok, off, n_docs, n_tok, dim, Uq, Ud, gsc_q, gsc_d);
  return hipGetLastError();
}

hipError_t launch_contrastive(const float* Uq, const float* gsc_q, const float* Ud,
                              const float* gsc_d, int nq, int64_t n_docs, int dim,
                              const int32_t* pos, float tau, float w_li, float w_c, float* dC,
                              float* terms, float* dqc, float* ddc, float* loss, int32_t* ctrl,
                              hipStream_t stream) {
  const float inv_tau = 1.0f / tau;
  const size_t lds_rows = ((size_t)(kClRowThreads / (dim / 4) + 1) * dim +
                           (n_docs <= kClRowLdsDocs ? (size_t)n_docs : 0)) * sizeof(float);
  hipLaunchKernelGGL(cl_rows_kernel, dim3((unsigned)nq), dim3(kClRowThreads), lds_rows, stream,
                     Uq, gsc_q, Ud, nq, n_docs, dim, pos, inv_tau, w_c, dC, terms, dqc, ctrl);
  const size_t lds = (size_t)(kClThreads / (dim / 4)) * dim * sizeof(float);
  hipLaunchKernelGGL(cl_docs_kernel, dim3((unsigned)n_docs), dim3(kClThreads), lds, stream, Uq,
                     Ud, gsc_d, nq, n_docs, dim, inv_tau, dC, terms, w_li, w_c, loss, ddc, ctrl);
  return hipGetLastError();
}

}  // namespace hpr
