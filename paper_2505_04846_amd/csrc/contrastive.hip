// ColTrast's pooled contrastive loss L_C (SimCSE-style InfoNCE on the cosines of mean-pooled
// embeddings) and its gradient, for the total loss L = (L_LI + L_C) / 2.
//
//   pool_kernel     one workgroup per document and per query: the mean of its token rows (fp32,
//                   fixed summation order) and the norm of that mean.  Reads the store once.
//   cl_rows_kernel  one workgroup per query: logits c[q, d] = cos(P_q, P_d) / tau, the row's
//                   log-sum-exp and loss term, w dL/dc (w: the loss weight), and the query side
//                   of the gradient, dL/dQ[q, i] = (dU_q - U_q <U_q, dU_q>) / (|P_q| lq) with
//                   dU_q = (1/tau) sum_d w dL/dc[q, d] U_d -- the same for every token i.
//   cl_docs_kernel  one workgroup per document: the document side, dL/dD[j] = (dU_d - U_d
//                   <U_d, dU_d>) / (|P_d| L_d) for every token j of d, with dU_d = (1/tau)
//                   sum_q w dL/dc[q, d] U_q; workgroup 0 also reduces the loss terms in query
//                   order and writes L_C and the total loss.
// Dimensions are spread over threads with the documents (or queries) split between thread
// groups whose partial sums are combined in a fixed order, so every result is deterministic.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

constexpr int kClThreads = 256;

__device__ float cl_block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  const float t = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return t;
}

__device__ float cl_block_max(float v, float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  const float t = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
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
    float* __restrict__ Pq, float* __restrict__ Pd, float* __restrict__ nrm_q,
    float* __restrict__ nrm_d) {
  extern __shared__ float cl_part[];  // [RG][dim]
  __shared__ float red[kClThreads / kWave];
  const int tid = threadIdx.x;
  const int CH = dim / 8, RG = kClThreads / CH;
  const int64_t b = blockIdx.x;
  const uint16_t* src;
  int64_t rows;
  float* dst;
  float* nrm;
  if (b < n_docs) {
    const int64_t last_tok = n_tok - 1;
    int64_t lo = off[b], hi = off[b + 1];
    lo = lo < 0 ? 0 : (lo > last_tok ? last_tok : lo);
    hi = hi <= lo ? lo + 1 : (hi > n_tok ? n_tok : hi);
    src = D + lo * dim;
    rows = hi - lo;
    dst = Pd + b * dim;
    nrm = nrm_d + b;
  } else {
    const int64_t q = b - n_docs;
    src = Q + q * lq * dim;
    rows = lq;
    dst = Pq + q * dim;
    nrm = nrm_q + q;
  }
  const int c = tid % CH, g = tid / CH;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (g < RG) {
    for (int64_t r = g; r < rows; r += RG) {
      const u32x4 v = load16(src + r * dim + 8 * c);
      acc[0] += bf16_lo(v.x);
      acc[1] += bf16_hi(v.x);
      acc[2] += bf16_lo(v.y);
      acc[3] += bf16_hi(v.y);
      acc[4] += bf16_lo(v.z);
      acc[5] += bf16_hi(v.z);
      acc[6] += bf16_lo(v.w);
      acc[7] += bf16_hi(v.w);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) cl_part[g * dim + 8 * c + k] = acc[k];
  }
  __syncthreads();
  const float inv_rows = 1.0f / (float)rows;
  float sq = 0.f;
  for (int k = tid; k < dim; k += kClThreads) {
    float s = 0.f;
    for (int gg = 0; gg < RG; ++gg) s += cl_part[gg * dim + k];
    const float m = s * inv_rows;
    dst[k] = m;
    sq += m * m;
  }
  sq = cl_block_sum(sq, red);
  if (tid == 0) *nrm = sqrtf(sq);
}

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
  for (int i = 1; i < kClThreads / kWave; ++i) t = red[i] < t ? red[i] : t;
  __syncthreads();
  return t;
}

// One workgroup per query q.  dC (the weighted dL/dc) doubles as the row's logit scratch.
__global__ __launch_bounds__(kClThreads) void cl_rows_kernel(
    const float* __restrict__ Pq, const float* __restrict__ nrm_q, const float* __restrict__ Pd,
    const float* __restrict__ nrm_d, int nq, int lq, int64_t n_docs, int dim,
    const int32_t* __restrict__ pos, float inv_tau, float w, float* __restrict__ dC,
    float* __restrict__ terms, float* __restrict__ dqc, int32_t* __restrict__ ctrl) {
  extern __shared__ float cl_sm[];  // u_q [dim], then dU partials [2][dim]
  __shared__ float red[kClThreads / kWave];
  __shared__ int64_t redi[kClThreads / kWave];
  const int tid = threadIdx.x;
  const int q = blockIdx.x;
  float* uq = cl_sm;
  float* du = cl_sm + dim;
  const float inv_nq = 1.0f / nrm_q[q];
  for (int k = tid; k < dim; k += kClThreads) uq[k] = Pq[(int64_t)q * dim + k] * inv_nq;
  __syncthreads();
  float* row = dC + (int64_t)q * n_docs;
  // logits, and the first index holding their maximum
  float M = -__builtin_huge_valf();
  for (int64_t d = tid; d < n_docs; d += kClThreads) {
    const float* pd = Pd + d * dim;
    float dot = 0.f;
    for (int k = 0; k < dim; ++k) dot += uq[k] * pd[k];
    const float cv = dot / nrm_d[d] * inv_tau;
    row[d] = cv;
    M = fmaxf(M, cv);
  }
  M = cl_block_max(M, red);
  int64_t dM = n_docs;
  for (int64_t d = tid; d < n_docs; d += kClThreads)
    if (row[d] == M && d < dM) dM = d;
  dM = cl_block_min(dM, redi);
  // log-sum-exp = M + log1p(sum over d != dM of exp(c - M)), accurate when one logit dominates
  float so = 0.f;
  for (int64_t d = tid; d < n_docs; d += kClThreads)
    if (d != dM) so += expf(row[d] - M);
  const float l1p = log1pf(cl_block_sum(so, red));
  const float lse = M + l1p;
  const int64_t p = pos[q];
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
  for (int64_t d = tid; d < n_docs; d += kClThreads) {
    const float pr = bad ? 0.f : expf(row[d] - lse);
    if (d != p) {
      row[d] = gs * pr;
      rest += pr;
    }
  }
  rest = cl_block_sum(rest, red);
  if (tid == 0 && !bad) row[p] = -gs * rest;
  __syncthreads();
  // dU_q[k] = (1/tau) sum_d dC[q, d] Pd[d, k] / |P_d|: column k per thread, two document halves
  const int G2 = kClThreads / dim >= 2 ? 2 : 1;
  const int k = tid % dim, gh = tid / dim;
  if (gh < G2 && tid < G2 * dim) {
    float s = 0.f;
    for (int64_t d = gh; d < n_docs; d += G2) s += row[d] * (Pd[d * dim + k] / nrm_d[d]);
    du[gh * dim + k] = s * inv_tau;
  }
  for (int kk = tid + G2 * dim; kk < dim; kk += kClThreads) {  // dim > 256: one group, rest
    float s = 0.f;
    for (int64_t d = 0; d < n_docs; ++d) s += row[d] * (Pd[d * dim + kk] / nrm_d[d]);
    du[kk] = s * inv_tau;
  }
  __syncthreads();
  float ud = 0.f;  // <u_q, dU_q>
  for (int kk = tid; kk < dim; kk += kClThreads) {
    const float dv = G2 == 2 ? du[kk] + du[dim + kk] : du[kk];
    ud += uq[kk] * dv;
  }
  ud = cl_block_sum(ud, red);
  const float scale = inv_nq / (float)lq;
  for (int kk = tid; kk < dim; kk += kClThreads) {
    const float dv = G2 == 2 ? du[kk] + du[dim + kk] : du[kk];
    dqc[(int64_t)q * dim + kk] = (dv - uq[kk] * ud) * scale;
  }
}

// One workgroup per document d (workgroup 0 also finishes the loss).
__global__ __launch_bounds__(kClThreads) void cl_docs_kernel(
    const float* __restrict__ Pq, const float* __restrict__ nrm_q, const float* __restrict__ Pd,
    const float* __restrict__ nrm_d, const int64_t* __restrict__ off, int nq, int64_t n_docs,
    int64_t n_tok, int dim, float inv_tau, const float* __restrict__ dC,
    const float* __restrict__ terms, float w_li, float w_c, float* __restrict__ loss,
    float* __restrict__ ddc, const int32_t* __restrict__ ctrl) {
  extern __shared__ float cl_sm[];  // u_d [dim], then dU partials [2][dim]
  __shared__ float red[kClThreads / kWave];
  const int tid = threadIdx.x;
  const int64_t d = blockIdx.x;
  float* ud_v = cl_sm;
  float* du = cl_sm + dim;
  const float inv_nd = 1.0f / nrm_d[d];
  for (int k = tid; k < dim; k += kClThreads) ud_v[k] = Pd[d * dim + k] * inv_nd;
  const int G2 = kClThreads / dim >= 2 ? 2 : 1;
  const int k = tid % dim, gh = tid / dim;
  if (gh < G2 && tid < G2 * dim) {
    float s = 0.f;
    for (int q = gh; q < nq; q += G2) s += dC[(int64_t)q * n_docs + d] * (Pq[(int64_t)q * dim + k] / nrm_q[q]);
    du[gh * dim + k] = s * inv_tau;
  }
  for (int kk = tid + G2 * dim; kk < dim; kk += kClThreads) {
    float s = 0.f;
    for (int q = 0; q < nq; ++q) s += dC[(int64_t)q * n_docs + d] * (Pq[(int64_t)q * dim + kk] / nrm_q[q]);
    du[kk] = s * inv_tau;
  }
  __syncthreads();
  float dot = 0.f;
  for (int kk = tid; kk < dim; kk += kClThreads) {
    const float dv = G2 == 2 ? du[kk] + du[dim + kk] : du[kk];
    dot += ud_v[kk] * dv;
  }
  dot = cl_block_sum(dot, red);
  const int64_t last_tok = n_tok - 1;
  int64_t lo = off[d], hi = off[d + 1];
  lo = lo < 0 ? 0 : (lo > last_tok ? last_tok : lo);
  hi = hi <= lo ? lo + 1 : (hi > n_tok ? n_tok : hi);
  const float scale = inv_nd / (float)(hi - lo);
  for (int kk = tid; kk < dim; kk += kClThreads) {
    const float dv = G2 == 2 ? du[kk] + du[dim + kk] : du[kk];
    ddc[d * dim + kk] = (dv - ud_v[kk] * dot) * scale;
  }
  if (d != 0) return;
  float acc = 0.f;  // fixed order: thread t sums queries t, t + 256, ...; then a fixed tree
  for (int qq = tid; qq < nq; qq += kClThreads) acc += terms[qq];
  acc = cl_block_sum(acc, red);
  if (tid == 0) {
    const float lc = ctrl[0] != 0 ? __builtin_nanf("") : acc / (float)nq;
    loss[2] = lc;
    loss[0] = w_li * loss[1] + w_c * lc;
  }
}

}  // namespace

hipError_t launch_pool(const uint16_t* q, int nq, int lq, const uint16_t* d_tok,
                       const int64_t* off, int64_t n_docs, int64_t n_tok, int dim, float* Pq,
                       float* Pd, float* nrm_q, float* nrm_d, hipStream_t stream) {
  const int CH = dim / 8, RG = kClThreads / CH;
  const size_t lds = (size_t)RG * dim * sizeof(float);
  hipLaunchKernelGGL(pool_kernel, dim3((unsigned)(n_docs + nq)), dim3(kClThreads), lds, stream,
                     q, nq, lq, d_tok, off, n_docs, n_tok, dim, Pq, Pd, nrm_q, nrm_d);
  return hipGetLastError();
}

hipError_t launch_contrastive(const float* Pq, const float* nrm_q, const float* Pd,
                              const float* nrm_d, const int64_t* off, int nq, int lq,
                              int64_t n_docs, int64_t n_tok, int dim, const int32_t* pos,
                              float tau, float w_li, float w_c, float* dC, float* terms,
                              float* dqc, float* ddc, float* loss, int32_t* ctrl,
                              hipStream_t stream) {
  const size_t lds = (size_t)3 * dim * sizeof(float);
  const float inv_tau = 1.0f / tau;
  hipLaunchKernelGGL(cl_rows_kernel, dim3((unsigned)nq), dim3(kClThreads), lds, stream, Pq,
                     nrm_q, Pd, nrm_d, nq, lq, n_docs, dim, pos, inv_tau, w_c, dC, terms, dqc,
                     ctrl);
  hipLaunchKernelGGL(cl_docs_kernel, dim3((unsigned)n_docs), dim3(kClThreads), lds, stream, Pq,
                     nrm_q, Pd, nrm_d, off, nq, n_docs, n_tok, dim, inv_tau, dC, terms, w_li, w_c,
                     loss, ddc, ctrl);
  return hipGetLastError();
}

}  // namespace hpr
