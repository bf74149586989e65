// In-batch InfoNCE over MaxSim scores (the L_LI half of the ColTrast loss) and its backward.
//
//   infonce_kernel  one workgroup: per query row the max logit, a log1p-form log-sum-exp, the
//                   loss term and G = dloss/dS; the batch mean is reduced in a fixed order.
//   grad_q_*        dQ[q,i,:] = sum_d G[q,d] * D[argmax token of (q,i,d)]: partial sums over
//                   XCD-local document ranges (the gathered rows hit L2), then a fixed-order
//                   sum over the ranges.
//   grad_d_kernel   dD: one workgroup per document.  The (q,i) entries are sorted by the token
//                   they selected (stable counting sort in LDS), then each token row is summed
//                   over its entries in entry order, so the result is deterministic without
//                   atomics; rows nobody selected are written as zeros.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

constexpr int kRowThreads = 256;
constexpr int kRowCache = 8;  // scores per thread kept in registers by infonce_kernel

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
                                                              float s, float gw, float* G,
                                                              float* terms, float* loss,
                                                              float* scores_out, int32_t* ctrl) {
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
  const float gscale = gw * s / (float)nq;  // gw: the loss's weight in a weighted sum

  // The row's first kRowCache * kRowThreads scores stay in registers for the three passes
  // (each later pass would otherwise be another round trip to L2); the rest are re-read.
  float sv[kRowCache];
#pragma unroll
  for (int c = 0; c < kRowCache; ++c) {
    const int64_t d = tid + (int64_t)c * kRowThreads;
    sv[c] = d < n ? Sq[d] : 0.f;
  }
  // f(d, S[q, d]) for this thread's d in increasing order (static register indices first)
  auto each = [&](auto f) {
#pragma unroll
    for (int c = 0; c < kRowCache; ++c) {
      const int64_t d = tid + (int64_t)c * kRowThreads;
      if (d < n) f(d, sv[c]);
    }
    for (int64_t d = tid + (int64_t)kRowCache * kRowThreads; d < n; d += kRowThreads) f(d, Sq[d]);
  };
  float M = -__builtin_huge_valf();
  int64_t dM = n;
  each([&](int64_t d, float sd) {
    const float l = (s * sd);
    if (l > M) {
      M = l;
      dM = d;
    }
  });
  block_argmax(M, dM, redf, redi);
  // log-sum-exp = M + log1p(sum over d != dM of exp(l - M)): keeps the loss accurate when one
  // logit dominates (the loss is then ~ the small sum, which log(1 + x) would lose).
  float so = 0.f;
  each([&](int64_t d, float sd) {
    if (d != dM) so += expf((s * sd) - M);
  });
  so = block_sum(so, redf);
  const float l1p = log1pf(so);
  const float lse = M + l1p;
  const int64_t p = pos[q];
  const bool bad = p < 0 || p >= n;
  float term = 0.f;
  if (bad) {
    each([&](int64_t d, float sd) {
      if (scores_out) scores_out[(int64_t)q * n + d] = sd;
      Gq[d] = 0.f;
    });
    if (tid == 0) atomicOr(&ctrl[0], 2);
  } else {
    term = (M - (s * Sq[p])) + l1p;
    // G[q,d] = (s/B) softmax; the positive gets -(s/B) * (sum of the other probabilities),
    // which equals (s/B) (p_pos - 1) without the cancellation of 1 - p_pos in fp32.
    float rest = 0.f;
    each([&](int64_t d, float sd) {
      if (scores_out) scores_out[(int64_t)q * n + d] = sd;
      if (d != p) {
        const float e = expf((s * sd) - lse);
        Gq[d] = gscale * e;
        rest += e;
      }
    });
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

constexpr int kGqWaves = 4;
constexpr int kGqThreads = 64 * kGqWaves;
constexpr int kGqEntries = 4 * kGqWaves;  // (q, i) entries per workgroup: 16 lanes each
constexpr int kGqBatch = 4;               // documents whose rows a lane gathers at once

// dQ, first pass: workgroup (r, g) sums, for the 16 entries e = q * lq + i of group g, the
// gathered rows G[q,d] * D[token a(q,i,d)] over the documents of range r.  Ranges are placed on
// XCDs so that a range's document rows are gathered from its L2.  Lane: entry (lane >> 4),
// 8 columns at 8 * ((lane & 15) + 16 cc).  Partials part[r][e][:] are summed by the second pass
// in range order, so the result does not depend on scheduling.
template <int CPL>
__global__ __launch_bounds__(kGqThreads, CPL == 1 ? 8 : 4) void grad_q_part_kernel(
    const uint16_t* __restrict__ D, const int64_t* __restrict__ off, int64_t n_docs,
    int64_t n_tok, int dim, int nq, int lq, const uint16_t* __restrict__ amax,
    const float* __restrict__ G, float* __restrict__ part, float* __restrict__ dq, int n_groups,
    int R, bool direct) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t lin = xcd_linear(blockIdx.x, (int64_t)n_groups * R);
  const int r = (int)(lin / n_groups);
  const int grp = (int)(lin - (int64_t)r * n_groups);
  const int64_t E = (int64_t)nq * lq;
  const int64_t e = (int64_t)grp * kGqEntries + wave * 4 + (lane >> 4);
  const bool active = e < E;
  const int c = lane & 15;
  const int64_t d0 = n_docs * r / R, d1 = n_docs * (r + 1) / R;
  const int64_t last_tok = n_tok - 1;

  float acc[CPL][8];
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc)
#pragma unroll
    for (int v = 0; v < 8; ++v) acc[cc][v] = 0.f;

  // Documents in chunks of 32.  First, lane l loads the row index and weight of two of the
  // wave's four entries (2 (l >> 5) and the next) against document l & 31 of the chunk -- one
  // round trip for the chunk's metadata -- into the wave's table in LDS; then each 16-lane
  // group gathers its entry's rows, kGqBatch documents at a time, reading each document's (row,
  // weight) with one LDS load that the group's lanes share.  Small batches keep the kernel
  // within 64 VGPRs at dim <= 128: eight waves per SIMD, so every workgroup of the training
  // step is resident at once.  Only the wave itself reads its
  // table, and a wave's LDS accesses complete in order.
  __shared__ int2 meta[kGqWaves][4][32];
  const int mu = lane & 31, mh = lane >> 5;
  const int k = lane >> 4;  // this lane's entry within the wave
  for (int64_t db = d0; db < d1; db += 32) {
    const int64_t dm = db + mu;
    const bool okd = dm < d1;
    int64_t base = okd ? off[dm] : 0;
    base = base < 0 ? 0 : (base > last_tok ? last_tok : base);
    int rowm[2];
    float gm[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int64_t ek = (int64_t)grp * kGqEntries + wave * 4 + 2 * mh + t;
      const bool ok = okd && ek < E;
      const int64_t rr = base + (ok ? amax[dm * E + ek] : 0);
      rowm[t] = (int)(rr > last_tok ? last_tok : rr);
      gm[t] = ok ? G[(ek / lq) * n_docs + dm] : 0.f;
      meta[wave][2 * mh + t][mu] = make_int2(rowm[t], __float_as_int(gm[t]));
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int part = 0; part < 32 / kGqBatch; ++part) {
      if (db + kGqBatch * part >= d1) break;  // uniform
      u32x4 w[kGqBatch][CPL];
      float g[kGqBatch];
#pragma unroll
      for (int uu = 0; uu < kGqBatch; ++uu) {
        const int2 mt = meta[wave][k][kGqBatch * part + uu];
        const int64_t row = mt.x;
        g[uu] = __int_as_float(mt.y);
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) {
          const int kk = 8 * (c + 16 * cc);
          w[uu][cc] = kk < dim ? load16(D + row * dim + kk) : u32x4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int uu = 0; uu < kGqBatch; ++uu)
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) {
          acc[cc][0] += g[uu] * bf16_lo(w[uu][cc].x);
          acc[cc][1] += g[uu] * bf16_hi(w[uu][cc].x);
          acc[cc][2] += g[uu] * bf16_lo(w[uu][cc].y);
          acc[cc][3] += g[uu] * bf16_hi(w[uu][cc].y);
          acc[cc][4] += g[uu] * bf16_lo(w[uu][cc].z);
          acc[cc][5] += g[uu] * bf16_hi(w[uu][cc].z);
          acc[cc][6] += g[uu] * bf16_lo(w[uu][cc].w);
          acc[cc][7] += g[uu] * bf16_hi(w[uu][cc].w);
        }
    }
    __builtin_amdgcn_wave_barrier();  // the table is rewritten by the next chunk
  }
  if (!active) return;
  float* dst = (direct ? dq : part + (int64_t)r * E * dim) + e * dim;  // direct: final sums
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc) {
    const int k = 8 * (c + 16 * cc);
    if (k < dim) {
      *reinterpret_cast<f32x4*>(dst + k) = f32x4{acc[cc][0], acc[cc][1], acc[cc][2], acc[cc][3]};
      *reinterpret_cast<f32x4*>(dst + k + 4) = f32x4{acc[cc][4], acc[cc][5], acc[cc][6], acc[cc][7]};
    }
  }
}

// dQ, second pass: dq[i] = sum over ranges r = 0, 1, ... of part[r][i], 4 values at a time.
// Run by its own kernel, or folded into the first lines of grad_d_kernel (the next launch of the
// call), whose workgroups each take one slice of the values.
// dqc (optional, [nq][dim]): a per-query term added to every token's row (the contrastive part
// of the total loss).
__device__ __forceinline__ void grad_q_sum_ranges(const float* __restrict__ part, int R,
                                                  int64_t i0, int64_t i1, int64_t n4,
                                                  float* __restrict__ dq,
                                                  const float* __restrict__ dqc, int lq,
                                                  int dim) {
  const f32x4* p = reinterpret_cast<const f32x4*>(part);
  for (int64_t i = i0 + threadIdx.x; i < i1; i += blockDim.x) {
    f32x4 s = p[i];
    if (dqc) {
      const int64_t e = 4 * i / dim;
      const int64_t k = 4 * i - e * dim;
      s += *reinterpret_cast<const f32x4*>(dqc + (e / lq) * dim + k);
    }
    int r = 1;
    for (; r + 8 <= R; r += 8) {  // eight ranges' loads in flight, then added in range order
      f32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = p[(int64_t)(r + u) * n4 + i];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; r < R; ++r) s += p[(int64_t)r * n4 + i];
    reinterpret_cast<f32x4*>(dq)[i] = s;
  }
}

__global__ void grad_q_reduce_kernel(const float* __restrict__ part, int R, int64_t n4,
                                     float* __restrict__ dq, const float* __restrict__ dqc,
                                     int lq, int dim) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x;
  const int64_t i1 = i0 + blockDim.x < n4 ? i0 + blockDim.x : n4;
  grad_q_sum_ranges(part, R, i0, i1, n4, dq, dqc, lq, dim);
}

constexpr int kGdRows = 512;        // rows of a document sorted per pass
constexpr int kGdMaxStageQ = 4096;  // G[:, d] is staged in LDS when nq is at most this

// TPE threads read one Q row, CPT chunks of 16 bytes (8 columns) each: chunk c + TPE i of the
// row belongs to thread c of its group (dim <= 8 TPE CPT); an NT-thread workgroup has NT / TPE
// groups.  Fewer, wider threads per entry spread the per-position bookkeeping over more
// columns.
__host__ __device__ inline int gd_cpt(int dim) { return dim <= 64 ? 1 : dim <= 128 ? 2 : 4; }
__host__ __device__ inline int gd_tpe(int dim) { return 8; }

// LDS layout of grad_d_kernel (bytes, each part 16-byte aligned).
struct GdLds {
  int keys, sorted, weight, cnt, rs, gcol, total;
};
__host__ __device__ inline GdLds gd_lds(int E, int nq, int waves) {
  GdLds l;
  l.keys = 0;  // the document's argmax entries, staged once
  l.sorted = (2 * E + 15) / 16 * 16;
  l.weight = l.sorted + 4 * E;
  l.cnt = l.weight + 4 * E;
  l.rs = l.cnt + waves * kGdRows * 4;  // per-wave histograms
  l.gcol = l.rs + ((kGdRows + 1) * 4 + 15) / 16 * 16;
  l.total = l.gcol + (nq <= kGdMaxStageQ ? (4 * nq + 15) / 16 * 16 : 0);
  return l;
}

// dD: one workgroup per document d.  Entry e = q * lq + i selected token a(e) = amax[d][e] of
// the document; dD[j] = sum over the entries with a(e) = j, in entry order, of G[q,d] Q[e].
// The argmax entries (and G[:, d]) are staged in LDS.  Per pass over kGdRows rows:
//   1. a stable counting sort of the entries by token -- per-wave histograms over contiguous
//      entry ranges, a prefix scan, a ballot-ranked scatter in entry order -- lists each row's
//      entries contiguously, in entry order, with their weights G[q,d];
//   2. the sorted list is cut into one contiguous slice per group of TPE threads, at row
//      boundaries, each slice holding about the same number of entries (a row never
//      straddles two slices);
//   3. each group walks its slice in order, gathering whole 256-byte Q rows (TPE x 16 bytes,
//      straight from L2) a batch of positions ahead of the ones it adds, and writes each row once
//      it is complete -- zeros (or the contrastive part) for rows nobody selected.
// Deterministic: every row sums its entries in entry order, with no atomics on floats.
template <int TPE, int CPT, int NT>
__global__ __launch_bounds__(NT, NT >= 512 ? 4 : 2) void grad_d_kernel(
    const uint16_t* __restrict__ Q, const int64_t* __restrict__ off, int64_t n_docs,
    int64_t n_tok, int dim, int nq, int lq, uint64_t lq_magic,
    const uint16_t* __restrict__ amax, const float* __restrict__ G, float* __restrict__ dd,
    const float* __restrict__ dq_part, int dq_R, float* __restrict__ dq,
    const float* __restrict__ dqc, const float* __restrict__ ddc) {
  extern __shared__ __attribute__((aligned(16))) unsigned char gd_smem[];
  constexpr int kGroups = NT / TPE;
  constexpr int kRpt = kGdRows / NT;  // rows per thread in the scan
  if (dq_part) {  // the dQ range sums, one slice per workgroup (independent of the rest)
    const int64_t n4 = (int64_t)nq * lq * dim / 4;
    const int64_t per = (n4 + gridDim.x - 1) / gridDim.x;
    const int64_t i0 = per * blockIdx.x;
    grad_q_sum_ranges(dq_part, dq_R, i0, i0 + per < n4 ? i0 + per : n4, n4, dq, dqc, lq, dim);
  }
  const int E = nq * lq;
  const GdLds L = gd_lds(E, nq, NT / 64);  // the same layout the launcher sized
  uint16_t* am = reinterpret_cast<uint16_t*>(gd_smem + L.keys);
  uint32_t* spk = reinterpret_cast<uint32_t*>(gd_smem + L.sorted);
  float* sw = reinterpret_cast<float*>(gd_smem + L.weight);
  int* cnt = reinterpret_cast<int*>(gd_smem + L.cnt);
  int* rs = reinterpret_cast<int*>(gd_smem + L.rs);
  float* gcol = reinterpret_cast<float*>(gd_smem + L.gcol);
  __shared__ int wave_tot[(NT / 64)];
  __shared__ int bounds[kGroups + 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t d = blockIdx.x;
  const bool g_staged = nq <= kGdMaxStageQ;
  {
    const uint16_t* src = amax + d * E;
    const int nvec = (E % 8 == 0) ? E / 8 : 0;  // 16-byte loads need 16-byte aligned rows
    for (int i = tid; i < nvec; i += NT)
      reinterpret_cast<u32x4*>(am)[i] = load16(src + 8 * i);
    for (int e = 8 * nvec + tid; e < E; e += NT) am[e] = src[e];
    if (g_staged)
      for (int q = tid; q < nq; q += NT) gcol[q] = G[(int64_t)q * n_docs + d];
  }

  const int64_t last_tok = n_tok - 1;
  int64_t lo = off[d], hi = off[d + 1];
  lo = lo < 0 ? 0 : (lo > last_tok ? last_tok : lo);
  hi = hi <= lo ? lo + 1 : (hi > n_tok ? n_tok : hi);
  const int64_t len = hi - lo;
  // this wave's entries [eb, ee): contiguous, whole 64-entry chunks except at the end
  const int epw = ((E + (NT / 64) - 1) / (NT / 64) + 63) / 64 * 64;
  const int eb = wave * epw < E ? wave * epw : E;
  const int ee = eb + epw < E ? eb + epw : E;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  const int grp = tid / TPE;
  const int c = tid - grp * TPE;  // this thread's chunks: columns 8 (c + TPE i) .. + 7
  bool cok[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) cok[i] = 8 * (c + TPE * i) < dim;
  // the document's contrastive part (the same for each of its rows), or zeros
  float init[8 * CPT];
#pragma unroll
  for (int v = 0; v < 8 * CPT; ++v) init[v] = 0.f;
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    if (ddc && cok[i]) {
      const float* src = ddc + d * dim + 8 * (c + TPE * i);
      const f32x4 v0 = *reinterpret_cast<const f32x4*>(src);
      const f32x4 v1 = *reinterpret_cast<const f32x4*>(src + 4);
      init[8 * i + 0] = v0.x; init[8 * i + 1] = v0.y; init[8 * i + 2] = v0.z;
      init[8 * i + 3] = v0.w; init[8 * i + 4] = v1.x; init[8 * i + 5] = v1.y;
      init[8 * i + 6] = v1.z; init[8 * i + 7] = v1.w;
    }
  }

  for (int64_t w0 = 0; w0 < len; w0 += kGdRows) {
    const int Wn = (int)(len - w0 < kGdRows ? len - w0 : kGdRows);
    int nbits = 0;
    while ((1 << nbits) < Wn) ++nbits;
    for (int k = lane; k < Wn; k += 64) cnt[wave * kGdRows + k] = 0;
    __syncthreads();
    // per-wave histogram of the pass's tokens
    for (int e = eb + lane; e < ee; e += 64) {
      const int key = (int)am[e] - (int)w0;
      if (key >= 0 && key < Wn) atomicAdd(&cnt[wave * kGdRows + key], 1);
    }
    __syncthreads();
    // exclusive scan over (token, wave) in token-major order; thread t owns kRpt tokens
    {
      const int r_begin = tid * kRpt;
      int tot[kRpt];
      int sum = 0;
#pragma unroll
      for (int i = 0; i < kRpt; ++i) {
        const int row = r_begin + i;
        tot[i] = 0;
        if (row < Wn)
          for (int w = 0; w < (NT / 64); ++w) tot[i] += cnt[w * kGdRows + row];
        sum += tot[i];
      }
      int incl = sum;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
      if (lane == 63) wave_tot[wave] = incl;
      __syncthreads();
      int before = 0;
      for (int w = 0; w < wave; ++w) before += wave_tot[w];
      int run = before + incl - sum;
#pragma unroll
      for (int i = 0; i < kRpt; ++i) {
        const int row = r_begin + i;
        if (row < Wn) {
          rs[row] = run;
          int r2 = run;
          for (int w = 0; w < (NT / 64); ++w) {
            const int cw = cnt[w * kGdRows + row];
            cnt[w * kGdRows + row] = r2;
            r2 += cw;
          }
          run += tot[i];
        }
      }
      if (tid == NT - 1) rs[Wn] = before + incl;
    }
    __syncthreads();
    // stable scatter: in entry order within the wave, ranked among equal tokens by ballots;
    // each position also receives its entry's weight
    for (int base = eb; base < ee; base += 64) {
      const int e = base + lane;
      int key = -1;
      if (e < ee) key = (int)am[e] - (int)w0;
      const bool valid = key >= 0 && key < Wn;
      uint64_t peers = __ballot(valid);
      for (int b = 0; b < nbits; ++b) {
        const bool bit = valid && ((key >> b) & 1);
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
      }
      if (valid) {
        const int rank = __popcll(peers & lt_mask);
        const int n = __popcll(peers);
        const int start = cnt[wave * kGdRows + key];
        const uint32_t qq = (uint32_t)(((uint64_t)e * lq_magic) >> 32);
        spk[start + rank] = (uint32_t)e | ((uint32_t)key << 16);
        sw[start + rank] = g_staged ? gcol[qq] : G[(int64_t)qq * n_docs + d];
        if (rank == 0) cnt[wave * kGdRows + key] = start + n;
      }
    }
    __syncthreads();
    // slices: group g takes rows [bounds[g], bounds[g + 1]), cut where the sorted positions
    // pass g / kGroups of the pass's entries
    if (tid <= kGroups) {
      const int n = rs[Wn];
      int r = tid == 0 ? 0 : Wn;
      if (tid > 0 && tid < kGroups) {
        const int target = (int)(((int64_t)tid * n + kGroups - 1) / kGroups);
        int a = 0, b = Wn;  // first row whose entries start at or after the target
        while (a < b) {
          const int mid = (a + b) >> 1;
          if (rs[mid] < target)
            a = mid + 1;
          else
            b = mid;
        }
        r = a;
      }
      bounds[tid] = r;
    }
    __syncthreads();

    // ---- the group's walk over its slice of positions [p0, p1), in order.  Every position
    // carries its entry and row; a row is written when the next position belongs to another
    // row.  Positions past the slice are padding (weight 0, row kNoRow) and write nothing.
    {
      constexpr uint32_t kNoRow = 0xffffu;
      const int p0 = rs[bounds[grp]];
      const int p1 = rs[bounds[grp + 1]];
      float* drow0 = dd + (lo + w0) * dim + 8 * c;
      auto write_row = [&](uint32_t row, const float (&v)[8 * CPT]) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
          if (cok[i]) {
            float* dst = drow0 + (int64_t)row * dim + 8 * TPE * i;
            *reinterpret_cast<f32x4*>(dst) =
                f32x4{v[8 * i], v[8 * i + 1], v[8 * i + 2], v[8 * i + 3]};
            *reinterpret_cast<f32x4*>(dst + 4) =
                f32x4{v[8 * i + 4], v[8 * i + 5], v[8 * i + 6], v[8 * i + 7]};
          }
        }
      };
      float acc[8 * CPT];
#pragma unroll
      for (int v = 0; v < 8 * CPT; ++v) acc[v] = init[v];
      // two batches of positions in flight: the next one is loaded while this one is added
      constexpr int kB = CPT >= 4 ? 4 : NT >= 512 ? 2 : 8;  // positions per batch
      u32x4 wb[2][kB][CPT];
      float gb[2][kB];
      uint32_t rb[2][kB];
      auto load_batch = [&](int slot, int pb) {
#pragma unroll
        for (int u = 0; u < kB; ++u) {
          const int pos = pb + u;
          const bool ok = pos < p1;
          const uint32_t pk = spk[ok ? pos : p0];
          rb[slot][u] = ok ? pk >> 16 : kNoRow;
          gb[slot][u] = ok ? sw[pos] : 0.f;
          const uint16_t* qrow = Q + (int64_t)(pk & 0xffffu) * dim;
#pragma unroll
          for (int i = 0; i < CPT; ++i) {  // columns past dim re-read the row's last chunk
            const int col = 8 * (c + TPE * i) < dim ? 8 * (c + TPE * i) : dim - 8;
            wb[slot][u][i] = load16(qrow + col);
          }
        }
      };
      auto add_batch = [&](int slot, uint32_t next_row) {
#pragma unroll
        for (int u = 0; u < kB; ++u) {
          const float g = gb[slot][u];
#pragma unroll
          for (int i = 0; i < CPT; ++i) {
            const u32x4 w = wb[slot][u][i];
            acc[8 * i + 0] += g * bf16_lo(w.x);
            acc[8 * i + 1] += g * bf16_hi(w.x);
            acc[8 * i + 2] += g * bf16_lo(w.y);
            acc[8 * i + 3] += g * bf16_hi(w.y);
            acc[8 * i + 4] += g * bf16_lo(w.z);
            acc[8 * i + 5] += g * bf16_hi(w.z);
            acc[8 * i + 6] += g * bf16_lo(w.w);
            acc[8 * i + 7] += g * bf16_hi(w.w);
          }
          const uint32_t row = rb[slot][u];
          const uint32_t nrow = u + 1 < kB ? rb[slot][u + 1] : next_row;
          if (row != nrow && row != kNoRow) {  // the row's last entry: write it
            write_row(row, acc);
#pragma unroll
            for (int v = 0; v < 8 * CPT; ++v) acc[v] = init[v];
          }
        }
      };
      if (p0 < p1) load_batch(0, p0);
      for (int pb = p0; pb < p1; pb += 2 * kB) {
        const bool more1 = pb + kB < p1;
        if (more1) load_batch(1, pb + kB);
        add_batch(0, more1 ? rb[1][0] : kNoRow);
        if (!more1) break;
        const bool more0 = pb + 2 * kB < p1;
        if (more0) load_batch(0, pb + 2 * kB);
        add_batch(1, more0 ? rb[0][0] : kNoRow);
      }
    }
    // rows nobody selected: their value is the document's contrastive part (or zero), one
    // thread per row
    for (int r = tid; r < Wn; r += NT) {
      if (rs[r] != rs[r + 1]) continue;
      float* dst = dd + (lo + w0 + r) * dim;
      for (int k = 0; k < dim; k += 4) {
        f32x4 v = {0.f, 0.f, 0.f, 0.f};
        if (ddc) v = *reinterpret_cast<const f32x4*>(ddc + d * dim + k);
        *reinterpret_cast<f32x4*>(dst + k) = v;
      }
    }
    __syncthreads();  // the pass's LDS is reused by the next one
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
                          float gw, float* G, float* terms, float* loss, float* scores_out,
                          int32_t* ctrl, hipStream_t stream) {
  hipLaunchKernelGGL(infonce_kernel, dim3((unsigned)nq), dim3(kRowThreads), 0, stream, S, nq,
                     n_docs, pos, scale, gw, G, terms, loss, scores_out, ctrl);
  return hipGetLastError();
}

int grad_d_lds_bytes(int nq, int lq) { return gd_lds(nq * lq, nq, 4).total; }

int grad_q_ranges(int64_t n_docs, int64_t n_tok, int64_t E, int dim) {
  // about 2 MiB of document rows per range (an XCD's L2 holds its ranges' rows), at most 32
  // ranges and 64 MiB of partial sums
  int64_t R = (n_tok * dim * 2 + (2 << 20) - 1) / (2 << 20);
  const int64_t by_mem = ((int64_t)64 << 20) / (E * dim * 4 > 0 ? E * dim * 4 : 1);
  if (R > by_mem) R = by_mem;
  if (R > 32) R = 32;
  if (R > n_docs) R = n_docs;
  return R < 1 ? 1 : (int)R;
}

hipError_t launch_grad_q(const uint16_t* d_tok, const int64_t* off, int64_t n_docs, int64_t n_tok,
                         int dim, int nq, int lq, const uint16_t* amax, const float* G,
                         float* part, float* dq, bool defer_sum, const float* dqc,
                         hipStream_t stream) {
  const int64_t E = (int64_t)nq * lq;
  const int R = grad_q_ranges(n_docs, n_tok, E, dim);
  const int n_groups = (int)((E + kGqEntries - 1) / kGqEntries);
  const unsigned blocks = (unsigned)((int64_t)n_groups * R);
  const bool direct = R == 1 && !dqc;  // one range and nothing to add: write the final sums
  if (dim <= 128)
    hipLaunchKernelGGL(grad_q_part_kernel<1>, dim3(blocks), dim3(kGqThreads), 0, stream, d_tok,
                       off, n_docs, n_tok, dim, nq, lq, amax, G, part, dq, n_groups, R, direct);
  else
    hipLaunchKernelGGL(grad_q_part_kernel<2>, dim3(blocks), dim3(kGqThreads), 0, stream, d_tok,
                       off, n_docs, n_tok, dim, nq, lq, amax, G, part, dq, n_groups, R, direct);
  if (!direct && !defer_sum) {
    const int64_t n4 = E * dim / 4;
    hipLaunchKernelGGL(grad_q_reduce_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0,
                       stream, part, R, n4, dq, dqc, lq, dim);
  }
  return hipGetLastError();
}

template <int TPE, int CPT, int NT>
hipError_t launch_grad_d_nt(const uint16_t* q, const int64_t* off, int64_t n_docs, int64_t n_tok,
                           int dim, int nq, int lq, uint64_t magic, const uint16_t* amax,
                           const float* G, float* dd, const float* dq_part, int dq_R, float* dq,
                           const float* dqc, const float* ddc, hipStream_t stream) {
  const int lds = gd_lds(nq * lq, nq, NT / 64).total;
  if (lds > 65536) {  // beyond the default dynamic LDS limit (large nq * lq only)
    const hipError_t e = hipFuncSetAttribute((const void*)grad_d_kernel<TPE, CPT, NT>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((grad_d_kernel<TPE, CPT, NT>), dim3((unsigned)n_docs), dim3(NT), lds, stream,
                     q, off, n_docs, n_tok, dim, nq, lq, magic, amax, G, dd, dq_part, dq_R, dq,
                     dqc, ddc);
  return hipGetLastError();
}

// Up to dim 128 a document takes 8 waves (two workgroups per CU, four waves per SIMD, within
// 128 VGPRs: two positions per gather batch) when its LDS layout still fits two workgroups per
// CU; otherwise, and at dim 256 (whose rows need the registers), 4 waves.
template <int TPE, int CPT>
hipError_t launch_grad_d_t(const uint16_t* q, const int64_t* off, int64_t n_docs, int64_t n_tok,
                           int dim, int nq, int lq, uint64_t magic, const uint16_t* amax,
                           const float* G, float* dd, const float* dq_part, int dq_R, float* dq,
                           const float* dqc, const float* ddc, hipStream_t stream) {
  if constexpr (CPT <= 2) {
    if (2 * gd_lds(nq * lq, nq, 8).total <= 160 * 1024)
      return launch_grad_d_nt<TPE, CPT, 512>(q, off, n_docs, n_tok, dim, nq, lq, magic, amax, G,
                                             dd, dq_part, dq_R, dq, dqc, ddc, stream);
  }
  return launch_grad_d_nt<TPE, CPT, 256>(q, off, n_docs, n_tok, dim, nq, lq, magic, amax, G, dd,
                                         dq_part, dq_R, dq, dqc, ddc, stream);
}

hipError_t launch_grad_d(const uint16_t* q, const int64_t* off, int64_t n_docs, int64_t n_tok,
                         int dim, int nq, int lq, const uint16_t* amax, const float* G, float* dd,
                         const float* dq_part, float* dq, const float* dqc, const float* ddc,
                         hipStream_t stream) {
  const int dq_R = dq_part ? grad_q_ranges(n_docs, n_tok, (int64_t)nq * lq, dim) : 0;
  if (dq_R <= 1 && !dqc) dq_part = nullptr;  // one range, nothing to add: grad_q wrote dq
  // floor(e / lq) = (e * ceil(2^32 / lq)) >> 32 for e < 2^14 and lq <= 128: the product
  // overshoots e / lq by less than e / 2^32 < 2^-18, below the 1 / lq gap to the next integer.
  const uint64_t magic = (0x100000000ull + (uint64_t)lq - 1) / (uint64_t)lq;
  switch (gd_tpe(dim) * 8 + gd_cpt(dim)) {
    case 8 * 8 + 1: return launch_grad_d_t<8, 1>(q, off, n_docs, n_tok, dim, nq, lq, magic, amax, G, dd, dq_part, dq_R, dq, dqc, ddc, stream);
    case 8 * 8 + 2: return launch_grad_d_t<8, 2>(q, off, n_docs, n_tok, dim, nq, lq, magic, amax, G, dd, dq_part, dq_R, dq, dqc, ddc, stream);
    case 8 * 8 + 4: return launch_grad_d_t<8, 4>(q, off, n_docs, n_tok, dim, nq, lq, magic, amax, G, dd, dq_part, dq_R, dq, dqc, ddc, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_scale(float* x, int64_t n, const float* scale, hipStream_t stream) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(scale_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, x, n, scale);
  return hipGetLastError();
}

}  // namespace hpr
