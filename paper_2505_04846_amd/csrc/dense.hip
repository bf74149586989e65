// Exact inner-product top-k over a dense fp16 store (pooled single-vector retrieval).
//
// s[q, r] = <Q[q], X[r]> (fp16 MFMA, fp32 accumulate); the k best rows per query under
// (score desc, row asc).  The score matrix is never materialised:
//
//   1. Sample.  Rows [0, S) are scored exactly into a workspace matrix and the row top-k of it
//      is taken (the radix select of topk.hip).  Its k-th score theta_q is a lower bound on the
//      final k-th score, and every sample row outside the sample top-k is beaten by k sample
//      rows, so it cannot be in the answer.
//   2. Scan.  Rows [S, n) are scored by the GEMM kernel below, whose epilogue appends a row to
//      its query's candidate list only when its key beats the query's bound.  With a random
//      sample the expected list length is about k (n - S) / S.
//   3. Merge.  Per query, the exact top-k of (sample top-k) U (candidates) under a unique
//      64-bit key (score key, ~row).  A query whose list overflowed its capacity is queued (its
//      bound raised to the k-th key found so far, still a valid bound: k rows reach it).
//   4. Exact fallback for the queued queries, decided on the device: the k-th largest key of
//      {keys >= bound} by a radix select over the GEMM itself -- 8 rescans of rows [S, n), each
//      counting one byte of the 64-bit keys into per-query 256-bin histograms (in LDS, then
//      added to global memory), with the sample's entries counted by the select step -- then
//      one rescan that collects the keys >= that k-th key (exactly k with the sample's: keys
//      are unique, so the list cannot overflow) and a final merge.  These launches use
//      persistent grids that read the number of queued queries from the device and exit at
//      once when it is 0, so the call never synchronises with the host and is capturable in a
//      HIP graph.
//
// GEMM tile: 256 queries x 256 rows per 8-wave workgroup (each wave 64 x 128 = 2 x 4 blocks of
// v_mfma_f32_32x32x16_f16; 128 x 128 per wave at one wave per SIMD measured 20 % slower); K advances 32 halves per stage through a 4-deep LDS ring filled by
// direct-to-LDS loads (global_load_lds_dwordx4, a wave-uniform base plus 32-bit lane offsets),
// so two to three stages of loads are in flight while one is multiplied.  The loop is software
// pipelined with one barrier per stage, placed between the stage's two k-steps: the next
// stage's first operands are read from LDS while the current stage's last MFMAs run.  LDS rows
// are 64 bytes with the 16-byte chunk c of row r stored at position c ^ ((r >> 2) & 3), which
// keeps the MFMA operand reads free of bank conflicts (measured: none).  Workgroups that share
// a row tile are placed on one XCD so its rows come from HBM about once.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

typedef __attribute__((ext_vector_type(16))) float f32x16;

// Workgroup tile geometry: TQ queries x 256 rows, WQ x WR waves, an NST-deep LDS ring of
// K stages (32 halves each) holding the query tile then the row tile.
template <int TQ, int WQ, int WR, int NST, int MIN_WG>
struct GemmGeom {
  static constexpr int kTQ = TQ;                    // queries per workgroup tile
  static constexpr int kTR = 256;                   // rows per workgroup tile
  static constexpr int kKC = 32;                    // halves of K per stage
  static constexpr int kStages = NST;               // LDS ring depth
  static constexpr int kWQ = WQ;                    // waves along queries
  static constexpr int kWR = WR;                    // waves along rows
  static constexpr int kBQ = kTQ / (32 * kWQ);      // 32-query blocks per wave
  static constexpr int kBR = kTR / (32 * kWR);      // 32-row blocks per wave
  static constexpr int kWaves = kWQ * kWR;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kMinWG = MIN_WG;             // resident workgroups per CU to allow
  static constexpr int kRowBytes = kKC * 2;         // 64
  static constexpr int kQTileBytes = kTQ * kRowBytes;
  static constexpr int kXTileBytes = kTR * kRowBytes;
  static constexpr int kStageBytes = kQTileBytes + kXTileBytes;
  static constexpr int kQLoads = kQTileBytes / 1024;              // 1 KiB wave-loads of queries
  static constexpr int kLoadsPerWave = kStageBytes / 1024 / kWaves;  // 16-byte loads per lane
  static_assert(kStageBytes % (1024 * kWaves) == 0, "a stage splits evenly over the waves");
};
// Many queries: 256 x 256 tiles, 8 waves of 64 x 128 (2 x 4 blocks), one workgroup per CU.
using GeomWide = GemmGeom<256, 4, 2, 4, 1>;
// At most 64 queries: 64 x 256 tiles, 4 waves of 64 x 64 (2 x 2 blocks), two workgroups per CU
// (2 x 80 KiB of LDS).  The row stream is the bound there; the wide tile would multiply up to
// 192 padding queries per row.
using GeomNarrow = GemmGeom<64, 1, 4, 4, 2>;

// 16 zero bytes in global memory: the source of the K-tail chunks past `dim`.
__device__ __attribute__((aligned(16))) const uint32_t kZero16[4] = {0u, 0u, 0u, 0u};

struct GemmArgs {
  const uint16_t* q;      // fp16 [nqa, dim]
  const uint16_t* x;      // fp16 [n, dim]
  const int32_t* qmap;    // local query -> global query (nullptr: identity)
  int nqa;                // queries of this launch
  int dim;
  int64_t r0, r1;         // rows [r0, r1) of X
  int n_qt, n_rt;         // tiles along queries / rows
  // store mode
  float* scores;          // [nqa, ld], column c = row r0 + c
  int64_t ld;
  // filter mode
  const float* theta;     // [nq] bound score per global query
  const int64_t* tie;     // [nq] rows <= tie[q] pass on an equal score (-1: none)
  int32_t* count;         // [nq] appended candidates
  float* cand_s;          // [nq, cap]
  uint32_t* cand_i;       // [nq, cap]
  int64_t cap;
  // persistent launches: the number of queries (rows of q, entries of qmap) is *m_dev
  const int32_t* m_dev;
  // histogram mode: per local query, 256 bins of byte `shift / 8` of the keys >= the bound
  // whose bits above that byte equal prefix[global query]
  uint32_t* hist;                       // [m, 256]
  const unsigned long long* prefix;     // [nq]
  int shift;
};

enum GemmMode { kStore = 0, kFilter = 1, kHist = 2 };

// One 256-row tile of X against query tile qt (queries [qt kTQ, qt kTQ + kTQ) of the nqa of
// the launch).
template <typename G, int MODE>
__device__ __forceinline__ void gemm_tile(const GemmArgs& a, int nqa, int qt, int rt,
                                          unsigned char* smem) {
  constexpr int kTQ = G::kTQ, kTR = G::kTR, kKC = G::kKC, kStages = G::kStages;
  constexpr int kWQ = G::kWQ, kBQ = G::kBQ, kBR = G::kBR;
  constexpr int kRowBytes = G::kRowBytes, kQTileBytes = G::kQTileBytes;
  constexpr int kStageBytes = G::kStageBytes, kLoadsPerWave = G::kLoadsPerWave;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wq = wave % kWQ;  // (32 kBQ)-query slice of the tile
  const int wr = wave / kWQ;  // (32 kBR)-row slice of the tile
  const int q_base = qt * kTQ;
  const int64_t row_base = a.r0 + (int64_t)rt * kTR;

  // ---- this lane's direct-to-LDS sources: load j of the wave fills slot g = (L w + j) 64 + l
  // of the stage (L loads per wave; the query tile's slots first, then the row tile's).  Whether
  // a load reads queries or rows is uniform per (wave, j).  The source is a per-load base (the
  // tile's first row, advanced by each stage's K offset) plus a 32-bit per-lane byte offset
  // (row within the tile, clamped to the last valid row, and chunk).
  const char* q_tile = reinterpret_cast<const char*>(a.q + (int64_t)q_base * a.dim);
  const char* x_tile = reinterpret_cast<const char*>(a.x + row_base * a.dim);
  const int64_t q_rows = (int64_t)(nqa - q_base), x_rows = a.r1 - row_base;
  uint32_t voff[kLoadsPerWave];
  int src_c[kLoadsPerWave];
  bool is_x[kLoadsPerWave];
#pragma unroll
  for (int j = 0; j < kLoadsPerWave; ++j) {
    const int wl = wave * kLoadsPerWave + j;  // uniform
    is_x[j] = wl >= G::kQLoads;
    const int local = (is_x[j] ? wl - G::kQLoads : wl) * 64 + lane;
    int r = local >> 2;
    const int c = (local & 3) ^ ((r >> 2) & 3);
    const int64_t rows = is_x[j] ? x_rows : q_rows;
    r = r < rows ? r : (int)rows - 1;
    voff[j] = (uint32_t)r * (uint32_t)a.dim * 2u + 16u * c;
    src_c[j] = 8 * c;
  }
  const bool k_tail = (a.dim % kKC) != 0;
  // Loads stage `src_kk` of K into the ring buffer of stage `kk` (src_kk < kk only for the
  // filler stages past the last one, which keep the number of stages in flight constant).
  auto issue_stage = [&](int kk, int src_kk) {
    unsigned char* st = smem + (kk % kStages) * kStageBytes;
    const int k0 = src_kk * kKC;
    const char* qb = q_tile + 2 * (int64_t)k0;
    const char* xb = x_tile + 2 * (int64_t)k0;
    if (!k_tail || k0 + kKC <= a.dim) {
#pragma unroll
      for (int j = 0; j < kLoadsPerWave; ++j)
        __builtin_amdgcn_global_load_lds((glb_void_t*)((is_x[j] ? xb : qb) + voff[j]),
                                         (lds_void_t*)(st + (wave * kLoadsPerWave + j) * 1024),
                                         16, 0, 0);
    } else {  // the last, partial K chunk: chunks past `dim` read 16 zero bytes
#pragma unroll
      for (int j = 0; j < kLoadsPerWave; ++j) {
        const void* p = (k0 + src_c[j] < a.dim) ? (const void*)((is_x[j] ? xb : qb) + voff[j])
                                                 : (const void*)kZero16;
        __builtin_amdgcn_global_load_lds((glb_void_t*)p,
                                         (lds_void_t*)(st + (wave * kLoadsPerWave + j) * 1024),
                                         16, 0, 0);
      }
    }
  };

  // ---- per-lane LDS offsets of the MFMA operands: row `col` of block b, chunk 2 s + half
  const int col = lane & 31, half = lane >> 5;
  uint32_t offq[kBQ][2], offx[kBR][2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int c = 2 * s + half;
#pragma unroll
    for (int b = 0; b < kBQ; ++b) {
      const int r = wq * 32 * kBQ + 32 * b + col;
      offq[b][s] = r * kRowBytes + 16 * (c ^ ((r >> 2) & 3));
    }
#pragma unroll
    for (int b = 0; b < kBR; ++b) {
      const int r = wr * 32 * kBR + 32 * b + col;
      offx[b][s] = kQTileBytes + r * kRowBytes + 16 * (c ^ ((r >> 2) & 3));
    }
  }

  f32x16 acc[kBQ][kBR];
#pragma unroll
  for (int i = 0; i < kBQ; ++i)
#pragma unroll
    for (int j = 0; j < kBR; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Software pipeline over the K stages.  Every iteration issues exactly one stage of loads
  // (past the last stage it reloads the last one into a buffer nobody reads again), so "stage
  // kk+1 has landed" is always "at most one stage of this wave's loads is still in flight".
  const int nk = (a.dim + kKC - 1) / kKC;
#pragma unroll
  for (int s = 0; s < kStages - 1; ++s) issue_stage(s, s < nk ? s : nk - 1);

  struct Frags {
    f16x8 a[kBQ], b[kBR];
  };
  auto read_frags = [&](int kk, int s, Frags& f) {
    const unsigned char* st = smem + (kk % kStages) * kStageBytes;
#pragma unroll
    for (int b = 0; b < kBQ; ++b) f.a[b] = as_f16x8(*reinterpret_cast<const u32x4*>(st + offq[b][s]));
#pragma unroll
    for (int b = 0; b < kBR; ++b) f.b[b] = as_f16x8(*reinterpret_cast<const u32x4*>(st + offx[b][s]));
  };
  auto mfma = [&](const Frags& f) {
#pragma unroll
    for (int i = 0; i < kBQ; ++i)
#pragma unroll
      for (int j = 0; j < kBR; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
  };
  auto barrier = [&]() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };

  Frags f0, f1;
  static_assert(kStages == 4, "the waits below assume two stages in flight");
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * kLoadsPerWave));  // stage 0 landed (this wave)
  barrier();                                                // ... and for every wave
  read_frags(0, 0, f0);
#pragma unroll 1
  for (int kk = 0; kk < nk; ++kk) {
    read_frags(kk, 1, f1);
    mfma(f0);
    // Stage kk+1 lands everywhere, and every wave's reads of stage kk-1 are complete (this
    // wave's LDS reads drain before the barrier), so that stage's buffer ((kk + 3) % 4) can
    // take stage kk+3.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(kLoadsPerWave));
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    barrier();
    const int nxt = kk + kStages - 1;
    issue_stage(nxt, nxt < nk ? nxt : nk - 1);
    read_frags(kk + 1 < nk ? kk + 1 : kk, 0, f0);
    __builtin_amdgcn_sched_barrier(0);  // the next stage's reads go out before these MFMAs
    mfma(f1);
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // no load may still target LDS when the kernel ends

  // ---- epilogue.  acc[i][j] register r: query q_base + 32 kBQ wq + 32 i + 8 (r / 4) +
  // 4 half + r % 4, row row_base + 32 kBR wr + 32 j + col.
  if constexpr (MODE == kHist) {
    // per-tile histograms in LDS (the ring is no longer read once every wave has passed the
    // barrier), then the non-zero bins added to the launch's histograms
    static_assert(kTQ * 256 * 4 <= G::kStages * kStageBytes, "histograms fit the LDS ring");
    uint32_t* hl = reinterpret_cast<uint32_t*>(smem);
    barrier();
    for (int e = tid; e < kTQ * 256; e += G::kThreads) hl[e] = 0u;
    barrier();
    const unsigned long long pmask = a.shift >= 56 ? 0ull : (~0ull << (a.shift + 8));
#pragma unroll
    for (int i = 0; i < kBQ; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qo = 32 * kBQ * wq + 32 * i + 8 * (r >> 2) + 4 * half + (r & 3);
        const int ql = q_base + qo;
        if (ql >= nqa) continue;
        const int gq = a.qmap[ql];
        const float th = a.theta[gq];
        const int64_t tie = a.tie[gq];
        const unsigned long long pre = a.prefix[gq];
#pragma unroll
        for (int j = 0; j < kBR; ++j) {
          const int64_t row = row_base + 32 * kBR * wr + 32 * j + col;
          const float v = acc[i][j][r];
          if (row < a.r1 && (v > th || (v == th && row <= tie))) {
            const unsigned long long key =
                ((unsigned long long)score_key(v) << 32) | (unsigned long long)(uint32_t)~(uint32_t)row;
            if (((key ^ pre) & pmask) == 0ull)
              atomicAdd(&hl[qo * 256 + (int)((key >> a.shift) & 255ull)], 1u);
          }
        }
      }
    }
    barrier();
    for (int e = tid; e < kTQ * 256; e += G::kThreads) {
      const uint32_t c = hl[e];
      if (c != 0u && q_base + (e >> 8) < nqa) atomicAdd(&a.hist[(int64_t)(q_base + (e >> 8)) * 256 + (e & 255)], c);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < kBQ; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int ql = q_base + 32 * kBQ * wq + 32 * i + 8 * (r >> 2) + 4 * half + (r & 3);
      if (ql >= nqa) continue;
      if (MODE == kStore) {
        float* dst = a.scores + (int64_t)ql * a.ld + (row_base - a.r0) + 32 * kBR * wr + col;
#pragma unroll
        for (int j = 0; j < kBR; ++j) {
          const int64_t row = row_base + 32 * kBR * wr + 32 * j + col;
          if (row < a.r1) dst[32 * j] = acc[i][j][r];
        }
      } else {
        const int gq = a.qmap ? a.qmap[ql] : ql;
        const float th = a.theta[gq];
        const int64_t tie = a.tie[gq];
#pragma unroll
        for (int j = 0; j < kBR; ++j) {
          const int64_t row = row_base + 32 * kBR * wr + 32 * j + col;
          const float v = acc[i][j][r];
          if (row < a.r1 && (v > th || (v == th && row <= tie))) {
            const int p = atomicAdd(&a.count[gq], 1);
            if (p < a.cap) {
              a.cand_s[(int64_t)gq * a.cap + p] = v;
              a.cand_i[(int64_t)gq * a.cap + p] = (uint32_t)row;
            }
          }
        }
      }
    }
  }
}

// One tile per workgroup (workgroups sharing a row tile on one XCD), or, when PERSIST, a grid
// that walks the tiles of the *m_dev queries of the launch (none when it is 0).
template <typename G, int MODE, bool PERSIST>
__global__ __launch_bounds__(G::kThreads, G::kMinWG) void dense_gemm_kernel(GemmArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  if constexpr (PERSIST) {
    const int nqa = __builtin_amdgcn_readfirstlane(*a.m_dev);
    if (nqa <= 0) return;
    const int n_qt = (nqa + G::kTQ - 1) / G::kTQ;
    const int64_t total = (int64_t)n_qt * a.n_rt;
    for (int64_t t = blockIdx.x; t < total; t += gridDim.x) {
      __syncthreads();  // the previous tile's LDS reads are complete before the ring refills
      const int rt = (int)(t / n_qt);
      gemm_tile<G, MODE>(a, nqa, (int)(t - (int64_t)rt * n_qt), rt, smem);
    }
  } else {
    const int64_t total = (int64_t)a.n_qt * a.n_rt;
    const int64_t lin = xcd_linear(blockIdx.x, total);
    const int rt = (int)(lin / a.n_qt);
    gemm_tile<G, MODE>(a, a.nqa, (int)(lin - (int64_t)rt * a.n_qt), rt, smem);
  }
}

// Bound of every query from its sample top-k: theta = k-th score, strict comparison; lists
// emptied; the queue of overflowing queries emptied.
__global__ void dense_init_kernel(const float* ss, int nq, int k, float* theta, int64_t* tie,
                                  int32_t* count, int32_t* n_queued) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q == 0) *n_queued = 0;
  if (q >= nq) return;
  theta[q] = ss[(int64_t)q * k + k - 1];
  tie[q] = -1;
  count[q] = 0;
}

// Queued queries (*m_dev of them): their Q rows are gathered into qc and their histograms
// zeroed.
__global__ void dense_fallback_prep_kernel(const uint16_t* q, int dim, const int32_t* qlist,
                                           const int32_t* m_dev, uint16_t* qc, uint32_t* hist) {
  const int m = *m_dev;
  for (int i = blockIdx.x; i < m; i += gridDim.x) {
    const int gq = qlist[i];
    const u32x4* s = reinterpret_cast<const u32x4*>(q + (int64_t)gq * dim);
    u32x4* d = reinterpret_cast<u32x4*>(qc + (int64_t)i * dim);
    for (int c = threadIdx.x; c < dim / 8; c += blockDim.x) d[c] = s[c];
    for (int c = threadIdx.x; c < 256; c += blockDim.x) hist[(int64_t)i * 256 + c] = 0u;
  }
}

// One radix step of the exact fallback for queued query i (one workgroup each; none past
// *m_dev): the query's scan histogram (hist[i], then zeroed for the next pass) plus its sample
// top-k entries with key >= the bound and the same prefix give the byte of the k-th key at
// `shift`; after the last byte (shift 0) the bound becomes that key, inclusive, and the list is
// emptied for the collecting rescan.
__global__ __launch_bounds__(256) void dense_radix_kernel(
    const int32_t* m_dev, const int32_t* qlist, int shift, const float* ss, const int64_t* si,
    int k, uint32_t* hist, unsigned long long* prefix, uint32_t* remaining, float* theta,
    int64_t* tie, int32_t* count) {
  __shared__ uint32_t h[256];
  __shared__ uint32_t sh_bin, sh_above;
  const int i = blockIdx.x;
  if (i >= *m_dev) return;  // uniform
  const int q = qlist[i];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const unsigned long long pmask = shift >= 56 ? 0ull : (~0ull << (shift + 8));
  const unsigned long long pre = prefix[q];
  const float th = theta[q];
  const int64_t tb = tie[q];
  h[tid] = hist[(int64_t)i * 256 + tid];
  hist[(int64_t)i * 256 + tid] = 0u;
  if (tid == 0) {
    sh_bin = 0u;
    sh_above = 0u;
  }
  __syncthreads();
  for (int e = tid; e < k; e += 256) {
    const float v = ss[(int64_t)q * k + e];
    const int64_t row = si[(int64_t)q * k + e];
    if (v > th || (v == th && row <= tb)) {
      const unsigned long long key =
          ((unsigned long long)score_key(v) << 32) | (unsigned long long)(uint32_t)~(uint32_t)row;
      if (((key ^ pre) & pmask) == 0ull) atomicAdd(&h[(int)((key >> shift) & 255ull)], 1u);
    }
  }
  __syncthreads();
  const uint32_t rem = remaining[q];
  if (wave == 0) {  // the bin holding the rem-th largest key, counting from bin 255 down
    uint32_t c[4], tot = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      c[j] = h[255 - 4 * lane - j];
      tot += c[j];
    }
    uint32_t incl = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    const uint32_t excl = incl - tot;
    if (excl < rem && rem <= incl) {
      uint32_t accu = excl;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (accu + c[j] >= rem) {
          sh_bin = 255u - 4u * lane - j;
          sh_above = accu;
          break;
        }
        accu += c[j];
      }
    }
  }
  __syncthreads();
  if (tid == 0) {
    const unsigned long long np = pre | ((unsigned long long)sh_bin << shift);
    prefix[q] = np;
    remaining[q] = rem - sh_above;
    if (shift == 0) {  // np is the k-th largest key: collect every key >= it
      theta[q] = key_score((uint32_t)(np >> 32));
      tie[q] = (int64_t)(uint32_t)~(uint32_t)np;
      count[q] = 0;
    }
  }
}

constexpr int kMergeThreads = 1024;
constexpr int kMergeMaxK = 1024;

// Exact top-k of (sample top-k of query q) U (its candidates) under the unique key
// (score key << 32) | ~row: 8 radix passes of 8 bits find the k-th key K, the elements with key
// >= K are gathered (exactly k: keys are unique) and bitonic-sorted.  With a queue
// (n_queued != nullptr), a query whose list overflowed gets its bound raised to K, its radix
// state reset (prefix 0, k keys to find) and is appended to qlist_out; its output is rewritten
// by the fallback.  With m_dev, block b merges queued query qsel[b] when b < *m_dev.
__global__ __launch_bounds__(kMergeThreads) void dense_merge_kernel(
    const float* ss, const int64_t* si, int k, const int32_t* count, const float* cand_s,
    const uint32_t* cand_i, int64_t cap, const int32_t* qsel, const int32_t* m_dev,
    float* out_s, int64_t* out_i, float* theta, int64_t* tie, int32_t* n_queued,
    int32_t* qlist_out, unsigned long long* q_prefix, uint32_t* q_remaining) {
  __shared__ uint32_t hist[256];
  __shared__ unsigned long long sk[kMergeMaxK];
  __shared__ uint32_t sh_bin, sh_above, sh_n;
  if (m_dev && (int)blockIdx.x >= *m_dev) return;  // uniform
  const int q = qsel ? qsel[blockIdx.x] : (int)blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int cnt = count[q];
  const int64_t m_c = cnt < cap ? cnt : cap;
  const int64_t m = k + m_c;
  auto key_at = [&](int64_t e) -> unsigned long long {
    float s;
    uint32_t row;
    if (e < k) {
      s = ss[(int64_t)q * k + e];
      row = (uint32_t)si[(int64_t)q * k + e];
    } else {
      s = cand_s[(int64_t)q * cap + (e - k)];
      row = cand_i[(int64_t)q * cap + (e - k)];
    }
    return ((unsigned long long)score_key(s) << 32) | (unsigned long long)(~row);
  };

  unsigned long long prefix = 0, pmask = 0;
  uint32_t remaining = (uint32_t)k;
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
    if (tid < 256) hist[tid] = 0;
    if (tid == 0) {
      sh_bin = 0;
      sh_above = 0;
    }
    __syncthreads();
    for (int64_t e = tid; e < m; e += kMergeThreads) {
      const unsigned long long key = key_at(e);
      if ((key & pmask) == prefix) atomicAdd(&hist[(uint32_t)(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      uint32_t c[4], tot = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = hist[255 - 4 * lane - j];
        tot += c[j];
      }
      uint32_t incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
      const uint32_t excl = incl - tot;
      if (excl < remaining && remaining <= incl) {
        uint32_t accu = excl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (accu + c[j] >= remaining) {
            sh_bin = 255u - 4u * lane - j;
            sh_above = accu;
            break;
          }
          accu += c[j];
        }
      }
    }
    __syncthreads();
    prefix |= (unsigned long long)sh_bin << shift;
    pmask |= 255ull << shift;
    remaining -= sh_above;
    __syncthreads();
  }
  const unsigned long long K = prefix;  // the k-th largest key

  if (tid == 0) sh_n = 0;
  __syncthreads();
  for (int64_t e = tid; e < m; e += kMergeThreads) {
    const unsigned long long key = key_at(e);
    if (key >= K) {
      const uint32_t p = atomicAdd(&sh_n, 1u);
      if (p < (uint32_t)k) sk[p] = key;
    }
  }
  __syncthreads();
  uint32_t P = 1;
  while (P < (uint32_t)k) P <<= 1;
  for (uint32_t i = k + tid; i < P; i += kMergeThreads) sk[i] = 0ull;
  for (uint32_t size = 2; size <= P; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      for (uint32_t i = tid; i < P; i += kMergeThreads) {
        const uint32_t j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;  // descending runs where `up`
          const unsigned long long ki = sk[i], kj = sk[j];
          if ((kj > ki) == up) {
            sk[i] = kj;
            sk[j] = ki;
          }
        }
      }
    }
  }
  __syncthreads();
  for (int p = tid; p < k; p += kMergeThreads) {
    out_s[(int64_t)q * k + p] = key_score((uint32_t)(sk[p] >> 32));
    out_i[(int64_t)q * k + p] = (int64_t)(uint32_t)~(uint32_t)sk[p];
  }
  if (n_queued && cnt > cap && tid == 0) {
    theta[q] = key_score((uint32_t)(K >> 32));
    tie[q] = (int64_t)(uint32_t)~(uint32_t)K;
    q_prefix[q] = 0ull;
    q_remaining[q] = (uint32_t)k;
    const int slot = atomicAdd(n_queued, 1);
    qlist_out[slot] = q;
  }
}

}  // namespace

namespace {

template <typename G, int MODE, bool PERSIST>
hipError_t launch_gemm_t(const GemmArgs& a, unsigned blocks, hipStream_t stream) {
  const int lds = G::kStages * G::kStageBytes;
  const void* fn = (const void*)dense_gemm_kernel<G, MODE, PERSIST>;
  const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((dense_gemm_kernel<G, MODE, PERSIST>), dim3(blocks), dim3(G::kThreads), lds,
                     stream, a);
  return hipGetLastError();
}

template <typename G, int MODE>
hipError_t launch_gemm_grid(GemmArgs a, int64_t n_rt, hipStream_t stream) {
  a.n_qt = (a.nqa + G::kTQ - 1) / G::kTQ;
  if (n_rt < 1 || n_rt > 0x7fffffffLL || (int64_t)a.n_qt * n_rt > 0xffffffffLL)
    return hipErrorInvalidValue;
  a.n_rt = (int)n_rt;
  return launch_gemm_t<G, MODE, false>(a, (unsigned)((int64_t)a.n_qt * n_rt), stream);
}

}  // namespace

hipError_t launch_dense_gemm(const DenseGemm& g, int n_cu, hipStream_t stream) {
  if (g.nqa < 1 || g.r1 <= g.r0) return hipErrorInvalidValue;
  GemmArgs a = {};
  a.q = g.q;
  a.x = g.x;
  a.qmap = g.qmap;
  a.nqa = g.nqa;
  a.dim = g.dim;
  a.r0 = g.r0;
  a.r1 = g.r1;
  a.scores = g.scores;
  a.ld = g.ld;
  a.theta = g.theta;
  a.tie = g.tie;
  a.count = g.count;
  a.cand_s = g.cand_s;
  a.cand_i = g.cand_i;
  a.cap = g.cap;
  a.m_dev = g.m_dev;
  a.hist = g.hist;
  a.prefix = g.prefix;
  a.shift = g.shift;
  const int64_t n_rt = (g.r1 - g.r0 + 255) / 256;
  if (g.m_dev) {  // persistent narrow-tile grid over the *m_dev queued queries
    if (n_rt > 0x7fffffffLL || !g.qmap) return hipErrorInvalidValue;
    a.n_rt = (int)n_rt;
    const unsigned blocks = (unsigned)((n_cu > 0 ? n_cu : 256) * GeomNarrow::kMinWG);
    if (g.mode == kHist) return launch_gemm_t<GeomNarrow, kHist, true>(a, blocks, stream);
    if (g.mode == kFilter) return launch_gemm_t<GeomNarrow, kFilter, true>(a, blocks, stream);
    return hipErrorInvalidValue;
  }
  const bool narrow = g.nqa <= GeomNarrow::kTQ;
  switch (g.mode) {
    case kStore:
      return narrow ? launch_gemm_grid<GeomNarrow, kStore>(a, n_rt, stream)
                    : launch_gemm_grid<GeomWide, kStore>(a, n_rt, stream);
    case kFilter:
      return narrow ? launch_gemm_grid<GeomNarrow, kFilter>(a, n_rt, stream)
                    : launch_gemm_grid<GeomWide, kFilter>(a, n_rt, stream);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_dense_init(const float* ss, int nq, int k, float* theta, int64_t* tie,
                             int32_t* count, int32_t* n_queued, hipStream_t stream) {
  hipLaunchKernelGGL(dense_init_kernel, dim3((nq + 255) / 256), dim3(256), 0, stream, ss, nq, k,
                     theta, tie, count, n_queued);
  return hipGetLastError();
}

hipError_t launch_dense_merge(const float* ss, const int64_t* si, int nq_grid, int k,
                              const int32_t* count, const float* cand_s, const uint32_t* cand_i,
                              int64_t cap, const int32_t* qsel, const int32_t* m_dev,
                              float* out_s, int64_t* out_i, float* theta, int64_t* tie,
                              int32_t* n_queued, int32_t* qlist_out, unsigned long long* prefix,
                              uint32_t* remaining, hipStream_t stream) {
  if (k < 1 || k > kMergeMaxK || nq_grid < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dense_merge_kernel, dim3((unsigned)nq_grid), dim3(kMergeThreads), 0, stream,
                     ss, si, k, count, cand_s, cand_i, cap, qsel, m_dev, out_s, out_i, theta, tie,
                     n_queued, qlist_out, prefix, remaining);
  return hipGetLastError();
}

hipError_t launch_dense_fallback_prep(const uint16_t* q, int dim, const int32_t* qlist,
                                      const int32_t* m_dev, uint16_t* qc, uint32_t* hist,
                                      int n_cu, hipStream_t stream) {
  hipLaunchKernelGGL(dense_fallback_prep_kernel, dim3((unsigned)(n_cu > 0 ? n_cu : 256)),
                     dim3(256), 0, stream, q, dim, qlist, m_dev, qc, hist);
  return hipGetLastError();
}

hipError_t launch_dense_radix(const int32_t* m_dev, const int32_t* qlist, int nq_grid, int shift,
                              const float* ss, const int64_t* si, int k, uint32_t* hist,
                              unsigned long long* prefix, uint32_t* remaining, float* theta,
                              int64_t* tie, int32_t* count, hipStream_t stream) {
  hipLaunchKernelGGL(dense_radix_kernel, dim3((unsigned)nq_grid), dim3(256), 0, stream, m_dev,
                     qlist, shift, ss, si, k, hist, prefix, remaining, theta, tie, count);
  return hipGetLastError();
}

}  // namespace hpr
