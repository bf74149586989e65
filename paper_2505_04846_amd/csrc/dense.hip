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
// v_mfma_f32_32x32x16_f16; 128 x 128 per wave at one wave per SIMD measured 20 % slower).  K
// advances 64 halves per stage through two 64 KiB LDS buffers filled by direct-to-LDS buffer
// loads (buffer_load_dwordx4 ... lds: a tile base in the resource, the stage's K offset as the
// scalar offset, a 32-bit lane offset), each wave load covering 8 whole 128-byte row segments:
// on this chip the direct-to-LDS path moves data at about twice the rate with whole cache lines
// as with the half lines of 32-half stages, and the copy into LDS, not the MFMA, is what bounds
// the loop (without it the same loop runs at the MFMA rate).  One barrier per stage, placed
// before the stage's last k-step, whose MFMAs run while the next stage's first operands are
// read.  In LDS the 16-byte chunk p of row r is stored at position p ^ ((r >> 2) & 3), which
// keeps the operand reads free of bank conflicts.  Calls with at most 64 queries use a narrow
// 64 x 256 tile (4 waves, two workgroups per CU, a 4-deep ring of 32-half stages): there the
// row stream from HBM is the bound.  The filter epilogue compacts the passing entries per lane
// in LDS and appends them with one round of list atomics per slot.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

typedef __attribute__((ext_vector_type(16))) float f32x16;

// Workgroup tile geometry: TQ queries x 256 rows, WQ x WR waves, an NST-deep LDS ring of
// K stages of KC halves each, holding the query tile then the row tile.
//
// LDS layout of a stage: 1 KiB blocks, one per 16-byte-per-lane wave load, each holding
// R = 512 / KC rows.  A block is KC / 32 sub-blocks, sub-block h holding halves
// [32 h, 32 h + 32) of the stage for the block's R rows as 64-byte rows; the 16-byte chunk p of
// row r is stored at position p ^ ((r >> 2) & 3).  With KC = 64 one wave load reads 8 whole
// 128-byte rows (full cache lines); with KC = 32, 16 half lines.
template <int TQ, int WQ, int WR, int KC, int NST, int MIN_WG>
struct GemmGeom {
  static constexpr int kTQ = TQ;                    // queries per workgroup tile
  static constexpr int kTR = 256;                   // rows per workgroup tile
  static constexpr int kKC = KC;                    // halves of K per stage
  static constexpr int kKSteps = KC / 16;           // MFMA k-steps per stage
  static constexpr int kRowsPerBlock = 512 / KC;    // rows per 1 KiB block
  static constexpr int kStages = NST;               // LDS ring depth
  static constexpr int kWQ = WQ;                    // waves along queries
  static constexpr int kWR = WR;                    // waves along rows
  static constexpr int kBQ = kTQ / (32 * kWQ);      // 32-query blocks per wave
  static constexpr int kBR = kTR / (32 * kWR);      // 32-row blocks per wave
  static constexpr int kWaves = kWQ * kWR;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kMinWG = MIN_WG;             // resident workgroups per CU to allow
  static constexpr int kRowBytes = kKC * 2;
  static constexpr int kQTileBytes = kTQ * kRowBytes;
  static constexpr int kXTileBytes = kTR * kRowBytes;
  static constexpr int kStageBytes = kQTileBytes + kXTileBytes;
  static constexpr int kQLoads = kQTileBytes / 1024;              // 1 KiB wave-loads of queries
  static constexpr int kLoadsPerWave = kStageBytes / 1024 / kWaves;  // 16-byte loads per lane
  static_assert(KC == 32 || KC == 64, "stages of 32 or 64 halves");
  static_assert(kStageBytes % (1024 * kWaves) == 0, "a stage splits evenly over the waves");
  static_assert(kQTileBytes % 1024 == 0, "no wave load straddles the two tiles");
  static_assert(32 * kBQ <= 64, "a wave's queries fit one lane each");
};
// Many queries: 256 x 256 tiles, 8 waves of 64 x 128 (2 x 4 blocks), one workgroup per CU; two
// 64 KiB stages of 64 halves.
using GeomWide = GemmGeom<256, 4, 2, 64, 2, 1>;
// At most 64 queries: 64 x 256 tiles, 4 waves of 64 x 64 (2 x 2 blocks), two workgroups per CU
// (2 x 80 KiB of LDS), a 4-deep ring of 20 KiB stages.  The row stream is the bound there; the
// wide tile would multiply up to 192 padding queries per row.
using GeomNarrow = GemmGeom<64, 1, 4, 32, 4, 2>;

// 16 zero bytes in global memory: the source of the K-tail chunks past `dim`.
__device__ __attribute__((aligned(16))) const uint32_t kZero16[4] = {0u, 0u, 0u, 0u};
// A raw buffer resource over `base` (stride 0, byte-sized records, 32-bit data format, range
// 2^31 - 1 bytes: the callers' offsets stay far below it).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff,
                                           0x00020000);
}
// 16 bytes per lane from base + voff + soff into LDS at lds + 16 lane (the wave's block).
__device__ __forceinline__ void buffer_load_lds16(__amdgpu_buffer_rsrc_t r, unsigned char* lds,
                                                  uint32_t voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)lds, 16, (int)voff, soff, 0, 0);
}

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
  constexpr int kWQ = G::kWQ, kBQ = G::kBQ, kBR = G::kBR, kKSteps = G::kKSteps;
  constexpr int kR = G::kRowsPerBlock, kQTileBytes = G::kQTileBytes;
  constexpr int kStageBytes = G::kStageBytes, kLoadsPerWave = G::kLoadsPerWave;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wq = wave % kWQ;  // (32 kBQ)-query slice of the tile
  const int wr = wave / kWQ;  // (32 kBR)-row slice of the tile
  const int q_base = qt * kTQ;
  const int64_t row_base = a.r0 + (int64_t)rt * kTR;

  // ---- filter bounds of the wave's queries, one per lane, loaded now so that their latency
  // hides behind the K loop: lane l holds query q_base + 32 kBQ wq + l.
  float th_l = 0.f;
  int64_t tie_l = -1;
  int gq_l = 0;
  if constexpr (MODE == kFilter) {
    const int ql = q_base + 32 * kBQ * wq + lane;
    if (lane < 32 * kBQ && ql < nqa) {
      gq_l = a.qmap ? a.qmap[ql] : ql;
      th_l = a.theta[gq_l];
      tie_l = a.tie[gq_l];
    }
  }

  // ---- this lane's direct-to-LDS sources: load j of the wave fills block (L w + j) of the
  // stage (L loads per wave; the query tile's blocks first, then the row tile's), lane l
  // writing 16 bytes at byte 16 l of the block: sub-block h = (l / 4) / R, row (l / 4) % R of
  // the block, position l % 4.  Whether a load reads queries or rows is uniform per (wave, j).
  // The source is a per-load base (the tile's first row, advanced by each stage's K offset)
  // plus a 32-bit per-lane byte offset (row within the tile, clamped to the last valid row, and
  // chunk).
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
    const int blk = is_x[j] ? wl - G::kQLoads : wl;
    int r = blk * kR + (lane >> 2) % kR;
    const int c = 4 * ((lane >> 2) / kR) + ((lane & 3) ^ ((r >> 2) & 3));
    const int64_t rows = is_x[j] ? x_rows : q_rows;
    r = r < rows ? r : (int)rows - 1;
    voff[j] = (uint32_t)r * (uint32_t)a.dim * 2u + 16u * c;
    src_c[j] = 8 * c;
  }
  // Loads K stage src_kk into ring buffer `buf`.  Whole stages use buffer loads (the tile's
  // first row as base, the stage's K offset as scalar offset, the lane's 32-bit offset); the
  // stage with the K tail, and any stage past the last (src_kk >= nk, which keeps the number of
  // loads in flight constant), use global loads whose chunks past `dim` read 16 zero bytes.
  const int nk = (a.dim + kKC - 1) / kKC;
  const int nk_full = a.dim / kKC;
  const __amdgpu_buffer_rsrc_t rs_q = buffer_rsrc(q_tile), rs_x = buffer_rsrc(x_tile);
  auto issue = [&](int buf, int src_kk) {
    unsigned char* st = smem + buf * kStageBytes;
    const int k0 = src_kk * kKC;
    if (src_kk < nk_full) {
#pragma unroll
      for (int j = 0; j < kLoadsPerWave; ++j)
        buffer_load_lds16(is_x[j] ? rs_x : rs_q, st + (wave * kLoadsPerWave + j) * 1024, voff[j],
                          2 * k0);
    } else {
      const char* qb = q_tile + 2 * (int64_t)k0;
      const char* xb = x_tile + 2 * (int64_t)k0;
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

  // ---- per-lane LDS offsets of the MFMA operands: row `col` of block b, chunk 2 s + half of
  // the stage's k-steps s = 0, 1 (steps 2 and 3 of a 64-half stage are the same positions one
  // 512-byte sub-block further)
  const int col = lane & 31, half = lane >> 5;
  auto lds_off = [&](int r, int c) {
    return (uint32_t)((r / kR) * 1024 + (r % kR) * 64 + 16 * (c ^ ((r >> 2) & 3)));
  };
  uint32_t offq[kBQ][2], offx[kBR][2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int c = 2 * s + half;
#pragma unroll
    for (int b = 0; b < kBQ; ++b) offq[b][s] = lds_off(wq * 32 * kBQ + 32 * b + col, c);
#pragma unroll
    for (int b = 0; b < kBR; ++b) offx[b][s] = kQTileBytes + lds_off(wr * 32 * kBR + 32 * b + col, c);
  }

  f32x16 acc[kBQ][kBR];
#pragma unroll
  for (int i = 0; i < kBQ; ++i)
#pragma unroll
    for (int j = 0; j < kBR; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  struct Frags {
    f16x8 a[kBQ], b[kBR];
  };
  // fragments of k-step s of stage kk
  auto read_frags = [&](int kk, int s, Frags& f) {
    const unsigned char* st = smem + (kk % kStages) * kStageBytes + (s >> 1) * (kR * 64);
#pragma unroll
    for (int b = 0; b < kBQ; ++b)
      f.a[b] = as_f16x8(*reinterpret_cast<const u32x4*>(st + offq[b][s & 1]));
#pragma unroll
    for (int b = 0; b < kBR; ++b)
      f.b[b] = as_f16x8(*reinterpret_cast<const u32x4*>(st + offx[b][s & 1]));
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
  if constexpr (kStages == 2) {
    // Two 64-half stages: stage kk+1's loads are issued when stage kk starts and complete while
    // its four k-steps run; one barrier per stage (stage kk+1 landed everywhere, every read of
    // stage kk done, so its buffer can take stage kk+2), placed before the last k-step's MFMAs
    // so that the next stage's first operands are read while they run.  Within the stage the
    // scheduling groups below make each k-step's MFMAs alternate with the reads of the next
    // k-step's operands (measured 2-5 % faster than the compiler's own order).
    static_assert(kKSteps == 4, "the schedule below is written for four k-steps");
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    barrier();
    read_frags(0, 0, f0);
#pragma unroll 1
    for (int kk = 0; kk < nk; ++kk) {
      issue((kk + 1) & 1, kk + 1);
      __builtin_amdgcn_sched_barrier(0);
      read_frags(kk, 1, f1);
      mfma(f0);
      read_frags(kk, 2, f0);
      mfma(f1);
      read_frags(kk, 3, f1);
      mfma(f0);
#pragma unroll
      for (int u = 0; u < 3; ++u) {
#pragma unroll
        for (int t = 0; t < kBQ + kBR; ++t) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
#pragma unroll
        for (int t = 0; t < kBQ * kBR - kBQ - kBR; ++t)
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      barrier();
      read_frags(kk + 1 < nk ? kk + 1 : kk, 0, f0);
      __builtin_amdgcn_sched_barrier(0);  // the next stage's reads go out before these MFMAs
      mfma(f1);
    }
  } else {
    // Software pipeline over a ring of 32-half stages.  Every iteration issues exactly one
    // stage of loads (past the last stage, zeros into a buffer nobody reads again), so "stage
    // kk+1 has landed" is always "at most kStages - 3 stages of this wave's loads are still in
    // flight".
    static_assert(kKSteps == 2 && kStages >= 3 && (kStages - 2) * kLoadsPerWave <= 63,
                  "two k-steps per stage; vmcnt range");
#pragma unroll
    for (int s = 0; s < kStages - 1; ++s) issue(s, s);
    // stage 0 landed (this wave): at most the kStages - 2 later stages still in flight
    __builtin_amdgcn_s_waitcnt(waitcnt_vm((kStages - 2) * kLoadsPerWave));
    barrier();  // ... and for every wave
    read_frags(0, 0, f0);
#pragma unroll 1
    for (int kk = 0; kk < nk; ++kk) {
      read_frags(kk, 1, f1);
      mfma(f0);
      // Stage kk+1 lands everywhere, and every wave's reads of stage kk-1 are complete (this
      // wave's LDS reads drain before the barrier), so that stage's buffer
      // ((kk + kStages - 1) % kStages) can take stage kk + kStages - 1.
      __builtin_amdgcn_s_waitcnt(waitcnt_vm((kStages - 3) * kLoadsPerWave));
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      barrier();
      const int nxt = kk + kStages - 1;
      issue(nxt % kStages, nxt);
      read_frags(kk + 1 < nk ? kk + 1 : kk, 0, f0);
      __builtin_amdgcn_sched_barrier(0);  // the next stage's reads go out before these MFMAs
      mfma(f1);
    }
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
  if constexpr (MODE == kStore) {
#pragma unroll
    for (int i = 0; i < kBQ; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ql = q_base + 32 * kBQ * wq + 32 * i + 8 * (r >> 2) + 4 * half + (r & 3);
        if (ql >= nqa) continue;
        float* dst = a.scores + (int64_t)ql * a.ld + (row_base - a.r0) + 32 * kBR * wr + col;
#pragma unroll
        for (int j = 0; j < kBR; ++j) {
          const int64_t row = row_base + 32 * kBR * wr + 32 * j + col;
          if (row < a.r1) dst[32 * j] = acc[i][j][r];
        }
      }
    }
    return;
  }
  // Filter: each lane records the entries that beat their query's bound in LDS slots of its
  // own (no atomics, no cross-lane traffic), then appends them to the global lists one slot
  // per round, so that the round trips of the list atomics overlap across the wave; a lane's
  // entries beyond kSlots (rare) are appended directly.  The query bounds come from the lanes
  // that loaded them, by readlane.  Per group of four entries (one query per half-wave) a
  // cheap test, score >= bound, selects the groups that need the exact test (bound, tie row,
  // tile edges); entries pass rarely.
  constexpr int kSlots = 16;
  constexpr int kT = G::kThreads;
  static_assert(kT * kSlots * 12 <= G::kStages * kStageBytes, "the slots fit the LDS ring");
  barrier();  // every wave's reads of the ring are done
  uint32_t* e_r = reinterpret_cast<uint32_t*>(smem);  // [kSlots][kT]
  float* e_v = reinterpret_cast<float*>(e_r + kSlots * kT);
  int* e_q = reinterpret_cast<int*>(e_v + kSlots * kT);
  const int th_bits = __float_as_int(th_l);
  const int tie_hi = (int)(tie_l >> 32), tie_lo = (int)(uint32_t)tie_l;
  int n_l = 0;  // this lane's entries
#pragma unroll
  for (int i = 0; i < kBQ; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int q0 = 32 * i + 8 * (r >> 2) + (r & 3);  // the wave's query of lanes 0-31
      const int th0 = __builtin_amdgcn_readlane(th_bits, q0);
      const int th1 = __builtin_amdgcn_readlane(th_bits, q0 + 4);
      const float th = __int_as_float(half ? th1 : th0);
      bool cand = false;
#pragma unroll
      for (int j = 0; j < kBR; ++j) cand |= acc[i][j][r] >= th;
      if (__ballot(cand) == 0) continue;  // wave-uniform
      const int ql = q_base + 32 * kBQ * wq + q0 + 4 * half;
      const int th0_hi = __builtin_amdgcn_readlane(tie_hi, q0);
      const int th1_hi = __builtin_amdgcn_readlane(tie_hi, q0 + 4);
      const int th0_lo = __builtin_amdgcn_readlane(tie_lo, q0);
      const int th1_lo = __builtin_amdgcn_readlane(tie_lo, q0 + 4);
      const int gq0 = __builtin_amdgcn_readlane(gq_l, q0);
      const int gq1 = __builtin_amdgcn_readlane(gq_l, q0 + 4);
      const int64_t tie = ((int64_t)(half ? th1_hi : th0_hi) << 32) |
                          (int64_t)(uint32_t)(half ? th1_lo : th0_lo);
      const int gq = half ? gq1 : gq0;
#pragma unroll
      for (int j = 0; j < kBR; ++j) {
        const int64_t row = row_base + 32 * kBR * wr + 32 * j + col;
        const float v = acc[i][j][r];
        if (ql < nqa && row < a.r1 && (v > th || (v == th && row <= tie))) {
          if (n_l < kSlots) {
            e_r[n_l * kT + tid] = (uint32_t)row;
            e_v[n_l * kT + tid] = v;
            e_q[n_l * kT + tid] = gq;
          } else {
            const int p = atomicAdd(&a.count[gq], 1);
            if (p < a.cap) {
              a.cand_s[(int64_t)gq * a.cap + p] = v;
              a.cand_i[(int64_t)gq * a.cap + p] = (uint32_t)row;
            }
          }
          ++n_l;
        }
      }
    }
  }
  const int m = n_l < kSlots ? n_l : kSlots;
#pragma unroll 1
  for (int sl = 0; __ballot(sl < m) != 0; ++sl) {
    if (sl < m) {
      const int gq = e_q[sl * kT + tid];
      const int p = atomicAdd(&a.count[gq], 1);
      if (p < a.cap) {
        a.cand_s[(int64_t)gq * a.cap + p] = e_v[sl * kT + tid];
        a.cand_i[(int64_t)gq * a.cap + p] = e_r[sl * kT + tid];
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
    // Tiles in groups of kQGroup query tiles: within a group the query tile varies fastest,
    // and each XCD takes a contiguous run of the order, so the 32 workgroups an XCD runs at a
    // time cover 4 query tiles x 8 row tiles (measured 6 % faster than all 16 query tiles x 2
    // row tiles: the operand slices of a K step are fetched into the XCD's L2 fewer times).
    constexpr int kQGroup = 4;
    const int64_t total = (int64_t)a.n_qt * a.n_rt;
    const int64_t lin = xcd_linear(blockIdx.x, total);
    const int64_t span = (int64_t)kQGroup * a.n_rt;
    const int grp = (int)(lin / span);
    const int64_t in = lin - (int64_t)grp * span;
    const int gs = min(kQGroup, a.n_qt - grp * kQGroup);
    const int rt = (int)(in / gs);
    gemm_tile<G, MODE>(a, a.nqa, grp * kQGroup + (int)(in - (int64_t)rt * gs), rt, smem);
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
