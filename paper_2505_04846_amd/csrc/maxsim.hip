// Late-interaction (MaxSim) scoring on gfx950 MFMA, with the max over document tokens fused in
// registers (the Lq x Ld similarity table never leaves the register file).
//
// Decomposition
//   * MFMA shape.  v_mfma_f32_32x32x16_bf16: measured on MI355X it sustains ~2.3 PFLOP/s from a
//     single wave per SIMD, twice what the 16x16x32 form delivers, so every tile is 32 x 32.
//   * Query side.  A wave owns NB blocks of 32 query-token "slots": whole queries of
//     lqp = round_up(lq, 32) slots each.  Their bf16 tokens stay in VGPRs for the whole kernel
//     as the B operand (K = 16 per step, KS steps; dim <= 16 KS).
//   * Document side.  Each document is cut into tiles of 32 consecutive tokens (the A operand,
//     rows = document tokens).  A tile never straddles two documents: rows past a document's
//     last token re-load that last token, which leaves the maximum unchanged (max is
//     idempotent), so no masking is needed.
//   * C layout (32x32): lane l holds column l % 32 (a query slot) and the 16 rows
//     8 (i / 4) + 4 (l / 32) + i % 4, i = 0..15 (document tokens).  The score folds each tile's
//     16 values into one running max per lane with v_max3 (8 instructions per tile and block).
//     At the end of a document the two half-waves are combined and the slot maxima summed per
//     query.  (The loss also needs the argmax token: maxsim_argmax.hip.)
//   * Workgroup = 4 waves on 4 query sets, all consuming the same stream of document tiles,
//     which the workgroup stages through LDS (double-buffered, one stage in flight).  Workgroups
//     sharing a document range are mapped onto the same XCD and start together, so the range is
//     read from HBM about once per XCD and served from its L2 to every query group: the tile
//     loads are ordinary (L2-allocating) loads, not streaming ones.  Ranges are short enough
//     (at most 262,144 tokens) that those workgroups stay within L2 reach of each other.
//   * Software pipeline.  Each tile's epilogue (the fold of its 16 values per lane into the
//     running maximum) is issued inside the next tile's MFMA stream, block by block, in the
//     shadow of the MFMA before it.
//   * K permutation.  Lane half h = l / 32 of step s carries contraction indices
//     16 s + 8 h .. 16 s + 8 h + 7 for both operands; A and B use the same rule, so every
//     product pairs matching indices whatever order the hardware reduces them in.
#include "maxsim_common.h"

namespace hpr {
namespace msim {

namespace {

// LDS geometry of one 32-token tile: rows of KS*32 bytes padded by 16, so that the A fragment
// of k-step s of a lane sits at a fixed offset 32 s from a per-lane base (immediate offsets, no
// per-read address arithmetic) and the 16 rows of a read phase start 16 bytes apart modulo the
// 256-byte bank width (conflict-free); a stage holds kTps tiles.
//
// DIRECT (dim 128 with 128 query slots per wave, the many-query grids): the tiles go straight
// from global memory into LDS (buffer loads with the LDS as destination), one tile per wave and
// stage, so a stage holds WPW tiles.  A wave load writes 1 KiB of consecutive LDS bytes, so a
// tile's region is rounded up to whole loads; the lanes that land on a row's padding or past
// the tile's 32 rows load row 0 of the tile into bytes nobody reads.
template <int KS, bool DIRECT = false, int WPW = 4>
struct TileGeom {
  static constexpr int kCpr = KS * 2;              // 16-byte chunks per row
  static constexpr int kRowB = KS * 32 + 16;       // bytes per (padded) row
  static constexpr int kTileB = 32 * kRowB;        // bytes per tile
  static constexpr int kLoads = (kTileB + 1023) / 1024;             // direct loads per tile
  static constexpr int kTileS = DIRECT ? kLoads * 1024 : kTileB;    // tile stride in a stage
  static constexpr int kTps = DIRECT ? WPW : KS >= 8 ? 2 : 4;       // tiles per stage
};


// Waves per SIMD the register allocation of the score kernel must allow: two (up to 256 VGPRs),
// which leaves the dim-128 variant room for 128 query slots per wave (half the LDS operand
// reads per MFMA of 64 slots and half the query groups, hence half the document-range
// re-reads).  Fewer query slots (small nq: NB = 1 or 2 blocks per wave) need fewer registers,
// and the allocation allows three or four waves per SIMD: the kernel is then bound by the
// store stream, which more resident workgroups keep in flight.
constexpr int maxsim_waves(int ks, int nb) {
  if (ks == 16) return 2;
  return nb >= 4 ? 2 : nb == 2 ? 3 : 4;
}
// Workgroups per CU: the register bound above, and the LDS of two stages plus the result
// buffers against the CU's 160 KiB.
constexpr int maxsim_resident(int ks, int nb) {
  const int stage = (ks >= 8 ? 2 : 4) * 32 * (ks * 32 + 16);
  const int by_lds = (160 * 1024) / (2 * stage + 4096);
  const int waves = maxsim_waves(ks, nb);
  return waves < by_lds ? waves : by_lds;
}

// MaxSim scores only (the retrieval path).
//
// Per tile: the NB x KS MFMAs, and the epilogue of the previous tile (each block's 16 values
// folded into its running maximum by eight v_max3) interleaved with them: block b's
// epilogue is issued just before block b's first MFMA of the new tile, in the shadow of the
// MFMA before it (sched_group_barrier), so no second accumulator set is needed.  When the
// previous tile ended its document, the document's scores are reduced (maximum over the
// half-waves, sum over each query's slots) after the new tile's MFMAs are issued.
template <int KS, int NB, int WPW, bool DIRECT = false>
__global__ __launch_bounds__(64 * WPW, (maxsim_waves(KS, NB) * 4 / WPW)) void maxsim_kernel(
    MaxsimArgs a, const int64_t* __restrict__ off, const int64_t* __restrict__ part) {
  using G = TileGeom<KS, DIRECT, WPW>;
  constexpr int kThreads = 64 * WPW;
  constexpr int kSlotsWG = WPW * NB * 32;
  constexpr int kTps = G::kTps;
  static_assert(!DIRECT || NB == 4, "direct staging: the many-query variant (ordinary loads)");
  // as many resident workgroups as the plan assumes (maxsim_resident): two stages and the ring
  static_assert((maxsim_waves(KS, NB) * 4 / WPW) *
                        (2 * kTps * G::kTileS + 3 * kTps * (kSlotsWG / 32) * 4) <=
                    160 * 1024,
                "LDS of the resident workgroups");
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][kTps * G::kTileS];
  // Per-document results, written to HBM after the barrier that follows the epilogue (a tile's
  // epilogue runs in the next tile's step, possibly in the next stage): a ring of three
  // stages, one slot per (tile, query of the workgroup).
  __shared__ float res_score[3][kTps][kSlotsWG / 32];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31;
  const int half = lane >> 5;

  // block -> (document range, query group); all uniform, kept in scalar registers.  Persistent
  // grid (one resident round per launch, one launch per pass of query groups): workgroup b runs
  // on XCD b % 8 and takes range b % 8 (the XCD's eighth of the store) for query group
  // qg_base + b / 8, so the workgroups of an XCD start together and read the same tiles at
  // about the same time, once from beyond the XCD's L2.  Otherwise one (range, query group)
  // per workgroup, the workgroups sharing a range placed on one XCD.
  int rng, qg;
  if (a.persist) {
    rng = (int)(blockIdx.x % (uint32_t)a.n_ranges);
    qg = a.qg_base + (int)(blockIdx.x / (uint32_t)a.n_ranges);
  } else {
    const uint32_t total = (uint32_t)a.n_qgroups * (uint32_t)a.n_ranges;
    const uint32_t lin = (uint32_t)xcd_linear(blockIdx.x, total);
    rng = (int)(lin / (uint32_t)a.n_qgroups);
    qg = (int)(lin - (uint32_t)rng * a.n_qgroups);
  }
  rng = __builtin_amdgcn_readfirstlane(rng);
  qg = __builtin_amdgcn_readfirstlane(qg);
  const int d_begin = __builtin_amdgcn_readfirstlane((int)part[rng]);
  const int d_end = __builtin_amdgcn_readfirstlane((int)part[rng + 1]);
  if (d_begin >= d_end || qg >= a.n_qgroups) return;  // uniform for the whole workgroup
  const int qwg = qg * WPW * a.qpw;  // first query of the workgroup
  const int q0 = qwg + wave * a.qpw;
  const bool wave_active = q0 < a.nq;  // idle waves still load tiles and meet the barriers

  // ---- query slots -> B operands (resident for the whole kernel)
  bf16x8 bq[NB][KS];
  int slot_row[NB];        // (q - qwg) * lq + i of this lane's slot in block b, or -1
  uint32_t my_blocks = 0;  // bit b set when block b belongs to query (q0 + lane)
  const int lqb = a.lqp >> 5;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int slot = b * 32 + col;
    const int ql = slot / a.lqp;
    const int i = slot - ql * a.lqp;
    const int qq = q0 + ql;
    const bool valid = wave_active && ql < a.qpw && qq < a.nq && i < a.lq;
    slot_row[b] = valid ? (qq - qwg) * a.lq + i : -1;
    if (b / lqb == lane) my_blocks |= 1u << b;
    const uint16_t* src = a.q + (valid ? (int64_t)qq * a.lq + i : 0) * a.dim;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int k = 16 * s + 8 * half;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (valid && k < a.dim) v = load16(src + k);
      bq[b][s] = as_bf16x8(v);
    }
  }

  const int n_tok = (int)a.n_tok;
  // Document bounds clamped into [0, n_tok) so that even an invalid CSR cannot make a load go
  // out of bounds; for a valid CSR they are exactly (off[d], off[d+1] - off[d]).  32-bit
  // scalar arithmetic only: a 64-bit offset is in range iff its high word is 0 and its low word
  // is below n_tok.
  auto open_doc = [&](TileCursor& c, int dd) {
    const int64_t lo64 = off[dd], hi64 = off[dd + 1];
    const uint32_t lo_hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)lo64 >> 32));
    const uint32_t lo_lo = __builtin_amdgcn_readfirstlane((uint32_t)lo64);
    const uint32_t hi_hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)hi64 >> 32));
    const uint32_t hi_lo = __builtin_amdgcn_readfirstlane((uint32_t)hi64);
    const int lo = (lo_hi == 0u && lo_lo < (uint32_t)n_tok) ? (int)lo_lo
                   : ((int32_t)lo_hi < 0 ? 0 : n_tok - 1);
    int hi = (hi_hi == 0u && hi_lo <= (uint32_t)n_tok) ? (int)hi_lo
             : ((int32_t)hi_hi < 0 ? 0 : n_tok);
    hi = hi > lo ? hi : lo + 1;
    c.d = dd;
    c.base = lo;
    c.len = hi - lo;
    c.t = 0;
    c.cnt = (c.len + 31) >> 5;
  };

  // ---- producer: the next stage's tiles, loaded into registers, then stored to LDS.  Thread
  // tid covers chunk c = tid % kCpr of rows r0 = tid / kCpr + kRp k (kRp = kThreads / kCpr
  // rows per pass) of the stage's tiles; unit m of a stage is pass m % kPpt of tile m / kPpt
  // (kPpt passes per tile).  When a pass spans several tiles (small dims) the tile also depends
  // on the wave.  Chunks past `dim` are never loaded nor stored: the LDS buffers are zeroed
  // once, so they read as zeros.
  constexpr int kRp = kThreads / G::kCpr;              // rows covered by one pass
  constexpr int kPpt = kRp >= 32 ? 1 : 32 / kRp;       // passes per tile
  constexpr int kTpp = kRp >= 32 ? kRp / 32 : 1;       // tiles per pass
  constexpr int kUpt = kTps * kPpt / kTpp;             // units per thread per stage
  TileCursor prod;
  open_doc(prod, d_begin);
  u32x4 stage_regs[DIRECT ? 1 : kUpt];
  const int lr = (tid / G::kCpr) & 31;            // row within the pass (within the tile)
  const int lt = __builtin_amdgcn_readfirstlane((tid / G::kCpr) >> 5);  // tile within the pass
  const int lc = tid % G::kCpr;
  const bool lok = 8 * lc < a.dim;
  const uint32_t lboff = 16u * lc;
  if (a.dim < 16 * KS) {  // chunks past dim are never stored: they must read as zeros
    for (int i = tid; i < (int)(sizeof(lds) / 16); i += kThreads)
      reinterpret_cast<u32x4*>(&lds[0][0])[i] = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
  }
  const uint32_t row_bytes = 2u * (uint32_t)a.dim;
  // direct staging: this lane's source offset within the tile for load q of the tile (rows
  // below 32 clamped to the tile's last row rmx; 0 for the lanes that fill padding)
  auto direct_off = [&](int q, uint32_t rmx) {
    const int p = q * 1024 + 16 * lane;
    const int row = p / G::kRowB;
    const int c = (p - row * G::kRowB) >> 4;
    const uint32_t r = (uint32_t)row < rmx ? (uint32_t)row : rmx;
    return (row < 32 && c < G::kCpr) ? r * (uint32_t)(32 * KS) + 16u * (uint32_t)c : 0u;
  };
  // direct staging: wave w loads tile w of the stage, whose first token is r0 and last row rmx
  // (the lane offsets are recomputed per stage: kept, they would cost registers this kernel
  // does not have)
  auto issue_tile = [&](int buf, int r0, uint32_t rmx) {
    const char* tptr = reinterpret_cast<const char*>(a.d) + (uint64_t)(uint32_t)r0 * row_bytes;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(tptr), (short)0, 0x7fffffff, 0x00020000);
    unsigned char* dst = &lds[buf][wave * G::kTileS];
#pragma unroll
    for (int q = 0; q < G::kLoads; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(dst + 1024 * q), 16,
                                               (int)direct_off(q, rmx), 0, 0, 0);
  };
  auto fetch_stage = [&](StageDesc& sd, int buf) {
    sd.d0 = prod.d;
    sd.t0 = prod.t;
    sd.valid = sd.last = sd.lng = 0u;
    bool my_ok = false;
    int my_r0 = 0;
    uint32_t my_rmx = 0u;
#pragma unroll
    for (int j = 0; j < kTps; ++j) {
      const bool ok = prod.d < d_end;
      const int r0 = ok ? prod.base + prod.t * 32 : 0;
      const uint32_t rmx = ok ? prod.len - prod.t * 32 - 1 : 0;  // later rows repeat the last
      const char* tptr = reinterpret_cast<const char*>(a.d) + (uint64_t)(uint32_t)r0 * row_bytes;
      if constexpr (DIRECT) {
        if (j == wave) {  // uniform
          my_ok = ok;
          my_r0 = r0;
          my_rmx = rmx;
        }
      } else if (j % kTpp == lt && lok) {  // this thread's units of tile j
#pragma unroll
        for (int p = 0; p < kPpt; ++p) {
          const uint32_t row = lr + kRp * p;
          const uint32_t r = row < rmx ? row : rmx;
          // Few-query variants (NB < 4) have one query group, so no other workgroup reads
          // the range: streaming loads keep it out of L2.  With several groups the range is
          // re-served from L2 and ordinary loads are faster.
          const char* src = tptr + (r * row_bytes + lboff);
          stage_regs[(j / kTpp) * kPpt + p] = NB < 4 ? load16_stream(src) : load16(src);
        }
      }
      if (ok) {
        sd.valid |= 1u << j;
        if (prod.t + 1 == prod.cnt) sd.last |= 1u << j;
        if (++prod.t == prod.cnt) {  // advance the producer to the next tile
          if (prod.d + 1 < d_end)
            open_doc(prod, prod.d + 1);
          else
            prod.d = d_end;
        }
      }
    }
    if constexpr (DIRECT)
      if (my_ok) issue_tile(buf, my_r0, my_rmx);
  };
  auto store_stage = [&](int buf) {
    if (!lok) return;
#pragma unroll
    for (int m = 0; m < kUpt; ++m) {
      const int j = (m / kPpt) * kTpp + lt;
      const uint32_t row = lr + kRp * (m % kPpt);
      *reinterpret_cast<u32x4*>(&lds[buf][j * G::kTileS + row * G::kRowB + lboff]) =
          stage_regs[m];
    }
  };

  // Running state per lane and block: rm[b], the maximum so far.
  float rm[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) rm[b] = -__builtin_huge_valf();
  const int n_wg_q = (a.nq - qwg) < WPW * a.qpw ? (a.nq - qwg) : WPW * a.qpw;
  const uint32_t a_lane = (uint32_t)(col * G::kRowB + half * 16);  // A: row col, chunk half
  auto frag = [&](int buf, int j, int s) {
    return as_bf16x8(
        *reinterpret_cast<const u32x4*>(&lds[buf][j * G::kTileS] + a_lane + 32 * s));
  };

  f32x16 acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = -__builtin_huge_valf();
  // One tile: its MFMAs into acc, and the previous tile's epilogue (acc folded into rm) issued
  // block by block just before the block's first MFMA of this tile.  fr[0] holds the tile's
  // k-step 0 fragment on entry and the next tile's (when in the same stage) on exit.
  auto step = [&](int buf, int j, bf16x8 (&fr)[2]) {
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      // the fragment of the next k-step (of the next tile after the last one, same stage)
      if (s + 1 < KS)
        fr[(s + 1) & 1] = frag(buf, j, s + 1);
      else if (j + 1 < kTps)
        fr[(s + 1) & 1] = frag(buf, j + 1, 0);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (s == 0) {  // eight v_max3 folding the 16 values into rm
          float m = rm[b];
#pragma unroll
          for (int r = 0; r < 16; r += 2) m = fmaxf(fmaxf(m, acc[b][r]), acc[b][r + 1]);
          rm[b] = m;
        }
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[s & 1], bq[b][s],
                                                         s == 0 ? f32x16{} : acc[b], 0, 0, 0);
      }
      if (s + 1 < KS || j + 1 < kTps) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (s == 0) __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);  // VALU
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                      // MFMA
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // The end of a document whose last tile's epilogue has run: maximum over the two half-waves
  // (rows), sum over the slots of each query in a fixed order, into LDS slot (rb, j).
  auto doc_end = [&](int rb, int j) {
    float qs = 0.f;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(rm[b]),
                                                       __float_as_uint(rm[b]), false, false);
      const float m = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      rm[b] = -__builtin_huge_valf();
      const float v = half32_sum(slot_row[b] >= 0 ? m : 0.f);
      if ((my_blocks >> b) & 1u) qs += v;
    }
    if (lane < a.qpw) res_score[rb][j][wave * a.qpw + lane] = qs;
  };

  // Results of the documents that ended in a stage (ring slot rb) -> HBM (coalesced per doc).
  // (the documents that end in a stage are consecutive from its first one, one per bit of
  // `last`)
  auto write_results = [&](const StageDesc& sd, int rb) {
    int d = sd.d0;
#pragma unroll 1
    for (uint32_t m = sd.last & sd.valid; m != 0u; m &= m - 1u, ++d) {
      const int j = __builtin_ctz(m);
      if (tid < n_wg_q) a.scores[(int64_t)(qwg + tid) * a.n_docs + d] = res_score[rb][j][tid];
    }
  };

  StageDesc cur, nxt, prv, prv2;
  fetch_stage(cur, 0);
  // The query operands and the first stage land together.  The operands must be resident
  // before the pipelined loop: otherwise their pending loads make the compiler wait for every
  // load in flight (the prefetch included) at each tile.
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  if constexpr (!DIRECT) store_stage(0);
  __syncthreads();
  bf16x8 fr[2];
  fr[0] = frag(0, 0, 0);

  // Persistent plans keep the workgroups of a range in step: every kSyncStages stages each
  // checks in on the range's counter (a.ctrl[8 pass + range], zeroed by the partition kernel
  // of the call) and waits until all n_sync workgroups of the range have, for at most kMaxSpins
  // sleeps; a workgroup whose wait runs out stops waiting for the rest of the launch (so a peer
  // that is not resident costs one wait, and no wait can hang).  Correctness never depends on
  // it: it only keeps the tiles of a range within reach of the XCD's L2.
  constexpr int kSyncStages = 256, kMaxSpins = 4096;
  int32_t* sync = nullptr;
  int n_sync = 0;
  __shared__ int sync_gave_up;  // written by thread 0 before the checkpoint's barrier
  if (tid == 0) sync_gave_up = 0;
  if (a.persist && a.n_ctrl > 0) {
    const int per_pass = (int)(gridDim.x / (uint32_t)a.n_ranges);
    const int pass = a.qg_base / per_pass;
    if (8 * pass + rng < a.n_ctrl) {
      sync = a.ctrl + 8 * pass + rng;
      n_sync = a.n_qgroups - a.qg_base < per_pass ? a.n_qgroups - a.qg_base : per_pass;
    }
  }
  // Pipeline state (uniform): whether the tile whose epilogue runs next ends its document, and
  // where that document's result goes.  (The first tile's "previous tile" is acc = -inf, whose
  // epilogue changes nothing: one code path, whose registers fit without spills.)
  bool pend_last = false;
  int pend_rb = 0, pend_j = 0;
  int stage = 0;
  for (;; ++stage) {
    const int buf = stage & 1;
    const int rb = stage % 3;
    const bool more = prod.d < d_end;
    // global loads in flight while this stage is computed (direct staging: into the other
    // buffer, idle since the last barrier)
    if (more) fetch_stage(nxt, buf ^ 1);
    // direct staging: the results of two stages ago go out while the tiles run, so that the
    // stage's closing wait for its loads finds the stores complete
    if constexpr (DIRECT)
      if (stage >= 2) write_results(prv2, (stage - 2) % 3);
    if (wave_active) {
#pragma unroll
      for (int j = 0; j < kTps; ++j) {
        if (!((cur.valid >> j) & 1u)) break;  // uniform: only the final stage is partial
        step(buf, j, fr);
        if (pend_last) doc_end(pend_rb, pend_j);
        pend_last = (cur.last >> j) & 1u;
        pend_rb = rb;
        pend_j = j;
      }
    }
    if constexpr (DIRECT) {
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's loads of the next stage landed
    } else {
      if (stage >= 2) write_results(prv2, (stage - 2) % 3);
      if (more) store_stage(buf ^ 1);
    }
    __syncthreads();
    if (!more) break;
    if (sync && (stage & (kSyncStages - 1)) == kSyncStages - 1) {
      // checkpoint: wait (bounded) until every workgroup of this range has reached it
      if (tid == 0) {
        const int target = (stage / kSyncStages + 1) * n_sync;
        atomicAdd(sync, 1);
        int spin = 0;
        while (__hip_atomic_load(sync, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target &&
               spin < kMaxSpins) {
          __builtin_amdgcn_s_sleep(8);
          ++spin;
        }
        sync_gave_up = spin == kMaxSpins ? 1 : 0;
      }
      __syncthreads();
      if (sync_gave_up) sync = nullptr;  // a peer never came: stop waiting (workgroup-uniform)
    }
    fr[0] = frag(buf ^ 1, 0, 0);
    prv2 = prv;
    prv = cur;
    cur = nxt;
  }
  // the last computed tile's epilogue and document end, then the final two stages' results
  if (wave_active) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      float m = fmaxf(acc[b][0], acc[b][1]);
#pragma unroll
      for (int r = 2; r < 16; r += 2) m = fmaxf(fmaxf(m, acc[b][r]), acc[b][r + 1]);
      rm[b] = fmaxf(rm[b], m);
    }
    if (pend_last) doc_end(pend_rb, pend_j);
  }
  __syncthreads();
  if (stage >= 1) write_results(prv, (stage - 1) % 3);
  write_results(cur, stage % 3);
}

__global__ void partition_kernel(const int64_t* off, int64_t n_docs, int64_t n_tok, int R,
                                 int64_t* part, int32_t* ctrl, int n_ctrl) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (ctrl)
    for (int i = r; i < n_ctrl; i += gridDim.x * blockDim.x) ctrl[i] = 0;
  if (r > R) return;
  if (r == R) {
    part[r] = n_docs;
    return;
  }
  const int64_t target = (n_tok / R) * r + (n_tok % R) * r / R;  // floor(n_tok * r / R)
  int64_t lo = 0, hi = n_docs;  // first d with off[d] >= target
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if (off[mid] < target)
      lo = mid + 1;
    else
      hi = mid;
  }
  part[r] = lo;
}

__global__ void csr_validate_kernel(const int64_t* off, int64_t n_docs, int64_t n_tok,
                                    unsigned long long* bad) {
  const int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (d >= n_docs) return;
  const int64_t lo = off[d], hi = off[d + 1];
  unsigned long long code = ~0ull;
  if ((d == 0 && lo != 0) || hi < lo || (d == n_docs - 1 && hi != n_tok))
    code = (unsigned long long)d * 2;
  else if (hi == lo)
    code = (unsigned long long)d * 2 + 1;
  if (code != ~0ull) atomicMin(bad, code);
}

__global__ void fill_u64_kernel(unsigned long long* p, unsigned long long v) { *p = v; }

template <int KS, int NB, int WPW, bool DIRECT = false>
hipError_t launch_t(const MaxsimPlan& plan, const MaxsimArgs& args, hipStream_t stream) {
  hipLaunchKernelGGL((maxsim_kernel<KS, NB, WPW, DIRECT>), dim3((unsigned)plan.grid),
                     dim3(64 * WPW), 0, stream, args, args.off, args.part);
  return hipGetLastError();
}
// Variants by k-steps of 16 (dim <= 16 KS) and query blocks per wave.  Query slots per wave:
// scores 128 (dim <= 128) or 64 (dim 256), fewer when the call has few query slots; argmax 64
// (dim <= 128) or 32 (dim 256).
hipError_t launch_variant(const MaxsimPlan& plan, const MaxsimArgs& args, bool argmax,
                          hipStream_t stream) {
  if (argmax) return launch_argmax_variant(plan, args, stream);
  switch (plan.ks * 8 + plan.nb) {
    case 2 * 8 + 1: return launch_t<2, 1, 4>(plan, args, stream);
    case 2 * 8 + 2: return launch_t<2, 2, 4>(plan, args, stream);
    case 2 * 8 + 4: return launch_t<2, 4, 4>(plan, args, stream);
    case 4 * 8 + 1: return launch_t<4, 1, 4>(plan, args, stream);
    case 4 * 8 + 2: return launch_t<4, 2, 4>(plan, args, stream);
    case 4 * 8 + 4: return launch_t<4, 4, 4>(plan, args, stream);
    case 8 * 8 + 1: return launch_t<8, 1, 4>(plan, args, stream);
    case 8 * 8 + 2: return launch_t<8, 2, 4>(plan, args, stream);
    case 8 * 8 + 4:
      if (args.dim == 128)
        return plan.wpw == 8 ? launch_t<8, 4, 8, true>(plan, args, stream)
                             : launch_t<8, 4, 4, true>(plan, args, stream);
      return plan.wpw == 8 ? launch_t<8, 4, 8>(plan, args, stream)
                           : launch_t<8, 4, 4>(plan, args, stream);
    case 16 * 8 + 1: return launch_t<16, 1, 4>(plan, args, stream);
    case 16 * 8 + 2: return launch_t<16, 2, 4>(plan, args, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

}  // namespace msim

using namespace msim;

constexpr int64_t kMaxRangeTokens = 262144;  // 64 MiB of bf16 tokens at dim 128

bool maxsim_plan(int nq, int lq, int64_t n_docs, int64_t n_tok, int dim, bool argmax, int n_cu,
                 MaxsimPlan* p) {
  if (dim < 8 || dim > 256 || dim % 8 != 0 || lq < 1 || nq < 1 || n_docs < 1) return false;
  p->ks = dim <= 32 ? 2 : dim <= 64 ? 4 : dim <= 128 ? 8 : 16;
  p->nb = argmax ? (p->ks == 16 ? 1 : 2) : (p->ks == 16 ? 2 : 4);
  if (!argmax) {  // few query slots: fewer blocks per wave (never fewer than one query needs)
    const int lqb = (lq + 31) / 32;
    const int64_t slots = (int64_t)nq * lqb * 32;
    int need = slots <= 32 * 4 ? 1 : slots <= 64 * 4 ? 2 : 4;
    if (need < lqb) need = lqb;
    need = need <= 1 ? 1 : need <= 2 ? 2 : 4;
    if (need < p->nb) p->nb = need;
  }
  p->wpw = 4;
  p->lqp = (lq + 31) / 32 * 32;
  if (p->lqp > p->nb * 32) return false;
  p->qpw = p->nb * 32 / p->lqp;
  const int64_t q_per_wg = (int64_t)p->qpw * p->wpw;
  p->n_qgroups = (int)((nq + q_per_wg - 1) / q_per_wg);
  // Workgroups: the plain score takes enough to fill every CU's resident slots 32 times over
  // (short ranges keep the workgroups sharing a range in step, so the range is served from L2);
  // the argmax variant, whose stores are short, takes one round of resident workgroups (fewer
  // per-workgroup prologues).  No range is shorter than ~1024 tokens (the query operands are
  // re-loaded by every workgroup).
  const int occ = argmax ? msim::argmax_resident(p->ks) : msim::maxsim_resident(p->ks, p->nb);
  const int64_t target_wg = (int64_t)(n_cu > 0 ? n_cu : 256) * occ * (argmax ? 1 : 32);
  int64_t R = (target_wg + p->n_qgroups - 1) / p->n_qgroups;
  // ... and, for the score kernel, ranges of at most kMaxRangeTokens tokens: the up to 64
  // workgroups of an XCD that read one range together drift apart over a long range, after
  // which its tiles are fetched again from beyond the XCD's L2 (a 7-million-token range at
  // 4,096 x 64 queries fetched ~195x the store per launch)
  if (!argmax) {
    const int64_t by_len = (n_tok + kMaxRangeTokens - 1) / kMaxRangeTokens;
    if (R < by_len) R = by_len;
  }
  const int64_t max_by_tokens = n_tok / 1024 > 0 ? n_tok / 1024 : 1;
  if (R > max_by_tokens) R = max_by_tokens;
  if (R > n_docs) R = n_docs;
  if (R > kMaxRanges) R = kMaxRanges;
  if (R < 1) R = 1;
  if ((int64_t)p->n_qgroups * R > 0x7fffffffLL) return false;
  p->n_ranges = (int)R;
  // Persistent grid for the score kernel when the query groups fill every resident slot of an
  // XCD at least twice, a whole number of times (or at least 8 times, the partial last pass
  // then costing at most an eighth): one range per XCD, one launch of one resident round per
  // pass.  (With a single pass the dynamically scheduled short ranges finish sooner: a long
  // persistent range waits for its slowest workgroup.)
  // The dim-128 variant then runs 8-wave workgroups (one per CU, the same two waves per SIMD):
  // every staged tile feeds twice the query slots, which halves the traffic from L2 into LDS
  // per MFMA (1.6-2.2 % faster at 4,096 x 64 queries; 2.4 % slower on the short-range grid).
  p->persist = false;
  p->grid = (int64_t)p->n_qgroups * p->n_ranges;
  auto fits = [](int64_t groups, int slots) {
    return slots > 0 && groups >= 2 * slots && (groups % slots == 0 || groups >= 8 * slots);
  };
  if (!argmax && n_cu > 0 && n_cu % 8 == 0 && (int64_t)n_tok >= 8 * 1024 && n_docs >= 8) {
    const int slots = n_cu / 8 * occ;  // resident workgroups per XCD
    if (fits(p->n_qgroups, slots)) {
      p->persist = true;
      p->n_ranges = 8;
      p->grid = (int64_t)8 * slots;
      if (p->ks == 8 && p->nb == 4 && occ % 2 == 0) {
        const int64_t groups8 = (nq + (int64_t)p->qpw * 8 - 1) / ((int64_t)p->qpw * 8);
        const int slots8 = slots / 2;
        if (fits(groups8, slots8)) {
          p->wpw = 8;
          p->n_qgroups = (int)groups8;
          p->grid = (int64_t)8 * slots8;
        }
      }
    }
  }
  return true;
}

hipError_t launch_partition(const int64_t* off, int64_t n_docs, int64_t n_tok, int n_ranges,
                            int64_t* part, int32_t* ctrl, int n_ctrl, hipStream_t stream) {
  const int threads = 256;
  const int blocks = (n_ranges + 1 + threads - 1) / threads;
  hipLaunchKernelGGL(partition_kernel, dim3(blocks), dim3(threads), 0, stream, off, n_docs,
                     n_tok, n_ranges, part, ctrl, n_ctrl);
  return hipGetLastError();
}

int maxsim_passes(const MaxsimPlan& plan) {
  if (!plan.persist) return 1;
  const int64_t per_pass = plan.grid / plan.n_ranges;
  return (int)((plan.n_qgroups + per_pass - 1) / per_pass);
}

hipError_t launch_maxsim(const MaxsimPlan& plan, int pass, const uint16_t* q, int nq, int lq,
                         const uint16_t* d_tok, const int64_t* off, int64_t n_docs,
                         int64_t n_tok, int dim, const int64_t* part, float* scores,
                         uint16_t* amax, int32_t* ctrl, int n_ctrl, hipStream_t stream) {
  MaxsimArgs args;
  args.q = q;
  args.d = d_tok;
  args.off = off;
  args.part = part;
  args.scores = scores;
  args.amax = amax;
  args.ctrl = ctrl;
  args.n_ctrl = ctrl != nullptr ? n_ctrl : 0;
  args.n_docs = n_docs;
  args.n_tok = n_tok;
  args.nq = nq;
  args.lq = lq;
  args.lqp = plan.lqp;
  args.qpw = plan.qpw;
  args.dim = dim;
  args.n_qgroups = plan.n_qgroups;
  args.n_ranges = plan.n_ranges;
  args.persist = plan.persist ? 1 : 0;
  args.qg_base = plan.persist ? pass * (int)(plan.grid / plan.n_ranges) : 0;
  return launch_variant(plan, args, amax != nullptr, stream);
}

hipError_t launch_csr_validate(const int64_t* off, int64_t n_docs, int64_t n_tok,
                               unsigned long long* bad, hipStream_t stream) {
  hipLaunchKernelGGL(fill_u64_kernel, dim3(1), dim3(1), 0, stream, bad, ~0ull);
  const int threads = 256;
  const int64_t blocks = (n_docs + threads - 1) / threads;
  hipLaunchKernelGGL(csr_validate_kernel, dim3((unsigned)blocks), dim3(threads), 0, stream, off,
                     n_docs, n_tok, bad);
  return hipGetLastError();
}

}  // namespace hpr
