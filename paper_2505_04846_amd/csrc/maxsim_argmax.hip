// MaxSim with the argmax (the forward of the loss), software-pipelined.  The epilogue of a tile
// (the running maximum, the packed argmax tile keys and their maximum) costs about half as many
// issue cycles as the tile's MFMAs, so each wave keeps two accumulator sets: the MFMAs of tile t
// are issued interleaved with the epilogue of tile t - 1 (sched_group_barrier pattern per
// region of at most 4 k-steps: the LDS reads of the next region's A fragments first, then a
// share of the epilogue's VALU instructions after each MFMA).  Two waves per SIMD: the second
// accumulator set needs the registers of a third resident wave.
//
// LDS rows are KS * 32 bytes padded by 16 (no swizzle): the A operand of k-step s sits at a
// fixed offset 32 s from a per-lane base, so the KS reads of a tile take immediate offsets; the
// 16 rows of a read phase start 16 bytes apart modulo the 256-byte bank width, which keeps the
// phase conflict-free.
//
// Results: the per-document scores and argmax tokens of a stage are written to LDS by the
// epilogues (the last tile of a stage finishes in the next stage), and to HBM two stages later,
// after a barrier has passed behind every epilogue of the stage: a ring of three result buffers.
//
// Staging.  At dim 128 the tiles go straight from global memory into LDS (buffer loads with
// the LDS as destination), four tiles per stage, wave w loading tile w: the loads of stage s + 1
// are issued when stage s starts, into the buffer stage s - 1 used, and each wave waits for its
// own before the stage's closing barrier.  Against staging through VGPRs (two tiles per stage,
// the registers the wider stage would need are not there) this halves the barriers and the
// per-stage bookkeeping per tile and drops the LDS stores.  The other dims keep the VGPR path.
//
// Everything else (query operands in VGPRs, the document tile stream, the C layout, the K
// permutation, XCD placement) is as in maxsim_kernel (maxsim.hip).
#include <type_traits>

#include "maxsim_common.h"

namespace hpr {
namespace msim {

namespace {

// DIRECT: the tiles are staged by direct-to-LDS buffer loads (only when dim = 16 KS, so that
// every chunk of a row is data), one tile per wave and four per stage.  A wave load writes 1 KiB
// of consecutive LDS bytes, 16 per lane, so a tile's region is rounded up to whole loads; the
// lane that lands on a row's padding or past the tile's 32 rows loads row 0 of the tile into
// bytes nobody reads.
template <int KS, bool DIRECT>
struct ArgGeom {
  static constexpr int kCpr = KS * 2;                  // 16-byte chunks per row
  static constexpr int kRowB = KS * 32 + 16;           // padded row
  static constexpr int kTileB = 32 * kRowB;
  static constexpr int kLoads = (kTileB + 1023) / 1024;  // direct loads per tile
  static constexpr int kTileS = DIRECT ? kLoads * 1024 : kTileB;  // tile stride in a stage
  static constexpr int kTps = DIRECT ? 4 : argmax_tps(KS);        // tiles per stage (even)
  static constexpr int kStageB = kTps * kTileS;
};

// What the epilogue of a computed tile needs: its tile index within the document, whether it
// ends the document, and where its document's results go (ring slot, tile within the stage).
struct PendTile {
  int t;
  int rb;
  int j;
  bool last;
};

// First document of token range r out of R equal ranges: the least d in [0, n_docs) with
// off[d] >= floor(n_tok * r / R), or n_docs when there is none or r = R (documents are never
// split; a range can be empty).  Lanes 0-31 answer for r = r0 and lanes 32-63 for r0 + 1, each
// half by a 32-way search that keeps the answer inside [lo, hi]: a round probes the last offset
// of each of 32 equal slices of [lo, hi); the probes below the target form a prefix (offsets
// ascend), and its length picks the slice that holds the answer.  A span S shrinks to at most
// ceil(S / 32) - 1 per round: two rounds for 1024 documents, four for 10^6.  Whatever the
// offsets hold, lo stays within [0, n_docs] and every probe within [0, n_docs).
__device__ int range_first_doc(const int64_t* __restrict__ off, int64_t n_docs, int64_t n_tok,
                               int R, int r0, int lane) {
  const int half = lane >> 5, i = lane & 31;
  // floor(n_tok * r / R) in 32 bits: n_tok < 2^31 and R <= 2^16, so (n_tok % R) * r < 2^32
  const uint32_t nt = (uint32_t)n_tok, ru = (uint32_t)R, qt = nt / ru, mt = nt % ru;
  const uint32_t r = (uint32_t)r0 + (uint32_t)half;
  const uint32_t t0 = qt * (uint32_t)r0 + mt * (uint32_t)r0 / ru;
  const uint32_t t1 = qt * (uint32_t)(r0 + 1) + mt * (uint32_t)(r0 + 1) / ru;
  const int64_t target = half ? t1 : t0;
  int64_t lo = r >= ru ? n_docs : 0, hi = n_docs;
  while (__ballot(lo < hi)) {
    const bool open = lo < hi;
    const int64_t step = (hi - lo + 31) >> 5;
    const int64_t last = hi - 1;
    int64_t p = lo + (int64_t)(i + 1) * step - 1;
    p = p < last ? p : last;
    const bool below = open && off[p] < target;
    const int c = __popc((uint32_t)(__ballot(below) >> (32 * half)));
    if (open) {
      const int64_t pl = lo + (int64_t)c * step - 1, ph = pl + step;
      const int64_t nlo = c > 0 ? (pl < last ? pl : last) + 1 : lo;
      hi = c < 32 ? (ph < last ? ph : last) : hi;
      lo = nlo;
    }
  }
  return (int)lo;
}

// A copy of a per-lane value that the compiler cannot see through: the ring addresses of the
// per-document results are formed from it where they are used (once per document) instead of
// being kept per (ring slot, tile) in registers that every stage would rotate.  Indexing the
// ring as one flat array keeps the slot arithmetic scalar.
__device__ __forceinline__ int opaque(int v) {
  int r;
  asm volatile("v_mov_b32 %0, %1" : "=v"(r) : "v"(v));
  return r;
}

template <int KS, int NB, int WPW, bool DIRECT>
__global__ __launch_bounds__(64 * WPW, 2) void maxsim_argmax_kernel(
    MaxsimArgs a, const int64_t* __restrict__ off) {
  using G = ArgGeom<KS, DIRECT>;
  static_assert(!DIRECT || G::kTps == WPW, "direct staging: one tile per wave");
  // two workgroups per CU (what the plan assumes for every variant): two stages and the ring
  static_assert(2 * (2 * G::kStageB + 3 * G::kTps * (WPW * NB * 4 + WPW * NB * 32 * 2)) <=
                    160 * 1024,
                "LDS of two resident workgroups");
  constexpr int kThreads = 64 * WPW;
  constexpr int kSlotsWG = WPW * NB * 32;
  constexpr int kTps = G::kTps;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][G::kStageB];
  __shared__ float res_score[3][kTps][kSlotsWG / 32];
  __shared__ uint16_t res_amax[3][kTps][kSlotsWG];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31;
  const int half = lane >> 5;

  const uint32_t total = (uint32_t)a.n_qgroups * (uint32_t)a.n_ranges;
  const uint32_t lin = (uint32_t)xcd_linear(blockIdx.x, total);
  const int rng = __builtin_amdgcn_readfirstlane((int)(lin / (uint32_t)a.n_qgroups));
  const int qg = __builtin_amdgcn_readfirstlane((int)(lin - (uint32_t)rng * a.n_qgroups));
  if (blockIdx.x == 0 && tid < a.n_ctrl) a.ctrl[tid] = 0;  // read only by later kernels
  const int qwg = qg * WPW * a.qpw;
  const int q0 = qwg + wave * a.qpw;
  const bool wave_active = q0 < a.nq;

  // ---- query slots -> B operands (resident)
  bf16x8 bq[NB][KS];
  int slot_row[NB];
  uint32_t my_blocks = 0;
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
  // (the query operands are waited for together with the first stage's tiles, below)

  // ---- this workgroup's documents: found while the query loads are in flight
  const int first = range_first_doc(off, a.n_docs, a.n_tok, a.n_ranges, rng, lane);
  const int d_begin = __builtin_amdgcn_readlane(first, 0);
  const int d_end = __builtin_amdgcn_readlane(first, 32);
  if (d_begin >= d_end) return;  // uniform for the whole workgroup

  const int n_tok = (int)a.n_tok;
  auto open_doc = [&](TileCursor& c, int dd) {  // bounds clamped as in maxsim_kernel
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

  // ---- producer (as in maxsim_kernel, unswizzled padded rows)
  constexpr int kRp = kThreads / G::kCpr;
  constexpr int kPpt = kRp >= 32 ? 1 : 32 / kRp;
  constexpr int kTpp = kRp >= 32 ? kRp / 32 : 1;
  constexpr int kUpt = kTps * kPpt / kTpp;
  TileCursor prod;
  open_doc(prod, d_begin);
  u32x4 stage_regs[DIRECT ? 1 : kUpt];
  const int lr = (tid / G::kCpr) & 31;
  const int lt = __builtin_amdgcn_readfirstlane((tid / G::kCpr) >> 5);
  const int lc = tid % G::kCpr;
  const bool lok = 8 * lc < a.dim;
  const uint32_t lboff = 16u * lc;
  if (a.dim < 16 * KS) {  // chunks past dim are never stored: they must read as zeros
    for (int i = tid; i < (int)(sizeof(lds) / 16); i += kThreads)
      reinterpret_cast<u32x4*>(&lds[0][0])[i] = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
  }
  const uint32_t row_bytes = 2u * (uint32_t)a.dim;
  // direct staging: this lane's source offset within the tile for each of the tile's loads
  // (rows below 32 of the tile's first token; 0 for the lanes that fill padding)
  auto direct_off = [&](int q, uint32_t rmx) {
    const int p = q * 1024 + 16 * lane;
    const int row = p / G::kRowB;
    const int c = (p - row * G::kRowB) >> 4;
    const uint32_t r = (uint32_t)row < rmx ? (uint32_t)row : rmx;
    return (row < 32 && c < G::kCpr) ? r * (uint32_t)(32 * KS) + 16u * (uint32_t)c : 0u;
  };
  uint32_t doff[DIRECT ? G::kLoads : 1];
  if constexpr (DIRECT) {
#pragma unroll
    for (int q = 0; q < G::kLoads; ++q) doff[q] = direct_off(q, 31u);
  }
  // direct staging: wave w loads tile w of the stage, whose first token is r0 and last row rmx
  auto issue_tile = [&](int buf, int r0, uint32_t rmx) {
    const char* tptr = reinterpret_cast<const char*>(a.d) + (uint64_t)(uint32_t)r0 * row_bytes;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(tptr), (short)0, 0x7fffffff, 0x00020000);
    unsigned char* dst = &lds[buf][wave * G::kTileS];
    if (rmx >= 31u) {
#pragma unroll
      for (int q = 0; q < G::kLoads; ++q)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(dst + 1024 * q), 16,
                                                 (int)doff[q], 0, 0, 0);
    } else {  // a document's last, partial tile: rows past its end repeat its last token
#pragma unroll
      for (int q = 0; q < G::kLoads; ++q)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(dst + 1024 * q), 16,
                                                 (int)direct_off(q, rmx), 0, 0, 0);
    }
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
      const uint32_t rmx = ok ? prod.len - prod.t * 32 - 1 : 0;
      if constexpr (DIRECT) {
        if (j == wave) {  // uniform
          my_ok = ok;
          my_r0 = r0;
          my_rmx = rmx;
        }
      } else if (j % kTpp == lt && lok) {
        const char* tptr =
            reinterpret_cast<const char*>(a.d) + (uint64_t)(uint32_t)r0 * row_bytes;
#pragma unroll
        for (int p = 0; p < kPpt; ++p) {
          const uint32_t row = lr + kRp * p;
          const uint32_t r = row < rmx ? row : rmx;
          stage_regs[(j / kTpp) * kPpt + p] = load16(tptr + (r * row_bytes + lboff));
        }
      }
      if (ok) {
        sd.valid |= 1u << j;
        if (prod.t + 1 == prod.cnt) sd.last |= 1u << j;
        if (prod.len > 65536) sd.lng |= 1u << j;
        if (++prod.t == prod.cnt) {
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
      *reinterpret_cast<u32x4*>(&lds[buf][j * G::kTileS + row * G::kRowB + lboff]) = stage_regs[m];
    }
  };

  // ---- consumer state (see maxsim_kernel): rm, bk, bt per block
  float rm[NB];
  int bk[NB], bt[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    rm[b] = -__builtin_huge_valf();
    bk[b] = INT32_MIN;
    bt[b] = 0;
  }
  const int64_t n_entries = (int64_t)a.nq * a.lq;
  const int n_wg_q = (a.nq - qwg) < WPW * a.qpw ? (a.nq - qwg) : WPW * a.qpw;
  const int n_wg_e = n_wg_q * a.lq;
  const int row_base = 4 * half;
  const uint32_t a_lane = (uint32_t)(col * G::kRowB + half * 16);  // A operand: row col, chunk half

  f32x16 accA[NB], accB[NB];

  // A operand fragment of k-step s of tile j in stage buffer `buf` (immediate offset 32 s).
  auto frag = [&](int buf, int j, int s) {
    return as_bf16x8(*reinterpret_cast<const u32x4*>(&lds[buf][j * G::kTileS] + a_lane + 32 * s));
  };
  // The tile is processed in kRegions scheduling regions of kRs k-steps each (at most 4, so
  // that only two sets of A fragments are live); region p of the epilogue covers registers
  // [kRv p, kRv (p + 1)) of every block of Y: the tile maximum mt, the packed argmax keys k (see
  // the tile keys above) and their maximum mk; the last region also updates the running
  // maximum.
  constexpr int kRs = KS / 2 < 4 ? KS / 2 : 4;
  constexpr int kRegions = KS / kRs;
  constexpr int kRv = 16 / kRegions;
  auto epi_part = [&](const f32x16 (&Y)[NB], int part, float (&mt)[NB], int (&k)[NB][16],
                      int (&mk)[NB]) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int r0 = kRv * part;
      float m = fmaxf(Y[b][r0], Y[b][r0 + 1]);
#pragma unroll
      for (int r = r0 + 2; r < r0 + kRv; r += 2) m = fmaxf(fmaxf(m, Y[b][r]), Y[b][r + 1]);
#pragma unroll
      for (int r = r0; r < r0 + kRv; ++r)
        k[b][r] = __builtin_amdgcn_bitop3_b32(__float_as_int(Y[b][r]), ~15, 15 - r, 0xea);
      int x = max(k[b][r0], k[b][r0 + 1]);
#pragma unroll
      for (int r = r0 + 2; r < r0 + kRv; r += 2) x = max3_i(x, k[b][r], k[b][r + 1]);
      mt[b] = part == 0 ? m : fmaxf(mt[b], m);
      mk[b] = part == 0 ? x : max(mk[b], x);
      if (part == kRegions - 1) rm[b] = fmaxf(rm[b], mt[b]);
    }
  };
  // Rest of the epilogue: lanes whose tile is all negative (one branch for every block, taken
  // by rare waves; it recomputes the keys from Y, whose registers are live until the next
  // step, so that the region's 16 keys per block need not stay live past it), the key update,
  // the end of a document.
  auto epi_finish = [&](const f32x16 (&Y)[NB], const float (&mt)[NB], int (&mk)[NB],
                        const PendTile& p) {
    bool neg = false;
#pragma unroll
    for (int b = 0; b < NB; ++b) neg |= mt[b] < 0.f;
    if (__ballot(neg) != 0) {  // a wave-uniform branch: no exec-mask save and restore
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        int kn[16];  // sign-flipped keys: ((bits ^ 0x7fffffff) & ~15) | (15 - r)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          kn[r] = __builtin_amdgcn_bitop3_b32(__float_as_int(Y[b][r]), ~15, 15 - r, 0xea) ^
                  0x7ffffff0;
        int x = max(kn[0], kn[1]);
#pragma unroll
        for (int r = 2; r < 16; r += 2) x = max3_i(x, kn[r], kn[r + 1]);
        mk[b] = mt[b] < 0.f ? x : mk[b];
      }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      // strictly larger truncated key <=> mk > (bk | 15): the earlier tile keeps ties
      const bool take = mk[b] > (bk[b] | 15);
      bk[b] = take ? mk[b] : bk[b];
      bt[b] = take ? p.t : bt[b];
    }
    if (p.last) {
      float qs = 0.f;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        // the two half-waves (rows 0-15 and 16-31 of the tile column) meet through
        // v_permlane32_swap: in the lanes of half 0, element 0 is the lane's own value and
        // element 1 its partner's (only those lanes' results are used)
        const auto sm = __builtin_amdgcn_permlane32_swap(__float_as_uint(rm[b]),
                                                         __float_as_uint(rm[b]), false, false);
        const float m = fmaxf(__uint_as_float(sm[0]), __uint_as_float(sm[1]));
        rm[b] = -__builtin_huge_valf();
        const int r = (bk[b] & 15) ^ 15;
        int x = bt[b] * 32 + row_base + r + (r & 12);  // row 8 (r / 4) + 4 half + r % 4
        const int tv = bk[b] & ~15;
        const int otv = (int)__builtin_amdgcn_permlane32_swap((uint32_t)tv, (uint32_t)tv,
                                                              false, false)[1];
        const int ox = (int)__builtin_amdgcn_permlane32_swap((uint32_t)x, (uint32_t)x, false,
                                                             false)[1];
        const bool tk = (otv > tv) | ((otv == tv) & (ox < x));
        x = tk ? ox : x;
        if (half == 0 && slot_row[b] >= 0)
          res_amax[0][0][opaque(slot_row[b]) + (p.rb * kTps + p.j) * kSlotsWG] = (uint16_t)x;
        bk[b] = INT32_MIN;
        const float v = half32_sum(slot_row[b] >= 0 ? m : 0.f);
        if ((my_blocks >> b) & 1u) qs += v;
      }
      if (lane < a.qpw)
        res_score[0][0][opaque(wave * a.qpw + lane) + (p.rb * kTps + p.j) * (kSlotsWG / 32)] = qs;
    }
  };
  // One pipelined step: the MFMAs of tile j (stage buffer `buf`) into X and, when HAS_Y, the
  // epilogue values of the previous tile Y interleaved with them.  Region p first issues the
  // LDS reads of the A fragments of region p + 1 (for the last region: region 0 of tile j + 1,
  // when that tile is in the same stage), then runs its MFMAs with a share of the epilogue's
  // VALU instructions after each; fr[p % 2] holds the fragments region p uses (fr[0] holds tile
  // j's region 0 on entry, tile j + 1's on exit).
  auto step = [&](auto has_y, f32x16 (&X)[NB], const f32x16 (&Y)[NB], int buf, int j,
                  bf16x8 (&fr)[2][kRs], float (&mt)[NB], int (&k)[NB][16], int (&mk)[NB]) {
    constexpr bool kHasY = decltype(has_y)::value;
    constexpr int kV = (kRv * 2 * NB + kRs * NB - 1) / (kRs * NB);  // VALU per MFMA
#pragma unroll
    for (int p = 0; p < kRegions; ++p) {
      const bool last_region = p + 1 == kRegions;
      const bool reads = !last_region || j + 1 < kTps;
#pragma unroll
      for (int s = 0; s < kRs; ++s) {
        if (!last_region)
          fr[(p + 1) & 1][s] = frag(buf, j, (p + 1) * kRs + s);
        else if (reads)
          fr[(p + 1) & 1][s] = frag(buf, j + 1, s);
      }
#pragma unroll
      for (int s = 0; s < kRs; ++s)
#pragma unroll
        for (int b = 0; b < NB; ++b)
          X[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              fr[p & 1][s], bq[b][p * kRs + s], (p == 0 && s == 0) ? f32x16{} : X[b], 0, 0, 0);
      if constexpr (kHasY) epi_part(Y, p, mt, k, mk);
      if (reads) __builtin_amdgcn_sched_group_barrier(0x100, kRs, 0);  // DS reads
#pragma unroll
      for (int i = 0; i < kRs * NB; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                // MFMA
        if constexpr (kHasY) __builtin_amdgcn_sched_group_barrier(0x002, kV, 0);  // VALU
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // the documents that end in a stage are consecutive from its first one, one per bit of `last`
  auto write_results = [&](const StageDesc& sd, int rb) {
    int d = sd.d0;
#pragma unroll 1
    for (uint32_t m = sd.last & sd.valid; m != 0u; m &= m - 1u, ++d) {
      const int j = __builtin_ctz(m);
      // a document too long for 16-bit argmax offsets scores NaN, which the loss carries on
      // (stored as the bit pattern: this file is compiled assuming no NaN arithmetic)
      const bool lng = (sd.lng >> j) & 1u;
      const int slot = rb * kTps + j;
      if (tid < n_wg_q)
        reinterpret_cast<uint32_t*>(a.scores)[(int64_t)(qwg + tid) * a.n_docs + d] =
            lng ? 0x7fc00000u
                : __float_as_uint(res_score[0][0][opaque(tid) + slot * (kSlotsWG / 32)]);
      uint16_t* dst = a.amax + (int64_t)d * n_entries + (int64_t)qwg * a.lq;
      for (int e = tid; e < n_wg_e; e += kThreads)
        dst[e] = res_amax[0][0][opaque(e) + slot * kSlotsWG];
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
  bf16x8 fr[2][kRs];  // see step; region 0 of a stage's first tile is read after its barrier
#pragma unroll
  for (int s = 0; s < kRs; ++s) fr[0][s] = frag(0, 0, s);

  // Pipeline state (uniform): whether a computed tile awaits its epilogue, which accumulator set
  // holds it (B after every full stage, since kTps is even), and its descriptor.
  bool pend = false;
  bool pend_in_a = false;
  PendTile pt = {0, 0, 0, false};
  int ct = 0;  // tile index within its document of the next tile to compute
  int stage = 0;
  for (;; ++stage) {
    const int buf = stage & 1;
    const int rb = stage % 3;
    const bool more = prod.d < d_end;
    if (more) fetch_stage(nxt, buf ^ 1);  // direct staging: into the other buffer, now idle
    // direct staging: the results of two stages ago go out while the tiles run, so that the
    // stage's closing wait for its loads finds the stores complete
    if constexpr (DIRECT)
      if (stage >= 2) write_results(prv2, (stage - 2) % 3);
    if (wave_active) {
#pragma unroll
      for (int j = 0; j < kTps; ++j) {
        if (!((cur.valid >> j) & 1u)) break;  // uniform: only the final stage is partial
        const bool last = (cur.last >> j) & 1u;
        f32x16 (&X)[NB] = (j & 1) ? accB : accA;
        f32x16 (&Y)[NB] = (j & 1) ? accA : accB;
        float mt[NB];
        int k[NB][16], mk[NB];
        if (pend) {
          step(std::true_type{}, X, Y, buf, j, fr, mt, k, mk);
          epi_finish(Y, mt, mk, pt);
        } else {
          step(std::false_type{}, X, Y, buf, j, fr, mt, k, mk);
        }
        pend = true;
        pend_in_a = !(j & 1);
        pt = PendTile{ct, rb, j, last};
        ct = last ? 0 : ct + 1;
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
#pragma unroll
    for (int s = 0; s < kRs; ++s) fr[0][s] = frag(buf ^ 1, 0, s);
    prv2 = prv;
    prv = cur;
    cur = nxt;
  }
  // the last computed tile's epilogue, then the results of the final two stages
  if (wave_active && pend) {
    float mt[NB];
    int k[NB][16], mk[NB];
    if (pend_in_a) {
#pragma unroll
      for (int p = 0; p < kRegions; ++p) epi_part(accA, p, mt, k, mk);
      epi_finish(accA, mt, mk, pt);
    } else {
#pragma unroll
      for (int p = 0; p < kRegions; ++p) epi_part(accB, p, mt, k, mk);
      epi_finish(accB, mt, mk, pt);
    }
  }
  __syncthreads();
  if (stage >= 1) write_results(prv, (stage - 1) % 3);
  write_results(cur, stage % 3);
}

template <int KS, int NB, int WPW, bool DIRECT = false>
hipError_t launch_argmax_t(const MaxsimPlan& plan, const MaxsimArgs& args, hipStream_t stream) {
  const int64_t blocks = (int64_t)plan.n_qgroups * plan.n_ranges;
  hipLaunchKernelGGL((maxsim_argmax_kernel<KS, NB, WPW, DIRECT>), dim3((unsigned)blocks),
                     dim3(64 * WPW), 0, stream, args, args.off);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_argmax_variant(const MaxsimPlan& plan, const MaxsimArgs& args,
                                 hipStream_t stream) {
  switch (plan.ks) {
    case 2: return launch_argmax_t<2, 2, 4>(plan, args, stream);
    case 4: return launch_argmax_t<4, 2, 4>(plan, args, stream);
    case 8:
      return args.dim == 128 ? launch_argmax_t<8, 2, 4, true>(plan, args, stream)
                             : launch_argmax_t<8, 2, 4>(plan, args, stream);
    case 16: return launch_argmax_t<16, 1, 4>(plan, args, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace msim
}  // namespace hpr
