// Late-interaction (MaxSim) scoring on gfx950 MFMA, with the max over document tokens fused in
// registers (the Lq x Ld similarity table never leaves the register file).
//
// Decomposition
//   * Query side.  A wave owns NB blocks of 16 query-token "slots" (NB*16 slots): whole queries
//     of lqp = round_up(lq, 16) slots each.  Their bf16 tokens stay in VGPRs for the whole
//     kernel as the B operand of v_mfma_f32_16x16x32_bf16 (K = 32 per step, KS steps).
//   * Document side.  Each document is cut into tiles of 16 consecutive tokens (the A operand,
//     rows = document tokens).  A tile never straddles two documents: rows past a document's
//     last token re-load that last token, which leaves the maximum unchanged (max is
//     idempotent), so no masking is needed.
//   * MFMA C layout (16x16): lane l holds column l % 16 (a query slot) and rows
//     4 * (l / 16) + r, r = 0..3 (document tokens), so the running max over document tokens is an
//     in-lane v_max per accumulator register; only at the end of a document are the 4 row
//     registers and the 4 lane groups reduced, and the slot maxima summed per query.
//   * Workgroup = 4 waves on 4 different query sets, all streaming the same document range, so
//     each document tile is fetched from L2 once per workgroup and hits in L1 for the other
//     waves.  Workgroups sharing a document range are mapped onto the same XCD.
//   * K permutation.  Lane group g = l / 16 of step s carries contraction indices
//     32 s + 8 g .. 32 s + 8 g + 7 for both operands; A and B use the same rule, so every
//     product pairs matching indices whatever order the hardware reduces them in.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

struct MaxsimArgs {
  const uint16_t* q;
  const uint16_t* d;
  const int64_t* off;
  const int64_t* part;
  float* scores;
  uint16_t* amax;
  int32_t* flag;
  int64_t n_docs, n_tok;
  int nq, lq, lqp, qpw, dim, n_qgroups, n_ranges;
};

// Tiles per LDS stage (a stage is loaded by the whole workgroup while the previous one is
// consumed), and the LDS geometry of one 16-token tile: rows of KS*64 bytes holding 16-byte
// chunks at XOR-swizzled positions so that the 16 lanes reading one chunk index from 16
// different rows hit 16 different bank groups.
template <int KS>
struct TileGeom {
  static constexpr int kCpr = KS * 4;            // 16-byte chunks per row
  static constexpr int kRowB = KS * 64;          // bytes per row
  static constexpr int kTileB = 16 * kRowB;      // bytes per tile
  static constexpr int kTps = KS >= 8 ? 4 : 8;   // tiles per stage
  static constexpr int kUnitsPerTile = 16 * kCpr;  // 16-byte units per tile
};

// Position of tile `t` of the current document stream; uniform across the workgroup.
struct TileCursor {
  int64_t d;      // document
  int64_t base;   // first token row (clamped)
  int64_t len;    // tokens (>= 1)
  int t;          // tile index within the document
  int cnt;        // tiles of the document
};

template <int KS, int NB, int WPW, bool ARGMAX>
__global__ __launch_bounds__(64 * WPW, (KS == 8 && ARGMAX) ? 1 : 2) void maxsim_kernel(MaxsimArgs a) {
  using G = TileGeom<KS>;
  constexpr int kThreads = 64 * WPW;
  // units loaded per thread for each tile of a stage
  constexpr int kRpt = G::kUnitsPerTile > kThreads ? G::kUnitsPerTile / kThreads : 1;
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][G::kTps * G::kTileB];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int col = lane & 15;
  const int grp = lane >> 4;

  const int64_t total = (int64_t)a.n_qgroups * a.n_ranges;
  const int64_t lin = xcd_linear(blockIdx.x, total);
  const int rng = (int)(lin / a.n_qgroups);
  const int qg = (int)(lin - (int64_t)rng * a.n_qgroups);
  const int64_t d_begin = a.part[rng], d_end = a.part[rng + 1];
  if (d_begin >= d_end) return;  // uniform for the whole workgroup
  const int q0 = (qg * WPW + wave) * a.qpw;
  const bool wave_active = q0 < a.nq;  // idle waves still load tiles and meet the barriers

  // ---- query slots -> B operands (resident for the whole kernel)
  bf16x8 bq[NB][KS];
  int slot_row[NB];        // q * lq + i of this lane's slot in block b, or -1 for padding
  uint32_t my_blocks = 0;  // bit b set when block b belongs to query (q0 + lane)
  const int lqb = a.lqp >> 4;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int slot = b * 16 + col;
    const int ql = slot / a.lqp;
    const int i = slot - ql * a.lqp;
    const int qq = q0 + ql;
    const bool valid = wave_active && ql < a.qpw && qq < a.nq && i < a.lq;
    slot_row[b] = valid ? qq * a.lq + i : -1;
    if (b / lqb == lane) my_blocks |= 1u << b;
    const uint16_t* src = a.q + (int64_t)(valid ? slot_row[b] : 0) * a.dim;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int k = 32 * s + 8 * grp;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (valid && k < a.dim) v = load16(src + k);
      bq[b][s] = as_bf16x8(v);
    }
  }

  const int64_t last_tok = a.n_tok - 1;
  // Document bounds clamped into [0, n_tok) so that even an invalid CSR cannot make a load go
  // out of bounds; for a valid CSR they are exactly (off[d], off[d+1] - off[d]).
  auto open_doc = [&](TileCursor& c, int64_t dd) {
    int64_t lo = a.off[dd], hi = a.off[dd + 1];
    lo = lo < 0 ? 0 : (lo > last_tok ? last_tok : lo);
    hi = hi <= lo ? lo + 1 : (hi > a.n_tok ? a.n_tok : hi);
    c.d = dd;
    c.base = lo;
    c.len = hi - lo;
    c.t = 0;
    c.cnt = (int)((c.len + 15) >> 4);
  };
  auto advance = [&](TileCursor& c) {  // to the next tile; c.d == d_end marks the end
    if (++c.t == c.cnt) {
      if (c.d + 1 < d_end)
        open_doc(c, c.d + 1);
      else
        c.d = d_end;
    }
  };

  // ---- producer: the next stage's tiles, loaded into registers, then stored to LDS.  Tile j
  // of a stage is loaded by units u = tid + kThreads m (row u / kCpr, chunk u % kCpr).
  TileCursor prod;
  open_doc(prod, d_begin);
  u32x4 stage_regs[G::kTps][kRpt];
  auto fetch_stage = [&]() {
#pragma unroll
    for (int j = 0; j < G::kTps; ++j) {
      const bool ok = prod.d < d_end;
      const int64_t base = prod.base, len = prod.len;
      const int t = prod.t;
#pragma unroll
      for (int m = 0; m < kRpt; ++m) {
        const int u = tid + kThreads * m;
        const int row = u / G::kCpr;
        const int c = u % G::kCpr;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (ok && u < G::kUnitsPerTile && 8 * c < a.dim) {
          int64_t r = (int64_t)t * 16 + row;
          r = r < len ? r : len - 1;  // rows past the end repeat the document's last token
          v = load16_stream(a.d + (base + r) * a.dim + 8 * c);
        }
        stage_regs[j][m] = v;
      }
      if (ok) advance(prod);
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int j = 0; j < G::kTps; ++j)
#pragma unroll
      for (int m = 0; m < kRpt; ++m) {
        const int u = tid + kThreads * m;
        if (u < G::kUnitsPerTile) {
          const int row = u / G::kCpr;
          const int c = u % G::kCpr;
          const int cs = c ^ (row & (G::kCpr - 1));
          *reinterpret_cast<u32x4*>(&lds[buf][j * G::kTileB + row * G::kRowB + cs * 16]) =
              stage_regs[j][m];
        }
      }
  };

  float rm[NB][4];
  int ra[NB][4];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      rm[b][r] = -__builtin_huge_valf();
      ra[b][r] = 0;
    }
  const int64_t n_entries = (int64_t)a.nq * a.lq;

  TileCursor cons;
  open_doc(cons, d_begin);

  fetch_stage();
  store_stage(0);
  __syncthreads();

  for (int stage = 0;; ++stage) {
    const int buf = stage & 1;
    const bool more = prod.d < d_end;
    if (more) fetch_stage();  // global loads in flight while this stage is computed

#pragma unroll 1
    for (int j = 0; j < G::kTps; ++j) {
      if (cons.d >= d_end) break;  // uniform
      if (wave_active) {
        // A operand: tile row `col`, k chunk 4 s + grp (swizzled position in LDS)
        bf16x8 av[KS];
        const unsigned char* tile = &lds[buf][j * G::kTileB + col * G::kRowB];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const int c = 4 * s + grp;
          av[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(tile + ((c ^ (col & (G::kCpr - 1))) * 16)));
        }
        f32x4 acc[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
          for (int b = 0; b < NB; ++b)
            acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[s], bq[b][s], acc[b], 0, 0, 0);
        const int t = cons.t;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = acc[b][r];
            if (ARGMAX) {
              const bool gt = v > rm[b][r];  // strict: the earlier tile keeps ties
              rm[b][r] = gt ? v : rm[b][r];
              ra[b][r] = gt ? t : ra[b][r];
            } else {
              rm[b][r] = fmaxf(rm[b][r], v);
            }
          }
        if (t + 1 == cons.cnt) {  // last tile of the document: reduce and emit
          const int64_t d = cons.d;
          float qs = 0.f;
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            float m = rm[b][0];
            int jx = ra[b][0] * 16 + grp * 4;
#pragma unroll
            for (int r = 1; r < 4; ++r) {
              const float v = rm[b][r];
              if (ARGMAX) {
                const int jj = ra[b][r] * 16 + grp * 4 + r;
                if (v > m || (v == m && jj < jx)) {
                  m = v;
                  jx = jj;
                }
              } else {
                m = fmaxf(m, v);
              }
            }
#pragma unroll
            for (int mask = 16; mask <= 32; mask <<= 1) {
              const float om = __shfl_xor(m, mask);
              if (ARGMAX) {
                const int oj = __shfl_xor(jx, mask);
                if (om > m || (om == m && oj < jx)) {
                  m = om;
                  jx = oj;
                }
              } else {
                m = fmaxf(m, om);
              }
            }
            if (ARGMAX && grp == 0 && slot_row[b] >= 0)
              a.amax[d * n_entries + slot_row[b]] = (uint16_t)jx;
            float v = slot_row[b] >= 0 ? m : 0.f;
            v += __shfl_xor(v, 1);
            v += __shfl_xor(v, 2);
            v += __shfl_xor(v, 4);
            v += __shfl_xor(v, 8);
            if ((my_blocks >> b) & 1u) qs += v;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              rm[b][r] = -__builtin_huge_valf();
              ra[b][r] = 0;
            }
          }
          if (lane < a.qpw && q0 + lane < a.nq) a.scores[(int64_t)(q0 + lane) * a.n_docs + d] = qs;
          if (ARGMAX && cons.len > 65536 && lane == 0) *a.flag = 1;
        }
      }
      advance(cons);
    }

    if (more) store_stage(buf ^ 1);
    __syncthreads();
    if (!more) break;
  }
}

__global__ void partition_kernel(const int64_t* off, int64_t n_docs, int64_t n_tok, int R,
                                 int64_t* part, int32_t* ctrl) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < 2 && ctrl) ctrl[r] = 0;
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

template <int KS, int NB, int WPW, bool ARGMAX>
hipError_t launch_t(const MaxsimPlan& plan, const MaxsimArgs& args, hipStream_t stream) {
  const int64_t blocks = (int64_t)plan.n_qgroups * plan.n_ranges;
  hipLaunchKernelGGL((maxsim_kernel<KS, NB, WPW, ARGMAX>), dim3((unsigned)blocks), dim3(64 * WPW),
                     0, stream, args);
  return hipGetLastError();
}

// Variants: (dim <= 32 * KS) x argmax.  The argmax variants keep fewer query slots per wave
// (NB = 4) and run 8 waves per workgroup so that two waves fit per SIMD and one wave's argmax
// VALU work overlaps another's MFMAs; the plain variants hold 128 slots per wave.
hipError_t launch_variant(const MaxsimPlan& plan, const MaxsimArgs& args, bool argmax,
                          hipStream_t stream) {
  if (argmax) {
    switch (plan.ks) {
      case 1: return launch_t<1, 4, 8, true>(plan, args, stream);
      case 2: return launch_t<2, 4, 8, true>(plan, args, stream);
      case 4: return launch_t<4, 4, 8, true>(plan, args, stream);
      case 8: return launch_t<8, 4, 4, true>(plan, args, stream);
      default: return hipErrorInvalidValue;
    }
  }
  switch (plan.ks) {
    case 1: return launch_t<1, 8, 4, false>(plan, args, stream);
    case 2: return launch_t<2, 8, 4, false>(plan, args, stream);
    case 4: return launch_t<4, 8, 4, false>(plan, args, stream);
    case 8: return launch_t<8, 4, 4, false>(plan, args, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool maxsim_plan(int nq, int lq, int64_t n_docs, int64_t n_tok, int dim, bool argmax, int n_cu,
                 MaxsimPlan* p) {
  if (dim < 8 || dim > 256 || dim % 8 != 0 || lq < 1 || nq < 1 || n_docs < 1) return false;
  p->ks = dim <= 32 ? 1 : dim <= 64 ? 2 : dim <= 128 ? 4 : 8;
  p->nb = (p->ks == 8 || argmax) ? 4 : 8;
  p->wpw = (argmax && p->ks < 8) ? 8 : 4;
  p->lqp = (lq + 15) / 16 * 16;
  if (p->lqp > p->nb * 16) return false;
  p->qpw = p->nb * 16 / p->lqp;
  const int64_t q_per_wg = (int64_t)p->qpw * p->wpw;
  p->n_qgroups = (int)((nq + q_per_wg - 1) / q_per_wg);
  // Enough workgroups to fill every CU twice over four times, but no range shorter than
  // ~1024 tokens (the query operands are re-loaded by every workgroup).
  const int64_t target_wg = (int64_t)(n_cu > 0 ? n_cu : 256) * 2 * 4;
  int64_t R = (target_wg + p->n_qgroups - 1) / p->n_qgroups;
  const int64_t max_by_tokens = n_tok / 1024 > 0 ? n_tok / 1024 : 1;
  if (R > max_by_tokens) R = max_by_tokens;
  if (R > n_docs) R = n_docs;
  if (R > kMaxRanges) R = kMaxRanges;
  if (R < 1) R = 1;
  if ((int64_t)p->n_qgroups * R > 0x7fffffffLL) return false;
  p->n_ranges = (int)R;
  return true;
}

hipError_t launch_partition(const int64_t* off, int64_t n_docs, int64_t n_tok, int n_ranges,
                            int64_t* part, int32_t* ctrl, hipStream_t stream) {
  const int threads = 256;
  const int blocks = (n_ranges + 1 + threads - 1) / threads;
  hipLaunchKernelGGL(partition_kernel, dim3(blocks), dim3(threads), 0, stream, off, n_docs,
                     n_tok, n_ranges, part, ctrl);
  return hipGetLastError();
}

hipError_t launch_maxsim(const MaxsimPlan& plan, const uint16_t* q, int nq, int lq,
                         const uint16_t* d_tok, const int64_t* off, int64_t n_docs,
                         int64_t n_tok, int dim, const int64_t* part, float* scores,
                         uint16_t* amax, int32_t* flag, hipStream_t stream) {
  MaxsimArgs args;
  args.q = q;
  args.d = d_tok;
  args.off = off;
  args.part = part;
  args.scores = scores;
  args.amax = amax;
  args.flag = flag;
  args.n_docs = n_docs;
  args.n_tok = n_tok;
  args.nq = nq;
  args.lq = lq;
  args.lqp = plan.lqp;
  args.qpw = plan.qpw;
  args.dim = dim;
  args.n_qgroups = plan.n_qgroups;
  args.n_ranges = plan.n_ranges;
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
