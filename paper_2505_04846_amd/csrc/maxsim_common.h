// Device-side pieces shared by the two MaxSim kernels (maxsim.hip: scores only;
// maxsim_argmax.hip: scores and the argmax for the loss): the launch arguments, the document
// cursor and stage descriptor of the LDS tile stream, cross-lane sums, and the packed argmax
// keys.
#pragma once

#include "common.h"
#include "kernels.h"

namespace hpr {
namespace msim {

typedef __attribute__((ext_vector_type(16))) float f32x16;

struct MaxsimArgs {
  const uint16_t* q;
  const uint16_t* d;
  const int64_t* off;
  const int64_t* part;  // range table of the score kernel (the argmax kernel finds its own)
  float* scores;
  uint16_t* amax;
  int32_t* ctrl;        // argmax kernel: control words of the call, zeroed by workgroup 0
  int64_t n_docs, n_tok;
  int nq, lq, lqp, qpw, dim, n_qgroups, n_ranges, n_ctrl;
  int persist;          // score kernel: persistent grid (see maxsim_kernel) ...
  int qg_base;          // ... and the first query group of the launch
};

// Position of tile `t` of the current document stream; uniform across the workgroup.  Token
// and document indices fit 32 bits (the host rejects stores of 2^31 tokens or more).
struct TileCursor {
  int d;      // document
  int base;   // first token row (clamped)
  int len;    // tokens (>= 1)
  int t;      // tile index within the document
  int cnt;    // tiles of the document
};

// Which tiles a stage holds, in scalar registers: the stage starts at tile t0 of document d0;
// bit j of `valid` / `last` / `lng` says that tile j exists / ends its document / belongs to a
// document of more than 65536 tokens.
struct StageDesc {
  int d0;
  int t0;
  uint32_t valid, last, lng;
};

// Argmax keys ("tile keys") of one 32x32 tile column: the lane's 16 values v_r (r = 0..15,
// rows ascending with r) as order-preserving integers o(v) (o(v) = bits of v for v >= 0,
// bits ^ 0x7fffffff below zero: increasing in v) with the low 4 bits replaced by 15 - r.  The
// signed maximum of the keys is then the largest o(v) & ~15 held by the lowest row, in one
// v_bitop3 per value ((bits & ~15) | (15 - r), truth table 0xea: a & b | c) plus one three-way
// max per two values (a compare-and-select search of the 16 rows costs about twice as many
// instructions).  The row selected is the first one whose value equals the maximum up to its 4
// lowest mantissa bits (a relative window below 2^-19); the score itself takes the exact
// maximum.  For v >= 0, o(v) = bits(v): a lane whose tile holds a non-negative value needs
// nothing else; a lane whose 16 values are all negative (its key is then negative) redoes the
// keys with the sign-flipped encoding, key ^ 0x7ffffff0.
__device__ __forceinline__ int max3_i(int a, int b, int c) { return max(max(a, b), c); }

// Cross-lane moves within a row of 16 lanes through DPP (no LDS round trip).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL,
                                                            0xf, 0xf, false));
}
constexpr int kDppQuadXor1 = 0xb1;    // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4e;    // quad_perm [2, 3, 0, 1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;

// Sum over the 32 lanes l, l ^ 1, ..., of each half-wave in a fixed order; every lane of the
// half gets the total.  The last step adds the two 16-lane rows of each half through
// v_permlane16_swap (no LDS round trip): with both operands v, element 0 holds the even row of
// each pair in both rows and element 1 the odd row, so their sum is the pair's total in every
// lane, the same bits whichever row a lane is in (addition being commutative).
__device__ __forceinline__ float half32_sum(float v) {
  v += dpp_f<kDppQuadXor1>(v);
  v += dpp_f<kDppQuadXor2>(v);
  v += dpp_f<kDppRowHalfMirror>(v);  // quad q with quad 1 - q of the same half row
  v += dpp_f<kDppRowMirror>(v);      // the two half rows: the 16-lane row total
  const auto sw = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                   false);
  return __uint_as_float(sw[0]) + __uint_as_float(sw[1]);  // the two rows of the half-wave
}

// Workgroups of maxsim_argmax_kernel per CU: two by registers (its launch bounds), fewer when
// two stages and the result ring do not fit the CU's 160 KiB of LDS twice.
constexpr int argmax_tps(int ks) { return ks >= 8 ? 2 : ks == 4 ? 4 : 8; }
constexpr int argmax_resident(int ks) {
  const int tile = 32 * (ks * 32 + 16);
  const int tps = argmax_tps(ks);
  const int nb = ks == 16 ? 1 : 2;
  const int res = 3 * tps * (4 * nb + 4 * nb * 32 * 2);
  const int by_lds = (160 * 1024) / (2 * tps * tile + res);
  return by_lds < 2 ? by_lds : 2;
}

// Launches the argmax kernel variant for plan.ks (maxsim_argmax.hip).
hipError_t launch_argmax_variant(const MaxsimPlan& plan, const MaxsimArgs& args,
                                 hipStream_t stream);

}  // namespace msim
}  // namespace hpr
