// Calibration kernels: what the chip sustains, measured, to set beside the published peaks.
//
//   mfma_calibration_kernel  every wave runs four independent accumulation chains of
//                            v_mfma_f32_32x32x16_bf16 on register operands (no memory traffic)
//                            for a fixed number of iterations: 4 * 32768 FLOP per iteration.
//                            The operands are either a fixed low-entropy pattern or random
//                            bf16 values of the magnitude of unit-vector components: the matrix
//                            cores' sustained rate depends on the operands' bits (their switching
//                            power sets the clock the chip can hold), so the second is the
//                            ceiling for embeddings.
//   read_calibration_kernel  a grid-stride stream of 16-byte streaming (non-temporal) loads
//                            over a buffer, folded with
//                            integer adds (so the loads cannot be dropped), one word per
//                            workgroup written: the sustained HBM read rate.
// Both end after a fixed amount of work; nothing they compute is meaningful beyond keeping the
// work alive.
#include "common.h"
#include "kernels.h"

namespace hpr {

namespace {

typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kCalThreads = 256;

// A random bf16 pair: signs and 7-bit mantissas uniform, exponents 2^-5 .. 2^-2.
__device__ uint32_t random_bf16_pair(uint32_t x) {
  x ^= x >> 16;  // murmur3's 32-bit finaliser
  x *= 0x85ebca6bu;
  x ^= x >> 13;
  x *= 0xc2b2ae35u;
  x ^= x >> 16;
  const uint32_t lo = (x & 0x807fu) | ((0x7au + ((x >> 7) & 3u)) << 7);
  const uint32_t hi = ((x >> 16) & 0x807fu) | ((0x7au + ((x >> 23) & 3u)) << 7);
  return lo | (hi << 16);
}

template <bool kRandom>
__global__ __launch_bounds__(kCalThreads) void mfma_calibration_kernel(float* sink, int64_t iters) {
  const int lane = threadIdx.x & 63;
  bf16x8 a[4], b[4];
  if constexpr (kRandom) {  // a different operand pair in every chain, lane and wave
    const uint32_t seed = (uint32_t)(blockIdx.x * kCalThreads + threadIdx.x) * 64u;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      u32x4 ra, rb;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        ra[w] = random_bf16_pair(seed + 8u * c + w);
        rb[w] = random_bf16_pair(seed + 8u * c + 4u + w);
      }
      a[c] = as_bf16x8(ra);
      b[c] = as_bf16x8(rb);
    }
  } else {  // operands from the lane index, so nothing is known at compile time
    u32x4 ra = {0x3c003c00u + lane, 0x3c003c01u, 0x3c003c02u + lane, 0x3c003c03u};
    u32x4 rb = {0x3c003c04u, 0x3c003c05u + lane, 0x3c003c06u, 0x3c003c07u + lane};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      a[c] = as_bf16x8(ra);
      b[c] = as_bf16x8(rb);
    }
  }
  f32x16 acc0 = {}, acc1 = {}, acc2 = {}, acc3 = {};
  for (int64_t i = 0; i < iters; ++i) {
    acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1], b[1], acc1, 0, 0, 0);
    acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[2], b[2], acc2, 0, 0, 0);
    acc3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[3], b[3], acc3, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += acc0[r] + acc1[r] + acc2[r] + acc3[r];
  if (s == 1234.5f) sink[blockIdx.x] = s;  // never true in practice; keeps the chains live
}

__global__ __launch_bounds__(kCalThreads) void read_calibration_kernel(const u32x4* __restrict__ p,
                                                                       int64_t n16,
                                                                       uint32_t* sink) {
  constexpr int kU = 4;  // loads in flight per thread (eight waves per SIMD)
  const int64_t stride = (int64_t)gridDim.x * kCalThreads;
  uint32_t acc = 0;
  for (int64_t base = (int64_t)blockIdx.x * kCalThreads + threadIdx.x; base < n16;
       base += stride * kU) {
    u32x4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int64_t i = base + u * stride;
      v[u] = i < n16 ? __builtin_nontemporal_load(p + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) acc += v[u].x + v[u].y + v[u].z + v[u].w;
  }
  acc = (uint32_t)wave_sum((float)acc);
  if (threadIdx.x == 0) sink[blockIdx.x] = acc;
}

}  // namespace

int64_t mfma_calibration_waves(int n_cu) { return (int64_t)(n_cu > 0 ? n_cu : 256) * 4 * 2; }

hipError_t launch_mfma_calibration(float* sink, int64_t iters, int n_cu, bool random_operands,
                                   hipStream_t stream) {
  const int64_t waves = mfma_calibration_waves(n_cu);
  const unsigned blocks = (unsigned)(waves / (kCalThreads / kWave));
  if (random_operands)
    hipLaunchKernelGGL(mfma_calibration_kernel<true>, dim3(blocks), dim3(kCalThreads), 0, stream,
                       sink, iters);
  else
    hipLaunchKernelGGL(mfma_calibration_kernel<false>, dim3(blocks), dim3(kCalThreads), 0, stream,
                       sink, iters);
  return hipGetLastError();
}

hipError_t launch_read_calibration(const void* buf, int64_t bytes, uint32_t* sink, int blocks,
                                   hipStream_t stream) {
  hipLaunchKernelGGL(read_calibration_kernel, dim3((unsigned)blocks), dim3(kCalThreads), 0, stream,
                     reinterpret_cast<const u32x4*>(buf), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace hpr
