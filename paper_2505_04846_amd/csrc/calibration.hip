// Calibration kernels: what the chip sustains, measured, to set beside the published peaks.
//
//   mfma_calibration_kernel  every wave runs four independent accumulation chains of
//                            v_mfma_f32_32x32x16_bf16 on register operands (no memory traffic)
//                            for a fixed number of iterations: 4 * 32768 FLOP per iteration.
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

__global__ __launch_bounds__(kCalThreads) void mfma_calibration_kernel(float* sink, int64_t iters) {
  const int lane = threadIdx.x & 63;
  // operands from the lane index, so nothing is known at compile time
  u32x4 ra = {0x3c003c00u + lane, 0x3c003c01u, 0x3c003c02u + lane, 0x3c003c03u};
  u32x4 rb = {0x3c003c04u, 0x3c003c05u + lane, 0x3c003c06u, 0x3c003c07u + lane};
  const bf16x8 a = as_bf16x8(ra), b = as_bf16x8(rb);
  f32x16 acc0 = {}, acc1 = {}, acc2 = {}, acc3 = {};
  for (int64_t i = 0; i < iters; ++i) {
    acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc1, 0, 0, 0);
    acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc2, 0, 0, 0);
    acc3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc3, 0, 0, 0);
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

hipError_t launch_mfma_calibration(float* sink, int64_t iters, int n_cu, hipStream_t stream) {
  const int64_t waves = mfma_calibration_waves(n_cu);
  const unsigned blocks = (unsigned)(waves / (kCalThreads / kWave));
  hipLaunchKernelGGL(mfma_calibration_kernel, dim3(blocks), dim3(kCalThreads), 0, stream, sink,
                     iters);
  return hipGetLastError();
}

hipError_t launch_read_calibration(const void* buf, int64_t bytes, uint32_t* sink, int blocks,
                                   hipStream_t stream) {
  hipLaunchKernelGGL(read_calibration_kernel, dim3((unsigned)blocks), dim3(kCalThreads), 0, stream,
                     reinterpret_cast<const u32x4*>(buf), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace hpr
