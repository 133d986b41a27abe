// Sustained bf16 MFMA rate of the part, for the benchmark's roofline (not
// part of the attention path).  Every wavefront keeps four independent
// 32x32 fp32 accumulators and runs v_mfma_f32_32x32x16_bf16 on operands held
// in registers, loaded once from caller-supplied data (random values, so the
// matrix cores toggle as they do on real inputs: constant operands draw less
// power and run faster than any real kernel can).  One workgroup of 8
// wavefronts per CU, the occupancy of the attention kernel: the workgroup
// reserves 96 KB of LDS, so that no second one fits on a CU and the grid (one
// workgroup per CU) spreads evenly.  The accumulators are reduced into `out`
// so that nothing is dead.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"

namespace sa {
namespace {

constexpr int kPeakWaves = 8;  // wavefronts per workgroup
constexpr int kPeakLdsWords = 96 * 1024 / 4;  // reserved, keeps one workgroup per CU
constexpr int kPeakAcc = 4;    // independent accumulators per wavefront

__global__ __launch_bounds__(64 * kPeakWaves, 1) void mfma_peak_kernel(
    const bf16x8* __restrict__ src, float* __restrict__ out, int iters) {
  __shared__ float reserve[kPeakLdsWords];
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * kPeakWaves + (threadIdx.x >> 6);
  bf16x8 a[kPeakAcc], b[kPeakAcc];
#pragma unroll
  for (int i = 0; i < kPeakAcc; ++i) {
    a[i] = src[i * 64 + lane];
    b[i] = src[(kPeakAcc + i) * 64 + lane];
  }
  f32x16 acc[kPeakAcc];
#pragma unroll
  for (int j = 0; j < kPeakAcc; ++j) acc[j] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < kPeakAcc; ++k)
#pragma unroll
      for (int j = 0; j < kPeakAcc; ++j)  // consecutive MFMAs are independent
        acc[j] = mfma32x32x16(a[k], b[(k + j) % kPeakAcc], acc[j]);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kPeakAcc; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  reserve[threadIdx.x * (kPeakLdsWords / (64 * kPeakWaves))] = s;  // the reservation is used
  __syncthreads();
  out[(int64_t)wave * 64 + lane] = reserve[(threadIdx.x ^ 64) * (kPeakLdsWords / (64 * kPeakWaves))];
}

}  // namespace
}  // namespace sa

// src: device bf16 [2 * 4 * 64 * 8] (random values); out: device float
// [n_wg * 8 * 64]; each of n_wg workgroups (one per CU) runs iters * 16 MFMAs
// per wavefront (32 x 32 x 16 each, 32768 flop).  Returns 0, or 1 on a bad
// argument or a launch error.  Asynchronous on `stream`.
extern "C" __attribute__((visibility("default"))) int sa_mfma_peak(const void* src, float* out,
                                                                  int n_wg, int iters,
                                                                  void* stream) {
  if (!src || !out || n_wg < 1 || iters < 1) return 1;
  hipLaunchKernelGGL(sa::mfma_peak_kernel, dim3(n_wg), dim3(64 * sa::kPeakWaves), 0,
                     (hipStream_t)stream, (const sa::bf16x8*)src, out, iters);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}
