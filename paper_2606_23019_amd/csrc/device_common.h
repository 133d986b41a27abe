// Device-side helpers for the gfx950 kernels: vector types, MFMA and LDS
// transpose-read wrappers, and small wavefront utilities.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define SA_LDS __attribute__((address_space(3)))

// D = A * B + C for a 32x32 fp32 tile with K = 16 bf16 (v_mfma_f32_32x32x16_bf16).
// Lane l supplies A[l % 32][8 * (l / 32) + e] and B[8 * (l / 32) + e][l % 32],
// e = 0..7, and holds C[8 * (i / 4) + 4 * (l / 32) + i % 4][l % 32] in register i.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ds_read_b64_tr_b16: inside each group of 16 lanes, lane j loads 4 bf16 from its
// own address; lane i of the group receives element (i % 4) of lane 4 r + i / 4
// for r = 0..3.  With lane j pointing at row (j / 4), columns 4 (j % 4) .. +3 of
// a row-major 4 x 16 tile, lane i receives column i (rows 0..3).
__device__ __forceinline__ bf16x4 lds_read_tr16_b64(const __bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((SA_LDS bf16x4*)(p));
}

__device__ __forceinline__ bf16x8 lds_read_b128(const __bf16* p) {
  return *(const SA_LDS bf16x8*)(p);
}

__device__ __forceinline__ void lds_write_b128(__bf16* p, u32x4 v) {
  *(SA_LDS u32x4*)(p) = v;
}

// Value held by lane l ^ 32.
__device__ __forceinline__ float other_half(float x) { return __shfl_xor(x, 32, 64); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

}  // namespace sa
