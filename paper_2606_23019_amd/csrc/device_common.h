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
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

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

// Max and sum of x over the lane pair (l, l ^ 32) with v_permlane32_swap,
// which exchanges lanes 32..63 of its first operand with lanes 0..31 of its
// second: with x in both, every lane ends up holding its own x and its
// partner's, one in each result, and a symmetric operation on the two needs
// no select.  Vector ALU only, unlike other_half (a ds_bpermute through the
// LDS, which waits behind other wavefronts' LDS traffic).  Both results are
// exactly those of x op other_half(x).
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Work layout for the XCDs.  Launch position pos runs on XCD pos mod 8 (the
// dispatcher deals workgroups round-robin), and each XCD takes its positions
// in increasing order.  Given n_units groups of n_qb items, ranked 0 ..
// n_units - 1, position pos = x + 8 j is item j of sequence x, where sequence
// x holds one chunk of every group in rank order.  The group of rank k gives
// sequence x q = n_qb / 8 items plus one when x is one of (k r + i) mod 8,
// i < r = n_qb mod 8 (the leftovers rotate, so every sequence is exactly as
// long as its share of positions), and the chunks are runs of consecutive u:
// sequence x takes the run at place (x + k) mod 8 in u order.  The rotation
// spreads the first and last query blocks of each group (whose key windows
// are cut short at the ends of the video) over all XCDs, so no XCD gets the
// light end chunks of every group.  Returns the rank k and writes the
// item's u.
constexpr int kXcds = 8;  // accelerator complex dies of an MI355X, one L2 each

// Items of sequence x in the groups of rank < k: k q plus the t < k r with
// t = x (mod 8), where q = n_qb / 8 and r = n_qb mod 8.
__device__ __forceinline__ int64_t xcd_prefix(int k, int x, int q, int r) {
  const int64_t t = (int64_t)k * r - x;
  return (int64_t)k * q + (t > 0 ? (t + kXcds - 1) / kXcds : 0);
}

// First u of sequence x's chunk of the group of rank k.  Its run is at
// place p = (x + k) mod 8, so u0 is p q plus the runs before it that hold a
// leftover item: the run at place p' belongs to sequence (p' - k) mod 8, which
// has one when p' = (k (r + 1) + i) mod 8 for an i < r.
__device__ __forceinline__ int xcd_chunk_u0(int k, int x, int q, int r) {
  const int p = (x + k) % kXcds;
  int before = 0;
#pragma unroll
  for (int i = 0; i < kXcds - 1; ++i) before += (i < r && ((k * (r + 1) + i) % kXcds) < p) ? 1 : 0;
  return p * q + before;
}

__device__ __forceinline__ int xcd_slice(int64_t pos, int n_units, int n_qb, int* u_out) {
  const int q = n_qb / kXcds;
  const int r = n_qb - q * kXcds;
  const int x = (int)(pos % kXcds);
  const int64_t j = pos / kXcds;
  // k0 = floor(8 j / n_qb) has prefix(k0) <= j (k0 q + ceil(k0 r / 8) <= j
  // since 8 k0 q + k0 r <= 8 j), and the rank is at most 1 + 7 / n_qb above
  // it, so a fixed number of forward steps finds it; the steps and the
  // leftover count are unrolled, so no loop is left in the code.
  const int64_t k_est = j * kXcds / n_qb;
  int k = (int)(k_est < n_units - 1 ? k_est : n_units - 1);
#pragma unroll
  for (int s = 0; s < kXcds; ++s)
    if (k + 1 < n_units && xcd_prefix(k + 1, x, q, r) <= j) ++k;
  *u_out = xcd_chunk_u0(k, x, q, r) + (int)(j - xcd_prefix(k, x, q, r));
  return k;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

}  // namespace sa
