// Mask instantiation from a threshold map (paper Sec. 4.1.2): the mask for a
// density threshold p is M_p = 1[T <= p], one comparison per block, stored in
// the CRM layout (LSB-first uint64 words per query-block row).
//
// One wavefront per row (h, u) and set of up to 16 thresholds, eight words at
// a time.  Lane l loads T[h][u][64 w + l] for the eight words of the group
// into registers (all loads in flight together); then for every threshold
// p[i][h] a wavefront ballot of the comparison is the word itself (ballot bit
// l is lane l's predicate, i.e. key block 64 w + l at bit l), lane k keeps
// word k, and the group's words leave in one 64-byte store.  The thresholds of
// a wavefront come in with one vector load, so no scalar load waits inside the
// threshold loop.  The map is read from memory once per 16 thresholds (a
// head's map serves every timestep of its layer; the re-reads hit in L2): 4
// bytes read per block, one bit written per block and threshold, three vector
// instructions per 64 bits (the compare and two lane writes).

#include "device_common.h"
#include "launch.h"

namespace sa {

namespace {

constexpr int kInstWaves = 4;

constexpr int kGroup = 8;     // words whose map entries a lane holds in registers at once
constexpr int kInstThr = 16;  // thresholds per wavefront (grid.y splits larger sets)

// lo and hi hold the two halves of a wavefront-uniform 64-bit word in lane K,
// other lanes unchanged (v_writelane_b32).  The word is a ballot just written
// by a vector compare, and a vector read of a vector-written scalar needs two
// wait states first; one statement keeps the two writes behind the wait.
template <int K>
__device__ __forceinline__ void write_lane_k(uint32_t& lo, uint32_t& hi, uint64_t word) {
  asm("s_nop 1\n\tv_writelane_b32 %0, %2, %4\n\tv_writelane_b32 %1, %3, %4"
      : "+v"(lo), "+v"(hi)
      : "s"((uint32_t)word), "s"((uint32_t)(word >> 32)), "n"(K));
}
// The same for a k < kGroup that is a constant once the caller's loop is
// unrolled.
static_assert(kGroup <= 8, "write_lane covers lanes 0..7");
__device__ __forceinline__ void write_lane(uint32_t& lo, uint32_t& hi, uint64_t word, int k) {
  switch (k) {
    case 0: write_lane_k<0>(lo, hi, word); break;
    case 1: write_lane_k<1>(lo, hi, word); break;
    case 2: write_lane_k<2>(lo, hi, word); break;
    case 3: write_lane_k<3>(lo, hi, word); break;
    case 4: write_lane_k<4>(lo, hi, word); break;
    case 5: write_lane_k<5>(lo, hi, word); break;
    case 6: write_lane_k<6>(lo, hi, word); break;
    default: write_lane_k<7>(lo, hi, word); break;
  }
}

__global__ __launch_bounds__(64 * kInstWaves) void mask_inst_kernel(
    const float* __restrict__ T, const float* __restrict__ p, int n_p, int H, int n_qb, int n_kb,
    int W, uint64_t* __restrict__ bits) {
  const int lane = threadIdx.x & 63;
  const int64_t rows = (int64_t)H * n_qb;
  const int64_t row = (int64_t)blockIdx.x * kInstWaves + (threadIdx.x >> 6);
  if (row >= rows) return;  // uniform per wavefront
  const int h = (int)(row / n_qb);
  const int i_first = blockIdx.y * kInstThr;
  const int n_thr = min(kInstThr, n_p - i_first);
  // this wavefront's thresholds, lane k holding p[i_first + k][h], read once
  // with one vector load and handed to the comparisons by readlane
  const float p_lane = lane < n_thr ? p[(int64_t)(i_first + lane) * H + h] : 0.f;
  const float* trow = T + row * n_kb;
  for (int w0 = 0; w0 < W; w0 += kGroup) {
    const int nw = min(kGroup, W - w0);
    // all loads of the group first (independent, in flight together)
    float t[kGroup];
#pragma unroll
    for (int k = 0; k < kGroup; ++k) {
      const int v = (w0 + k) * 64 + lane;
      t[k] = (k < nw && v < n_kb) ? trow[v] : __builtin_nanf("");  // NaN: never on
    }
    for (int i = 0; i < n_thr; ++i) {  // uniform trip count
      const float pi = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, p_lane), i));
      uint32_t lo = 0, hi = 0;  // lane k ends up holding word w0 + k
#pragma unroll
      for (int k = 0; k < kGroup; ++k) {
        if (k < nw) {  // uniform
          const uint64_t word = __ballot(t[k] <= pi);
          write_lane(lo, hi, word, k);
        }
      }
      if (lane < nw)
        bits[((int64_t)(i_first + i) * rows + row) * W + w0 + lane] =
            ((uint64_t)hi << 32) | lo;
    }
  }
}

}  // namespace

hipError_t launch_mask_instantiate(const float* T, const float* p, int n_p, int H, int n_qb,
                                   int n_kb, uint64_t* bits, hipStream_t stream) {
  const int64_t rows = (int64_t)H * n_qb;
  const int W = (n_kb + 63) / 64;
  const int64_t grid = (rows + kInstWaves - 1) / kInstWaves;
  const int chunks = (n_p + kInstThr - 1) / kInstThr;
  if (chunks > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(mask_inst_kernel, dim3((unsigned)grid, (unsigned)chunks), dim3(64 * kInstWaves),
                     0, stream, T, p, n_p, H, n_qb, n_kb, W, bits);
  return hipGetLastError();
}

}  // namespace sa
