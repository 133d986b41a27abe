// Conservative resize of threshold maps and block masks between resolutions
// (paper Sec. 4.3.1, Eq. 7).  Target block (u, v) samples the base map at
// x = u n_q / n_q', y = v n_k / n_k' (exact rationals: integer quotient and
// remainder); the bilinear neighbours with positive weight are base rows
// floor(x) and, if the remainder is non-zero, floor(x) + 1 (clamped to the
// last row), and likewise for columns.
//  * mask: the ceiling of the bilinear interpolation of a 0/1 mask is 1 iff a
//    positively weighted neighbour is 1, i.e. the OR of those <= 4 bits;
//  * threshold map: the minimum over the same neighbours, which makes
//    instantiation and resizing commute (1[T' <= p] is the resized 1[T <= p]).
// Both are streams over the target with cached reads of the base: in the map
// kernel a thread writes one column of eight target rows; in the mask kernel
// a wavefront takes a target row, stages its two source rows in LDS and forms
// each CRM word with a ballot.

#include "device_common.h"
#include "launch.h"

namespace sa {

namespace {

struct AxisPt {
  int i0, i1;
  bool two;  // the second neighbour has a positive weight
};

// floor(t n_base / n_target) and whether the remainder is non-zero, without a
// 64-bit division: t n_base < 2^32 and the quotient is < 2^16, so the single-
// precision estimate num * (1 / n_target) is within 3 * 2^-24 * 2^16 < 0.02 of
// the true quotient and one integer remainder step fixes it.
__device__ __forceinline__ AxisPt axis_point(int t, int n_base, int n_target, float inv_target) {
  const int64_t num = (int64_t)t * n_base;
  int q = (int)((float)num * inv_target);
  int64_t rem = num - (int64_t)q * n_target;
  if (rem < 0) {
    --q;
    rem += n_target;
  } else if (rem >= n_target) {
    ++q;
    rem -= n_target;
  }
  return AxisPt{q, min(q + 1, n_base - 1), rem > 0};
}

constexpr int kMapRowsPerThread = 8;

// grid: (target columns / 256, target rows / 8, heads); each thread writes one
// column of eight consecutive target rows (few, well-filled workgroups).
__global__ __launch_bounds__(256) void resize_map_kernel(const float* __restrict__ T, int nq,
                                                         int nk, float* __restrict__ out, int tq,
                                                         int tk) {
  const int v = blockIdx.x * 256 + threadIdx.x;
  if (v >= tk) return;
  const int h = blockIdx.z;
  const AxisPt b = axis_point(v, nk, tk, 1.0f / (float)tk);
  const float inv_tq = 1.0f / (float)tq;
  const float* Th = T + (int64_t)h * nq * nk;
  const int u_end = min(tq, (int)(blockIdx.y + 1) * kMapRowsPerThread);
  for (int u = blockIdx.y * kMapRowsPerThread; u < u_end; ++u) {
    const AxisPt a = axis_point(u, nq, tq, inv_tq);
    float m = Th[(int64_t)a.i0 * nk + b.i0];
    if (b.two) m = fminf(m, Th[(int64_t)a.i0 * nk + b.i1]);  // fminf skips NaN
    if (a.two) {
      m = fminf(m, Th[(int64_t)a.i1 * nk + b.i0]);
      if (b.two) m = fminf(m, Th[(int64_t)a.i1 * nk + b.i1]);
    }
    out[((int64_t)h * tq + u) * tk + v] = m;
  }
}

__device__ __forceinline__ uint32_t crm_bit(const uint64_t* row, int j) {
  return (uint32_t)((row[j >> 6] >> (j & 63)) & 1ull);
}

constexpr int kResizeWaves = 4;

// One wavefront per target row; the two source rows are staged in LDS first so
// that the per-bit lookups are LDS reads, not dependent global loads.
__global__ __launch_bounds__(64 * kResizeWaves) void resize_mask_kernel(
    const uint64_t* __restrict__ bits, int H, int nq, int nk, int W, uint64_t* __restrict__ out,
    int tq, int tk, int Wt) {
  extern __shared__ uint64_t rows_lds[];  // [waves][2][W]
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * kResizeWaves + wave;
  if (row >= (int64_t)H * tq) return;  // uniform per wavefront; no workgroup barrier below
  const int h = (int)(row / tq);
  const int u = (int)(row - (int64_t)h * tq);
  const AxisPt a = axis_point(u, nq, tq, 1.0f / (float)tq);
  const float inv_tk = 1.0f / (float)tk;
  const uint64_t* g0 = bits + ((int64_t)h * nq + a.i0) * W;
  const uint64_t* g1 = bits + ((int64_t)h * nq + a.i1) * W;
  uint64_t* r0 = rows_lds + (int64_t)wave * 2 * W;
  uint64_t* r1 = r0 + W;
  for (int w = lane; w < W; w += 64) {
    r0[w] = g0[w];
    r1[w] = g1[w];
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  uint64_t* orow = out + row * Wt;
  for (int w0 = 0; w0 < Wt; w0 += 64) {
    const int nw = min(64, Wt - w0);
    uint64_t mine = 0;
    for (int w = 0; w < nw; ++w) {
      const int v = (w0 + w) * 64 + lane;
      uint32_t on = 0;
      if (v < tk) {
        const AxisPt b = axis_point(v, nk, tk, inv_tk);
        on = crm_bit(r0, b.i0) | (b.two ? crm_bit(r0, b.i1) : 0u);
        if (a.two) on |= crm_bit(r1, b.i0) | (b.two ? crm_bit(r1, b.i1) : 0u);
      }
      const uint64_t word = __ballot(on != 0);
      if (lane == w) mine = word;
    }
    if (lane < nw) orow[w0 + lane] = mine;
  }
}

}  // namespace

hipError_t launch_resize_map(const float* T, int H, int nq, int nk, float* out, int tq, int tk,
                             hipStream_t stream) {
  hipLaunchKernelGGL(resize_map_kernel,
                     dim3((tk + 255) / 256, (tq + kMapRowsPerThread - 1) / kMapRowsPerThread, H),
                     dim3(256), 0, stream, T, nq, nk, out, tq, tk);
  return hipGetLastError();
}

hipError_t launch_resize_mask(const uint64_t* bits, int H, int nq, int nk, uint64_t* out, int tq,
                              int tk, hipStream_t stream) {
  const int64_t rows = (int64_t)H * tq;
  hipLaunchKernelGGL(resize_mask_kernel, dim3((unsigned)((rows + kResizeWaves - 1) / kResizeWaves)),
                     dim3(64 * kResizeWaves), kResizeWaves * 2 * ((nk + 63) / 64) * 8, stream, bits,
                     H, nq, nk, (nk + 63) / 64, out, tq, tk, (tk + 63) / 64);
  return hipGetLastError();
}

}  // namespace sa
