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
// a wavefront takes target rows, stages the OR of each one's two source rows
// in LDS and forms each CRM word with a ballot, the column sample points
// coming from a table the workgroup shares.

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
// column of eight consecutive target rows (few, well-filled workgroups).  The
// row sample points are uniform over the workgroup; all loads of the eight
// rows go out before the first minimum is formed, so their latencies overlap.
__global__ __launch_bounds__(256) void resize_map_kernel(const float* __restrict__ T, int nq,
                                                         int nk, float* __restrict__ out, int tq,
                                                         int tk) {
  const int v = blockIdx.x * 256 + threadIdx.x;
  if (v >= tk) return;
  const int h = blockIdx.z;
  const AxisPt b = axis_point(v, nk, tk, 1.0f / (float)tk);
  const float inv_tq = 1.0f / (float)tq;
  const float* Th = T + (int64_t)h * nq * nk;
  const int u0 = blockIdx.y * kMapRowsPerThread;
  float x[kMapRowsPerThread][4];
#pragma unroll
  for (int r = 0; r < kMapRowsPerThread; ++r) {
    const int u = min(u0 + r, tq - 1);  // rows past the end repeat the last (not stored)
    const AxisPt a = axis_point(u, nq, tq, inv_tq);
    const float* r0 = Th + (int64_t)a.i0 * nk;
    const float* r1 = Th + (int64_t)a.i1 * nk;
    x[r][0] = r0[b.i0];
    x[r][1] = r0[b.i1];
    x[r][2] = r1[b.i0];
    x[r][3] = r1[b.i1];
    x[r][3] = a.two ? x[r][3] : x[r][0];
    x[r][2] = a.two ? x[r][2] : x[r][0];
  }
#pragma unroll
  for (int r = 0; r < kMapRowsPerThread; ++r) {
    // fminf skips NaN; neighbours with zero weight are replaced by the first
    float m = fminf(x[r][0], b.two ? x[r][1] : x[r][0]);
    m = fminf(m, fminf(x[r][2], b.two ? x[r][3] : x[r][2]));
    if (u0 + r < tq) out[((int64_t)h * tq + u0 + r) * tk + v] = m;
  }
}

constexpr int kResizeWaves = 4;
constexpr int kResizeRowsPerWave = 4;
// Target widths up to this many blocks keep their column sample points in a
// per-workgroup LDS table (32 KB); wider targets compute them per word.
constexpr int kResizeTableMax = 8192;

// A wavefront per target row, kResizeRowsPerWave rows per wavefront.  The
// target row's two base rows are ORed into one (the ceiling is the OR of the
// positively weighted neighbours, and the row and column choices combine
// independently), staged in LDS; the column sample points of the target
// width are shared by every row of the workgroup (TABLE: entry
// i0 | two << 31 per column).  Lane l of output word w takes target column
// 64 w + l; a ballot forms the word, and lane w keeps word w of a group of 64.
template <bool TABLE>
__global__ __launch_bounds__(64 * kResizeWaves) void resize_mask_kernel(
    const uint64_t* __restrict__ bits, int H, int nq, int nk, int W, uint64_t* __restrict__ out,
    int tq, int tk, int Wt) {
  extern __shared__ uint64_t lds_words[];  // [waves][W] ORed base rows, then the column table
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  uint32_t* table = (uint32_t*)(lds_words + kResizeWaves * W);
  const float inv_tk = 1.0f / (float)tk;
  if (TABLE) {
    for (int v = threadIdx.x; v < tk; v += 64 * kResizeWaves) {
      const AxisPt b = axis_point(v, nk, tk, inv_tk);
      table[v] = (uint32_t)b.i0 | (b.two ? 0x80000000u : 0u);
    }
    __syncthreads();
  }
  uint64_t* rr = lds_words + wave * W;
  const int64_t rows = (int64_t)H * tq;
  const int64_t row_first = ((int64_t)blockIdx.x * kResizeWaves + wave) * kResizeRowsPerWave;
  for (int k = 0; k < kResizeRowsPerWave; ++k) {
    const int64_t row = row_first + k;
    if (row >= rows) break;  // uniform per wavefront; no workgroup barrier below
    const int h = (int)(row / tq);
    const int u = (int)(row - (int64_t)h * tq);
    const AxisPt a = axis_point(u, nq, tq, 1.0f / (float)tq);
    const uint64_t* g0 = bits + ((int64_t)h * nq + a.i0) * W;
    const uint64_t* g1 = bits + ((int64_t)h * nq + a.i1) * W;
    __builtin_amdgcn_wave_barrier();  // the previous row's reads of rr are done
    for (int w = lane; w < W; w += 64) rr[w] = g0[w] | (a.two ? g1[w] : 0ull);
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
          int i0;
          bool two;
          if (TABLE) {
            const uint32_t e = table[v];
            i0 = (int)(e & 0x7fffffffu);
            two = (e >> 31) != 0;
          } else {
            const AxisPt b = axis_point(v, nk, tk, inv_tk);
            i0 = b.i0;
            two = b.two;
          }
          const int i1 = min(i0 + 1, nk - 1);
          on = (uint32_t)(rr[i0 >> 6] >> (i0 & 63)) & 1u;
          if (two) on |= (uint32_t)(rr[i1 >> 6] >> (i1 & 63)) & 1u;
        }
        const uint64_t word = __ballot(on != 0);
        if (lane == w) mine = word;
      }
      if (lane < nw) orow[w0 + lane] = mine;
    }
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
  const int W = (nk + 63) / 64, Wt = (tk + 63) / 64;
  const int64_t per_wg = (int64_t)kResizeWaves * kResizeRowsPerWave;
  const dim3 grid((unsigned)((rows + per_wg - 1) / per_wg));
  const size_t rows_bytes = (size_t)kResizeWaves * W * 8;
  if (tk <= kResizeTableMax)
    hipLaunchKernelGGL(resize_mask_kernel<true>, grid, dim3(64 * kResizeWaves),
                       rows_bytes + (size_t)tk * 4, stream, bits, H, nq, nk, W, out, tq, tk, Wt);
  else
    hipLaunchKernelGGL(resize_mask_kernel<false>, grid, dim3(64 * kResizeWaves), rows_bytes,
                       stream, bits, H, nq, nk, W, out, tq, tk, Wt);
  return hipGetLastError();
}

}  // namespace sa
