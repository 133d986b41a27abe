// Fidelity profiling of threshold-map masks on sampled rows (paper Sec. 4.2.1
// and 4.2.3): for a sampled query row with dense softmax P, and the sparse row
// P~ of a mask M_p = 1[T <= p] (the softmax over the keys of enabled blocks,
// which is what block-sparse attention computes), the Hellinger distance of
// Eq. 3 depends on one number only, the mass m that P puts on the enabled
// blocks:  sum_j sqrt(p_j q_j) = sqrt(m) when q = p / m on the kept keys, so
//   H = sqrt(1 - sqrt(m)) = sqrt(x / (1 + sqrt(1 - x))),   x = 1 - m.
// The second form uses the dropped mass x directly and has no cancellation
// when little is dropped.  The profile therefore needs, per sampled row, the
// dense row's mass on each key block; every candidate threshold is then a
// masked sum over blocks.
//
// Kernel 1 (block masses, bound by reading K): workgroup = (b, h, chunk of key
// blocks), 4 wavefronts, one key block at a time per wavefront.  S^T = K Q^T
// on v_mfma_f32_32x32x16_bf16 with the (up to 32) sampled rows as the 32
// columns: Q^T fragments stay in registers (the B operand), K rows are loaded
// straight from global memory as the A operand.  Each lane then holds one
// row's logits for its half of the keys; the block's log-sum-exp is a lane
// reduction plus one exchange between the half-wavefronts.
// Kernel 2 (one wavefront per sampled row, one lane per candidate): the row's
// dense log-normaliser from its block log-masses, then for each candidate p
// the dropped mass over blocks with !(T <= p) and H from the closed form above.  Kernel 3 averages
// 1 - H over a head's rows into the Fidelity Score (Eq. 4).

#include <math.h>

#include "device_common.h"
#include "launch.h"

namespace sa {

namespace {

constexpr float kLog2eF = 1.4426950408889634f;
constexpr float kLn2F = 0.6931471805599453f;
constexpr int kFidWaves = 4;
constexpr int kFidBlocksPerWave = 4;  // key blocks per wavefront per workgroup

template <int D>
__global__ __launch_bounds__(64 * kFidWaves) void fid_block_mass_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const int32_t* __restrict__ rows,
    int R, int H, int N, int blk, int n_kb, float c_log2, float* __restrict__ blk_lse) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int half = lane >> 5;
  const int l32 = lane & 31;
  const int bh = blockIdx.y;
  const int h = bh % H;
  const int64_t base = (int64_t)bh * N * D;

  // Q^T fragments of the sampled rows: column l32 is row rows[h][l32] (zero past R)
  bf16x8 qf[D / 16];
  {
    int r = l32 < R ? rows[(int64_t)h * R + l32] : 0;
    r = min(max(r, 0), N - 1);
#pragma unroll
    for (int dc = 0; dc < D / 16; ++dc)
      qf[dc] = l32 < R ? *(const bf16x8*)(Q + base + (int64_t)r * D + dc * 16 + half * 8)
                       : bf16x8{};
  }

  // This wavefront's key blocks are v_first + t * kFidWaves + wave; they are
  // walked as one stream of 32-key groups, and the next group's K fragments
  // are requested before the current group's MFMAs so that loads overlap.
  const int v_first = blockIdx.x * (kFidWaves * kFidBlocksPerWave) + wave;
  int n_blocks = 0;  // blocks of this wavefront that exist
  while (n_blocks < kFidBlocksPerWave && v_first + n_blocks * kFidWaves < n_kb) ++n_blocks;
  if (n_blocks == 0) return;  // uniform per wavefront; no workgroup barrier below
  const int gpb = blk / 32;   // 32-key groups per block

  auto group_key0 = [&](int j) { return (v_first + (j / gpb) * kFidWaves) * blk + (j % gpb) * 32; };
  auto load_group = [&](int j, bf16x8 (&kf)[D / 16]) {
    const int key = min(group_key0(j) + l32, N - 1);
    const __bf16* krow = K + base + (int64_t)key * D;
#pragma unroll
    for (int dc = 0; dc < D / 16; ++dc) kf[dc] = *(const bf16x8*)(krow + dc * 16 + half * 8);
  };

  const int n_groups = n_blocks * gpb;
  bf16x8 kf[D / 16], kn[D / 16];
  load_group(0, kf);
  float mx = -INFINITY;
  float sum = 0.f;  // sum of exp2(s - mx) over this lane's keys of the current block
  for (int j = 0; j < n_groups; ++j) {
    if (j + 1 < n_groups) load_group(j + 1, kn);
    const int v = v_first + (j / gpb) * kFidWaves;
    const int key_hi = min((v + 1) * blk, N);
    const int g0 = group_key0(j);
    f32x16 s = {};
    if (g0 < key_hi) {  // uniform; groups wholly past N hold no key
#pragma unroll
      for (int dc = 0; dc < D / 16; ++dc) s = mfma32x32x16(kf[dc], qf[dc], s);
      // register i: key g0 + 8 (i / 4) + 4 half + i % 4 of this lane's row
      float gmx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int kk = g0 + 8 * (i >> 2) + 4 * half + (i & 3);
        s[i] = kk < key_hi ? s[i] * c_log2 : -INFINITY;
        gmx = fmaxf(gmx, s[i]);
      }
      const float nmx = fmaxf(mx, gmx);
      if (nmx != -INFINITY) {  // a lane may see only masked keys of a ragged block
        float gs = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) gs += fast_exp2(s[i] - nmx);
        sum = (mx == -INFINITY ? 0.f : sum * fast_exp2(mx - nmx)) + gs;
        mx = nmx;
      }
    }
    if (j % gpb == gpb - 1) {  // last group of block v: combine the half-wavefronts
      const float omx = other_half(mx);
      const float osum = other_half(sum);
      const float tmx = fmaxf(mx, omx);
      const float tsum = (mx == -INFINITY ? 0.f : sum * fast_exp2(mx - tmx)) +
                         (omx == -INFINITY ? 0.f : osum * fast_exp2(omx - tmx));
      if (half == 0 && l32 < R)
        blk_lse[((int64_t)bh * R + l32) * n_kb + v] = (tmx + fast_log2(tsum)) * kLn2F;
      mx = -INFINITY;
      sum = 0.f;
    }
#pragma unroll
    for (int dc = 0; dc < D / 16; ++dc) kf[dc] = kn[dc];
  }
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

constexpr int kFidMaxR = 32;
constexpr int kFidMaxK = 64;

// One wavefront per sampled row (b, h, i); lane c owns candidate c (K <= 64).
// The row's dense log-normaliser comes from its block log-masses (lanes over
// blocks), then every lane walks all blocks: the block's mass and map entry
// are the same for the whole wavefront, and lane c adds the mass when the
// block is off for its threshold.  Each block costs a few instructions
// whatever the number of candidates, and no per-candidate reduction is left.
__global__ __launch_bounds__(64 * kFidWaves) void fid_row_kernel(
    const float* __restrict__ blk_lse, const int32_t* __restrict__ rows, int R,
    const float* __restrict__ T, const float* __restrict__ p, int K, int H, int N, int blk,
    int n_qb, int n_kb, float* __restrict__ hel) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.y * kFidWaves + (threadIdx.x >> 6);
  if (i >= R) return;  // uniform per wavefront
  const int bh = blockIdx.x;
  const int h = bh % H;
  const float* lrow = blk_lse + ((int64_t)bh * R + i) * n_kb;
  const int r = min(max(rows[(int64_t)h * R + i], 0), N - 1);
  const float* trow = T + ((int64_t)h * n_qb + r / blk) * n_kb;
  float mx = -INFINITY;
  for (int v = lane; v < n_kb; v += 64) mx = fmaxf(mx, lrow[v]);
  mx = wave_max(mx);
  float z = 0.f;
  for (int v = lane; v < n_kb; v += 64) z += __expf(lrow[v] - mx);
  const float lse = mx + __logf(wave_sum(z));
  const float pc = lane < K ? p[lane] : 0.f;
  float dropped = 0.f;
  bool kept = false;
#pragma unroll 8
  for (int v = 0; v < n_kb; ++v) {
    const float t = trow[v];                 // wavefront-uniform address
    const float mass = __expf(lrow[v] - lse);
    if (t <= pc)                             // NaN on either side: block off
      kept = true;
    else
      dropped += mass;
  }
  dropped = fminf(fmaxf(dropped, 0.f), 1.f);
  if (lane < K)
    hel[((int64_t)bh * R + i) * K + lane] = kept ? sqrtf(dropped / (1.f + sqrtf(1.f - dropped))) : 1.f;
}

// Fidelity Score per (b, h, candidate): 1 - mean over the sampled rows.
__global__ __launch_bounds__(256) void fid_mean_kernel(const float* __restrict__ hel, int R, int K,
                                                       int64_t n_out, float* __restrict__ fid) {
  const int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;  // o = bh * K + c
  if (o >= n_out) return;
  const int64_t bh = o / K;
  const int c = (int)(o - bh * K);
  float acc = 0.f;
  for (int i = 0; i < R; ++i) acc += hel[(bh * R + i) * K + c];
  fid[o] = 1.f - acc / (float)R;
}

}  // namespace

bool fidelity_supported(int R, int K) { return R >= 1 && R <= kFidMaxR && K >= 1 && K <= kFidMaxK; }

hipError_t launch_fidelity(const void* q, const void* k, const int32_t* rows, int R, const float* T,
                           const float* p, int K, float* blk_lse, float* hel, float* fid, int B,
                           int H, int N, int d, int blk, float scale, hipStream_t stream) {
  const int n_qb = (N + blk - 1) / blk;
  const int n_kb = n_qb;
  const int per_wg = kFidWaves * kFidBlocksPerWave;
  const dim3 grid1((n_kb + per_wg - 1) / per_wg, B * H);
  const float c_log2 = scale * kLog2eF;
  if (d == 128)
    hipLaunchKernelGGL(fid_block_mass_kernel<128>, grid1, dim3(64 * kFidWaves), 0, stream,
                       (const __bf16*)q, (const __bf16*)k, rows, R, H, N, blk, n_kb, c_log2, blk_lse);
  else
    hipLaunchKernelGGL(fid_block_mass_kernel<64>, grid1, dim3(64 * kFidWaves), 0, stream,
                       (const __bf16*)q, (const __bf16*)k, rows, R, H, N, blk, n_kb, c_log2, blk_lse);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(fid_row_kernel, dim3(B * H, (R + kFidWaves - 1) / kFidWaves),
                     dim3(64 * kFidWaves), 0, stream, blk_lse, rows, R, T, p, K, H, N, blk, n_qb,
                     n_kb, hel);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n_out = (int64_t)B * H * K;
  hipLaunchKernelGGL(fid_mean_kernel, dim3((unsigned)((n_out + 255) / 256)), dim3(256), 0, stream,
                     hel, R, K, n_out, fid);
  return hipGetLastError();
}

}  // namespace sa
