// Block-sparse attention forward for gfx950 (CDNA4).
//
// What it computes (paper Sec. 4.3.2): FlashAttention's forward pass with the
// dense key-block loop replaced by a walk over the key blocks enabled in the
// query block's Compressed Row Mask row.  Each executed block is a dense
// 128 x 128 (or 64 x 64) tile, so both contractions run on the matrix cores.
//
// Work item = (b, h, query block u), BQ / 32 wavefronts per item, each owning
// 32 query rows.  Items of 128 query rows, and the maskless path wherever
// the tiles fit in LDS, run 2 (or 4) items per 8-wavefront workgroup in
// ping-pong (bsattn_fwd_pp_kernel, described there); masked items of 64 rows
// run one item per workgroup (bsattn_fwd_kernel).  Per enabled key block kb:
//
//   1. the workgroup copies K[kb] and V[kb] (BK x D bf16, row-major) from
//      global memory into LDS (16-byte chunks, XOR-swizzled per row);
//   2. every wavefront computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16:
//      Q^T (its 32 queries) stays in registers as the B operand (read once
//      per item, in the ping-pong kernel through LDS where the tiles are
//      square), K rows come from LDS as the A operand.  In the transposed product each lane owns
//      one query column, so the row statistics of the softmax are lane-local
//      apart from one exchange between the two half-wavefronts;
//   3. online softmax in fp32 in the log2 domain: running max m and sum l,
//      p = exp2(s * scale * log2(e) - m), the accumulator rescaled by
//      exp2(m_old - m_new);
//   4. O^T += V^T P^T, again 32x32x16 MFMA: P (rounded to bf16) is already
//      in the B-operand layout -- the K rows were fed to the first product
//      in an order that makes this so -- and V^T comes from LDS through the
//      gfx950 transposing read ds_read_b64_tr_b16.
//
// Epilogue: out = O / l rounded to bf16 (or kept in fp32 for the fp32-output
// entry points), lse = (m + log2 l) ln 2; the rows go out through the free
// K/V tiles in LDS so that stores write whole rows (store_rows_staged).
// The same kernels with DENSE = true are the maskless path (every key block).
// Keys past N (ragged last block) are loaded as zeros and get -inf logits.

#include <math.h>

#include "device_common.h"
#include "launch.h"

namespace sa {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int BQ, int BK, int D>
struct Tile {
  static constexpr int kWaves = BQ / 32;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kChunksPerRow = D / 8;  // 16-byte chunks
  // a tile is copied by wave-wide 1 KB direct-to-LDS loads (64 lanes x 16 B)
  static constexpr int kLoadsPerWave = BK * kChunksPerRow / 64 / kWaves;
  static_assert(BQ % 32 == 0 && BK % 32 == 0 && D % 32 == 0, "tile shape");
  static_assert((BK * kChunksPerRow) % (64 * kWaves) == 0, "copy split");
};

// XOR applied to the 16-byte chunk index of LDS row r (same for K and V
// tiles).  LDS is read 256 bytes (64 banks of 4 bytes) per cycle: 16 lanes of
// a 16-byte read, or 32 lanes of an 8-byte transposing read.
//  d = 128 (a row is one 256-byte bank line, 16 chunks): K operand reads put
//  16 different rows at one logical chunk per cycle -> the XOR must be a
//  bijection on r mod 16; V transposing reads put rows 4k .. 4k + 3 at 4
//  adjacent chunks -> the XORs of those rows must differ in bits 2..3.
//  d = 64 (two rows share a bank line, 8 chunks): the same conditions applied
//  separately to even and odd rows.
template <int D>
__device__ __forceinline__ int swz(int r) {
  static_assert(D == 64 || D == 128, "head dim");
  if constexpr (D == 128)
    return ((r & 3) << 2) | ((r >> 2) & 3);
  else
    return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// Key (within a 32-key group) fed to MFMA row m: bits 2 and 3 of m swapped.
// With this order, register i of the S^T accumulator of lane l holds key
// 16 * (i / 8) + 8 * (l / 32) + (i % 8): eight consecutive keys per half
// wavefront, exactly the B-operand layout of the following P V product.
__device__ __forceinline__ int key_of_row(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

// Workgroup barrier after this wave's LDS reads have completed.  Unlike
// __syncthreads() it does not wait for outstanding global->LDS copies.  The
// memory clobber keeps the compiler from moving memory accesses across it.
__device__ __forceinline__ void barrier_lds_reads_done() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Workgroup barrier once all but the VM most recent global->LDS copies of
// every wave have landed (copies complete in issue order).
template <int VM>
__device__ __forceinline__ void barrier_copies_landed() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(VM) : "memory");
}

// One wave-wide direct-to-LDS copy: lane l reads 16 bytes at base + voff and
// writes them to LDS byte address m0 + 16 l.  Issued as inline assembly so
// that the compiler does not add conservative vmcnt waits before unrelated
// LDS reads; completion is awaited explicitly with barrier_copies_landed().
__device__ __forceinline__ void copy16_to_lds(uint32_t lds_byte_addr, const void* base,
                                              uint32_t voff) {
  asm volatile("global_load_lds_dwordx4 %0, %1"
               ::"v"(voff), "s"(base), "{m0}"(__builtin_amdgcn_readfirstlane(lds_byte_addr))
               : "memory");
}

// Per-lane byte offsets of a tile copy.  Lane l of load i writes the 16-byte
// LDS chunk 64 (i + kLoadsPerWave * wave) + l, i.e. row r = R (kLoadsPerWave
// wave + i) + l / C and physical chunk p = l mod C (C chunks per row, R = 64 / C
// rows per load); the XOR swizzle is applied by reading source chunk
// p ^ swz(r).  Source rows are sn elements apart (d for [B][H][N][d] tensors,
// H d for [B][N][H][d]).  The swizzle depends on r mod 16 only, so the lane's
// part of the offset repeats with period 4 in the load index n = kLoadsPerWave
// wave + i, and the rest, R n sn elements, is uniform over the wavefront:
// a plan holds 4 lane offsets, and each load adds its uniform row offset to
// the scalar base address.  (Every real row is congruent mod 16 to the row
// used for its swizzle: R (n - n mod 4) is a multiple of 16.)
template <typename T, int D>
struct CopyPlan {
  static constexpr int kRowsPerLoad = 64 / T::kChunksPerRow;
  uint32_t lane_off[4];  // byte offset of the lane's chunk for loads with n mod 4 = m
  __device__ __forceinline__ void init(int wave, int lane, int sn) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = (wave * T::kLoadsPerWave + j) & 3;  // n mod 4 of load j, j + 4, ...
      const int lr = lane / T::kChunksPerRow;
      const int p = lane % T::kChunksPerRow;
      const int r = m * kRowsPerLoad + lr;  // row relative to load n - n mod 4
      lane_off[j] = (uint32_t)(r * sn + ((p ^ swz<D>(r)) << 3)) * 2u;
    }
  }
  // wavefront-uniform byte offset of load i: rows R (n - n mod 4)
  __device__ __forceinline__ static int64_t row_off(int wave, int i, int sn) {
    const int n = wave * T::kLoadsPerWave + i;
    return (int64_t)((n & ~3) * kRowsPerLoad) * sn * 2;
  }
};

// Loads i0 .. i0 + count - 1 of a copy of rows key0 .. key0 + BK - 1 (rows sn
// elements apart) into an LDS tile with global_load_lds_dwordx4 (no
// registers; completion is tracked by vmcnt).  count and i0 are compile-time
// constants wherever this is inlined into an unrolled loop.  In a ragged last
// block, rows past N repeat row N - 1: finite values whose logits are masked
// and whose probabilities are exactly zero.
template <typename T, int BK, int D>
__device__ __forceinline__ void issue_tile_slice(__bf16* lds, const __bf16* src, int key0, int N,
                                                 int sn, int wave_u, int lane,
                                                 const CopyPlan<T, D>& cp, int i0, int count) {
  const char* tile = (const char*)(src + (int64_t)key0 * sn);
  const uint32_t lds0 =
      (uint32_t)(uintptr_t)(SA_LDS void*)lds + (uint32_t)(wave_u * T::kLoadsPerWave * 1024);
  if (key0 + BK <= N) {
#pragma unroll
    for (int i = i0; i < i0 + count; ++i)
      copy16_to_lds(lds0 + i * 1024, tile + CopyPlan<T, D>::row_off(wave_u, i, sn),
                    cp.lane_off[i & 3]);
  } else {
    // Row R n + lr of the tile is read from row min(R n + lr, last), addressed
    // from the tile start: lane_off covers rows R (n mod 4) + lr, so the rows
    // still to add are min(R (n - n mod 4), last - R (n mod 4) - lr), which is
    // negative when the clamped row lies below row R (n - n mod 4).  The sum
    // is taken mod 2^32 and equals the true offset, which is non-negative and
    // inside the tile.  (Adding a negative row count to the uniform base of a
    // full-tile load instead would wrap the 32-bit lane offset.)
    const int last = N - 1 - key0;  // last real row of this tile
    int lr = lane / T::kChunksPerRow;
    // opaque to the optimiser: keeps the per-load row sums below from being
    // hoisted out of the block loop, where they would hold 4 registers
    asm volatile("" : "+v"(lr));
#pragma unroll
    for (int i = i0; i < i0 + count; ++i) {
      const int n = wave_u * T::kLoadsPerWave + i;
      constexpr int R = CopyPlan<T, D>::kRowsPerLoad;
      const int rows = min((n & ~3) * R, last - (n & 3) * R - lr);
      copy16_to_lds(lds0 + i * 1024, tile, cp.lane_off[i & 3] + (uint32_t)(rows * sn) * 2u);
    }
  }
}

// A whole tile copy.
template <typename T, int BK, int D>
__device__ __forceinline__ void issue_tile_copy(__bf16* lds, const __bf16* src, int key0, int N,
                                                int sn, int wave_u, int lane,
                                                const CopyPlan<T, D>& cp) {
  issue_tile_slice<T, BK, D>(lds, src, key0, N, sn, wave_u, lane, cp, 0, T::kLoadsPerWave);
}

// Four consecutive outputs of a row: bf16 (round to nearest even) or fp32.
__device__ __forceinline__ void store_out4(__bf16* p, float a, float b, float c, float d) {
  *(bf16x4*)p = bf16x4{(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
}
__device__ __forceinline__ void store_out4(float* p, float a, float b, float c, float d) {
  *(f32x4*)p = f32x4{a, b, c, d};
}

// Output epilogue through LDS.  In the accumulator layout lane l holds 64
// values of query row l mod 32, so a direct store instruction writes 16
// bytes into each of 32 rows.  Here the wavefront's 32 rows, normalised and
// converted, go into a free LDS slice in row-major order (16-byte chunk c of
// row r at chunk c ^ (r mod C), C chunks per row, conflict-free both ways)
// and are read back so that each lane stores 16 contiguous bytes and a store
// instruction covers whole rows.  The slice is this wavefront's own and
// wavefront-local LDS accesses complete in order, so no barrier is needed.
// out0 is row 0 of the wavefront's rows (rows sn elements apart); rows at or
// past n_rows are not stored.
template <int D, typename OutT>
__device__ __forceinline__ void store_rows_staged(const f32x16 (&o)[D / 32], float inv,
                                                  char* slice, OutT* out0, int sn, int n_rows,
                                                  int lane) {
  constexpr int kChunk = 16 / (int)sizeof(OutT);  // elements per 16-byte chunk
  constexpr int C = D / kChunk;                   // chunks per row
  constexpr int kRowBytes = D * (int)sizeof(OutT);
  const int r = lane & 31;
  const int half = lane >> 5;
#pragma unroll
  for (int dg = 0; dg < D / 32; ++dg)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      // elements d = 32 dg + 8 r4 + 4 half + 0..3 of row r
      const float a = o[dg][4 * r4 + 0] * inv, b = o[dg][4 * r4 + 1] * inv;
      const float c = o[dg][4 * r4 + 2] * inv, d = o[dg][4 * r4 + 3] * inv;
      if constexpr (sizeof(OutT) == 2) {
        const int ch = 4 * dg + r4;
        *(SA_LDS bf16x4*)(slice + r * kRowBytes + ((ch ^ (r % C)) << 4) + 8 * half) =
            bf16x4{(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
      } else {
        const int ch = 8 * dg + 2 * r4 + half;
        *(SA_LDS f32x4*)(slice + r * kRowBytes + ((ch ^ (r % C)) << 4)) = f32x4{a, b, c, d};
      }
    }
  constexpr int kRowsPerStore = 64 / C;
  constexpr int kStores = 32 / kRowsPerStore;
  const int cl = lane % C;
  const int rl = lane / C;
  // All read-backs go out before the first store: the empty asm takes each
  // value where it is read, so the reads are not sunk into the guarded
  // stores below, where each would wait for its own LDS round trip.
  u32x4 v[kStores];
#pragma unroll
  for (int j = 0; j < kStores; ++j) {
    const int row = j * kRowsPerStore + rl;
    v[j] = *(const SA_LDS u32x4*)(slice + row * kRowBytes + ((cl ^ (row % C)) << 4));
  }
#pragma unroll
  for (int j = 0; j < kStores; ++j) asm volatile("" : "+v"(v[j]));
#pragma unroll
  for (int j = 0; j < kStores; ++j) {
    const int row = j * kRowsPerStore + rl;
    if (row < n_rows) *(u32x4*)(out0 + ((uint32_t)(row * sn) + (uint32_t)(cl * kChunk))) = v[j];
  }
}

// The staged epilogue needs 32 D sizeof(OutT) bytes per wavefront out of the
// item's K and V tiles (2 BK D bf16).
template <int BQ, int BK, int D, typename OutT>
constexpr bool kStagedStore = BQ * (int)sizeof(OutT) <= 4 * BK;

// DENSE = true is the maskless path: every key block 0 .. n_kb - 1 is enabled
// (counts, lists and order unused) and the items are laid out for the XCDs
// as the schedule lays them out, with the (b, h) groups in index order.
// Occupancy hint (waves per SIMD): two, except for 64 x 128 tiles with d = 128
// (two wavefronts own 128 keys of S and P each), which need more than 256
// registers per wave and run one.
template <int BQ, int BK, int D>
constexpr int kWavesPerSimd = (BQ == 64 && BK == 128 && D == 128) ? 1 : 2;

template <int BQ, int BK, int D, bool DENSE, typename OutT>
__global__ __launch_bounds__(BQ / 32 * 64, (kWavesPerSimd<BQ, BK, D>)) void bsattn_fwd_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ lists,
    const int32_t* __restrict__ order, OutT* __restrict__ O, float* __restrict__ LSE, int H,
    int N, int n_qb, int n_kb, float c_log2, int64_t sb, int64_t sh, int sn) {
  using T = Tile<BQ, BK, D>;
  constexpr int kL = T::kLoadsPerWave;
  __shared__ __attribute__((aligned(1024))) __bf16 Ks[BK * D];
  __shared__ __attribute__((aligned(1024))) __bf16 Vs[BK * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int half = lane >> 5;
  const int l32 = lane & 31;

  // Work item, row count and key blocks come from caller-visible buffers
  // (sa_bsattn_fwd_prepared): they are clamped into range, so malformed
  // input gives wrong values but never an access outside the tensors.
  const int n_items = (int)gridDim.x;
  int item;
  if (DENSE) {  // every group costs the same: the XCD layout of the schedule, groups in index order
    int uu;
    const int unit = xcd_slice(blockIdx.x, n_items / n_qb, n_qb, &uu);
    item = min(max(unit * n_qb + uu, 0), n_items - 1);
  } else {
    item = min(max(order[blockIdx.x], 0), n_items - 1);
  }
  const int bh = item / n_qb;
  const int u = item - bh * n_qb;
  const int h = bh % H;
  const int row = h * n_qb + u;
  const int cnt = DENSE ? n_kb : min(max(counts[row], 0), n_kb);
  const int32_t* list = DENSE ? nullptr : lists + (int64_t)row * n_kb;
  // key block of the t-th enabled block (ascending, as the CRM walk yields them)
  auto kblk = [&](int t) { return DENSE ? t : min(max(list[t], 0), n_kb - 1); };
  const int64_t base = (int64_t)(bh / H) * sb + (int64_t)h * sh;  // element (b, h, token 0, 0)
  const __bf16* Qb = Q + base;
  const __bf16* Kb = K + base;
  const __bf16* Vb = V + base;

  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  CopyPlan<T, D> cp;
  cp.init(wave_u, lane, sn);
  if (cnt > 0) issue_tile_copy<T, BK, D>(Ks, Kb, kblk(0) * BK, N, sn, wave_u, lane, cp);

  // Q^T fragments (B operand): lane holds Q[qrow][16 dc + 8 half .. +7].
  // (Staging them through the V tile as the ping-pong kernel does measured
  // 0.2-0.6 % slower here: two more barriers against 16 KB of Q per item.)
  const int qrow = u * BQ + wave * 32 + l32;
  bf16x8 qf[D / 16];
#pragma unroll
  for (int dc = 0; dc < D / 16; ++dc) {
    if (qrow < N)
      qf[dc] = *(const bf16x8*)(Qb + (int64_t)qrow * sn + dc * 16 + half * 8);
    else
      qf[dc] = bf16x8{};
  }

  // Q and the first tiles have landed: the loop below starts with no
  // outstanding vector loads that the compiler would otherwise wait for.
  __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0)

  f32x16 o[D / 32];
#pragma unroll
  for (int dg = 0; dg < D / 32; ++dg) o[dg] = f32x16{};
  float m_run = -INFINITY;  // running max of the log2-domain logits
  float l_run = 0.f;        // this lane's share of the running sum

  const int g = lane >> 4;
  const int j = lane & 15;

  // Copies are issued in slices between compute steps rather than in one
  // burst per tile: V[t] in BK / 32 slices between the key groups of S[t]
  // (its buffer is free once P V[t-1] is done), K[t+1] in two halves inside
  // the softmax of block t (its buffer is free once S[t] is done).  Bursts of
  // copies queue behind each other at issue and hold up the wavefront.
  constexpr int kVSlice = kL / (BK / 32);
  static_assert(kL % (BK / 32) == 0 && kL % 2 == 0, "copy slices");
  for (int t = 0; t < cnt; ++t) {
    const int key0 = kblk(t) * BK;
    const bool more = t + 1 < cnt;
    const int key1 = more ? kblk(t + 1) * BK : 0;

    barrier_copies_landed<0>();  // K[t] landed (no younger copy is in flight)

    // S^T = K Q^T, one 32-key group per accumulator.
    f32x16 s[BK / 32];
#pragma unroll
    for (int kg = 0; kg < BK / 32; ++kg) {
      s[kg] = f32x16{};
      const int kr = kg * 32 + key_of_row(l32);
#pragma unroll
      for (int dc = 0; dc < D / 16; ++dc) {
        const bf16x8 a = lds_read_b128(Ks + kr * D + (((2 * dc + half) ^ swz<D>(kr)) << 3));
        s[kg] = mfma32x32x16(a, qf[dc], s[kg]);
      }
      issue_tile_slice<T, BK, D>(Vs, Vb, key0, N, sn, wave_u, lane, cp, kg * kVSlice, kVSlice);
    }

    barrier_lds_reads_done();  // every wave is done with Ks

    if (key0 + BK > N) {  // ragged last block: keys >= N do not exist
#pragma unroll
      for (int kg = 0; kg < BK / 32; ++kg)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = key0 + kg * 32 + 16 * (i >> 3) + 8 * half + (i & 7);
          if (key >= N) s[kg][i] = -INFINITY;
        }
    }

    float mx = -INFINITY;
#pragma unroll
    for (int kg = 0; kg < BK / 32; ++kg)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kg][i]);
    mx = pair_max(mx) * c_log2;
    if (more) issue_tile_slice<T, BK, D>(Ks, Kb, key1, N, sn, wave_u, lane, cp, 0, kL / 2);
    // Rescale only when some row's maximum grew.  Keeping the exact running
    // maximum (rather than a stale one) makes each row's largest probability
    // exactly 1, which bf16 represents without error.
    const bool grow = mx > m_run;  // always true on the first block
    if (__any(grow)) {
      const float m_new = grow ? mx : m_run;
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dg = 0; dg < D / 32; ++dg) o[dg] *= alpha;
    }

    bf16x8 pf[BK / 16];
    float lsum = 0.f;
#pragma unroll
    for (int kg = 0; kg < BK / 32; ++kg) {
#pragma unroll
      for (int j8 = 0; j8 < 2; ++j8)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float p = fast_exp2(fmaf(s[kg][8 * j8 + e], c_log2, -m_run));
          lsum += p;
          pf[2 * kg + j8][e] = (__bf16)p;
        }
      if (kg == (BK / 32 - 1) / 2 && more)
        issue_tile_slice<T, BK, D>(Ks, Kb, key1, N, sn, wave_u, lane, cp, kL / 2, kL / 2);
    }
    l_run += lsum;

    if (more)
      barrier_copies_landed<kL>();  // V[t] landed; K[t+1] may still be in flight
    else
      barrier_copies_landed<0>();

    // O^T += V^T P^T.  Lane group g = lane / 16 covers d0 = 32 dg + 16 (g & 1)
    // and keys 16 c + 8 (g >> 1) + 0..7 (two transposing reads of 4 rows).
#pragma unroll
    for (int dg = 0; dg < D / 32; ++dg) {
      const int dd = dg * 32 + 16 * (g & 1) + (j & 3) * 4;
#pragma unroll
      for (int c = 0; c < BK / 16; ++c) {
        const int r0 = c * 16 + 8 * (g >> 1) + (j >> 2);
        const int r1 = r0 + 4;
        const bf16x4 lo = lds_read_tr16_b64(Vs + r0 * D + (((dd >> 3) ^ swz<D>(r0)) << 3) + (dd & 7));
        const bf16x4 hi = lds_read_tr16_b64(Vs + r1 * D + (((dd >> 3) ^ swz<D>(r1)) << 3) + (dd & 7));
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        o[dg] = mfma32x32x16(a, pf[c], o[dg]);
      }
    }

    barrier_lds_reads_done();  // every wave is done with Vs
  }

  // Epilogue addresses are rebuilt from the wave-uniform row base and a lane
  // id recomputed here (mbcnt), so that nothing formed before the loop has to
  // stay live across it.
  const float l_tot = pair_sum(l_run);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  const int lane_e = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int l32_e = lane_e & 31;
  const int half_e = lane_e >> 5;
  const int row0 = u * BQ + wave_u * 32;  // first query row of this wavefront
  if constexpr (kStagedStore<BQ, BK, D, OutT>) {
    // the loop's last barrier follows every wave's last LDS read, and no copy
    // is outstanding: wavefront w stages its rows in bytes [w S, (w + 1) S)
    // of [Ks | Vs], S = 32 D sizeof(OutT)
    if (half_e == 0 && row0 + l32_e < N)
      LSE[(int64_t)bh * N + row0 + l32_e] = l_tot > 0.f ? (m_run + fast_log2(l_tot)) * kLn2 : -INFINITY;
    constexpr int kSlice = 32 * D * (int)sizeof(OutT);
    constexpr int kTileBytes = BK * D * 2;
    const int off = wave_u * kSlice;
    char* slice = off < kTileBytes ? (char*)Ks + off : (char*)Vs + (off - kTileBytes);
    store_rows_staged<D, OutT>(o, inv, slice, O + base + (int64_t)row0 * sn, sn, N - row0, lane_e);
  } else if (row0 + l32_e < N) {
    if (half_e == 0)
      LSE[(int64_t)bh * N + row0 + l32_e] = l_tot > 0.f ? (m_run + fast_log2(l_tot)) * kLn2 : -INFINITY;
    OutT* orow = (O + base + (int64_t)row0 * sn) + (uint32_t)(l32_e * sn);
#pragma unroll
    for (int dg = 0; dg < D / 32; ++dg)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
        store_out4(orow + dg * 32 + 8 * r4 + 4 * half_e, o[dg][4 * r4 + 0] * inv,
                   o[dg][4 * r4 + 1] * inv, o[dg][4 * r4 + 2] * inv, o[dg][4 * r4 + 3] * inv);
  }
}


// Ping-pong workgroups: 8 wavefronts in two groups of 4; a group holds
// 128 / BQ items (one of 128 query rows or two of 64), each item with its own
// K and V tiles in LDS.  Used where those tiles fit the 160 KB of LDS.
template <int BQ, int BK, int D>
struct PingPong {
  static constexpr int kItems = 8 / (BQ / 32);  // items per workgroup
  static constexpr int kLdsBytes = kItems * 2 * BK * D * 2;
  static constexpr bool kFits = kLdsBytes <= 160 * 1024;
};

// Where ping-pong is used: items of 128 query rows (two per workgroup), and
// the maskless path wherever the tiles fit.  Masked items of 64 rows keep one
// item per workgroup: four masked items in lockstep over the largest of their
// counts measured 7-10 % slower than separate workgroups at densities of 0.1
// and 0.25, while the maskless 64 x 64 path gained 5 %.
template <int BQ, int BK, int D, bool DENSE>
constexpr bool kUsePingPong = PingPong<BQ, BK, D>::kFits && (BQ == 128 || DENSE);

// Ping-pong kernel.  An 8-wavefront workgroup runs 2 items of 128 query rows
// (or 4 of 64): wavefronts 0-3 and 4-7 form two groups, each item with its
// own K and V tiles in LDS (128 KB at 128 x 128, d = 128: one workgroup per
// CU).  Every SIMD holds one wavefront of each group.  A group's block loop
// alternates two phases separated by workgroup barriers:
//   MFMA phase t:    P V of block t - 1, then S of block t (the MFMAs of a
//                    step rotate over independent accumulators);
//   softmax phase t: copies of V[t] and K[t + 1] issued, then the softmax of
//                    block t; the phase ends once this group's copies landed.
// The second group starts one barrier later, so on every SIMD one group's
// softmax (vector ALU) runs beside the other group's MFMAs: gfx950 co-issues
// the two from different wavefronts, not from one wavefront whose softmax
// depends on its own S.  Both groups pass the same number of barriers: each
// runs max(counts) + 1 MFMA phases and max(counts) softmax phases over the
// workgroup's items, idle where its own item has no block, plus one offset
// barrier.  The items are neighbours in one XCD's sequence of the schedule,
// so they share most key blocks and have similar counts.
template <int BQ, int BK, int D, bool DENSE, typename OutT>
__global__ __launch_bounds__(512, 1) void bsattn_fwd_pp_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ lists,
    const int32_t* __restrict__ order, OutT* __restrict__ O, float* __restrict__ LSE, int H,
    int N, int n_qb, int n_kb, float c_log2, int64_t sb, int64_t sh, int sn, int n_items) {
  using T = Tile<BQ, BK, D>;
  constexpr int kItems = PingPong<BQ, BK, D>::kItems;  // items per workgroup
  __shared__ __attribute__((aligned(1024))) __bf16 Ks_all[kItems][BK * D];
  __shared__ __attribute__((aligned(1024))) __bf16 Vs_all[kItems][BK * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int grp = __builtin_amdgcn_readfirstlane(wave >> 2);
  const int slot = __builtin_amdgcn_readfirstlane(wave / T::kWaves);  // this wave's item
  const int gwave = wave % T::kWaves;  // wavefront inside its item
  const int half = lane >> 5;
  const int l32 = lane & 31;
  __bf16* Ks = Ks_all[slot];
  __bf16* Vs = Vs_all[slot];

  // Workgroup b on XCD b mod 8 takes items kItems (b / 8) .. + kItems - 1 of
  // that XCD's sequence: the launch positions x + 8 j of the one-item layout.
  auto pos_of = [&](int sl) -> int64_t {
    return (int64_t)(blockIdx.x % kXcds) + kXcds * (kItems * (int64_t)(blockIdx.x / kXcds) + sl);
  };
  // The look-ups are branch-free (positions clamped, validity applied after
  // the loads), so that the scalar loads of all items go out together:
  // every order entry, then every count and this item's first key block, in
  // two rounds of memory latency instead of one chain per item.
  int it_of[kItems];
#pragma unroll
  for (int sl = 0; sl < kItems; ++sl) {
    const int64_t pos = min(pos_of(sl), (int64_t)n_items - 1);
    if (DENSE) {
      int uu;
      const int unit = xcd_slice(pos, n_items / n_qb, n_qb, &uu);
      it_of[sl] = min(max(unit * n_qb + uu, 0), n_items - 1);
    } else {
      it_of[sl] = order[pos];
    }
  }
  __builtin_amdgcn_sched_barrier(0);  // all order loads issued before any is used
  int c_of[kItems];
  int item = 0;
#pragma unroll
  for (int sl = 0; sl < kItems; ++sl) {
    const int it = min(max(it_of[sl], 0), n_items - 1);
    c_of[sl] = DENSE ? n_kb : counts[(it / n_qb) % H * n_qb + it % n_qb];
    if (sl == slot) item = it;
  }
  const int bh = item / n_qb;
  const int u = item - bh * n_qb;
  const int h = bh % H;
  const int row = h * n_qb + u;
  const int32_t* list = DENSE ? nullptr : lists + (int64_t)row * n_kb;
  auto kblk = [&](int t) { return DENSE ? t : min(max(list[t], 0), n_kb - 1); };
  int first = kblk(0);  // in range for every row (n_kb >= 1): read before cnt is known
  asm volatile("" : "+s"(first));     // keeps that load here, not inside the cnt > 0 branch
  __builtin_amdgcn_sched_barrier(0);  // counts and the first key block issued together
  // every item's count: all groups run max(counts) iterations
  int cnt = 0, n_iter = 0;
#pragma unroll
  for (int sl = 0; sl < kItems; ++sl) {
    const int c = pos_of(sl) < n_items ? min(max(c_of[sl], 0), n_kb) : 0;
    n_iter = max(n_iter, c);
    if (sl == slot) cnt = c;
  }
  const bool has_item = pos_of(slot) < n_items;

  const int64_t base = (int64_t)(bh / H) * sb + (int64_t)h * sh;
  const __bf16* Qb = Q + base;
  const __bf16* Kb = K + base;
  const __bf16* Vb = V + base;

  const int gwave_u = __builtin_amdgcn_readfirstlane(gwave);
  CopyPlan<T, D> cp;
  cp.init(gwave_u, lane, sn);
  if (cnt > 0) issue_tile_copy<T, BK, D>(Ks, Kb, first * BK, N, sn, gwave_u, lane, cp);

  // Q^T fragments (B operand): lane holds Q[row gwave 32 + l32 of the item]
  // [16 dc + 8 half .. +7].  With square tiles the item's Q rows come in as
  // one more tile copy, into its V tile (free until the first softmax phase
  // issues V[0]), and are read from there after the barriers below: rows of
  // 256 contiguous bytes per four lanes instead of 32 rows per load
  // instruction.  In a ragged last query block, rows past N hold row N - 1
  // (their outputs are not stored); a workgroup slot without an item copies
  // the clamped item's rows and stores nothing.
  constexpr bool kStageQ = BQ == BK;
  const int qrow = u * BQ + gwave * 32 + l32;
  bf16x8 qf[D / 16];
  if constexpr (kStageQ) {
    issue_tile_copy<T, BK, D>(Vs, Qb, u * BQ, N, sn, gwave_u, lane, cp);
  } else {
#pragma unroll
    for (int dc = 0; dc < D / 16; ++dc) {
      if (has_item && qrow < N)
        qf[dc] = *(const bf16x8*)(Qb + (int64_t)qrow * sn + dc * 16 + half * 8);
      else
        qf[dc] = bf16x8{};
    }
  }
  __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): Q and K[0] landed

  f32x16 o[D / 32];
#pragma unroll
  for (int dg = 0; dg < D / 32; ++dg) o[dg] = f32x16{};
  float m_run = -INFINITY;
  float l_run = 0.f;
  const int g = lane >> 4;
  const int j = lane & 15;
  bf16x8 pf[BK / 16];
#pragma unroll
  for (int c = 0; c < BK / 16; ++c) pf[c] = bf16x8{};

  if (grp == 1) barrier_lds_reads_done();  // the second group runs one phase behind
  barrier_lds_reads_done();                // both groups' K[0] (and Q) tiles are in LDS
  if constexpr (kStageQ) {
    // every wavefront's Q copy landed before the first barrier; the group's
    // reads complete before the barrier that ends its first MFMA phase,
    // after which its first softmax phase reuses the tile for V[0]
    const int qr = gwave * 32 + l32;
#pragma unroll
    for (int dc = 0; dc < D / 16; ++dc)
      qf[dc] = lds_read_b128(Vs + qr * D + (((2 * dc + half) ^ swz<D>(qr)) << 3));
  }

  for (int t = 0; t <= n_iter; ++t) {
    // ---- MFMA phase: P V of block t - 1, then S of block t
    if (t >= 1 && t - 1 < cnt) {
#pragma unroll
      for (int c = 0; c < BK / 16; ++c) {
#pragma unroll
        for (int dg = 0; dg < D / 32; ++dg) {
          const int dd = dg * 32 + 16 * (g & 1) + (j & 3) * 4;
          const int r0 = c * 16 + 8 * (g >> 1) + (j >> 2);
          const int r1 = r0 + 4;
          const bf16x4 lo = lds_read_tr16_b64(Vs + r0 * D + (((dd >> 3) ^ swz<D>(r0)) << 3) + (dd & 7));
          const bf16x4 hi = lds_read_tr16_b64(Vs + r1 * D + (((dd >> 3) ^ swz<D>(r1)) << 3) + (dd & 7));
          const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          o[dg] = mfma32x32x16(a, pf[c], o[dg]);
        }
      }
    }
    f32x16 s[BK / 32];
#pragma unroll
    for (int kg = 0; kg < BK / 32; ++kg) s[kg] = f32x16{};
    const bool do_s = t < cnt;
    if (do_s) {
#pragma unroll
      for (int dc = 0; dc < D / 16; ++dc) {
#pragma unroll
        for (int kg = 0; kg < BK / 32; ++kg) {
          const int kr = kg * 32 + key_of_row(l32);
          const bf16x8 a = lds_read_b128(Ks + kr * D + (((2 * dc + half) ^ swz<D>(kr)) << 3));
          s[kg] = mfma32x32x16(a, qf[dc], s[kg]);
        }
      }
    }
    barrier_lds_reads_done();  // this group's Ks and Vs are free
    if (t == n_iter) break;

    // ---- softmax phase of block t; copies of V[t] and K[t + 1]
    if (do_s) {
      const int key0 = kblk(t) * BK;
      const bool more = t + 1 < cnt;
      issue_tile_copy<T, BK, D>(Vs, Vb, key0, N, sn, gwave_u, lane, cp);
      if (key0 + BK > N) {
#pragma unroll
        for (int kg = 0; kg < BK / 32; ++kg)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = key0 + kg * 32 + 16 * (i >> 3) + 8 * half + (i & 7);
            if (key >= N) s[kg][i] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kg = 0; kg < BK / 32; ++kg)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kg][i]);
      mx = pair_max(mx) * c_log2;
      if (more) issue_tile_copy<T, BK, D>(Ks, Kb, kblk(t + 1) * BK, N, sn, gwave_u, lane, cp);
      const bool grow = mx > m_run;
      if (__any(grow)) {
        const float m_new = grow ? mx : m_run;
        const float alpha = fast_exp2(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int dg = 0; dg < D / 32; ++dg) o[dg] *= alpha;
      }
      float lsum = 0.f;
#pragma unroll
      for (int kg = 0; kg < BK / 32; ++kg)
#pragma unroll
        for (int j8 = 0; j8 < 2; ++j8)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float p = fast_exp2(fmaf(s[kg][8 * j8 + e], c_log2, -m_run));
            lsum += p;
            pf[2 * kg + j8][e] = (__bf16)p;
          }
      l_run += lsum;
    }
    barrier_copies_landed<0>();  // this group's V[t] and K[t + 1] landed
  }
  if (grp == 0) barrier_lds_reads_done();  // matches the second group's extra barrier

  const float l_tot = pair_sum(l_run);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  const int lane_e = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int l32_e = lane_e & 31;
  const int half_e = lane_e >> 5;
  const int row0 = u * BQ + gwave_u * 32;
  if constexpr (kStagedStore<BQ, BK, D, OutT>) {
    // every wavefront's LDS reads and copies are over (the last barrier
    // above), so this item's K and V tiles are free: wavefront w of the item
    // stages its rows in bytes [w S, (w + 1) S) of [Ks | Vs], S = 32 D sizeof(OutT)
    if (has_item) {
      if (half_e == 0 && row0 + l32_e < N)
        LSE[(int64_t)bh * N + row0 + l32_e] = l_tot > 0.f ? (m_run + fast_log2(l_tot)) * kLn2 : -INFINITY;
      constexpr int kSlice = 32 * D * (int)sizeof(OutT);
      constexpr int kTileBytes = BK * D * 2;
      const int off = gwave_u * kSlice;
      char* slice = off < kTileBytes ? (char*)Ks + off : (char*)Vs + (off - kTileBytes);
      store_rows_staged<D, OutT>(o, inv, slice, O + base + (int64_t)row0 * sn, sn, N - row0, lane_e);
    }
  } else if (has_item && row0 + l32_e < N) {
    if (half_e == 0)
      LSE[(int64_t)bh * N + row0 + l32_e] = l_tot > 0.f ? (m_run + fast_log2(l_tot)) * kLn2 : -INFINITY;
    OutT* orow = (O + base + (int64_t)row0 * sn) + (uint32_t)(l32_e * sn);
#pragma unroll
    for (int dg = 0; dg < D / 32; ++dg)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
        store_out4(orow + dg * 32 + 8 * r4 + 4 * half_e, o[dg][4 * r4 + 0] * inv,
                   o[dg][4 * r4 + 1] * inv, o[dg][4 * r4 + 2] * inv, o[dg][4 * r4 + 3] * inv);
  }
}

template <int BQ, int BK, int D, bool DENSE, typename OutT>
hipError_t launch_tile(const AttnArgs& a, hipStream_t stream) {
  const int64_t n_items = (int64_t)a.B * a.H * a.n_qb;
  if constexpr (kUsePingPong<BQ, BK, D, DENSE>) {
    // kItems consecutive items of one XCD's sequence per workgroup
    constexpr int kItems = PingPong<BQ, BK, D>::kItems;
    const int64_t seq0 = (n_items + kXcds - 1) / kXcds;  // longest XCD sequence
    const int64_t n_wg = kXcds * ((seq0 + kItems - 1) / kItems);
    hipLaunchKernelGGL((bsattn_fwd_pp_kernel<BQ, BK, D, DENSE, OutT>), dim3((unsigned)n_wg),
                       dim3(512), 0, stream, (const __bf16*)a.q,
                       (const __bf16*)a.k, (const __bf16*)a.v, a.counts, a.lists, a.order,
                       (OutT*)a.out, a.lse, a.H, a.N, a.n_qb, a.n_kb, a.scale * kLog2e, a.sb,
                       a.sh, a.sn, (int)n_items);
  } else {
    hipLaunchKernelGGL((bsattn_fwd_kernel<BQ, BK, D, DENSE, OutT>), dim3((unsigned)n_items),
                       dim3(Tile<BQ, BK, D>::kThreads), 0, stream, (const __bf16*)a.q,
                       (const __bf16*)a.k, (const __bf16*)a.v, a.counts, a.lists, a.order,
                       (OutT*)a.out, a.lse, a.H, a.N, a.n_qb, a.n_kb, a.scale * kLog2e, a.sb,
                       a.sh, a.sn);
  }
  return hipGetLastError();
}

template <int BQ, int BK, bool DENSE, typename OutT>
hipError_t launch_d(const AttnArgs& a, hipStream_t stream) {
  if (a.d == 128) return launch_tile<BQ, BK, 128, DENSE, OutT>(a, stream);
  if (a.d == 64) return launch_tile<BQ, BK, 64, DENSE, OutT>(a, stream);
  return hipErrorInvalidValue;
}

template <bool DENSE, typename OutT>
hipError_t launch_any(const AttnArgs& a, hipStream_t stream) {
  if (a.blk_q == 128 && a.blk_k == 128) return launch_d<128, 128, DENSE, OutT>(a, stream);
  if (a.blk_q == 64 && a.blk_k == 64) return launch_d<64, 64, DENSE, OutT>(a, stream);
  if (a.blk_q == 128 && a.blk_k == 64) return launch_d<128, 64, DENSE, OutT>(a, stream);
  if (a.blk_q == 64 && a.blk_k == 128) return launch_d<64, 128, DENSE, OutT>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream) {
  return a.out_f32 ? launch_any<false, float>(a, stream) : launch_any<false, __bf16>(a, stream);
}

hipError_t launch_attention_dense(const AttnArgs& a, hipStream_t stream) {
  if (a.out_f32) return hipErrorInvalidValue;  // the maskless path writes bf16 only
  return launch_any<true, __bf16>(a, stream);
}

}  // namespace sa
