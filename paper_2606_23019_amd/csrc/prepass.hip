// Mask pre-pass and work schedule.
//
// Pre-pass: the paper walks each Compressed Row Mask inside the attention
// kernel with a bit-scan iterator (Sec. 4.3.2 and the appendix "CRM Forward
// Iterator": skip empty segments, report base + count-trailing-zeros, clear
// the lowest bit).  Masks are static, so here the walk runs once per row in
// a separate kernel: one wavefront per row walks the row's words in order;
// lane l owns bit l of a word, and the popcount of the word's lower bits is
// its place after the blocks already written, so the enabled key blocks of a
// word leave in ascending order in one store.
// The attention kernel then reads a dense list instead of decoding bits.
//
// Schedule: heads have very different densities, so (b, h) groups are
// started heaviest first, and the order is laid out for the 8 XCDs, each
// with its own L2.  Workgroups are dealt to the XCDs round-robin (launch
// position p runs on XCD p mod 8, in increasing p), so the order is written
// as 8 interleaved sequences: sequence x holds one chunk of every group, the
// groups heaviest first, where a group's n_qb query blocks are cut into 8
// runs of n_qb / 8 consecutive blocks (the n_qb mod 8 leftover items rotate
// over the XCDs from group to group, which makes every sequence exactly as
// long as the positions p = x mod 8) and sequence x takes the run at place
// (x + k) mod 8 for the group of rank k.  Each XCD thus works on a few groups
// at a time, on neighbouring query blocks that share most key blocks in
// structured masks, so their K/V tiles are reused from its L2, and every XCD
// gets an equal share of every group and, over the groups, of every part of
// the sequence (the first and last query blocks of a video have fewer key
// blocks), so the load stays balanced.  One workgroup computes each group's
// total enabled blocks, ranks the groups in LDS (by counting smaller keys, or
// with a bitonic network beyond 512 groups) and writes the order, each chunk
// in ascending u; a second kernel then sorts every window of up to 128 places
// of a chunk by enabled-block count, so that the items the attention kernel
// runs side by side have similar counts.

#include "device_common.h"
#include "launch.h"

namespace sa {

namespace {

constexpr int kPrepassWaves = 4;

__global__ __launch_bounds__(64 * kPrepassWaves) void prepass_kernel(
    const uint64_t* __restrict__ mask, int rows, int n_kb, int W, int32_t* __restrict__ counts,
    int32_t* __restrict__ lists) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kPrepassWaves + (threadIdx.x >> 6);
  if (row >= rows) return;  // uniform per wavefront
  const uint64_t* mrow = mask + (int64_t)row * W;
  int32_t* lrow = lists + (int64_t)row * n_kb;
  // Word by word: lane l owns bit l of the word (key block 64 w + l); its
  // place in the list is the number of set bits below it (a popcount of the
  // masked word), so each word's entries leave in one store, in ascending
  // order, whatever the number of set bits.
  const uint64_t below = (1ull << lane) - 1ull;  // bits below this lane's
  int done = 0;  // blocks already written for this row
  for (int w0 = 0; w0 < W; w0 += 64) {
    // 64 words at a time, lane i loading word w0 + i (one round of latency),
    // then handed to the whole wavefront one by one with readlane
    uint64_t mine = 0;
    if (w0 + lane < W) {
      mine = mrow[w0 + lane];
      const int real = n_kb - (w0 + lane) * 64;  // bits of this word that name a real key block
      if (real < 64) mine &= (1ull << real) - 1ull;  // real >= 1 for w < W
    }
    const int nw = min(64, W - w0);
    for (int i = 0; i < nw; ++i) {
      const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)mine, i);
      const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(mine >> 32), i);
      const uint64_t word = ((uint64_t)hi << 32) | lo;
      if ((word >> lane) & 1ull) lrow[done + __popcll(word & below)] = (w0 + i) * 64 + lane;
      done += __popcll(word);
    }
  }
  if (lane == 0) counts[row] = done;
}

constexpr int kSchedThreads = 1024;
constexpr int kRankSortMax = 512;  // groups ranked by counting; more use the bitonic network
constexpr int kSchedWindow = 128;  // two places per lane of one wavefront

__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(const int32_t* __restrict__ counts,
                                                                  int B, int H, int n_qb,
                                                                  int32_t* __restrict__ order) {
  __shared__ uint64_t keys[kScheduleMaxUnits];
  __shared__ uint32_t head_cost[kScheduleMaxUnits];
  __shared__ uint32_t rank_unit[kScheduleMaxUnits];  // group index by rank
  const int tid = threadIdx.x;
  const int n_units = B * H;
  const int64_t n_items = (int64_t)n_units * n_qb;
  if (n_units > kScheduleMaxUnits) {
    for (int64_t i = tid; i < n_items; i += kSchedThreads) order[i] = (int32_t)i;
    return;
  }
  // Per-head cost: `parts` threads per head each sum a strided share of the
  // head's rows, then add it into LDS (few loads per thread instead of n_qb
  // dependent-latency loads by one thread).  The share's loads go out eight
  // at a time before any is added, so their latencies overlap instead of
  // adding up.
  for (int h = tid; h < H; h += kSchedThreads) head_cost[h] = 0;
  __syncthreads();
  const int parts = H < kSchedThreads ? kSchedThreads / H : 1;
  for (int w = tid; w < H * parts; w += kSchedThreads) {
    const int h = w / parts;
    const int32_t* hrow = counts + (int64_t)h * n_qb;
    uint32_t c = 0;
    for (int u0 = w - h * parts; u0 < n_qb; u0 += 8 * parts) {
      int32_t v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int u = u0 + i * parts;
        v[i] = u < n_qb ? hrow[u] : 0;
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) c += (uint32_t)v[i];
    }
    atomicAdd(&head_cost[h], c);
  }
  __syncthreads();
  // Ascending order of the keys (~cost, index): decreasing cost, ties by
  // increasing index; the keys are distinct.  Up to kRankSortMax groups, each
  // thread ranks its group by counting the smaller keys (one pass, one
  // barrier); beyond that a bitonic network over the keys in LDS.
  if (n_units <= kRankSortMax) {
    for (int i = tid; i < n_units; i += kSchedThreads)
      keys[i] = ((uint64_t)(0xFFFFFFFFu - head_cost[i % H]) << 32) | (uint32_t)i;
    __syncthreads();
    for (int i = tid; i < n_units; i += kSchedThreads) {
      const uint64_t mine = keys[i];
      int rank = 0;
      for (int o = 0; o < n_units; ++o) rank += keys[o] < mine ? 1 : 0;
      rank_unit[rank] = (uint32_t)i;
    }
  } else {
    int P = 1;
    while (P < n_units) P <<= 1;
    for (int i = tid; i < P; i += kSchedThreads) {
      keys[i] = (i < n_units)
                    ? ((uint64_t)(0xFFFFFFFFu - head_cost[i % H]) << 32) | (uint32_t)i
                    : ~0ull;
    }
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int i = tid; i < P; i += kSchedThreads) {
          const int p = i ^ j;
          if (p > i) {
            const uint64_t a = keys[i], b = keys[p];
            const bool up = (i & k) == 0;
            if ((a > b) == up) {
              keys[i] = b;
              keys[p] = a;
            }
          }
        }
        __syncthreads();
      }
    }
    for (int i = tid; i < n_units; i += kSchedThreads) rank_unit[i] = (uint32_t)(keys[i] & 0xFFFFFFFFu);
  }
  __syncthreads();
  // Ascending u inside each chunk here; window_sort_kernel then reorders
  // each window of a chunk by count.  One wavefront per group rank k: the
  // group's 8 chunks interleave into one run of launch positions, from
  // 8 prefix(k, 7) (prefix is non-increasing in x) to 8 prefix(k + 1, 0) + 7,
  // so the lanes write consecutive positions, each keeping the positions
  // whose place j = pos / 8 lies in chunk (pos mod 8, k).  The few positions
  // at either end that belong to a neighbouring rank are written by that
  // rank's wavefront.
  const int q = n_qb / kXcds;
  const int r = n_qb - q * kXcds;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  for (int k = wave; k < n_units; k += kSchedThreads / 64) {
    const int64_t p_lo = kXcds * xcd_prefix(k, kXcds - 1, q, r);
    const int64_t p_hi = min(kXcds * xcd_prefix(k + 1, 0, q, r) + kXcds, n_items);
    const int base = (int)rank_unit[k] * n_qb;
    for (int64_t pos = p_lo + lane; pos < p_hi; pos += 64) {
      const int x = (int)(pos % kXcds);
      const int64_t j = pos / kXcds;
      const int64_t j0 = xcd_prefix(k, x, q, r);
      if (j >= j0 && j < xcd_prefix(k + 1, x, q, r))
        order[pos] = base + xcd_chunk_u0(k, x, q, r) + (int)(j - j0);
    }
  }
}

// Chunk (x, k) of sequence x holds the group of rank k's query blocks
// u0 .. u0 + len - 1 at sequence places prefix(k) .. + len - 1.  The attention
// kernel runs neighbouring places of a sequence side by side (two per
// ping-pong workgroup, in lockstep over the larger count), so each chunk is
// cut into windows of up to 128 places, and inside a window the query blocks
// are placed by enabled-block count: decreasing in the even windows of the
// chunk, increasing in its odd ones, so that a pair which straddles two
// windows of a chunk meets counts from the same end, and decreasing in the
// sequence's last window whatever its parity, so that every XCD ends its
// work on its lightest items, which shortens the tail of the launch.  Every
// chunk thus starts on its heaviest items: while the light end of one group
// finishes, the next group's long items start, and fewer groups' K/V tiles
// compete for an XCD's L2 at a time than when every other chunk started light
// (L2 fetches over the fabric per launch measured 12.8 against 23.9 GB at
// 14B-480p, 5.3 against 8.2 GB at density 0.1 with structured masks; the
// pair balance is the same).  A window still holds the same consecutive
// query blocks.  The places of window (x, k, wi) depend on k only, not on which
// group has rank k, so this runs after schedule_kernel on the order it wrote,
// one wavefront per window across the whole chip: lane l reads the items at
// the window's places t = l and l + 64, keys each as (count << 7) | (127 - t)
// (distinct keys, larger for larger counts and, among equal counts, for
// smaller t), counts the larger keys of the window from a key row in LDS, and
// writes each item back at its rank's place.  Each window's places are read and written by its
// own wavefront only, so the permutation happens in place.
constexpr int kWindowSortWaves = 4;

__global__ __launch_bounds__(64 * kWindowSortWaves) void window_sort_kernel(
    const int32_t* __restrict__ counts, int H, int n_qb, int n_units, int32_t* __restrict__ order) {
  __shared__ __attribute__((aligned(16))) int32_t key_rows[kWindowSortWaves][kSchedWindow];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q = n_qb / kXcds;
  const int r = n_qb - q * kXcds;
  const int win_per_chunk = (q + 1 + kSchedWindow - 1) / kSchedWindow;
  const int64_t w = (int64_t)blockIdx.x * kWindowSortWaves + wave;
  if (w >= (int64_t)kXcds * n_units * win_per_chunk) return;  // uniform per wavefront
  const int x = (int)(w % kXcds);
  const int rest = (int)(w / kXcds);
  const int k = rest / win_per_chunk;
  const int wi = rest - k * win_per_chunk;
  const int64_t j0 = xcd_prefix(k, x, q, r);
  const int len = (int)(xcd_prefix(k + 1, x, q, r) - j0);
  const int L = min(kSchedWindow, len - wi * kSchedWindow);
  if (L <= 0) return;  // uniform per wavefront
  const int64_t first = j0 + (int64_t)wi * kSchedWindow;  // the window's first place
  // lane l holds places l and l + 64 of the window; places past L hold -1,
  // below every key
  int item[2] = {0, 0}, key[2] = {-1, -1};
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int t = lane + 64 * h;
    if (t < L) {
      item[h] = order[x + kXcds * (first + t)];
      const int64_t row = (int64_t)(item[h] / n_qb % H) * n_qb + item[h] % n_qb;
      key[h] = (min(max(counts[row], 0), (1 << 23) - 1) << 7) | (127 - t);
    }
  }
  int32_t* key_row = key_rows[wave];
  key_row[lane] = key[0];
  key_row[lane + 64] = key[1];
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the wavefront's keys are in LDS
  int rank[2] = {0, 0};  // window members placed before each of the lane's two
#pragma unroll 4
  for (int i = 0; i < L; i += 4) {  // keys past L (up to a multiple of 4) are -1
    const i32x4 kv = *(const SA_LDS i32x4*)(key_row + i);
#pragma unroll
    for (int h = 0; h < 2; ++h)
      rank[h] += (kv[0] > key[h] ? 1 : 0) + (kv[1] > key[h] ? 1 : 0) +
                 (kv[2] > key[h] ? 1 : 0) + (kv[3] > key[h] ? 1 : 0);
  }
  // direction: by the window's parity inside its chunk; the last window of
  // the last chunk (the sequence's last) is decreasing
  const bool last = k == n_units - 1 && (wi + 1) * kSchedWindow >= len;
  const bool increasing = (wi & 1) && !last;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int t = increasing ? L - 1 - rank[h] : rank[h];
    if (lane + 64 * h < L) order[x + kXcds * (first + t)] = item[h];
  }
}

}  // namespace

hipError_t launch_prepass(const uint64_t* mask_bits, int H, int n_qb, int n_kb, int32_t* counts,
                          int32_t* lists, hipStream_t stream) {
  const int rows = H * n_qb;
  const int W = (n_kb + 63) / 64;
  const int grid = (rows + kPrepassWaves - 1) / kPrepassWaves;
  hipLaunchKernelGGL(prepass_kernel, dim3(grid), dim3(64 * kPrepassWaves), 0, stream, mask_bits,
                     rows, n_kb, W, counts, lists);
  return hipGetLastError();
}

hipError_t launch_schedule(const int32_t* counts, int B, int H, int n_qb, int32_t* order,
                           hipStream_t stream) {
  hipLaunchKernelGGL(schedule_kernel, dim3(1), dim3(kSchedThreads), 0, stream, counts, B, H, n_qb,
                     order);
  const int n_units = B * H;
  if (n_units <= kScheduleMaxUnits) {  // otherwise the order is the identity
    const int q = n_qb / kXcds;
    const int64_t n_windows = (int64_t)kXcds * n_units * ((q + 1 + kSchedWindow - 1) / kSchedWindow);
    const int64_t grid = (n_windows + kWindowSortWaves - 1) / kWindowSortWaves;
    hipLaunchKernelGGL(window_sort_kernel, dim3((unsigned)grid), dim3(64 * kWindowSortWaves), 0,
                       stream, counts, H, n_qb, n_units, order);
  }
  return hipGetLastError();
}

}  // namespace sa
