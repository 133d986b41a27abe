/*
 * sa_bsattn.h -- block-sparse scaled-dot-product attention forward for
 * MI355X (gfx950), C ABI.
 *
 * The operation is the forward pass of the paper's CRM kernel (Sec. 4.3.2,
 * "CRM Kernel: Bit-wise Block-Sparse Attention Execution"): attention over
 * flattened video tokens in which every head follows a static bit-packed
 * block mask, and only the key blocks whose bit is set are computed.  For
 * batch b, head h and query token i (query block u = i / blk_q):
 *
 *   K_i   = { j < N : bit(h, u, j / blk_k) = 1 }
 *   s_ij  = scale * <q_i, k_j>
 *   lse_i = log sum_{j in K_i} exp(s_ij)             (natural log)
 *   out_i = sum_{j in K_i} exp(s_ij - lse_i) v_j
 *
 * A query block with no set bit gets out = 0 and lse = -inf.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are DEVICE pointers on the current HIP device.  The
 *   caller owns every buffer; the library never frees or retains them.
 * - q, k, v, out: bfloat16 (stored as uint16), contiguous [B][H][N][d],
 *   16-byte aligned.  lse: float32, contiguous [B][H][N], 4-byte aligned.
 *   out and lse must not overlap any input.
 * - mask_bits: the Compressed Row Mask of Sec. 4.3.2 stored as little-endian
 *   uint64 words, contiguous [H][n_qb][W] with n_qb = ceil(N / blk_q),
 *   n_kb = ceil(N / blk_k), W = ceil(n_kb / 64).  Key block v of row (h, u)
 *   is bit (v mod 64) of word v / 64 (LSB-first, the enumeration order of the
 *   paper's CRM forward iterator).  Bits at positions >= n_kb are ignored.
 *   One mask per head, shared by all batch entries.  8-byte aligned.
 * - stream: a hipStream_t passed as void* (NULL = the default stream).  All
 *   work is enqueued on it; no call synchronises unless its comment says so.
 *   Execution errors surface at the caller's next synchronisation.
 * - Supported shapes: d in {64, 128}; blk_q and blk_k each in {64, 128}
 *   (the paper uses 128 x 128 blocks; a query block of 128 rows may also walk
 *   64-key blocks and vice versa); B, H, N >= 1; n_kb <= 65535;
 *   B * H * n_qb < 2^31.  scale must be finite and > 0.
 * - Every argument is validated before anything is enqueued: a non-zero
 *   return means nothing was launched and no output was written.
 */
#ifndef SA_BSATTN_H
#define SA_BSATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SA_API __attribute__((visibility("default")))

/* Status codes. */
#define SA_OK 0
#define SA_ERR_INVALID_ARG 1 /* null/misaligned pointer, bad size, bad scale, aliasing */
#define SA_ERR_UNSUPPORTED 2 /* shape outside the supported set above */
#define SA_ERR_HIP 3         /* a HIP allocation or launch failed */
#define SA_ERR_TOO_LARGE 4   /* workspace beyond SA_NOALLOC_SCRATCH_BYTES (sa_bsattn_fwd_noalloc) */

/* Human-readable text for a status code (static storage, never NULL). */
SA_API const char* sa_status_string(int status);

/* Library version, major * 10000 + minor * 100 + patch. */
SA_API int sa_version(void);

/*
 * One-shot forward pass (Sec. 4.3.2): runs the mask pre-pass, the schedule
 * and the attention kernel on `stream`.  Internal workspace (per-row counts
 * and key-block lists, the work order) is taken with stream-ordered
 * hipMallocAsync and released with hipFreeAsync on the same stream.
 * Returns SA_OK, SA_ERR_INVALID_ARG, SA_ERR_UNSUPPORTED or SA_ERR_HIP.
 */
SA_API int sa_bsattn_fwd(const void* q, const void* k, const void* v,
                         const uint64_t* mask_bits, void* out, float* lse,
                         int B, int H, int N, int d, int blk_q, int blk_k,
                         float scale, void* stream);

/*
 * One-shot forward pass as sa_bsattn_fwd that allocates nothing, for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  The workspace of the
 * pre-pass and the schedule (counts, lists and order: 4 H n_qb +
 * 4 H n_qb n_kb + 4 B H n_qb bytes, each part rounded up to 256) lives in a
 * fixed array of SA_NOALLOC_SCRATCH_BYTES in the library's device memory,
 * one per GPU, held from the library's load onto that GPU until the process
 * ends.  A larger workspace returns SA_ERR_TOO_LARGE before anything is
 * enqueued (14B-like 720p, H 40 and 591 x 591 blocks, needs 56 MB).
 * The first call on a device looks the array's address up there
 * (hipGetSymbolAddress).  Every call on one GPU shares that GPU's array:
 * calls whose work overlaps in time on one GPU (other streams, other host
 * threads) race on it and give wrong results, so order them (one stream, or
 * events).  Nothing in the array needs to start at zero: each call writes
 * every entry it reads.  Arguments, layout, results and the other errors as
 * sa_bsattn_fwd; the result is bit for bit that of sa_bsattn_fwd.
 */
#define SA_NOALLOC_SCRATCH_BYTES (64u << 20)

SA_API int sa_bsattn_fwd_noalloc(const void* q, const void* k, const void* v,
                                 const uint64_t* mask_bits, void* out, float* lse,
                                 int B, int H, int N, int d, int blk_q, int blk_k,
                                 float scale, void* stream);

/*
 * One-shot forward pass as sa_bsattn_fwd, with out in float32 (contiguous
 * [B][H][N][d], 16-byte aligned; q, k, v stay bf16 and lse float32): the
 * kernel's fp32 accumulator divided by the row sum, with no bf16 rounding of
 * the result.  For callers that need the 2e-2 absolute bound on out even
 * where |out| >= 8, where half a bf16 ulp alone is 0.03.  The arithmetic up
 * to that last step is the same as sa_bsattn_fwd's, so the bf16 out of
 * sa_bsattn_fwd is the round-to-nearest-even of this out, and lse is bit for
 * bit the same.  Costs 2 more bytes of HBM writes per output element.
 */
SA_API int sa_bsattn_fwd_f32out(const void* q, const void* k, const void* v,
                                const uint64_t* mask_bits, float* out, float* lse, int B, int H,
                                int N, int d, int blk_q, int blk_k, float scale, void* stream);

/* Tensor layouts accepted by sa_bsattn_fwd_layout. */
#define SA_LAYOUT_BHND 0 /* [B][H][N][d]: heads outermost (the other entry points) */
#define SA_LAYOUT_BNHD 1 /* [B][N][H][d]: tokens outermost, as a DiT's projections emit */

/*
 * One-shot forward pass as sa_bsattn_fwd, with q, k, v and out in the layout
 * named by `layout` (all four alike; lse stays float32 [B][H][N]).  In
 * SA_LAYOUT_BNHD the rows of one head are H * d elements apart, so attention
 * runs straight on the projection output without a transpose.  The result is
 * bit-for-bit that of sa_bsattn_fwd on the transposed tensors.  Returns
 * SA_ERR_INVALID_ARG for an unknown layout and SA_ERR_UNSUPPORTED when
 * H * d * max(blk_q, blk_k) * 2 >= 2^31.
 */
SA_API int sa_bsattn_fwd_layout(const void* q, const void* k, const void* v,
                                const uint64_t* mask_bits, void* out, float* lse, int B, int H,
                                int N, int d, int blk_q, int blk_k, float scale, int layout,
                                void* stream);

/*
 * Mask pre-pass alone (the CRM walk of the paper's appendix "CRM Forward
 * Iterator", done once per row instead of inside the attention loop):
 * for each row r = h * n_qb + u writes counts[r] = number of set bits
 * (positions < n_kb) and lists[r * n_kb + 0 .. counts[r]-1] = the enabled key
 * blocks in ascending order.  Entries past counts[r] are left untouched.
 * counts: device int32 [H * n_qb]; lists: device int32 [H * n_qb * n_kb]
 * (int32 so that the attention kernel reads them with scalar loads).
 * Requires 1 <= n_kb <= 65535.
 */
SA_API int sa_mask_prepass(const uint64_t* mask_bits, int H, int n_qb, int n_kb,
                           int32_t* counts, int32_t* lists, void* stream);

/*
 * Mask instantiation from a threshold map (Sec. 4.1.2, Eq. 2 and the mask
 * M_p = 1[T <= p] that follows it): WEST's map T holds, per head and block,
 * the smallest density threshold at which the block is active; FAST chooses
 * a threshold per layer, timestep and head (Sec. 4.2.2).  For every
 * threshold set i and head h this writes the CRM row bits
 *   bit (v mod 64) of mask_bits[i][h][u][v / 64] = 1[T[h][u][v] <= p[i][h]]
 * with bits past n_kb zero; a NaN in T or p leaves the block off.  The
 * output of set i is exactly the mask_bits argument of sa_bsattn_fwd.
 * T: device float32 [H][n_qb][n_kb]; p: device float32 [n_p][H];
 * mask_bits: device uint64 [n_p][H][n_qb][W], W = ceil(n_kb / 64), every word
 * written.  mask_bits must not overlap T or p.  Requires n_p, H, n_qb >= 1,
 * n_p <= 1048560 and 1 <= n_kb <= 65535.
 */
SA_API int sa_mask_instantiate(const float* T, const float* p, int n_p, int H, int n_qb, int n_kb,
                               uint64_t* mask_bits, void* stream);

/*
 * Conservative resize between resolutions (Sec. 4.3.1, Eq. 7): masks and
 * maps are built once at a base resolution and resized for others.  Target
 * block (u, v) samples the base at x = u * n_qb / n_qb_out,
 * y = v * n_kb / n_kb_out (exact rationals); its bilinear neighbours with a
 * positive weight are base rows floor(x) and, if x is not whole,
 * floor(x) + 1 (the last row repeats past the end), likewise for columns.
 *
 * sa_resize_mask: CRM bits [H][n_qb][W] -> [H][n_qb_out][W_out]; a target
 * bit is the ceiling of the bilinear interpolation of the 0/1 mask, i.e. the
 * OR of its positively weighted neighbours.  Every output word is written
 * (bits past n_kb_out zero).
 *
 * sa_resize_threshold_map: float32 [H][n_qb][n_kb] -> [H][n_qb_out][n_kb_out];
 * a target entry is the minimum of its positively weighted neighbours (NaN
 * entries skipped), the reading of Eq. 7 for threshold maps under which
 * sa_mask_instantiate(resized map, p) == sa_resize_mask(sa_mask_instantiate
 * (map, p)) for every p.
 *
 * Meant for upscaling (every active base block survives); a smaller target
 * samples only some base rows.  Outputs must not overlap inputs.  All sizes
 * (H included) >= 1 and <= 65535.
 */
SA_API int sa_resize_mask(const uint64_t* mask_bits, int H, int n_qb, int n_kb, uint64_t* mask_out,
                          int n_qb_out, int n_kb_out, void* stream);

SA_API int sa_resize_threshold_map(const float* T, int H, int n_qb, int n_kb, float* T_out,
                                   int n_qb_out, int n_kb_out, void* stream);

/*
 * Work schedule (balances heads of uneven density and keeps K/V reuse inside
 * each XCD's L2): writes order[0 .. B*H*n_qb-1], a permutation of the work
 * items it = (b * H + h) * n_qb + u; the attention kernel runs item order[p]
 * at launch position p, and position p runs on XCD p mod 8.  The (b, h)
 * groups are ranked by decreasing total enabled blocks (ties by index).
 * With q = n_qb / 8 and r = n_qb mod 8, the group of rank k is cut into 8
 * chunks of consecutive u, chunk x holding q items plus one more when x is one
 * of (k r + i) mod 8, i < r; in u order the chunks follow by place
 * (x + k) mod 8.  Positions x, x + 8, x + 16, ... (sequence x) hold chunk x of
 * every group in rank order.  Each chunk is cut into windows of up to 128
 * consecutive u; the i-th window of a chunk holds its query blocks by
 * decreasing enabled-block count (ties by u) when i is even or the window is
 * the sequence's last, increasing otherwise, so that neighbouring positions
 * of a sequence, which the attention kernel runs side by side, have similar
 * counts.  counts: device int32
 * [H * n_qb] from the pre-pass (any values give a permutation).  order:
 * device int32 [B * H * n_qb].  With more than 4096 (b, h) groups the order
 * is the identity.
 */
SA_API int sa_schedule(const int32_t* counts, int B, int H, int n_qb,
                       int32_t* order, void* stream);

/*
 * Attention kernel alone, on a pre-computed pre-pass and schedule (the
 * static-mask case: masks are built once and reused for every prompt,
 * Sec. 4 overview figure, "Reuse for All Prompts").  counts/lists/order as produced
 * by sa_mask_prepass and sa_schedule for the same (B, H, N, blk_q, blk_k),
 * 4-byte aligned.  Entries out of range are clamped on the device (work item
 * to [0, B H n_qb), count to [0, n_kb], key block to [0, n_kb)): the result
 * of malformed buffers is unspecified, but nothing outside the tensors is
 * read or written.
 */
SA_API int sa_bsattn_fwd_prepared(const void* q, const void* k, const void* v,
                                  const int32_t* counts, const int32_t* lists,
                                  const int32_t* order, void* out, float* lse,
                                  int B, int H, int N, int d, int blk_q, int blk_k,
                                  float scale, void* stream);

/*
 * Maskless dense attention: the same kernel with every key block enabled and
 * no mask machinery (no pre-pass, no schedule, no workspace, no allocation).
 * It is the 0 %-sparsity baseline against which the CRM path's overhead is
 * measured (the paper's appendix "Detailed Kernel Overhead Analysis" compares
 * its kernel at 0 % sparsity with a dense FlashAttention kernel).  The result
 * equals sa_bsattn_fwd with an all-ones mask bit for bit.  blk is the tile
 * size (64 or 128, used for both query and key blocks).  Arguments and errors otherwise as
 * sa_bsattn_fwd.
 */
SA_API int sa_dense_attn_fwd(const void* q, const void* k, const void* v, void* out, float* lse,
                             int B, int H, int N, int d, int blk, float scale, void* stream);

/*
 * Fidelity profile of threshold-map masks on sampled query rows (FAST's
 * offline profiling: Hellinger distance Sec. 4.2.1 Eq. 3, Fidelity Score
 * Eq. 4, stratified row sampling Sec. 4.2.3).  For batch b, head h, sampled
 * row i (query token r = rows[h][i], query block u = r / blk) and candidate
 * threshold p[c], with P the dense softmax row of token r over all N keys and
 * P~ the softmax over the keys of the blocks v with T[h][u][v] <= p[c] (zero
 * elsewhere):
 *   hellinger[b][h][i][c] = H(P, P~)                 (1 if no block is kept)
 *   fidelity[b][h][c]     = 1 - mean_i hellinger[b][h][i][c]
 *   blk_lse[b][h][i][v]   = log sum_{j in block v} exp(scale <q_r, k_j>)
 * (blk_lse is also the working buffer between the two kernels.)
 * q, k: bf16 [B][H][N][d] as above; rows: device int32 [H][R], entries
 * clamped to [0, N); T: device float32 [H][n_qb][n_kb] (n_qb = n_kb =
 * ceil(N / blk)); p: device float32 [K]; outputs float32 as shown.  Outputs
 * must not overlap inputs or each other.  Requires 1 <= R <= 32,
 * 1 <= K <= 64, B * H <= 65535, d in {64, 128}, blk in {64, 128}.
 */
SA_API int sa_fidelity_profile(const void* q, const void* k, const int32_t* rows, int R,
                               const float* T, const float* p, int K, float* blk_lse,
                               float* hellinger, float* fidelity, int B, int H, int N, int d,
                               int blk, float scale, void* stream);

/*
 * Plan API for static masks (the paper's masks are built offline and reused
 * for every prompt: Sec. 4 overview figure, "Reuse for All Prompts"; the
 * executed blocks are those of Sec. 4.3.2's CRM rows).  A plan holds the
 * result of the CRM walk (the pre-pass) and the work schedule for one mask,
 * so that each forward pass runs only the attention kernel.
 * sa_bsattn_plan_create allocates the plan's
 * device buffers with hipMalloc, runs the pre-pass and schedule on `stream`,
 * then SYNCHRONISES `stream` to record the executed-block count.  The plan
 * keeps no pointer to mask_bits.  A plan is bound to the device that was
 * current at creation and is read-only after creation, so concurrent
 * sa_bsattn_fwd_plan calls (any streams) may share it; destroying it while
 * such calls are in flight is the caller's error.
 */
typedef struct sa_plan* sa_plan_t;

SA_API int sa_bsattn_plan_create(const uint64_t* mask_bits, int B, int H, int N,
                                 int blk_q, int blk_k, void* stream, sa_plan_t* plan);

/*
 * Attention with a plan (Sec. 4.3.2, on the plan's precomputed block lists;
 * on the device that was current at creation, else
 * SA_ERR_INVALID_ARG): only the attention kernel is enqueued (no
 * allocation, memset or synchronisation), so the call may be captured into a
 * HIP graph and replayed; the plan and the tensors must outlive the graph.
 */
SA_API int sa_bsattn_fwd_plan(sa_plan_t plan, const void* q, const void* k, const void* v,
                              void* out, float* lse, int d, float scale, void* stream);

/* sa_bsattn_fwd_plan with a float32 out, as sa_bsattn_fwd_f32out. */
SA_API int sa_bsattn_fwd_plan_f32out(sa_plan_t plan, const void* q, const void* k, const void* v,
                                     float* out, float* lse, int d, float scale, void* stream);

/* Total executed (b, h, u, v) blocks of the plan: B * sum of all row counts
 * (the blocks whose CRM bit is set, Sec. 4.3.2). */
SA_API int sa_bsattn_plan_stats(sa_plan_t plan, int64_t* executed_blocks);

/* Frees the plan (hipFree, which waits for outstanding work on the device). */
SA_API int sa_bsattn_plan_destroy(sa_plan_t plan);

#ifdef __cplusplus
}
#endif

#endif /* SA_BSATTN_H */
