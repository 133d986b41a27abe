// C ABI of the block-sparse attention library (declared in include/sa_bsattn.h).
//
// Every entry point validates all arguments before enqueuing anything, so a
// non-zero status means no kernel ran and no output was written.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <new>

#include "../../include/sa_bsattn.h"
#include "launch.h"

namespace {

constexpr int kVersion = 300;  // 0.3.0: allocation-free one-shot entry point

struct Dims {
  int n_qb, n_kb, W;
};

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

inline bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return na && nb && x < y + nb && y < x + na;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Shape checks shared by every entry point that takes (B, H, N, blk_q, blk_k).
int check_shape(int B, int H, int N, int blk_q, int blk_k, Dims* dims) {
  if (B < 1 || H < 1 || N < 1) return SA_ERR_INVALID_ARG;
  if ((blk_q != 64 && blk_q != 128) || (blk_k != 64 && blk_k != 128)) return SA_ERR_UNSUPPORTED;
  const int n_qb = (int)(((int64_t)N + blk_q - 1) / blk_q);
  const int n_kb = (int)(((int64_t)N + blk_k - 1) / blk_k);
  if (n_kb > 65535) return SA_ERR_UNSUPPORTED;
  if ((int64_t)B * H * n_qb >= ((int64_t)1 << 31)) return SA_ERR_UNSUPPORTED;
  dims->n_qb = n_qb;
  dims->n_kb = n_kb;
  dims->W = (n_kb + 63) / 64;
  return SA_OK;
}

int check_tensors(const void* q, const void* k, const void* v, const void* mask_bits, size_t mask_words,
                  const void* out, const float* lse, int B, int H, int N, int d, float scale,
                  size_t out_elem = 2) {
  if (d != 64 && d != 128) return SA_ERR_UNSUPPORTED;
  if (!(scale > 0.f) || !isfinite(scale)) return SA_ERR_INVALID_ARG;
  if (!q || !k || !v || !out || !lse) return SA_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(lse, 4))
    return SA_ERR_INVALID_ARG;
  const size_t tensor_bytes = (size_t)B * H * N * d * 2;
  const size_t out_bytes = (size_t)B * H * N * d * out_elem;
  const size_t lse_bytes = (size_t)B * H * N * 4;
  const size_t mask_bytes = (size_t)mask_words * 8;
  const void* ins[4] = {q, k, v, mask_bits};
  const size_t in_bytes[4] = {tensor_bytes, tensor_bytes, tensor_bytes, mask_bytes};
  for (int i = 0; i < 4; ++i) {
    if (!ins[i]) continue;
    if (overlap(out, out_bytes, ins[i], in_bytes[i])) return SA_ERR_INVALID_ARG;
    if (overlap(lse, lse_bytes, ins[i], in_bytes[i])) return SA_ERR_INVALID_ARG;
  }
  if (overlap(out, out_bytes, lse, lse_bytes)) return SA_ERR_INVALID_ARG;
  return SA_OK;
}

struct Workspace {
  size_t counts_off, lists_off, order_off, total;
};

Workspace plan_workspace(int B, int H, const Dims& dm) {
  Workspace w;
  const size_t rows = (size_t)H * dm.n_qb;
  w.counts_off = 0;
  w.lists_off = align_up(rows * 4, 256);
  w.order_off = w.lists_off + align_up(rows * dm.n_kb * 4, 256);
  w.total = w.order_off + align_up((size_t)B * H * dm.n_qb * 4, 256);
  return w;
}

}  // namespace

struct sa_plan {
  int B, H, N, blk_q, blk_k;
  Dims dims;
  int device;
  void* buf;
  int32_t* counts;
  int32_t* lists;
  int32_t* order;
  int64_t executed;
};

extern "C" {

SA_API const char* sa_status_string(int status) {
  switch (status) {
    case SA_OK: return "ok";
    case SA_ERR_INVALID_ARG: return "invalid argument";
    case SA_ERR_UNSUPPORTED: return "unsupported shape";
    case SA_ERR_HIP: return "HIP runtime error";
    case SA_ERR_TOO_LARGE: return "workspace larger than the fixed scratch of the allocation-free entry point";
    default: return "unknown status";
  }
}

SA_API int sa_version(void) { return kVersion; }

SA_API int sa_mask_prepass(const uint64_t* mask_bits, int H, int n_qb, int n_kb, int32_t* counts,
                           int32_t* lists, void* stream) {
  if (!mask_bits || !counts || !lists || H < 1 || n_qb < 1 || n_kb < 1) return SA_ERR_INVALID_ARG;
  if (!aligned(mask_bits, 8) || !aligned(counts, 4) || !aligned(lists, 4)) return SA_ERR_INVALID_ARG;
  if (n_kb > 65535 || (int64_t)H * n_qb >= ((int64_t)1 << 31)) return SA_ERR_UNSUPPORTED;
  const hipError_t e =
      sa::launch_prepass(mask_bits, H, n_qb, n_kb, counts, lists, (hipStream_t)stream);
  return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

SA_API int sa_mask_instantiate(const float* T, const float* p, int n_p, int H, int n_qb, int n_kb,
                               uint64_t* mask_bits, void* stream) {
  if (!T || !p || !mask_bits || n_p < 1 || H < 1 || n_qb < 1 || n_kb < 1) return SA_ERR_INVALID_ARG;
  if (!aligned(T, 4) || !aligned(p, 4) || !aligned(mask_bits, 8)) return SA_ERR_INVALID_ARG;
  if (n_kb > 65535 || n_p > 16 * 65535) return SA_ERR_UNSUPPORTED;
  const int64_t rows = (int64_t)H * n_qb;
  const int64_t W = (n_kb + 63) / 64;
  if (rows >= ((int64_t)1 << 31) || (int64_t)n_p * rows * W >= ((int64_t)1 << 40))
    return SA_ERR_UNSUPPORTED;
  const size_t t_bytes = (size_t)rows * n_kb * 4;
  const size_t p_bytes = (size_t)n_p * H * 4;
  const size_t b_bytes = (size_t)n_p * rows * W * 8;
  if (overlap(mask_bits, b_bytes, T, t_bytes) || overlap(mask_bits, b_bytes, p, p_bytes))
    return SA_ERR_INVALID_ARG;
  const hipError_t e =
      sa::launch_mask_instantiate(T, p, n_p, H, n_qb, n_kb, mask_bits, (hipStream_t)stream);
  return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

static int check_resize(const void* in, size_t in_align, int H, int nq, int nk, const void* out,
                        size_t out_align, int tq, int tk) {
  if (!in || !out || H < 1 || nq < 1 || nk < 1 || tq < 1 || tk < 1) return SA_ERR_INVALID_ARG;
  if (!aligned(in, in_align) || !aligned(out, out_align)) return SA_ERR_INVALID_ARG;
  if (nq > 65535 || nk > 65535 || tq > 65535 || tk > 65535 || H > 65535) return SA_ERR_UNSUPPORTED;
  if ((int64_t)H * tq * tk >= ((int64_t)1 << 40) || (int64_t)H * nq >= ((int64_t)1 << 31) ||
      (int64_t)H * tq >= ((int64_t)1 << 31))
    return SA_ERR_UNSUPPORTED;
  return SA_OK;
}

SA_API int sa_resize_threshold_map(const float* T, int H, int n_qb, int n_kb, float* T_out,
                                   int n_qb_out, int n_kb_out, void* stream) {
  int st = check_resize(T, 4, H, n_qb, n_kb, T_out, 4, n_qb_out, n_kb_out);
  if (st != SA_OK) return st;
  if (overlap(T_out, (size_t)H * n_qb_out * n_kb_out * 4, T, (size_t)H * n_qb * n_kb * 4))
    return SA_ERR_INVALID_ARG;
  const hipError_t e =
      sa::launch_resize_map(T, H, n_qb, n_kb, T_out, n_qb_out, n_kb_out, (hipStream_t)stream);
  return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

SA_API int sa_resize_mask(const uint64_t* mask_bits, int H, int n_qb, int n_kb, uint64_t* mask_out,
                          int n_qb_out, int n_kb_out, void* stream) {
  int st = check_resize(mask_bits, 8, H, n_qb, n_kb, mask_out, 8, n_qb_out, n_kb_out);
  if (st != SA_OK) return st;
  const size_t in_bytes = (size_t)H * n_qb * ((n_kb + 63) / 64) * 8;
  const size_t out_bytes = (size_t)H * n_qb_out * ((n_kb_out + 63) / 64) * 8;
  if (overlap(mask_out, out_bytes, mask_bits, in_bytes)) return SA_ERR_INVALID_ARG;
  const hipError_t e = sa::launch_resize_mask(mask_bits, H, n_qb, n_kb, mask_out, n_qb_out,
                                              n_kb_out, (hipStream_t)stream);
  return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

SA_API int sa_schedule(const int32_t* counts, int B, int H, int n_qb, int32_t* order, void* stream) {
  if (!counts || !order || B < 1 || H < 1 || n_qb < 1) return SA_ERR_INVALID_ARG;
  if (!aligned(counts, 4) || !aligned(order, 4)) return SA_ERR_INVALID_ARG;
  if ((int64_t)B * H * n_qb >= ((int64_t)1 << 31)) return SA_ERR_UNSUPPORTED;
  const hipError_t e = sa::launch_schedule(counts, B, H, n_qb, order, (hipStream_t)stream);
  return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

// Attention kernel alone on a prepared pre-pass and schedule; out is bf16 or,
// with out_f32, fp32.
static int fwd_prepared(const void* q, const void* k, const void* v, const int32_t* counts,
                        const int32_t* lists, const int32_t* order, void* out, float* lse, int B,
                        int H, int N, int d, int blk_q, int blk_k, float scale, bool out_f32,
                        void* stream) {
  Dims dm;
  int st = check_shape(B, H, N, blk_q, blk_k, &dm);
  if (st != SA_OK) return st;
  st = check_tensors(q, k, v, nullptr, 0, out, lse, B, H, N, d, scale, out_f32 ? 4 : 2);
  if (st != SA_OK) return st;
  if (!counts || !lists || !order) return SA_ERR_INVALID_ARG;
  if (!aligned(counts, 4) || !aligned(lists, 4) || !aligned(order, 4)) return SA_ERR_INVALID_ARG;
  sa::AttnArgs a{q, k, v, counts, lists, order, out, lse, B, H, N, d, blk_q, blk_k,
                 dm.n_qb, dm.n_kb, scale,
                 (int64_t)H * N * d, (int64_t)N * d, d};
  a.out_f32 = out_f32;
  return sa::launch_attention(a, (hipStream_t)stream) == hipSuccess ? SA_OK : SA_ERR_HIP;
}

SA_API int sa_bsattn_fwd_prepared(const void* q, const void* k, const void* v,
                                  const int32_t* counts, const int32_t* lists,
                                  const int32_t* order, void* out, float* lse, int B, int H, int N,
                                  int d, int blk_q, int blk_k, float scale, void* stream) {
  return fwd_prepared(q, k, v, counts, lists, order, out, lse, B, H, N, d, blk_q, blk_k, scale,
                      false, stream);
}

// Checks of a one-shot call (either tensor layout; out bf16 or, with out_f32,
// fp32), before anything is enqueued.
static int check_oneshot(const void* q, const void* k, const void* v, const uint64_t* mask_bits,
                         const void* out, const float* lse, int B, int H, int N, int d, int blk_q,
                         int blk_k, float scale, int layout, bool out_f32, Dims* dm) {
  int st = check_shape(B, H, N, blk_q, blk_k, dm);
  if (st != SA_OK) return st;
  if (!mask_bits || !aligned(mask_bits, 8)) return SA_ERR_INVALID_ARG;
  if (layout != SA_LAYOUT_BHND && layout != SA_LAYOUT_BNHD) return SA_ERR_INVALID_ARG;
  st = check_tensors(q, k, v, mask_bits, (size_t)H * dm->n_qb * dm->W, out, lse, B, H, N, d, scale,
                     out_f32 ? 4 : 2);
  if (st != SA_OK) return st;
  const int sn = layout == SA_LAYOUT_BNHD ? H * d : d;
  // tile copies address a tile with 32-bit byte offsets
  if ((int64_t)sn * (blk_k > blk_q ? blk_k : blk_q) * 2 >= ((int64_t)1 << 31)) return SA_ERR_UNSUPPORTED;
  return SA_OK;
}

// Pre-pass, schedule and attention of a checked one-shot call, with the
// workspace laid out by plan_workspace at ws.
static hipError_t launch_oneshot(const void* q, const void* k, const void* v,
                                 const uint64_t* mask_bits, void* out, float* lse, int B, int H,
                                 int N, int d, int blk_q, int blk_k, float scale, int layout,
                                 bool out_f32, const Dims& dm, void* ws, hipStream_t s) {
  const Workspace w = plan_workspace(B, H, dm);
  char* base = (char*)ws;
  int32_t* counts = (int32_t*)(base + w.counts_off);
  int32_t* lists = (int32_t*)(base + w.lists_off);
  int32_t* order = (int32_t*)(base + w.order_off);
  const bool bnhd = layout == SA_LAYOUT_BNHD;
  const int sn = bnhd ? H * d : d;
  hipError_t e = sa::launch_prepass(mask_bits, H, dm.n_qb, dm.n_kb, counts, lists, s);
  if (e == hipSuccess) e = sa::launch_schedule(counts, B, H, dm.n_qb, order, s);
  if (e == hipSuccess) {
    sa::AttnArgs a{q, k, v, counts, lists, order, out, lse, B, H, N, d, blk_q, blk_k,
                   dm.n_qb, dm.n_kb, scale,
                   (int64_t)H * N * d, bnhd ? (int64_t)d : (int64_t)N * d, sn};
    a.out_f32 = out_f32;
    e = sa::launch_attention(a, s);
  }
  return e;
}

// One-shot forward with a stream-ordered workspace.
static int fwd_oneshot(const void* q, const void* k, const void* v, const uint64_t* mask_bits,
                       void* out, float* lse, int B, int H, int N, int d, int blk_q, int blk_k,
                       float scale, int layout, bool out_f32, void* stream) {
  Dims dm;
  const int st = check_oneshot(q, k, v, mask_bits, out, lse, B, H, N, d, blk_q, blk_k, scale,
                               layout, out_f32, &dm);
  if (st != SA_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  const Workspace w = plan_workspace(B, H, dm);
  void* ws = nullptr;
  if (hipMallocAsync(&ws, w.total, s) != hipSuccess || !ws) return SA_ERR_HIP;
  const hipError_t e = launch_oneshot(q, k, v, mask_bits, out, lse, B, H, N, d, blk_q, blk_k,
                                      scale, layout, out_f32, dm, ws, s);
  const hipError_t ef = hipFreeAsync(ws, s);
  return (e == hipSuccess && ef == hipSuccess) ? SA_OK : SA_ERR_HIP;
}

// Scratch of the allocation-free entry point: the workspace (counts, lists,
// order) of one call, in the library's own device memory.  Each GPU holds its
// copy from the library's load onto it until the process ends.  In host code
// `scratch` only names the symbol; its device address on the current device
// comes from hipGetSymbolAddress, looked up once per device and kept below.
static __device__ __align__(256) unsigned char scratch[SA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static void* g_scratch_ptr[kMaxDevices];
static std::mutex g_scratch_mu;

// Device address of `scratch` on the current device (set up on the first call
// there, with that device current).
static int scratch_on_current_device(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SA_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SA_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SA_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return SA_OK;
}

SA_API int sa_bsattn_fwd(const void* q, const void* k, const void* v, const uint64_t* mask_bits,
                         void* out, float* lse, int B, int H, int N, int d, int blk_q, int blk_k,
                         float scale, void* stream) {
  return fwd_oneshot(q, k, v, mask_bits, out, lse, B, H, N, d, blk_q, blk_k, scale,
                     SA_LAYOUT_BHND, false, stream);
}

SA_API int sa_bsattn_fwd_noalloc(const void* q, const void* k, const void* v,
                                 const uint64_t* mask_bits, void* out, float* lse, int B, int H,
                                 int N, int d, int blk_q, int blk_k, float scale, void* stream) {
  Dims dm;
  int st = check_oneshot(q, k, v, mask_bits, out, lse, B, H, N, d, blk_q, blk_k, scale,
                         SA_LAYOUT_BHND, false, &dm);
  if (st != SA_OK) return st;
  if (plan_workspace(B, H, dm).total > (size_t)SA_NOALLOC_SCRATCH_BYTES) return SA_ERR_TOO_LARGE;
  void* ws = nullptr;
  st = scratch_on_current_device(&ws);
  if (st != SA_OK) return st;
  // Nothing in the scratch has to start at zero: the pre-pass writes every
  // count and every list entry up to the count, the schedule every order entry.
  const hipError_t e = launch_oneshot(q, k, v, mask_bits, out, lse, B, H, N, d, blk_q, blk_k,
                                      scale, SA_LAYOUT_BHND, false, dm, ws, (hipStream_t)stream);
  return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

SA_API int sa_bsattn_fwd_f32out(const void* q, const void* k, const void* v,
                                const uint64_t* mask_bits, float* out, float* lse, int B, int H,
                                int N, int d, int blk_q, int blk_k, float scale, void* stream) {
  return fwd_oneshot(q, k, v, mask_bits, out, lse, B, H, N, d, blk_q, blk_k, scale,
                     SA_LAYOUT_BHND, true, stream);
}

SA_API int sa_bsattn_fwd_layout(const void* q, const void* k, const void* v,
                                const uint64_t* mask_bits, void* out, float* lse, int B, int H,
                                int N, int d, int blk_q, int blk_k, float scale, int layout,
                                void* stream) {
  return fwd_oneshot(q, k, v, mask_bits, out, lse, B, H, N, d, blk_q, blk_k, scale, layout, false,
                     stream);
}

SA_API int sa_dense_attn_fwd(const void* q, const void* k, const void* v, void* out, float* lse,
                             int B, int H, int N, int d, int blk, float scale, void* stream) {
  Dims dm;
  int st = check_shape(B, H, N, blk, blk, &dm);
  if (st != SA_OK) return st;
  st = check_tensors(q, k, v, nullptr, 0, out, lse, B, H, N, d, scale);
  if (st != SA_OK) return st;
  sa::AttnArgs a{q, k, v, nullptr, nullptr, nullptr, out, lse, B, H, N, d, blk, blk,
                 dm.n_qb, dm.n_kb, scale,
                 (int64_t)H * N * d, (int64_t)N * d, d};
  return sa::launch_attention_dense(a, (hipStream_t)stream) == hipSuccess ? SA_OK : SA_ERR_HIP;
}

SA_API int sa_fidelity_profile(const void* q, const void* k, const int32_t* rows, int R,
                               const float* T, const float* p, int K, float* blk_lse,
                               float* hellinger, float* fidelity, int B, int H, int N, int d,
                               int blk, float scale, void* stream) {
  Dims dm;
  int st = check_shape(B, H, N, blk, blk, &dm);
  if (st != SA_OK) return st;
  if (d != 64 && d != 128) return SA_ERR_UNSUPPORTED;
  if (!(scale > 0.f) || !isfinite(scale)) return SA_ERR_INVALID_ARG;
  if (!q || !k || !rows || !T || !p || !blk_lse || !hellinger || !fidelity) return SA_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(rows, 4) || !aligned(T, 4) ||
      !aligned(p, 4) || !aligned(blk_lse, 4) || !aligned(hellinger, 4) || !aligned(fidelity, 4))
    return SA_ERR_INVALID_ARG;
  if (R < 1 || K < 1) return SA_ERR_INVALID_ARG;
  if (!sa::fidelity_supported(R, K) || (int64_t)B * H > 65535) return SA_ERR_UNSUPPORTED;
  const size_t tensor_bytes = (size_t)B * H * N * d * 2;
  const size_t rows_bytes = (size_t)H * R * 4;
  const size_t t_bytes = (size_t)H * dm.n_qb * dm.n_kb * 4;
  const size_t p_bytes = (size_t)K * 4;
  const size_t lse_bytes = (size_t)B * H * R * dm.n_kb * 4;
  const size_t hel_bytes = (size_t)B * H * R * K * 4;
  const size_t fid_bytes = (size_t)B * H * K * 4;
  const void* ins[5] = {q, k, rows, T, p};
  const size_t in_bytes[5] = {tensor_bytes, tensor_bytes, rows_bytes, t_bytes, p_bytes};
  const void* outs[3] = {blk_lse, hellinger, fidelity};
  const size_t out_bytes[3] = {lse_bytes, hel_bytes, fid_bytes};
  for (int o = 0; o < 3; ++o) {
    for (int i = 0; i < 5; ++i)
      if (overlap(outs[o], out_bytes[o], ins[i], in_bytes[i])) return SA_ERR_INVALID_ARG;
    for (int o2 = o + 1; o2 < 3; ++o2)
      if (overlap(outs[o], out_bytes[o], outs[o2], out_bytes[o2])) return SA_ERR_INVALID_ARG;
  }
  const hipError_t e = sa::launch_fidelity(q, k, rows, R, T, p, K, blk_lse, hellinger, fidelity, B,
                                           H, N, d, blk, scale, (hipStream_t)stream);
  return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

SA_API int sa_bsattn_plan_create(const uint64_t* mask_bits, int B, int H, int N, int blk_q,
                                 int blk_k, void* stream, sa_plan_t* plan) {
  if (!plan) return SA_ERR_INVALID_ARG;
  *plan = nullptr;
  Dims dm;
  int st = check_shape(B, H, N, blk_q, blk_k, &dm);
  if (st != SA_OK) return st;
  if (!mask_bits || !aligned(mask_bits, 8)) return SA_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  sa_plan* p = new (std::nothrow) sa_plan();
  if (!p) return SA_ERR_HIP;
  p->B = B; p->H = H; p->N = N; p->blk_q = blk_q; p->blk_k = blk_k; p->dims = dm;
  if (hipGetDevice(&p->device) != hipSuccess) { delete p; return SA_ERR_HIP; }
  const Workspace w = plan_workspace(B, H, dm);
  if (hipMalloc(&p->buf, w.total) != hipSuccess) { delete p; return SA_ERR_HIP; }
  char* base = (char*)p->buf;
  p->counts = (int32_t*)(base + w.counts_off);
  p->lists = (int32_t*)(base + w.lists_off);
  p->order = (int32_t*)(base + w.order_off);
  hipError_t e = sa::launch_prepass(mask_bits, H, dm.n_qb, dm.n_kb, p->counts, p->lists, s);
  if (e == hipSuccess) e = sa::launch_schedule(p->counts, B, H, dm.n_qb, p->order, s);
  int32_t* host_counts = nullptr;
  const size_t rows = (size_t)H * dm.n_qb;
  if (e == hipSuccess) {
    host_counts = new (std::nothrow) int32_t[rows];
    if (!host_counts) e = hipErrorOutOfMemory;
  }
  if (e == hipSuccess) e = hipMemcpyAsync(host_counts, p->counts, rows * 4, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    delete[] host_counts;
    (void)hipFree(p->buf);
    delete p;
    return SA_ERR_HIP;
  }
  int64_t tot = 0;
  for (size_t i = 0; i < rows; ++i) tot += host_counts[i];
  delete[] host_counts;
  p->executed = tot * B;
  *plan = p;
  return SA_OK;
}

static int fwd_plan(sa_plan_t plan, const void* q, const void* k, const void* v, void* out,
                    float* lse, int d, float scale, bool out_f32, void* stream) {
  if (!plan) return SA_ERR_INVALID_ARG;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SA_ERR_HIP;
  if (dev != plan->device) return SA_ERR_INVALID_ARG;  // the plan's buffers live on its device
  return fwd_prepared(q, k, v, plan->counts, plan->lists, plan->order, out, lse, plan->B, plan->H,
                      plan->N, d, plan->blk_q, plan->blk_k, scale, out_f32, stream);
}

SA_API int sa_bsattn_fwd_plan(sa_plan_t plan, const void* q, const void* k, const void* v,
                              void* out, float* lse, int d, float scale, void* stream) {
  return fwd_plan(plan, q, k, v, out, lse, d, scale, false, stream);
}

SA_API int sa_bsattn_fwd_plan_f32out(sa_plan_t plan, const void* q, const void* k, const void* v,
                                     float* out, float* lse, int d, float scale, void* stream) {
  return fwd_plan(plan, q, k, v, out, lse, d, scale, true, stream);
}

SA_API int sa_bsattn_plan_stats(sa_plan_t plan, int64_t* executed_blocks) {
  if (!plan || !executed_blocks) return SA_ERR_INVALID_ARG;
  *executed_blocks = plan->executed;
  return SA_OK;
}

SA_API int sa_bsattn_plan_destroy(sa_plan_t plan) {
  if (!plan) return SA_ERR_INVALID_ARG;
  const hipError_t e = hipFree(plan->buf);
  delete plan;
  return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

}  // extern "C"
