// Internal host-side launchers shared by the C ABI (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

// Largest B * H for which the schedule sorts (b, h) groups by cost; larger
// problems keep the natural item order.
constexpr int kScheduleMaxUnits = 4096;

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* counts;
  const int32_t* lists;
  const int32_t* order;
  void* out;
  float* lse;
  int B, H, N, d, blk_q, blk_k, n_qb, n_kb;
  float scale;
  // element strides of q, k, v and out: batch, head, token (the head-dim is contiguous)
  int64_t sb, sh;
  int sn;
  bool out_f32 = false;  // out is fp32 instead of bf16 (masked path only)
};

hipError_t launch_prepass(const uint64_t* mask_bits, int H, int n_qb, int n_kb, int32_t* counts,
                          int32_t* lists, hipStream_t stream);

hipError_t launch_schedule(const int32_t* counts, int B, int H, int n_qb, int32_t* order,
                           hipStream_t stream);

hipError_t launch_mask_instantiate(const float* T, const float* p, int n_p, int H, int n_qb,
                                   int n_kb, uint64_t* bits, hipStream_t stream);

hipError_t launch_resize_map(const float* T, int H, int nq, int nk, float* out, int tq, int tk,
                             hipStream_t stream);

hipError_t launch_resize_mask(const uint64_t* bits, int H, int nq, int nk, uint64_t* out, int tq,
                              int tk, hipStream_t stream);

bool fidelity_supported(int R, int K);

hipError_t launch_fidelity(const void* q, const void* k, const int32_t* rows, int R, const float* T,
                           const float* p, int K, float* blk_lse, float* hel, float* fid, int B,
                           int H, int N, int d, int blk, float scale, hipStream_t stream);

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream);

// Maskless variant: every key block enabled; counts, lists and order unused.
hipError_t launch_attention_dense(const AttnArgs& a, hipStream_t stream);

}  // namespace sa
