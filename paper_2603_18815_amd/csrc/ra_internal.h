// Host-side launch interface between the C ABI layer and the kernel files.
// Every launcher assumes the arguments were validated by the ABI layer and
// returns the hipError_t of its launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ra {

struct PagedKV {
  uint16_t *k_pool;
  uint16_t *v_pool;
  const int32_t *block_table;
  int32_t num_pages;
  int32_t bt_stride;
  int32_t hkv;
};

// ---- decode (split over pages, then combine) ----
struct DecodePlan {
  int32_t split_tokens;   // tokens per split, a multiple of 128
  int32_t max_splits;     // splits of the longest row
};
DecodePlan decode_plan(int32_t B, int32_t hkv, int32_t max_kv_len);
size_t decode_workspace_bytes(int32_t B, int32_t hq, const DecodePlan &plan);

hipError_t launch_decode(const uint16_t *q, const PagedKV &kv, const int32_t *kv_lens, int32_t B,
                         int32_t hq, int32_t max_kv_len, float scale, float *out, float *lse,
                         void *workspace, const DecodePlan &plan, hipStream_t stream);

// ---- append (causal chunked prefill against the cache) ----
hipError_t launch_append(const uint16_t *q, const int32_t *cu_q, const int32_t *ctx_lens,
                         const PagedKV &kv, int32_t B, int32_t hq, int32_t total_q,
                         int32_t max_q_len, int32_t max_kv_len, float scale, float *out,
                         float *lse, hipStream_t stream);

// ---- page write / gather ----
hipError_t launch_page_write(const uint16_t *k_new, const uint16_t *v_new, const int32_t *cu_new,
                             const int32_t *start_pos, const PagedKV &kv, int32_t B,
                             int32_t total_new, int32_t max_new, int32_t max_pos,
                             hipStream_t stream);

hipError_t launch_page_gather(const PagedKV &kv, const int32_t *lens, const int32_t *cu_out,
                              int32_t B, int32_t total, int32_t max_len, uint16_t *k_out,
                              uint16_t *v_out, hipStream_t stream);

}  // namespace ra
