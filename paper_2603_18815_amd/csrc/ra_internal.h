// Host-side launch interface between the C ABI layer and the kernel files.
// Every launcher assumes the arguments were validated by the ABI layer and
// returns the hipError_t of its launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ra {

// Pools hold bf16 elements, or E4M3 codes (fp8) whose value is code * scale;
// k_pool / v_pool then point at bytes.
struct PagedKV {
  uint16_t *k_pool;
  uint16_t *v_pool;
  const int32_t *block_table;
  int32_t num_pages;
  int32_t bt_stride;
  int32_t hkv;
  bool fp8;
  float k_scale, v_scale;   // fp8 pools only (1 for bf16)
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

// ---- shared-prefix decode (rows of a group share their first prefix pages) ----
int32_t prefix_slots(const DecodePlan &plan, int32_t max_prefix_len);
// Work of one call, all in one launch of grid (Hkv, max_splits, prefix_planes
// + row_z): prefix_items (group chunk of rows_per_chunk rows, prefix split)
// pairs folded over the first prefix_planes planes, then one plane per (group,
// row slot). Both kinds of item use `tiles` 16-column tiles.
struct SharedPrefixShape {
  int32_t rows_per_chunk, tiles, chunks;
  int64_t prefix_items, prefix_planes, row_z;
};
SharedPrefixShape shared_prefix_shape(int32_t group, int32_t num_groups, int32_t max_group_rows,
                                      const DecodePlan &plan, int32_t max_prefix_len);
size_t shared_prefix_workspace_bytes(int32_t B, int32_t hq, const DecodePlan &plan,
                                     int32_t max_prefix_len);
hipError_t launch_decode_shared_prefix(const uint16_t *q, const PagedKV &kv,
                                       const int32_t *kv_lens, const int32_t *group_start,
                                       const int32_t *prefix_len, int32_t B, int32_t hq,
                                       int32_t num_groups, int32_t max_group_rows,
                                       int32_t max_prefix_len, int32_t max_kv_len, float scale,
                                       float *out, float *lse, void *workspace,
                                       const DecodePlan &plan, hipStream_t stream);

// ---- append, and the mixed step (decode rows and append rows), in one
// planned persistent launch; append alone is the mixed step without decode
// rows. Workspace: a header, the append row order, the append tile list, the
// decode split list and the decode partial results, each at a 256-byte
// aligned offset.
struct MixedLayout {
  DecodePlan plan;            // decode splits
  int32_t qblocks;            // query blocks of the longest append chunk
  int64_t max_tiles;          // bound on append tile entries
  int64_t max_splits;         // bound on decode split entries
  size_t tiles_offset, splits_offset, partials_offset, bytes;
};
MixedLayout mixed_layout(int32_t B_decode, int32_t B_append, int32_t hq, int32_t hkv_decode,
                         int32_t hkv_append, int32_t max_kv_len_decode, int32_t max_q_len);
int32_t mixed_hkv_limit();   // KV heads an entry can name
hipError_t launch_mixed(const uint16_t *q_decode, const PagedKV &kv_decode,
                        const int32_t *kv_lens, int32_t B_decode, int32_t max_kv_len_decode,
                        float *out_decode, float *lse_decode, const uint16_t *q_append,
                        const int32_t *cu_q, const int32_t *ctx_lens, const PagedKV &kv_append,
                        int32_t B_append, int32_t total_q, int32_t max_q_len,
                        int32_t max_kv_len_append, float *out_append, float *lse_append,
                        int32_t hq, float scale, void *workspace, const MixedLayout &layout,
                        hipStream_t stream, const uint16_t *k_new = nullptr,
                        const uint16_t *v_new = nullptr, const float *cos_sin = nullptr,
                        int32_t rope_rows = 0);

// ---- per-token log-probabilities under an LM head ----
int32_t logprob_chunks(int32_t N, int32_t V);
size_t logprob_workspace_bytes(int32_t N, int32_t V, int32_t D);
int64_t logprob_grid(int32_t N, int32_t V);
hipError_t launch_logprob(const uint16_t *h, const uint16_t *W, const int32_t *targets, int32_t N,
                          int32_t V, int32_t D, float scale, float *logp, float *lse,
                          void *workspace, bool packed, hipStream_t stream);
size_t logprob_packed_bytes(int32_t V, int32_t D);
hipError_t launch_logprob_pack(const uint16_t *W, int32_t V, int32_t D, uint16_t *Wp,
                               hipStream_t stream);

// ---- page write / gather ----
hipError_t launch_page_write(const uint16_t *k_new, const uint16_t *v_new, const int32_t *cu_new,
                             const int32_t *start_pos, const PagedKV &kv, int32_t B,
                             int32_t total_new, int32_t max_new, int32_t max_pos,
                             hipStream_t stream, const float *cos_sin = nullptr,
                             int32_t rope_rows = 0);

hipError_t launch_page_gather(const PagedKV &kv, const int32_t *lens, const int32_t *cu_out,
                              int32_t B, int32_t total, int32_t max_len, uint16_t *k_out,
                              uint16_t *v_out, hipStream_t stream);

}  // namespace ra
