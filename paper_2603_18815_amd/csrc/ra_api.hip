// C ABI of the rollout-attention library: argument validation (before any HIP
// call), launch planning and status codes. See include/rollout_attn.h.
#include "rollout_attn.h"

#include <atomic>
#include <cmath>
#include <mutex>

#include "ra_internal.h"

namespace {

constexpr int32_t kMaxGridYZ = 65535;

bool valid_status(int s) { return s >= RA_OK && s <= RA_ERR_HIP; }

bool valid_pool_scale(float s) { return std::isfinite(s) && s > 0.f && std::isfinite(1.0f / s); }

// Common checks on the paged cache descriptor.
int check_kv(const ra_paged_kv *kv) {
  if (!kv) return RA_ERR_NULL;
  if (kv->page_size != RA_PAGE_SIZE || kv->head_dim != RA_HEAD_DIM) return RA_ERR_UNSUPPORTED;
  if (kv->num_kv_heads <= 0 || kv->num_pages <= 0 || kv->bt_stride <= 0) return RA_ERR_SHAPE;
  if (kv->num_kv_heads > kMaxGridYZ) return RA_ERR_UNSUPPORTED;
  if (kv->kv_dtype != RA_KV_BF16 && kv->kv_dtype != RA_KV_FP8_E4M3) return RA_ERR_UNSUPPORTED;
  // fp8 scales: finite, positive, and with a finite fp32 reciprocal (the
  // page write multiplies by it)
  if (kv->kv_dtype == RA_KV_FP8_E4M3 && !(valid_pool_scale(kv->k_scale) &&
                                          valid_pool_scale(kv->v_scale)))
    return RA_ERR_SHAPE;
  if (!kv->k_pool || !kv->v_pool || !kv->block_table) return RA_ERR_NULL;
  return RA_OK;
}

bool is_fp8(const ra_paged_kv *kv) { return kv->kv_dtype == RA_KV_FP8_E4M3; }

bool positions_fit(const ra_paged_kv *kv, int32_t max_pos) {
  return max_pos >= 0 && (int64_t)max_pos <= (int64_t)kv->bt_stride * RA_PAGE_SIZE;
}

ra::PagedKV to_internal(const ra_paged_kv *kv) {
  ra::PagedKV p;
  p.k_pool = static_cast<uint16_t *>(kv->k_pool);
  p.v_pool = static_cast<uint16_t *>(kv->v_pool);
  p.block_table = kv->block_table;
  p.num_pages = kv->num_pages;
  p.bt_stride = kv->bt_stride;
  p.hkv = kv->num_kv_heads;
  p.fp8 = is_fp8(kv);
  p.k_scale = p.fp8 ? kv->k_scale : 1.f;
  p.v_scale = p.fp8 ? kv->v_scale : 1.f;
  return p;
}

int hip_status(hipError_t e) { return e == hipSuccess ? RA_OK : RA_ERR_HIP; }

// Device scratch of rollout_attn_decode_noalloc: the decode split partials of
// one call. Each GPU the library runs on holds its own copy for the life of
// the process. In host code `scratch` names a host-side stand-in, not device
// memory: only the per-device address from hipGetSymbolAddress is used.
__device__ __align__(256) unsigned char scratch[RA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

// Address of the current device's scratch, looked up once per device (with
// that device current) and kept.
hipError_t device_scratch(void **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void *p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return hipSuccess;
}

// Checks shared by rollout_attn_decode and rollout_attn_decode_noalloc.
int check_decode(const void *q, const ra_paged_kv *kv, const int32_t *kv_lens, int32_t B,
                 int32_t Hq, int32_t max_kv_len, float scale, const float *out) {
  if (B < 0 || Hq <= 0 || max_kv_len < 0 || !std::isfinite(scale)) return RA_ERR_SHAPE;
  int s = check_kv(kv);
  if (s != RA_OK) return s;
  if (!q || !kv_lens || !out) return RA_ERR_NULL;
  if (Hq % kv->num_kv_heads != 0) return RA_ERR_SHAPE;
  if (Hq / kv->num_kv_heads > 32 || B > kMaxGridYZ) return RA_ERR_UNSUPPORTED;
  if (!positions_fit(kv, max_kv_len)) return RA_ERR_SHAPE;
  return RA_OK;
}

}  // namespace

extern "C" {

int ra_abi_version(void) { return RA_ABI_VERSION; }

const char *ra_status_string(int status) {
  static const char *names[] = {"RA_OK", "RA_ERR_NULL", "RA_ERR_SHAPE", "RA_ERR_UNSUPPORTED",
                                "RA_ERR_WORKSPACE", "RA_ERR_HIP"};
  return valid_status(status) ? names[status] : "RA_UNKNOWN_STATUS";
}

size_t rollout_attn_decode_workspace_size(int32_t B, int32_t Hq, int32_t Hkv,
                                          int32_t max_kv_len) {
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || max_kv_len < 0) return 0;
  return ra::decode_workspace_bytes(B, Hq, ra::decode_plan(B, Hkv, max_kv_len));
}

int rollout_attn_decode(const void *q, const ra_paged_kv *kv, const int32_t *kv_lens, int32_t B,
                        int32_t Hq, int32_t max_kv_len, float scale, float *out, float *lse,
                        void *workspace, size_t workspace_bytes, hipStream_t stream) {
  const int s = check_decode(q, kv, kv_lens, B, Hq, max_kv_len, scale, out);
  if (s != RA_OK) return s;
  if (B == 0) return RA_OK;
  const ra::DecodePlan plan = ra::decode_plan(B, kv->num_kv_heads, max_kv_len);
  if (!workspace || workspace_bytes < ra::decode_workspace_bytes(B, Hq, plan))
    return RA_ERR_WORKSPACE;
  return hip_status(ra::launch_decode(static_cast<const uint16_t *>(q), to_internal(kv), kv_lens,
                                      B, Hq, max_kv_len, scale, out, lse, workspace, plan,
                                      stream));
}

int rollout_attn_decode_noalloc(const void *q, const ra_paged_kv *kv, const int32_t *kv_lens,
                                int32_t B, int32_t Hq, int32_t max_kv_len, float scale,
                                float *out, float *lse, hipStream_t stream) {
  const int s = check_decode(q, kv, kv_lens, B, Hq, max_kv_len, scale, out);
  if (s != RA_OK) return s;
  if (B == 0) return RA_OK;
  const ra::DecodePlan plan = ra::decode_plan(B, kv->num_kv_heads, max_kv_len);
  if (ra::decode_workspace_bytes(B, Hq, plan) > RA_NOALLOC_SCRATCH_BYTES) return RA_ERR_WORKSPACE;
  void *ws = nullptr;
  const hipError_t e = device_scratch(&ws);
  if (e != hipSuccess) return RA_ERR_HIP;
  return hip_status(ra::launch_decode(static_cast<const uint16_t *>(q), to_internal(kv), kv_lens,
                                      B, Hq, max_kv_len, scale, out, lse, ws, plan, stream));
}

size_t rollout_attn_decode_shared_prefix_workspace_size(int32_t B, int32_t Hq, int32_t Hkv,
                                                        int32_t max_kv_len,
                                                        int32_t max_prefix_len) {
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || max_kv_len < 0 || max_prefix_len < 0) return 0;
  return ra::shared_prefix_workspace_bytes(B, Hq, ra::decode_plan(B, Hkv, max_kv_len),
                                           max_prefix_len);
}

int rollout_attn_decode_shared_prefix(const void *q, const ra_paged_kv *kv,
                                      const int32_t *kv_lens, const int32_t *group_start,
                                      const int32_t *prefix_len, int32_t B, int32_t Hq,
                                      int32_t num_groups, int32_t max_group_rows,
                                      int32_t max_prefix_len, int32_t max_kv_len, float scale,
                                      float *out, float *lse, void *workspace,
                                      size_t workspace_bytes, hipStream_t stream) {
  if (B < 0 || Hq <= 0 || max_kv_len < 0 || num_groups < 0 || max_group_rows < 0 ||
      max_prefix_len < 0 || !std::isfinite(scale))
    return RA_ERR_SHAPE;
  int s = check_kv(kv);
  if (s != RA_OK) return s;
  if (!q || !kv_lens || !out || !group_start || !prefix_len) return RA_ERR_NULL;
  if (Hq % kv->num_kv_heads != 0) return RA_ERR_SHAPE;
  if (Hq / kv->num_kv_heads > 32 || B > kMaxGridYZ) return RA_ERR_UNSUPPORTED;
  if (!positions_fit(kv, max_kv_len) || max_prefix_len > max_kv_len) return RA_ERR_SHAPE;
  if (B == 0) return RA_OK;
  if (num_groups == 0 || max_group_rows == 0 || max_group_rows > B || num_groups > B)
    return RA_ERR_SHAPE;
  const ra::DecodePlan plan = ra::decode_plan(B, kv->num_kv_heads, max_kv_len);
  const ra::SharedPrefixShape sh = ra::shared_prefix_shape(Hq / kv->num_kv_heads, num_groups,
                                                           max_group_rows, plan, max_prefix_len);
  // grid z holds the prefix planes and the row planes; prefix item indices
  // (plane x max_splits + split) must fit an int
  if (sh.prefix_planes + sh.row_z > kMaxGridYZ ||
      sh.prefix_planes * plan.max_splits > INT32_MAX)
    return RA_ERR_UNSUPPORTED;
  if (!workspace ||
      workspace_bytes < ra::shared_prefix_workspace_bytes(B, Hq, plan, max_prefix_len))
    return RA_ERR_WORKSPACE;
  return hip_status(ra::launch_decode_shared_prefix(
      static_cast<const uint16_t *>(q), to_internal(kv), kv_lens, group_start, prefix_len, B, Hq,
      num_groups, max_group_rows, max_prefix_len, max_kv_len, scale, out, lse, workspace, plan,
      stream));
}

size_t rollout_attn_append_workspace_size(int32_t B, int32_t Hq, int32_t Hkv,
                                          int32_t max_q_len) {
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || max_q_len < 0 || Hq % Hkv != 0 || Hq / Hkv > 256)
    return 0;
  return ra::mixed_layout(0, B, Hq, Hkv, Hkv, 0, max_q_len).bytes;
}

int rollout_attn_append(const void *q, const int32_t *cu_q, const int32_t *ctx_lens,
                        const ra_paged_kv *kv, int32_t B, int32_t Hq, int32_t total_q,
                        int32_t max_q_len, int32_t max_kv_len, float scale, float *out,
                        float *lse, void *workspace, size_t workspace_bytes,
                        hipStream_t stream) {
  if (B < 0 || Hq <= 0 || total_q < 0 || max_q_len < 0 || max_kv_len < 0 || !std::isfinite(scale))
    return RA_ERR_SHAPE;
  int s = check_kv(kv);
  if (s != RA_OK) return s;
  if (!q || !cu_q || !ctx_lens || !out) return RA_ERR_NULL;
  if (Hq % kv->num_kv_heads != 0) return RA_ERR_SHAPE;
  if (Hq / kv->num_kv_heads > 256 || B > kMaxGridYZ) return RA_ERR_UNSUPPORTED;
  if (!positions_fit(kv, max_kv_len) || max_q_len > max_kv_len) return RA_ERR_SHAPE;
  if (B == 0 || total_q == 0 || max_q_len == 0) return RA_OK;
  const ra::PagedKV k = to_internal(kv);
  if (k.hkv > ra::mixed_hkv_limit()) return RA_ERR_UNSUPPORTED;
  const ra::MixedLayout layout = ra::mixed_layout(0, B, Hq, k.hkv, k.hkv, 0, max_q_len);
  if (layout.max_tiles > 0x7fffffff - 0xffff || layout.qblocks >= (1 << 23))
    return RA_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < layout.bytes) return RA_ERR_WORKSPACE;
  return hip_status(ra::launch_mixed(nullptr, k, nullptr, 0, 0, nullptr, nullptr,
                                     static_cast<const uint16_t *>(q), cu_q, ctx_lens, k, B,
                                     total_q, max_q_len, max_kv_len, out, lse, Hq, scale,
                                     workspace, layout, stream));
}

}  // extern "C"

namespace {

// rollout_attn_append_write, with an optional rotary table (cos_sin null: none;
// otherwise checked by the caller).
int append_write_impl(const void *q, const void *k_new, const void *v_new, const int32_t *cu_q,
                      const int32_t *ctx_lens, const ra_paged_kv *kv, int32_t B, int32_t Hq,
                      int32_t total_q, int32_t max_q_len, int32_t max_kv_len, float scale,
                      const float *cos_sin, int32_t rope_rows, float *out, float *lse,
                      void *workspace, size_t workspace_bytes, hipStream_t stream) {
  if (B < 0 || Hq <= 0 || total_q < 0 || max_q_len < 0 || max_kv_len < 0 || !std::isfinite(scale))
    return RA_ERR_SHAPE;
  int s = check_kv(kv);
  if (s != RA_OK) return s;
  if (!q || !k_new || !v_new || !cu_q || !ctx_lens || !out) return RA_ERR_NULL;
  if (Hq % kv->num_kv_heads != 0) return RA_ERR_SHAPE;
  if (Hq / kv->num_kv_heads > 256 || B > kMaxGridYZ) return RA_ERR_UNSUPPORTED;
  if (!positions_fit(kv, max_kv_len) || max_q_len > max_kv_len) return RA_ERR_SHAPE;
  if (B == 0 || total_q == 0 || max_q_len == 0) return RA_OK;
  const ra::PagedKV k = to_internal(kv);
  if (k.hkv > ra::mixed_hkv_limit()) return RA_ERR_UNSUPPORTED;
  const ra::MixedLayout layout = ra::mixed_layout(0, B, Hq, k.hkv, k.hkv, 0, max_q_len);
  if (layout.max_tiles > 0x7fffffff - 0xffff || layout.qblocks >= (1 << 23))
    return RA_ERR_UNSUPPORTED;
  // the write runs as (row, page, head) blocks, four per workgroup
  if ((int64_t)B * k.hkv * ((int64_t)max_q_len / RA_PAGE_SIZE + 2) / 4 > 0x7ffffff0)
    return RA_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < layout.bytes) return RA_ERR_WORKSPACE;
  return hip_status(ra::launch_mixed(
      nullptr, k, nullptr, 0, 0, nullptr, nullptr, static_cast<const uint16_t *>(q), cu_q,
      ctx_lens, k, B, total_q, max_q_len, max_kv_len, out, lse, Hq, scale, workspace, layout,
      stream, static_cast<const uint16_t *>(k_new), static_cast<const uint16_t *>(v_new), cos_sin,
      rope_rows));
}

// kv_page_write, with an optional rotary table for K.
int page_write_impl(const void *k_new, const void *v_new, const int32_t *cu_new,
                    const int32_t *start_pos, const ra_paged_kv *kv, int32_t B, int32_t total_new,
                    int32_t max_new, int32_t max_pos, const float *cos_sin, int32_t rope_rows,
                    hipStream_t stream) {
  if (B < 0 || total_new < 0 || max_new < 0 || max_pos < 0) return RA_ERR_SHAPE;
  int s = check_kv(kv);
  if (s != RA_OK) return s;
  if (!k_new || !v_new || !cu_new || !start_pos) return RA_ERR_NULL;
  if (B > kMaxGridYZ) return RA_ERR_UNSUPPORTED;
  if (!positions_fit(kv, max_pos) || max_new > max_pos) return RA_ERR_SHAPE;
  if (B == 0 || total_new == 0 || max_new == 0) return RA_OK;
  return hip_status(ra::launch_page_write(static_cast<const uint16_t *>(k_new),
                                          static_cast<const uint16_t *>(v_new), cu_new, start_pos,
                                          to_internal(kv), B, total_new, max_new, max_pos, stream,
                                          cos_sin, rope_rows));
}

// A rotary table must cover every position the call uses: [0, max_pos).
int check_rope(const float *cos_sin, int32_t rope_rows, int32_t max_pos) {
  if (rope_rows <= 0 || max_pos > rope_rows) return RA_ERR_SHAPE;
  if (!cos_sin) return RA_ERR_NULL;
  return RA_OK;
}

}  // namespace

extern "C" {

int rollout_attn_append_write(const void *q, const void *k_new, const void *v_new,
                              const int32_t *cu_q, const int32_t *ctx_lens, const ra_paged_kv *kv,
                              int32_t B, int32_t Hq, int32_t total_q, int32_t max_q_len,
                              int32_t max_kv_len, float scale, float *out, float *lse,
                              void *workspace, size_t workspace_bytes, hipStream_t stream) {
  return append_write_impl(q, k_new, v_new, cu_q, ctx_lens, kv, B, Hq, total_q, max_q_len,
                           max_kv_len, scale, nullptr, 0, out, lse, workspace, workspace_bytes,
                           stream);
}

int rollout_attn_append_write_rope(const void *q, const void *k_new, const void *v_new,
                                   const int32_t *cu_q, const int32_t *ctx_lens,
                                   const ra_paged_kv *kv, int32_t B, int32_t Hq, int32_t total_q,
                                   int32_t max_q_len, int32_t max_kv_len, float scale,
                                   const float *cos_sin, int32_t rope_rows, float *out, float *lse,
                                   void *workspace, size_t workspace_bytes, hipStream_t stream) {
  const int r = check_rope(cos_sin, rope_rows, max_kv_len);
  if (r != RA_OK) return r;
  return append_write_impl(q, k_new, v_new, cu_q, ctx_lens, kv, B, Hq, total_q, max_q_len,
                           max_kv_len, scale, cos_sin, rope_rows, out, lse, workspace,
                           workspace_bytes, stream);
}

size_t rollout_attn_mixed_workspace_size(int32_t B_decode, int32_t B_append, int32_t Hq,
                                         int32_t Hkv_decode, int32_t Hkv_append,
                                         int32_t max_kv_len_decode, int32_t max_q_len) {
  if (B_decode < 0 || B_append < 0 || Hq <= 0 || max_kv_len_decode < 0 || max_q_len < 0)
    return 0;
  if (B_decode > 0 && (Hkv_decode <= 0 || Hq % Hkv_decode != 0)) return 0;
  if (B_append > 0 && (Hkv_append <= 0 || Hq % Hkv_append != 0)) return 0;
  if (B_decode == 0) Hkv_decode = B_append > 0 ? Hkv_append : 1;
  if (B_append == 0) Hkv_append = Hkv_decode;
  if (Hq / Hkv_append > 256) return 0;
  return ra::mixed_layout(B_decode, B_append, Hq, Hkv_decode, Hkv_append, max_kv_len_decode,
                          B_append > 0 ? max_q_len : 0)
      .bytes;
}

int rollout_attn_mixed(const void *q_decode, const ra_paged_kv *kv_decode,
                       const int32_t *kv_lens, int32_t B_decode, int32_t max_kv_len_decode,
                       float *out_decode, float *lse_decode, const void *q_append,
                       const int32_t *cu_q, const int32_t *ctx_lens, const ra_paged_kv *kv_append,
                       int32_t B_append, int32_t total_q, int32_t max_q_len,
                       int32_t max_kv_len_append, float *out_append, float *lse_append,
                       int32_t Hq, float scale, void *workspace, size_t workspace_bytes,
                       hipStream_t stream) {
  if (B_decode < 0 || B_append < 0 || Hq <= 0 || max_kv_len_decode < 0 || total_q < 0 ||
      max_q_len < 0 || max_kv_len_append < 0 || !std::isfinite(scale))
    return RA_ERR_SHAPE;
  const bool dec = B_decode > 0;
  const bool app = B_append > 0 && total_q > 0 && max_q_len > 0;
  int s;
  if (dec) {
    if ((s = check_kv(kv_decode)) != RA_OK) return s;
    if (!q_decode || !kv_lens || !out_decode) return RA_ERR_NULL;
    if (Hq % kv_decode->num_kv_heads != 0) return RA_ERR_SHAPE;
    if (Hq / kv_decode->num_kv_heads > 32 || B_decode > kMaxGridYZ) return RA_ERR_UNSUPPORTED;
    if (!positions_fit(kv_decode, max_kv_len_decode)) return RA_ERR_SHAPE;
  }
  if (app) {
    if ((s = check_kv(kv_append)) != RA_OK) return s;
    if (!q_append || !cu_q || !ctx_lens || !out_append) return RA_ERR_NULL;
    if (Hq % kv_append->num_kv_heads != 0) return RA_ERR_SHAPE;
    if (Hq / kv_append->num_kv_heads > 256) return RA_ERR_UNSUPPORTED;
    if (!positions_fit(kv_append, max_kv_len_append) || max_q_len > max_kv_len_append)
      return RA_ERR_SHAPE;
  }
  if (!dec && !app) return RA_OK;
  // one element type per call (the kernel is built for one)
  if (dec && app && is_fp8(kv_decode) != is_fp8(kv_append)) return RA_ERR_UNSUPPORTED;
  // an empty side borrows the other side's cache descriptor (never read)
  const ra::PagedKV kd = to_internal(dec ? kv_decode : kv_append);
  const ra::PagedKV ka = to_internal(app ? kv_append : kv_decode);
  if (kd.hkv > ra::mixed_hkv_limit() || ka.hkv > ra::mixed_hkv_limit())
    return RA_ERR_UNSUPPORTED;
  const int32_t Bd = dec ? B_decode : 0, Ba = app ? B_append : 0;
  const ra::MixedLayout layout = ra::mixed_layout(Bd, Ba, Hq, kd.hkv, ka.hkv, max_kv_len_decode,
                                                  app ? max_q_len : 0);
  // entries are named by int32 indices (and the counter runs one past the
  // end per workgroup); query blocks and splits by 23 bits
  if (layout.max_tiles + layout.max_splits > 0x7fffffff - 0xffff ||
      layout.qblocks >= (1 << 23) || layout.plan.max_splits >= (1 << 23))
    return RA_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < layout.bytes) return RA_ERR_WORKSPACE;
  return hip_status(ra::launch_mixed(
      static_cast<const uint16_t *>(q_decode), kd, kv_lens, Bd, max_kv_len_decode, out_decode,
      lse_decode, static_cast<const uint16_t *>(q_append), cu_q, ctx_lens, ka, Ba, total_q,
      max_q_len, max_kv_len_append, out_append, lse_append, Hq, scale, workspace, layout,
      stream));
}

size_t token_logprob_workspace_size(int32_t N, int32_t V, int32_t D) {
  if (N <= 0 || V <= 0 || D <= 0 || D % 64 != 0) return 0;
  return ra::logprob_workspace_bytes(N, V, D);
}

int token_logprob(const void *h, const void *W, const int32_t *targets, int32_t N, int32_t V,
                  int32_t D, float scale, float *logprob, float *lse, void *workspace,
                  size_t workspace_bytes, hipStream_t stream) {
  if (N < 0 || V <= 0 || D <= 0 || !std::isfinite(scale)) return RA_ERR_SHAPE;
  if (!h || !W || !targets || !logprob) return RA_ERR_NULL;
  if (D % 64 != 0) return RA_ERR_UNSUPPORTED;
  if (N == 0) return RA_OK;
  if (ra::logprob_grid(N, V) > 0x7fffffff) return RA_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < ra::logprob_workspace_bytes(N, V, D)) return RA_ERR_WORKSPACE;
  return hip_status(ra::launch_logprob(static_cast<const uint16_t *>(h),
                                       static_cast<const uint16_t *>(W), targets, N, V, D, scale,
                                       logprob, lse, workspace, false, stream));
}

size_t token_logprob_packed_weight_size(int32_t V, int32_t D) {
  if (V <= 0 || D <= 0 || D % 64 != 0) return 0;
  return ra::logprob_packed_bytes(V, D);
}

int token_logprob_pack_weight(const void *W, int32_t V, int32_t D, void *W_packed,
                              size_t packed_bytes, hipStream_t stream) {
  if (V <= 0 || D <= 0) return RA_ERR_SHAPE;
  if (!W || !W_packed) return RA_ERR_NULL;
  if (D % 64 != 0) return RA_ERR_UNSUPPORTED;
  if (packed_bytes < ra::logprob_packed_bytes(V, D)) return RA_ERR_WORKSPACE;
  return hip_status(ra::launch_logprob_pack(static_cast<const uint16_t *>(W), V, D,
                                            static_cast<uint16_t *>(W_packed), stream));
}

int token_logprob_packed(const void *h, const void *W_packed, const int32_t *targets, int32_t N,
                         int32_t V, int32_t D, float scale, float *logprob, float *lse,
                         void *workspace, size_t workspace_bytes, hipStream_t stream) {
  if (N < 0 || V <= 0 || D <= 0 || !std::isfinite(scale)) return RA_ERR_SHAPE;
  if (!h || !W_packed || !targets || !logprob) return RA_ERR_NULL;
  if (D % 64 != 0) return RA_ERR_UNSUPPORTED;
  if (N == 0) return RA_OK;
  if (ra::logprob_grid(N, V) > 0x7fffffff) return RA_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < ra::logprob_workspace_bytes(N, V, D)) return RA_ERR_WORKSPACE;
  return hip_status(ra::launch_logprob(static_cast<const uint16_t *>(h),
                                       static_cast<const uint16_t *>(W_packed), targets, N, V, D,
                                       scale, logprob, lse, workspace, true, stream));
}

int kv_page_write(const void *k_new, const void *v_new, const int32_t *cu_new,
                  const int32_t *start_pos, const ra_paged_kv *kv, int32_t B, int32_t total_new,
                  int32_t max_new, int32_t max_pos, hipStream_t stream) {
  return page_write_impl(k_new, v_new, cu_new, start_pos, kv, B, total_new, max_new, max_pos,
                         nullptr, 0, stream);
}

int kv_page_write_rope(const void *k_new, const void *v_new, const int32_t *cu_new,
                       const int32_t *start_pos, const ra_paged_kv *kv, int32_t B,
                       int32_t total_new, int32_t max_new, int32_t max_pos, const float *cos_sin,
                       int32_t rope_rows, hipStream_t stream) {
  const int r = check_rope(cos_sin, rope_rows, max_pos);
  if (r != RA_OK) return r;
  return page_write_impl(k_new, v_new, cu_new, start_pos, kv, B, total_new, max_new, max_pos,
                         cos_sin, rope_rows, stream);
}

int kv_page_gather(const ra_paged_kv *kv, const int32_t *lens, const int32_t *cu_out, int32_t B,
                   int32_t total, int32_t max_len, void *k_out, void *v_out,
                   hipStream_t stream) {
  if (B < 0 || total < 0 || max_len < 0) return RA_ERR_SHAPE;
  int s = check_kv(kv);
  if (s != RA_OK) return s;
  if (!lens || !cu_out || !k_out || !v_out) return RA_ERR_NULL;
  if (B > kMaxGridYZ) return RA_ERR_UNSUPPORTED;
  if (!positions_fit(kv, max_len)) return RA_ERR_SHAPE;
  if (B == 0 || total == 0 || max_len == 0) return RA_OK;
  return hip_status(ra::launch_page_gather(to_internal(kv), lens, cu_out, B, total, max_len,
                                           static_cast<uint16_t *>(k_out),
                                           static_cast<uint16_t *>(v_out), stream));
}

}  // extern "C"
