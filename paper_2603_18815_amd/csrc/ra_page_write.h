// Page write of one (row, page, KV head) block of K/V, shared by the page
// write kernel and the planned append launch that writes the chunks itself.
// 256 threads move one block: K rows go to the token-major page 16 source
// bytes per lane; V tokens go through LDS so that the dim-major page is
// written in 8- or 16-byte pieces per lane as well (partial pages: element
// stores on the touched slots only).
// bf16 pools: bit copies. fp8 pools (kFp8): each bf16 element is stored as
// its E4M3 code of x * fp32(1 / scale) (round to nearest even, saturated).
// With a rotary table (kRope), each K row is first rotated at its position
// (rope8: dims i and i + 64 paired, fp32 products and sum, bf16 result) and
// the rotated row is written as above; V is written as it comes.
#pragma once

#include "ra_device.h"
#include "ra_internal.h"

namespace ra {
namespace pwrite {

constexpr int kItemThreads = 256;
constexpr int kVPitch = kHeadDim + 8;   // LDS row pitch (elements) of the staged V slots

struct WriteArgs {
  const uint16_t *k_new, *v_new;       // bf16 [total_new][Hkv][128]
  const int32_t *cu_new, *start_pos;
  uint16_t *k_pool, *v_pool;           // bf16 elements, or E4M3 bytes (fp8 pools)
  const int32_t *block_table;
  int32_t bt_stride, num_pages, hkv, total_new, max_new, max_pos;
  bool fp8;                            // the pools hold E4M3 codes
  float k_inv, v_inv;                  // fp8 pools: fp32(1 / k_scale), fp32(1 / v_scale)
  const float *cos_sin;                // rotary table [rope_rows][128] (cos | sin), or null
  int32_t rope_rows;
};

// Write arguments for pool kv (the reciprocal scales are taken in fp32, as
// the quantization rule states).
inline WriteArgs write_args(const uint16_t *k_new, const uint16_t *v_new, const int32_t *cu_new,
                            const int32_t *start_pos, const PagedKV &kv, int32_t total_new,
                            int32_t max_new, int32_t max_pos, const float *cos_sin = nullptr,
                            int32_t rope_rows = 0) {
  WriteArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.cu_new = cu_new;
  a.start_pos = start_pos;
  a.k_pool = kv.k_pool;
  a.v_pool = kv.v_pool;
  a.block_table = kv.block_table;
  a.bt_stride = kv.bt_stride;
  a.num_pages = kv.num_pages;
  a.hkv = kv.hkv;
  a.total_new = total_new;
  a.max_new = max_new;
  a.max_pos = max_pos;
  a.fp8 = kv.fp8;
  a.k_inv = kv.fp8 ? 1.0f / kv.k_scale : 1.f;
  a.v_inv = kv.fp8 ? 1.0f / kv.v_scale : 1.f;
  a.cos_sin = cos_sin;
  a.rope_rows = rope_rows;
  return a;
}

// The block: row b's page s / 16 + chunk (row-relative), KV head g; tokens
// [lo, hi) of that page are written (positions), cu0 + (pos - s) the source.
struct WriteItem {
  bool active;
  int cu0, s, pg, lo, hi, id;
};

// Row extent clamped so that no access leaves the caller's arrays.
__device__ __forceinline__ WriteItem write_item(const WriteArgs &a, int chunk, int b) {
  WriteItem it;
  it.active = false;
  it.cu0 = min(max(a.cu_new[b], 0), a.total_new);
  const int n = min(min(max(a.cu_new[b + 1] - it.cu0, 0), a.max_new), a.total_new - it.cu0);
  if (n <= 0) return it;
  it.s = min(max(a.start_pos[b], 0), a.max_pos - n);
  if (it.s < 0) return it;
  it.pg = it.s / kPage + chunk;
  if (it.pg > (it.s + n - 1) / kPage) return it;
  it.lo = max(it.s, it.pg * kPage);
  it.hi = min(it.s + n, it.pg * kPage + kPage);
  it.id = clamp_page(a.block_table[(size_t)b * a.bt_stride + it.pg], a.num_pages);
  it.active = true;
  return it;
}

// Phase 1 (thread t of 256): K rows to the page, V tokens into LDS.
template <bool kFp8, bool kRope = false>
__device__ __forceinline__ void write_phase1(const WriteArgs &a, const WriteItem &it, int g,
                                             int t, uint16_t (*sv)[kVPitch]) {
  const int slot = t >> 4, ch = t & 15;            // token slot, 8-element chunk
  const int pos = it.pg * kPage + slot;
  if (pos >= it.lo && pos < it.hi) {
    const size_t row = ((size_t)(it.cu0 + pos - it.s) * a.hkv + g) * kHeadDim;
    const size_t src = row + ch * 8;
    const size_t dst = (((size_t)it.id * a.hkv + g) * kPage + slot) * kHeadDim + ch * 8;
    u32x4 k = load_u32x4(a.k_new + src);
    if constexpr (kRope) {
      // this chunk's dims 8 ch + 0..7 pair with chunk ch ^ 8; frequency index
      // 8 (ch % 8) + 0..7
      const u32x4 partner = load_u32x4(a.k_new + row + (ch ^ 8) * 8);
      const float *cs = a.cos_sin + (size_t)min(pos, a.rope_rows - 1) * kHeadDim + (ch & 7) * 8;
      const f32x8 c = *reinterpret_cast<const f32x8 *>(cs);
      const f32x8 sn = *reinterpret_cast<const f32x8 *>(cs + kHeadDim / 2);
      k = __builtin_bit_cast(u32x4, rope8(__builtin_bit_cast(bf16x8, k),
                                          __builtin_bit_cast(bf16x8, partner), c, sn, ch >= 8));
    }
    if constexpr (kFp8)
      *reinterpret_cast<u32x2 *>(reinterpret_cast<uint8_t *>(a.k_pool) + dst) =
          quantize8(k, a.k_inv);
    else
      store_u32x4(a.k_pool + dst, k);
    *reinterpret_cast<u32x4 *>(&sv[slot][ch * 8]) = load_u32x4(a.v_new + src);
  }
}

// Phase 2 (after a barrier): the V page is [d][slot]; thread t -> one d row,
// eight slots.
template <bool kFp8>
__device__ __forceinline__ void write_phase2(const WriteArgs &a, const WriteItem &it, int g,
                                             int t, const uint16_t (*sv)[kVPitch]) {
  const int d = t >> 1, s0 = (t & 1) * 8;
  const size_t off = (((size_t)it.id * a.hkv + g) * kHeadDim + d) * kPage + s0;
  const int p0 = it.pg * kPage + s0;
  u32x4 w;
#pragma unroll
  for (int e = 0; e < 4; ++e)
    w[e] = (uint32_t)sv[s0 + 2 * e][d] | ((uint32_t)sv[s0 + 2 * e + 1][d] << 16);
  const bool whole = p0 >= it.lo && p0 + 8 <= it.hi;
  if constexpr (kFp8) {
    uint8_t *dst = reinterpret_cast<uint8_t *>(a.v_pool) + off;
    const u32x2 q = quantize8(w, a.v_inv);
    if (whole) {
      *reinterpret_cast<u32x2 *>(dst) = q;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (p0 + e >= it.lo && p0 + e < it.hi) dst[e] = (uint8_t)(q[e >> 2] >> (8 * (e & 3)));
    }
  } else {
    uint16_t *dst = a.v_pool + off;
    if (whole) {
      store_u32x4(dst, w);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (p0 + e >= it.lo && p0 + e < it.hi) dst[e] = sv[s0 + e][d];
    }
  }
}

}  // namespace pwrite
}  // namespace ra
