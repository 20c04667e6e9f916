// Page write of one (row, page, KV head) block of bf16 K/V, shared by the
// page write kernel and the planned append launch that writes the chunks
// itself. 256 threads move one block: K rows are copied 16 bytes per lane
// into the token-major page; V tokens go through LDS so that the dim-major
// page is written 16 bytes per lane as well (partial pages: 2-byte stores on
// the touched slots only).
#pragma once

#include "ra_device.h"

namespace ra {
namespace pwrite {

constexpr int kItemThreads = 256;
constexpr int kVPitch = kHeadDim + 8;   // LDS row pitch (elements) of the staged V slots

struct WriteArgs {
  const uint16_t *k_new, *v_new;       // bf16 [total_new][Hkv][128]
  const int32_t *cu_new, *start_pos;
  uint16_t *k_pool, *v_pool;
  const int32_t *block_table;
  int32_t bt_stride, num_pages, hkv, total_new, max_new, max_pos;
};

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
__device__ __forceinline__ void write_phase1(const WriteArgs &a, const WriteItem &it, int g,
                                             int t, uint16_t (*sv)[kVPitch]) {
  const int slot = t >> 4, ch = t & 15;            // token slot, 16-byte chunk
  const int pos = it.pg * kPage + slot;
  if (pos >= it.lo && pos < it.hi) {
    const size_t src = ((size_t)(it.cu0 + pos - it.s) * a.hkv + g) * kHeadDim + ch * 8;
    const size_t dst = (((size_t)it.id * a.hkv + g) * kPage + slot) * kHeadDim + ch * 8;
    store_u32x4(a.k_pool + dst, load_u32x4(a.k_new + src));
    *reinterpret_cast<u32x4 *>(&sv[slot][ch * 8]) = load_u32x4(a.v_new + src);
  }
}

// Phase 2 (after a barrier): the V page is [d][slot]; thread t -> one d row,
// eight slots.
__device__ __forceinline__ void write_phase2(const WriteArgs &a, const WriteItem &it, int g,
                                             int t, const uint16_t (*sv)[kVPitch]) {
  const int d = t >> 1, s0 = (t & 1) * 8;
  uint16_t *dst = a.v_pool + (((size_t)it.id * a.hkv + g) * kHeadDim + d) * kPage + s0;
  const int p0 = it.pg * kPage + s0;
  if (p0 >= it.lo && p0 + 8 <= it.hi) {
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = (uint32_t)sv[s0 + 2 * e][d] | ((uint32_t)sv[s0 + 2 * e + 1][d] << 16);
    store_u32x4(dst, w);
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (p0 + e >= it.lo && p0 + e < it.hi) dst[e] = sv[s0 + e][d];
  }
}

}  // namespace pwrite
}  // namespace ra
