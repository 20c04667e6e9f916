// Page write and page gather between packed token-major K/V rows and the
// paged pools (K pages token-major [16][128], V pages dim-major [128][16]).
// One workgroup moves one (row, page, KV head) block per pool; V goes through
// LDS so that both sides are accessed in 8- or 16-byte pieces per lane.
// bf16 pools: bit copies. fp8 pools: the write quantizes each bf16 element to
// its E4M3 code (x * fp32(1 / scale), round to nearest even, saturated; the
// block code is shared with the fused append launch), the gather copies the
// codes out.
#include "ra_device.h"
#include "ra_internal.h"
#include "ra_page_write.h"

namespace ra {
namespace {

constexpr int kThreads = 256;
constexpr int kVPitch = kHeadDim + 8;  // LDS row pitch (elements) of the staged V slots

// One (row, page, KV head) block per workgroup.
template <bool kFp8, bool kRope>
__global__ __launch_bounds__(pwrite::kItemThreads) void page_write_kernel(pwrite::WriteArgs a) {
  const pwrite::WriteItem it = pwrite::write_item(a, blockIdx.x, blockIdx.z);
  if (!it.active) return;
  __shared__ uint16_t sv[kPage][pwrite::kVPitch];
  pwrite::write_phase1<kFp8, kRope>(a, it, blockIdx.y, threadIdx.x, sv);
  __syncthreads();
  pwrite::write_phase2<kFp8>(a, it, blockIdx.y, threadIdx.x, sv);
}

__global__ __launch_bounds__(kThreads) void page_gather_kernel(
    const uint16_t *__restrict__ k_pool, const uint16_t *__restrict__ v_pool,
    const int32_t *__restrict__ block_table, int bt_stride, int num_pages, int hkv,
    const int32_t *__restrict__ lens, const int32_t *__restrict__ cu_out, int total, int max_len,
    uint16_t *__restrict__ k_out, uint16_t *__restrict__ v_out) {
  const int pg = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int cu0 = min(max(cu_out[b], 0), total);
  const int L = min(min(max(lens[b], 0), max_len), total - cu0);
  if (pg * kPage >= L) return;
  const int id = clamp_page(block_table[(size_t)b * bt_stride + pg], num_pages);

  __shared__ uint16_t sv[kPage][kVPitch];
  {
    const int d = tid >> 1, s0 = (tid & 1) * 8;
    const u32x4 w = load_u32x4(v_pool + (((size_t)id * hkv + g) * kHeadDim + d) * kPage + s0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sv[s0 + 2 * e][d] = (uint16_t)(w[e] & 0xffffu);
      sv[s0 + 2 * e + 1][d] = (uint16_t)(w[e] >> 16);
    }
  }
  __syncthreads();
  const int slot = tid >> 4, ch = tid & 15;
  const int pos = pg * kPage + slot;
  if (pos < L) {
    const size_t dst = ((size_t)(cu0 + pos) * hkv + g) * kHeadDim + ch * 8;
    const size_t src = (((size_t)id * hkv + g) * kPage + slot) * kHeadDim + ch * 8;
    store_u32x4(k_out + dst, load_u32x4(k_pool + src));
    store_u32x4(v_out + dst, *reinterpret_cast<const u32x4 *>(&sv[slot][ch * 8]));
  }
}

__global__ __launch_bounds__(kThreads) void page_gather_fp8_kernel(
    const uint8_t *__restrict__ k_pool, const uint8_t *__restrict__ v_pool,
    const int32_t *__restrict__ block_table, int bt_stride, int num_pages, int hkv,
    const int32_t *__restrict__ lens, const int32_t *__restrict__ cu_out, int total, int max_len,
    uint8_t *__restrict__ k_out, uint8_t *__restrict__ v_out) {
  const int pg = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int cu0 = min(max(cu_out[b], 0), total);
  const int L = min(min(max(lens[b], 0), max_len), total - cu0);
  if (pg * kPage >= L) return;
  const int id = clamp_page(block_table[(size_t)b * bt_stride + pg], num_pages);

  __shared__ uint8_t sv[kPage][kHeadDim + 16];
  {
    const int d = tid >> 1, s0 = (tid & 1) * 8;
    const u32x2 w = *reinterpret_cast<const u32x2 *>(
        v_pool + (((size_t)id * hkv + g) * kHeadDim + d) * kPage + s0);
#pragma unroll
    for (int e = 0; e < 8; ++e) sv[s0 + e][d] = (uint8_t)(w[e >> 2] >> (8 * (e & 3)));
  }
  __syncthreads();
  const int slot = tid >> 4, ch = tid & 15;
  const int pos = pg * kPage + slot;
  if (pos < L) {
    const size_t dst = ((size_t)(cu0 + pos) * hkv + g) * kHeadDim + ch * 8;
    const size_t src = (((size_t)id * hkv + g) * kPage + slot) * kHeadDim + ch * 8;
    *reinterpret_cast<u32x2 *>(k_out + dst) = *reinterpret_cast<const u32x2 *>(k_pool + src);
    *reinterpret_cast<u32x2 *>(v_out + dst) = *reinterpret_cast<const u32x2 *>(&sv[slot][ch * 8]);
  }
}

}  // namespace

hipError_t launch_page_write(const uint16_t *k_new, const uint16_t *v_new, const int32_t *cu_new,
                             const int32_t *start_pos, const PagedKV &kv, int32_t B,
                             int32_t total_new, int32_t max_new, int32_t max_pos,
                             hipStream_t stream, const float *cos_sin, int32_t rope_rows) {
  // A run of n tokens touches at most (n - 1) / 16 + 2 pages.
  const dim3 grid((unsigned)(((int64_t)max_new + kPage - 1) / kPage + 1), kv.hkv, B);
  const pwrite::WriteArgs a = pwrite::write_args(k_new, v_new, cu_new, start_pos, kv, total_new,
                                                 max_new, max_pos, cos_sin, rope_rows);
  const dim3 block(pwrite::kItemThreads);
  if (kv.fp8 && cos_sin)
    hipLaunchKernelGGL((page_write_kernel<true, true>), grid, block, 0, stream, a);
  else if (kv.fp8)
    hipLaunchKernelGGL((page_write_kernel<true, false>), grid, block, 0, stream, a);
  else if (cos_sin)
    hipLaunchKernelGGL((page_write_kernel<false, true>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((page_write_kernel<false, false>), grid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_page_gather(const PagedKV &kv, const int32_t *lens, const int32_t *cu_out,
                              int32_t B, int32_t total, int32_t max_len, uint16_t *k_out,
                              uint16_t *v_out, hipStream_t stream) {
  const dim3 grid((unsigned)(((int64_t)max_len + kPage - 1) / kPage), kv.hkv, B);
  if (kv.fp8)
    hipLaunchKernelGGL(page_gather_fp8_kernel, grid, dim3(kThreads), 0, stream,
                       reinterpret_cast<const uint8_t *>(kv.k_pool),
                       reinterpret_cast<const uint8_t *>(kv.v_pool), kv.block_table, kv.bt_stride,
                       kv.num_pages, kv.hkv, lens, cu_out, total, max_len,
                       reinterpret_cast<uint8_t *>(k_out), reinterpret_cast<uint8_t *>(v_out));
  else
    hipLaunchKernelGGL(page_gather_kernel, grid, dim3(kThreads), 0, stream, kv.k_pool, kv.v_pool,
                       kv.block_table, kv.bt_stride, kv.num_pages, kv.hkv, lens, cu_out, total,
                       max_len, k_out, v_out);
  return hipGetLastError();
}

}  // namespace ra
