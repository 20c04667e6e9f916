// Planned persistent launches: append rows alone, or one rollout step's
// decode rows (one new token each) and append rows (a chunk of new
// observation tokens each) together, against their paged caches.
//
// A plan kernel (one workgroup) lists the work of the call from the
// device-resident lengths, in one queue per XCD; queue q takes KV heads
// q, q + 8, q + 16, ...:
//   - append tiles (row, query block, KV head): the rows sorted by the key
//     blocks of their longest (last) tile, longest first (a counting sort),
//     each row's query blocks last first. The long tiles start early and the
//     short ones fill the end, and the tiles of one row and head follow each
//     other, so that the CUs of an XCD walk the same pages of K/V at about
//     the same time and share them through the XCD's L2;
//   - decode splits (row, split, KV head), row by row.
// The attention kernel then runs one workgroup of 8 waves per CU. Workgroups
// are placed on the XCDs round robin, so workgroup w starts on queue w mod 8
// and, once that queue is used up, takes what is left in the others. In each
// queue the workgroups take the next entry of one merged order from a device
// counter. The merged order places the decode splits at even spacing among
// the append tiles, so that a few CUs stream KV pages for decode (bound by
// HBM) while the rest run the append tiles' matrix products (bound by the
// matrix cores). Entry j of a queue's merged order (n entries, nd of them
// decode splits) is decode split floor(j nd / n) when
// floor((j + 1) nd / n) > floor(j nd / n), else append tile
// j - floor(j nd / n).
// A decode split is computed as by the decode split kernel but with 8 waves;
// the decode combine follows as in plain decode. Results do not depend on
// the order in which entries are taken.
#include <atomic>

#include "ra_append_tile.h"
#include "ra_decode_split.h"
#include "ra_internal.h"
#include "ra_page_write.h"

namespace ra {
namespace {

constexpr int kMixWaves = 8;
constexpr int kMixThreads = kMixWaves * kWave;
static_assert(kMixThreads == atile::kThreads, "append tiles take the whole workgroup");
constexpr int kPlanThreads = 1024;
constexpr int kCostBuckets = 4096;   // key-block counts above this share the last bucket
constexpr int kHeadBits = 8;         // entry = {row, index << kHeadBits | KV head}
constexpr int kQueues = 8;           // one work queue per XCD

struct MixedArgs {
  atile::AppendArgs ap;
  dsplit::DecodeArgs de;
  int2 *tiles;      // append tiles, one segment per queue
  int2 *splits;     // decode splits, one segment per queue
  int32_t *order;   // append rows, longest chunk end first
  int32_t *header;  // per queue q: [q] next entry, [8+q] tiles, [16+q] splits,
                    // [24+q] tile segment start, [32+q] split segment start
  int32_t B_append, qblocks;
};

// Exclusive prefix sum of v over the kPlanThreads threads of the workgroup;
// *total receives the sum of all. Every thread calls it.
__device__ int block_exclusive_scan(int v, int *s, int *total) {
  const int tid = threadIdx.x;
  s[tid] = v;
  __syncthreads();
  for (int off = 1; off < kPlanThreads; off *= 2) {
    const int t = tid >= off ? s[tid - off] : 0;
    __syncthreads();
    s[tid] += t;
    __syncthreads();
  }
  const int incl = s[tid];
  *total = s[kPlanThreads - 1];
  __syncthreads();   // s may be reused by the caller
  return incl - v;
}

// KV heads g = q, q + 8, ... below hkv go to queue q.
__device__ __forceinline__ int heads_of_queue(int hkv, int q) {
  return q < hkv ? (hkv - 1 - q) / kQueues + 1 : 0;
}

// Query blocks of row b with work (0 for an empty row).
__device__ __forceinline__ int row_qblocks(const atile::AppendArgs &ap, const atile::AppendRow &r) {
  if (r.T <= 0 || r.ctx < 0) return 0;
  return (r.T + ap.q_per_block - 1) / ap.q_per_block;
}

// Workgroup 0 plans. With the page write fused in (write_chunks > 0), every
// other workgroup writes four (row, page, KV head) blocks of the chunks' K/V
// meanwhile; the attention kernel after this one reads them from the pool.
__global__ __launch_bounds__(kPlanThreads) void mixed_plan_kernel(MixedArgs m, pwrite::WriteArgs w,
                                                                  int32_t write_chunks) {
  if (blockIdx.x > 0) {
    constexpr int kPer = kPlanThreads / pwrite::kItemThreads;
    __shared__ uint16_t sv[kPer][kPage][pwrite::kVPitch];
    const int part = threadIdx.x / pwrite::kItemThreads, t = threadIdx.x % pwrite::kItemThreads;
    const int64_t item = (int64_t)(blockIdx.x - 1) * kPer + part;   // (row, head, page)
    pwrite::WriteItem it;
    it.active = false;
    int g = 0;
    if (item < (int64_t)m.B_append * w.hkv * write_chunks) {
      const int64_t bg = item / write_chunks;
      g = (int)(bg % w.hkv);
      it = pwrite::write_item(w, (int)(item % write_chunks), (int)(bg / w.hkv));
    }
    if (it.active) {
      if (w.fp8 && w.cos_sin)
        pwrite::write_phase1<true, true>(w, it, g, t, sv[part]);
      else if (w.fp8)
        pwrite::write_phase1<true, false>(w, it, g, t, sv[part]);
      else if (w.cos_sin)
        pwrite::write_phase1<false, true>(w, it, g, t, sv[part]);
      else
        pwrite::write_phase1<false, false>(w, it, g, t, sv[part]);
    }
    __syncthreads();
    if (it.active) {
      if (w.fp8)
        pwrite::write_phase2<true>(w, it, g, t, sv[part]);
      else
        pwrite::write_phase2<false>(w, it, g, t, sv[part]);
    }
    return;
  }
  __shared__ int count[kCostBuckets];   // rows per key-block count, then write cursors
  __shared__ int s_scan[kPlanThreads];
  __shared__ int s_total;
  const int tid = threadIdx.x;
  const int hkv_a = m.ap.hkv, hkv_d = m.de.hkv;
  for (int c = tid; c < kCostBuckets; c += kPlanThreads) count[c] = 0;
  if (tid == 0) s_total = 0;
  __syncthreads();

  // ---- append rows, by the key blocks of their longest (last) tile, longest first
  for (int b = tid; b < m.B_append; b += kPlanThreads) {
    const atile::AppendRow r = atile::append_row(m.ap, b);
    const int nq = row_qblocks(m.ap, r);
    if (nq == 0) continue;
    const int nb = atile::append_tile_blocks(m.ap, r, nq - 1);
    atomicAdd(&count[min(nb, kCostBuckets) - 1], 1);
    atomicAdd(&s_total, nq);
  }
  __syncthreads();
  const int total_nq = s_total;
  constexpr int kPer = kCostBuckets / kPlanThreads;
  int own[kPer], sum = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    own[k] = count[kCostBuckets - 1 - (kPer * tid + k)];
    sum += own[k];
  }
  int n_rows;
  int cursor = block_exclusive_scan(sum, s_scan, &n_rows);
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    count[kCostBuckets - 1 - (kPer * tid + k)] = cursor;
    cursor += own[k];
  }
  __syncthreads();
  for (int b = tid; b < m.B_append; b += kPlanThreads) {
    const atile::AppendRow r = atile::append_row(m.ap, b);
    const int nq = row_qblocks(m.ap, r);
    if (nq == 0) continue;
    const int nb = atile::append_tile_blocks(m.ap, r, nq - 1);
    m.order[atomicAdd(&count[min(nb, kCostBuckets) - 1], 1)] = b;
  }
  __syncthreads();
  // ---- tiles: queue q holds heads q, q + 8, ...; in it, rows in the order
  // above, each row's query blocks last first, then its heads
  int seg_a[kQueues], acc = 0;
#pragma unroll
  for (int q = 0; q < kQueues; ++q) {
    seg_a[q] = acc;
    acc += heads_of_queue(hkv_a, q) * total_nq;
  }
  int done = 0;   // query blocks of the rows ranked before this chunk
  for (int k0 = 0; k0 < n_rows; k0 += kPlanThreads) {
    const int k = k0 + tid;
    const int b = k < n_rows ? m.order[k] : 0;
    const int nq = k < n_rows ? row_qblocks(m.ap, atile::append_row(m.ap, b)) : 0;
    int chunk;
    const int before = done + block_exclusive_scan(nq, s_scan, &chunk);
    for (int i = 0; i < nq; ++i) {
      const int qb = nq - 1 - i;
      for (int g = 0; g < hkv_a; ++g) {
        const int q = g % kQueues, hq = heads_of_queue(hkv_a, q);
        m.tiles[(size_t)seg_a[q] + (size_t)(before + i) * hq + g / kQueues] =
            make_int2(b, qb << kHeadBits | g);
      }
    }
    done += chunk;
  }

  // ---- decode splits: queue q holds heads q, q + 8, ...; rows in order
  int total_ns = 0;
  const int S = m.de.split_tokens;
  for (int r0 = 0; r0 < m.de.B; r0 += kPlanThreads) {
    const int b = r0 + tid;
    const int ns = b < m.de.B ? (dsplit::row_len(m.de, b) + S - 1) / S : 0;
    int chunk;
    block_exclusive_scan(ns, s_scan, &chunk);
    total_ns += chunk;
  }
  int seg_d[kQueues];
  acc = 0;
#pragma unroll
  for (int q = 0; q < kQueues; ++q) {
    seg_d[q] = acc;
    acc += heads_of_queue(hkv_d, q) * total_ns;
  }
  done = 0;
  for (int r0 = 0; r0 < m.de.B; r0 += kPlanThreads) {
    const int b = r0 + tid;
    const int ns = b < m.de.B ? (dsplit::row_len(m.de, b) + S - 1) / S : 0;
    int chunk;
    const int before = done + block_exclusive_scan(ns, s_scan, &chunk);
    for (int s = 0; s < ns; ++s)
      for (int g = 0; g < hkv_d; ++g) {
        const int q = g % kQueues, hq = heads_of_queue(hkv_d, q);
        m.splits[(size_t)seg_d[q] + (size_t)(before + s) * hq + g / kQueues] =
            make_int2(b, s << kHeadBits | g);
      }
    done += chunk;
  }
  if (tid < kQueues) {
    m.header[tid] = 0;
    m.header[8 + tid] = heads_of_queue(hkv_a, tid) * total_nq;
    m.header[16 + tid] = heads_of_queue(hkv_d, tid) * total_ns;
    m.header[24 + tid] = seg_a[tid];
    m.header[32 + tid] = seg_d[tid];
  }
}

// kDecode: the call has decode rows (otherwise every entry is an append tile).
// kFp8: the pools hold E4M3 codes. kRope: the append rows' q is rotated at its
// position (append-only calls). kDecodeTiles: 16-column tiles of a decode
// split (2 for groups of 17 to 32 query heads).
template <bool kPosScale, bool kDecode, bool kFp8, bool kRope = false, int kDecodeTiles = 1>
__global__ __launch_bounds__(kMixThreads, 1) void mixed_kernel(MixedArgs m) {
  __shared__ union {
    atile::AppendLds ap;
    dsplit::DecodeLds<kDecodeTiles, kMixWaves> de;
  } lds;
  __shared__ int s_next;
  // workgroups are placed on the XCDs round robin: start with this XCD's
  // queue, then take what is left in the others
  const int x = blockIdx.x % kQueues;
  for (int qi = 0; qi < kQueues; ++qi) {
    const int q = (x + qi) % kQueues;
    const int na = m.header[8 + q], nd = m.header[16 + q];
    const int64_t n = (int64_t)na + nd;
    const int2 *tiles = m.tiles + m.header[24 + q];
    const int2 *splits = m.splits + m.header[32 + q];
    for (;;) {
      __syncthreads();   // the previous entry is done with LDS and s_next
      if (threadIdx.x == 0) s_next = n > 0 ? atomicAdd(&m.header[q], 1) : 0;
      __syncthreads();
      const int j = __builtin_amdgcn_readfirstlane(s_next);
      if (j >= n) break;
      const int dj = (int)((int64_t)j * nd / n);
      if (kDecode && (int)(((int64_t)j + 1) * nd / n) > dj) {
        const int2 e = splits[dj];
        dsplit::decode_split<kDecodeTiles, false, kMixWaves, kFp8>(m.de,
                                                                   e.y & ((1 << kHeadBits) - 1),
                                                        e.y >> kHeadBits, e.x, lds.de);
      } else {
        const int2 e = tiles[j - dj];
        atile::append_tile<kPosScale, kFp8, kRope>(m.ap, e.y >> kHeadBits,
                                            e.y & ((1 << kHeadBits) - 1), e.x, lds.ap);
      }
    }
  }
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Compute units of the current device, queried once per device (a device's
// count never changes; racing first calls store the same value).
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];
hipError_t device_cus(int *cus) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices)
    return hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
  int n = g_cus[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if ((e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
      return e;
    g_cus[dev].store(n, std::memory_order_relaxed);
  }
  *cus = n;
  return hipSuccess;
}

}  // namespace

MixedLayout mixed_layout(int32_t B_decode, int32_t B_append, int32_t hq, int32_t hkv_decode,
                         int32_t hkv_append, int32_t max_kv_len_decode, int32_t max_q_len) {
  MixedLayout l;
  l.plan = decode_plan(B_decode > 0 ? B_decode : 1, hkv_decode, max_kv_len_decode);
  const int32_t qpb = atile::kRowsPerGroup / (hq / hkv_append);
  l.qblocks = max_q_len > 0 ? (int32_t)(((int64_t)max_q_len + qpb - 1) / qpb) : 0;
  l.max_tiles = (int64_t)B_append * l.qblocks * hkv_append;
  l.max_splits = (int64_t)B_decode * l.plan.max_splits * hkv_decode;
  l.tiles_offset = kAlign + align_up((size_t)(B_append > 0 ? B_append : 0) * sizeof(int32_t));
  l.splits_offset = l.tiles_offset + align_up((size_t)l.max_tiles * sizeof(int2));
  l.partials_offset = l.splits_offset + align_up((size_t)l.max_splits * sizeof(int2));
  l.bytes = l.partials_offset +
            (B_decode > 0 ? decode_workspace_bytes(B_decode, hq, l.plan) : 0);
  return l;
}

int32_t mixed_hkv_limit() { return 1 << kHeadBits; }

hipError_t launch_mixed(const uint16_t *q_decode, const PagedKV &kv_decode,
                        const int32_t *kv_lens, int32_t B_decode, int32_t max_kv_len_decode,
                        float *out_decode, float *lse_decode, const uint16_t *q_append,
                        const int32_t *cu_q, const int32_t *ctx_lens, const PagedKV &kv_append,
                        int32_t B_append, int32_t total_q, int32_t max_q_len,
                        int32_t max_kv_len_append, float *out_append, float *lse_append,
                        int32_t hq, float scale, void *workspace, const MixedLayout &layout,
                        hipStream_t stream, const uint16_t *k_new, const uint16_t *v_new,
                        const float *cos_sin, int32_t rope_rows) {
  char *ws = static_cast<char *>(workspace);
  MixedArgs m;
  m.ap = atile::make_append_args(q_append, cu_q, ctx_lens, kv_append, hq, total_q, max_q_len,
                                 max_kv_len_append, scale, out_append, lse_append);
  m.ap.cos_sin = cos_sin;   // q of the append rows rotated at their positions (or not)
  m.ap.rope_rows = rope_rows;
  m.de = dsplit::make_decode_args(q_decode, kv_decode, kv_lens, B_decode, hq,
                                  max_kv_len_decode, scale, ws + layout.partials_offset,
                                  layout.plan.max_splits, layout.plan);
  m.header = reinterpret_cast<int32_t *>(ws);
  m.tiles = reinterpret_cast<int2 *>(ws + layout.tiles_offset);
  m.order = reinterpret_cast<int32_t *>(ws + kAlign);
  m.splits = reinterpret_cast<int2 *>(ws + layout.splits_offset);
  m.B_append = B_append;
  m.qblocks = layout.qblocks;

  // the fused page write (append rows only): the chunks' tokens at ctx_lens
  const pwrite::WriteArgs w = pwrite::write_args(k_new, v_new, cu_q, ctx_lens, kv_append, total_q,
                                                 max_q_len, max_kv_len_append, cos_sin, rope_rows);
  const int32_t write_chunks = k_new ? (int32_t)(((int64_t)max_q_len + kPage - 1) / kPage + 1) : 0;
  const int64_t write_blocks =
      ((int64_t)B_append * kv_append.hkv * write_chunks + 3) / (kPlanThreads / pwrite::kItemThreads);
  hipLaunchKernelGGL(mixed_plan_kernel, dim3((unsigned)(1 + write_blocks)), dim3(kPlanThreads), 0,
                     stream, m, w, write_chunks);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // One workgroup per CU: the kernel's registers allow one 8-wave
  // workgroup per CU, and every workgroup runs until the entries run out.
  int cus = 0;
  if ((e = device_cus(&cus)) != hipSuccess) return e;
  const int64_t entries = layout.max_tiles + layout.max_splits;
  const unsigned grid = (unsigned)(entries < cus ? (entries > 0 ? entries : 1) : cus);
  const dim3 g(grid), b(kMixThreads);
  const bool pos = m.ap.scale_log2 > 0.f || B_append == 0;
  const bool fp8 = kv_decode.fp8 || kv_append.fp8;   // the ABI layer allows one element type
  // rotated queries come only with append-only calls (the fused rotated write)
  if (cos_sin && B_decode > 0) return hipErrorInvalidValue;
  if (B_decode > 0 && m.de.group > 16) {   // two-tile decode splits
    const int v2 = (pos ? 2 : 0) | (fp8 ? 1 : 0);
    if (v2 == 0) hipLaunchKernelGGL((mixed_kernel<false, true, false, false, 2>), g, b, 0, stream, m);
    if (v2 == 1) hipLaunchKernelGGL((mixed_kernel<false, true, true, false, 2>), g, b, 0, stream, m);
    if (v2 == 2) hipLaunchKernelGGL((mixed_kernel<true, true, false, false, 2>), g, b, 0, stream, m);
    if (v2 == 3) hipLaunchKernelGGL((mixed_kernel<true, true, true, false, 2>), g, b, 0, stream, m);
  } else {
    const int variant = (cos_sin ? 8 : 0) | (pos ? 4 : 0) | (B_decode > 0 ? 2 : 0) | (fp8 ? 1 : 0);
    switch (variant) {
#define RA_MIXED_CASE(V, P, D, F, R)                                                  \
  case V:                                                                             \
    hipLaunchKernelGGL((mixed_kernel<P, D, F, R>), g, b, 0, stream, m);               \
    break;
      RA_MIXED_CASE(0, false, false, false, false)
      RA_MIXED_CASE(1, false, false, true, false)
      RA_MIXED_CASE(2, false, true, false, false)
      RA_MIXED_CASE(3, false, true, true, false)
      RA_MIXED_CASE(4, true, false, false, false)
      RA_MIXED_CASE(5, true, false, true, false)
      RA_MIXED_CASE(6, true, true, false, false)
      RA_MIXED_CASE(7, true, true, true, false)
      RA_MIXED_CASE(8, false, false, false, true)
      RA_MIXED_CASE(9, false, false, true, true)
      RA_MIXED_CASE(12, true, false, false, true)
      RA_MIXED_CASE(13, true, false, true, true)
#undef RA_MIXED_CASE
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (B_decode == 0) return hipSuccess;
  hipLaunchKernelGGL(dsplit::decode_combine_kernel, dim3(hq, B_decode), dim3(kHeadDim), 0, stream,
                     m.de, out_decode, lse_decode);
  return hipGetLastError();
}

}  // namespace ra
