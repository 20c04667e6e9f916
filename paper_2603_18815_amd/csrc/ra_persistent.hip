// Planned persistent launches: append rows alone, or one rollout step's
// decode rows (one new token each) and append rows (a chunk of new
// observation tokens each) together, against their paged caches.
//
// A plan kernel (one workgroup) lists the work of the call from the
// device-resident lengths:
//   - append tiles (row, query block, KV head), sorted by the number of
//     64-key blocks they walk, longest first (a counting sort over the key
//     block counts), so that the long tiles start early and the short ones
//     fill the end instead of leaving CUs idle behind one long tile;
//   - decode splits (row, split, KV head), row by row.
// The attention kernel then runs one workgroup of 8 waves per CU; each
// workgroup takes the next entry of one merged order from a device counter
// until the order is used up. The merged order places the decode splits at
// even spacing among the append tiles, so that at any time a few CUs stream
// KV pages for decode (bound by HBM) while the rest run the append tiles'
// matrix products (bound by the matrix cores): the decode bytes are read
// while the matrix cores are busy instead of in a phase of their own. Entry
// j of the merged order (n entries, nd of them decode splits) is decode
// split floor(j nd / n) when floor((j + 1) nd / n) > floor(j nd / n), else
// append tile j - floor(j nd / n).
// A decode split is computed as by the decode split kernel but with 8 waves;
// the decode combine follows as in plain decode. Results do not depend on
// the order in which entries are taken.
#include "ra_append_tile.h"
#include "ra_decode_split.h"
#include "ra_internal.h"

namespace ra {
namespace {

constexpr int kMixWaves = 8;
constexpr int kMixThreads = kMixWaves * kWave;
static_assert(kMixThreads == atile::kThreads, "append tiles take the whole workgroup");
constexpr int kPlanThreads = 1024;
constexpr int kCostBuckets = 4096;   // key-block counts above this share the last bucket
constexpr int kHeadBits = 8;         // entry = {row, index << kHeadBits | KV head}

struct MixedArgs {
  atile::AppendArgs ap;
  dsplit::DecodeArgs de;
  int2 *tiles;      // append tiles, longest first
  int2 *splits;     // decode splits
  int32_t *header;  // [0] next merged entry, [1] append tiles, [2] decode splits
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

__global__ __launch_bounds__(kPlanThreads) void mixed_plan_kernel(MixedArgs m) {
  __shared__ int count[kCostBuckets];   // tiles per key-block count, then write cursors
  __shared__ int s_scan[kPlanThreads];
  const int tid = threadIdx.x;
  const int hkv_a = m.ap.hkv, hkv_d = m.de.hkv;
  for (int c = tid; c < kCostBuckets; c += kPlanThreads) count[c] = 0;
  __syncthreads();

  // ---- append tiles: bucket c holds the (row, query block) pairs that walk
  // c + 1 key blocks (or more, in the last bucket)
  const int pairs = m.B_append * m.qblocks;
  for (int i = tid; i < pairs; i += kPlanThreads) {
    const int b = i / m.qblocks, qb = i - b * m.qblocks;
    const int nb = atile::append_tile_blocks(m.ap, atile::append_row(m.ap, b), qb);
    if (nb > 0) atomicAdd(&count[min(nb, kCostBuckets) - 1], 1);
  }
  __syncthreads();
  // cursors: bucket c starts after every bucket above it (longest first);
  // thread t owns buckets kCostBuckets - 1 - (kPer t + k), k < kPer
  constexpr int kPer = kCostBuckets / kPlanThreads;
  int own[kPer], sum = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    own[k] = count[kCostBuckets - 1 - (kPer * tid + k)];
    sum += own[k];
  }
  int n_pairs;
  int cursor = block_exclusive_scan(sum, s_scan, &n_pairs);
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    count[kCostBuckets - 1 - (kPer * tid + k)] = cursor;
    cursor += own[k];
  }
  __syncthreads();
  for (int i = tid; i < pairs; i += kPlanThreads) {
    const int b = i / m.qblocks, qb = i - b * m.qblocks;
    const int nb = atile::append_tile_blocks(m.ap, atile::append_row(m.ap, b), qb);
    if (nb <= 0) continue;
    const int p = atomicAdd(&count[min(nb, kCostBuckets) - 1], 1);
    for (int g = 0; g < hkv_a; ++g)
      m.tiles[(size_t)p * hkv_a + g] = make_int2(b, qb << kHeadBits | g);
  }

  // ---- decode splits, row by row, KV head fastest
  const int S = m.de.split_tokens;
  int n_split_rows = 0;   // (row, split) pairs listed so far
  for (int r0 = 0; r0 < m.de.B; r0 += kPlanThreads) {
    const int b = r0 + tid;
    const int ns = b < m.de.B ? (dsplit::row_len(m.de, b) + S - 1) / S : 0;
    int chunk_total;
    const int first = n_split_rows + block_exclusive_scan(ns, s_scan, &chunk_total);
    for (int s = 0; s < ns; ++s)
      for (int g = 0; g < hkv_d; ++g)
        m.splits[(size_t)(first + s) * hkv_d + g] = make_int2(b, s << kHeadBits | g);
    n_split_rows += chunk_total;
  }
  if (tid == 0) {
    m.header[0] = 0;
    m.header[1] = n_pairs * hkv_a;
    m.header[2] = n_split_rows * hkv_d;
  }
}

// kDecode: the call has decode rows (otherwise every entry is an append tile).
template <bool kPosScale, bool kDecode>
__global__ __launch_bounds__(kMixThreads, 1) void mixed_kernel(MixedArgs m) {
  __shared__ union {
    atile::AppendLds ap;
    dsplit::DecodeLds<1, kMixWaves> de;
  } lds;
  __shared__ int s_next;
  const int na = m.header[1], nd = m.header[2];
  const int64_t n = (int64_t)na + nd;
  for (;;) {
    __syncthreads();   // the previous entry is done with LDS and s_next
    if (threadIdx.x == 0) s_next = atomicAdd(&m.header[0], 1);
    __syncthreads();
    const int j = __builtin_amdgcn_readfirstlane(s_next);
    if (j >= n) break;
    const int dj = (int)((int64_t)j * nd / n);
    if (kDecode && (int)(((int64_t)j + 1) * nd / n) > dj) {
      const int2 e = m.splits[dj];
      dsplit::decode_split<1, false, kMixWaves>(m.de, e.y & ((1 << kHeadBits) - 1),
                                                e.y >> kHeadBits, e.x, lds.de);
    } else {
      const int2 e = m.tiles[j - dj];
      atile::append_tile<kPosScale>(m.ap, e.y >> kHeadBits, e.y & ((1 << kHeadBits) - 1), e.x,
                                    lds.ap);
    }
  }
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

}  // namespace

MixedLayout mixed_layout(int32_t B_decode, int32_t B_append, int32_t hq, int32_t hkv_decode,
                         int32_t hkv_append, int32_t max_kv_len_decode, int32_t max_q_len) {
  MixedLayout l;
  l.plan = decode_plan(B_decode > 0 ? B_decode : 1, hkv_decode, max_kv_len_decode);
  const int32_t qpb = atile::kRowsPerGroup / (hq / hkv_append);
  l.qblocks = max_q_len > 0 ? (max_q_len + qpb - 1) / qpb : 0;
  l.max_tiles = (int64_t)B_append * l.qblocks * hkv_append;
  l.max_splits = (int64_t)B_decode * l.plan.max_splits * hkv_decode;
  l.tiles_offset = kAlign;
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
                        hipStream_t stream) {
  char *ws = static_cast<char *>(workspace);
  MixedArgs m;
  m.ap = atile::make_append_args(q_append, cu_q, ctx_lens, kv_append, hq, total_q, max_q_len,
                                 max_kv_len_append, scale, out_append, lse_append);
  m.de = dsplit::make_decode_args(q_decode, kv_decode, kv_lens, B_decode, hq,
                                  max_kv_len_decode, scale, ws + layout.partials_offset,
                                  layout.plan.max_splits, layout.plan);
  m.header = reinterpret_cast<int32_t *>(ws);
  m.tiles = reinterpret_cast<int2 *>(ws + layout.tiles_offset);
  m.splits = reinterpret_cast<int2 *>(ws + layout.splits_offset);
  m.B_append = B_append;
  m.qblocks = layout.qblocks;

  hipLaunchKernelGGL(mixed_plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, m);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // One workgroup per CU: the kernel's registers allow one 8-wave
  // workgroup per CU, and every workgroup runs until the entries run out.
  int dev = 0, cus = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) !=
      hipSuccess)
    return e;
  const int64_t entries = layout.max_tiles + layout.max_splits;
  const unsigned grid = (unsigned)(entries < cus ? (entries > 0 ? entries : 1) : cus);
  const dim3 g(grid), b(kMixThreads);
  const bool pos = m.ap.scale_log2 > 0.f || B_append == 0;
  if (B_decode == 0) {
    if (pos)
      hipLaunchKernelGGL((mixed_kernel<true, false>), g, b, 0, stream, m);
    else
      hipLaunchKernelGGL((mixed_kernel<false, false>), g, b, 0, stream, m);
  } else {
    if (pos)
      hipLaunchKernelGGL((mixed_kernel<true, true>), g, b, 0, stream, m);
    else
      hipLaunchKernelGGL((mixed_kernel<false, true>), g, b, 0, stream, m);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (B_decode == 0) return hipSuccess;
  hipLaunchKernelGGL(dsplit::decode_combine_kernel, dim3(hq, B_decode), dim3(kHeadDim), 0, stream,
                     m.de, out_decode, lse_decode);
  return hipGetLastError();
}

}  // namespace ra
