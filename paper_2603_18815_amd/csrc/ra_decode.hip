// Decode attention over paged KV caches: split-K over pages, then combine.
// The split and the combine are described with decode_split in the header.
#include <stdlib.h>

#include "ra_decode_split.h"
#include "ra_internal.h"

namespace ra {
namespace {

using namespace dsplit;

constexpr int kSplitWaves = 4;

// KV head fastest: the Hkv workgroups of one (item, split) are dispatched
// together, so the Hkv adjacent 4 KiB blocks of every page they read are
// requested close in time (DRAM row locality).
template <int NT, bool kPrefix, bool kFp8>
__global__ __launch_bounds__(kSplitWaves * kWave, 2) void decode_split_kernel(DecodeArgs a) {
  __shared__ DecodeLds<NT, kSplitWaves> lds;
  decode_split<NT, kPrefix, kSplitWaves, kFp8>(a, blockIdx.x, blockIdx.y, blockIdx.z, lds);
}

// Shared-prefix decode in one launch. Planes z < prefix_planes hold the
// prefix items, item i = z * gridDim.y + y, with the chunks of one (group,
// prefix split) adjacent so that the workgroups reading the same prefix pages
// run close together (the later ones mostly hit the cache); the planes after
// hold the row items as in plain decode. One launch lets the few prefix items
// run beside the many row items instead of before them, in a pass of their own
// that leaves most of the machine idle.
template <int NT, bool kFp8>
__global__ __launch_bounds__(kSplitWaves * kWave, 2) void decode_shared_kernel(
    DecodeArgs a, int32_t prefix_planes, int32_t chunks, int32_t prefix_items) {
  __shared__ DecodeLds<NT, kSplitWaves> lds;
  const int z = blockIdx.z;
  if (z < prefix_planes) {
    const int i = z * gridDim.y + blockIdx.y;
    if (i >= prefix_items) return;
    const int sub = i % chunks, gs = i / chunks;
    const int split = gs % a.prefix_slots, grp = gs / a.prefix_slots;
    DecodeArgs p = a;
    p.zdiv = chunks;
    decode_split<NT, true, kSplitWaves, kFp8>(p, blockIdx.x, split, grp * chunks + sub, lds);
  } else {
    decode_split<NT, false, kSplitWaves, kFp8>(a, blockIdx.x, blockIdx.y, z - prefix_planes, lds);
  }
}

template <int NT>
void launch_shared(bool fp8, dim3 grid, const DecodeArgs &a, const SharedPrefixShape &sh,
                   hipStream_t stream) {
  const int32_t planes = (int32_t)sh.prefix_planes, items = (int32_t)sh.prefix_items;
  if (fp8)
    hipLaunchKernelGGL((decode_shared_kernel<NT, true>), grid, dim3(kSplitWaves * kWave), 0,
                       stream, a, planes, sh.chunks, items);
  else
    hipLaunchKernelGGL((decode_shared_kernel<NT, false>), grid, dim3(kSplitWaves * kWave), 0,
                       stream, a, planes, sh.chunks, items);
}

template <int NT, bool kPrefix>
void launch_split(bool fp8, dim3 grid, const DecodeArgs &a, hipStream_t stream) {
  if (fp8)
    hipLaunchKernelGGL((decode_split_kernel<NT, kPrefix, true>), grid, dim3(kSplitWaves * kWave),
                       0, stream, a);
  else
    hipLaunchKernelGGL((decode_split_kernel<NT, kPrefix, false>), grid, dim3(kSplitWaves * kWave),
                       0, stream, a);
}

// Split length forced by the environment (RA_SPLIT_TOKENS, for testing the
// split and combine paths), read once per process: a decimal number of keys
// in [128, 65536], rounded up to a multiple of 128; anything else (absent,
// not a number, out of range) leaves the planned length. 0 when unset.
int64_t split_override() {
  static const int64_t value = [] {
    const char *env = getenv("RA_SPLIT_TOKENS");
    if (!env || !*env) return (int64_t)0;
    char *end = nullptr;
    const long long v = strtoll(env, &end, 10);
    if (*end != '\0' || v < 128 || v > 65536) return (int64_t)0;
    return (int64_t)((v + 127) / 128 * 128);
  }();
  return value;
}

}  // namespace

DecodePlan decode_plan(int32_t B, int32_t hkv, int32_t max_kv_len) {
  // Aim for about 8k (row, KV head, split) items on the longest-row bound:
  // enough workgroups to balance rows of different lengths over 256 CUs,
  // long enough splits that the partial results stay well under 1 % of the
  // KV bytes. Split lengths are powers of two in [512, 4096] keys, multiples
  // of 128 keys (4 waves x one page pair), and depend only on the host-side
  // sizes, never on page ids.
  int64_t work = (int64_t)B * hkv * (int64_t)(max_kv_len > 0 ? max_kv_len : 1);
  int64_t split = 512;
  while (split < 4096 && work / split > 8192) split *= 2;
  if (const int64_t forced = split_override()) split = forced;
  DecodePlan p;
  p.split_tokens = (int32_t)split;
  p.max_splits = (int32_t)((max_kv_len + split - 1) / split);
  if (p.max_splits < 1) p.max_splits = 1;
  return p;
}

size_t decode_workspace_bytes(int32_t B, int32_t hq, const DecodePlan &plan) {
  const size_t parts = (size_t)B * hq * plan.max_splits;
  return parts * (kHeadDim + 2) * sizeof(float);
}

int32_t prefix_slots(const DecodePlan &plan, int32_t max_prefix_len) {
  return (int32_t)((max(max_prefix_len, 0) + (int64_t)plan.split_tokens - 1) / plan.split_tokens);
}

size_t shared_prefix_workspace_bytes(int32_t B, int32_t hq, const DecodePlan &plan,
                                     int32_t max_prefix_len) {
  const size_t parts = (size_t)B * hq * (plan.max_splits + prefix_slots(plan, max_prefix_len));
  return parts * (kHeadDim + 2) * sizeof(float);
}

hipError_t launch_decode(const uint16_t *q, const PagedKV &kv, const int32_t *kv_lens, int32_t B,
                         int32_t hq, int32_t max_kv_len, float scale, float *out, float *lse,
                         void *workspace, const DecodePlan &plan, hipStream_t stream) {
  const DecodeArgs a =
      make_decode_args(q, kv, kv_lens, B, hq, max_kv_len, scale, workspace, plan.max_splits, plan);
  // the G query heads of a KV head are the columns of one 16-column tile, or
  // of two for groups of 17 to 32 heads
  if (a.group > 16)
    launch_split<2, false>(kv.fp8, dim3(kv.hkv, plan.max_splits, B), a, stream);
  else
    launch_split<1, false>(kv.fp8, dim3(kv.hkv, plan.max_splits, B), a, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_combine_kernel, dim3(hq, B), dim3(kHeadDim), 0, stream, a, out, lse);
  return hipGetLastError();
}

SharedPrefixShape shared_prefix_shape(int32_t group, int32_t num_groups, int32_t max_group_rows,
                                      const DecodePlan &plan, int32_t max_prefix_len) {
  SharedPrefixShape sh;
  // as many rows per prefix chunk as fill the row items' tiles (one tile,
  // two for groups of 17 to 32 heads), so that both kinds of item share one
  // register and LDS budget
  sh.tiles = group > 16 ? 2 : 1;
  sh.rows_per_chunk = max(1, min(max_group_rows, 16 * sh.tiles / group));
  sh.chunks = (max_group_rows + sh.rows_per_chunk - 1) / sh.rows_per_chunk;
  sh.prefix_items = (int64_t)num_groups * sh.chunks * prefix_slots(plan, max_prefix_len);
  sh.prefix_planes = (sh.prefix_items + plan.max_splits - 1) / plan.max_splits;
  sh.row_z = (int64_t)num_groups * max_group_rows;
  return sh;
}

hipError_t launch_decode_shared_prefix(const uint16_t *q, const PagedKV &kv,
                                       const int32_t *kv_lens, const int32_t *group_start,
                                       const int32_t *prefix_len, int32_t B, int32_t hq,
                                       int32_t num_groups, int32_t max_group_rows,
                                       int32_t max_prefix_len, int32_t max_kv_len, float scale,
                                       float *out, float *lse, void *workspace,
                                       const DecodePlan &plan, hipStream_t stream) {
  const int32_t ps = prefix_slots(plan, max_prefix_len);
  DecodeArgs a = make_decode_args(q, kv, kv_lens, B, hq, max_kv_len, scale, workspace,
                           plan.max_splits + ps, plan);
  const SharedPrefixShape sh =
      shared_prefix_shape(a.group, num_groups, max_group_rows, plan, max_prefix_len);
  a.group_start = group_start;
  a.prefix_len = prefix_len;
  a.prefix_slots = ps;
  a.rows_per_chunk = sh.rows_per_chunk;
  a.zdiv = max_group_rows;
  const dim3 grid(kv.hkv, plan.max_splits, (unsigned)(sh.prefix_planes + sh.row_z));
  if (sh.tiles == 2)
    launch_shared<2>(kv.fp8, grid, a, sh, stream);
  else
    launch_shared<1>(kv.fp8, grid, a, sh, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_combine_kernel, dim3(hq, (unsigned)sh.row_z), dim3(kHeadDim), 0, stream,
                     a, out, lse);
  return hipGetLastError();
}

}  // namespace ra
