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

SharedPrefixShape shared_prefix_shape(int32_t group, int32_t num_groups, int32_t max_group_rows) {
  SharedPrefixShape sh;
  sh.rows_per_chunk = min(max_group_rows, 2 * 16 / group);
  sh.tiles = (sh.rows_per_chunk * group + 15) / 16;
  sh.chunks = (max_group_rows + sh.rows_per_chunk - 1) / sh.rows_per_chunk;
  sh.prefix_z = (int64_t)num_groups * sh.chunks;
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
  const SharedPrefixShape sh = shared_prefix_shape(a.group, num_groups, max_group_rows);
  a.group_start = group_start;
  a.prefix_len = prefix_len;
  a.prefix_slots = ps;
  a.rows_per_chunk = sh.rows_per_chunk;
  hipError_t e = hipSuccess;
  if (ps > 0) {
    a.zdiv = sh.chunks;
    const dim3 grid(kv.hkv, ps, (unsigned)sh.prefix_z);
    if (sh.tiles == 1)
      launch_split<1, true>(kv.fp8, grid, a, stream);
    else
      launch_split<2, true>(kv.fp8, grid, a, stream);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  a.zdiv = max_group_rows;
  const dim3 rows_grid(kv.hkv, plan.max_splits, (unsigned)sh.row_z);
  if (a.group > 16)
    launch_split<2, false>(kv.fp8, rows_grid, a, stream);
  else
    launch_split<1, false>(kv.fp8, rows_grid, a, stream);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(decode_combine_kernel, dim3(hq, (unsigned)sh.row_z), dim3(kHeadDim), 0, stream,
                     a, out, lse);
  return hipGetLastError();
}

}  // namespace ra
