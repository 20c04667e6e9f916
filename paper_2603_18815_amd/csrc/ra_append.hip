// Append attention: causal chunked prefill of new observation tokens against
// each trajectory's paged cache. One workgroup per (query block, KV head,
// row); the tile itself is described with append_tile.
#include "ra_append_tile.h"
#include "ra_internal.h"

namespace ra {
namespace {

using namespace atile;

template <bool kPosScale>
__global__ __launch_bounds__(kThreads, 1) void append_kernel(AppendArgs a) {
  __shared__ AppendLds lds;
  append_tile<kPosScale>(a, blockIdx.x, blockIdx.y, blockIdx.z, lds);
}

}  // namespace

hipError_t launch_append(const uint16_t *q, const int32_t *cu_q, const int32_t *ctx_lens,
                         const PagedKV &kv, int32_t B, int32_t hq, int32_t total_q,
                         int32_t max_q_len, int32_t max_kv_len, float scale, float *out,
                         float *lse, hipStream_t stream) {
  const AppendArgs a = make_append_args(q, cu_q, ctx_lens, kv, hq, total_q, max_q_len,
                                        max_kv_len, scale, out, lse);
  const int qblocks = (max_q_len + a.q_per_block - 1) / a.q_per_block;
  const dim3 grid(qblocks, kv.hkv, B);
  if (a.scale_log2 > 0.f)
    hipLaunchKernelGGL(append_kernel<true>, grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(append_kernel<false>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ra
