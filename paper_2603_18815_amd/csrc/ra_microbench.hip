// Hardware ceilings measured on the GPU: matrix-core rate and shader clock,
// LDS read bandwidth, streaming and paged HBM read rates. Declared in
// include/ra_microbench.h.
#include "ra_microbench.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 4;   // independent accumulators per wave

__device__ __forceinline__ void clock_pair(int64_t *dst) {
  dst[0] = (int64_t)__builtin_amdgcn_s_memtime();
  dst[1] = (int64_t)__builtin_amdgcn_s_memrealtime();
}

__global__ __launch_bounds__(RA_MB_MFMA_THREADS) void mfma_kernel(const uint16_t *operands,
                                                                  int iters, float *sink,
                                                                  int64_t *clocks) {
  const int tid = threadIdx.x;
  bf16x8 a[kChains], b[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) {
    a[c] = *reinterpret_cast<const bf16x8 *>(operands + (tid * 2 * kChains + c) * 8);
    b[c] = *reinterpret_cast<const bf16x8 *>(operands + (tid * 2 * kChains + kChains + c) * 8);
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x16{};
  const bool timer = blockIdx.x == 0 && tid == 0;
  int64_t t[4];
  if (timer) clock_pair(t);
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[c], b[c], acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  if (timer) {
    clock_pair(t + 2);
#pragma unroll
    for (int k = 0; k < 4; ++k) clocks[k] = t[k];
  }
  sink[(size_t)blockIdx.x * RA_MB_MFMA_THREADS + tid] = s;
}

constexpr int kLdsWords = 4096;   // 16-byte words of LDS read (64 KiB)

__global__ __launch_bounds__(RA_MB_LDS_THREADS) void lds_kernel(int iters, uint32_t *sink,
                                                                int64_t *clocks) {
  __shared__ u32x4 buf[kLdsWords];
  const int tid = threadIdx.x;
  for (int k = tid; k < kLdsWords; k += RA_MB_LDS_THREADS)
    buf[k] = u32x4{(uint32_t)k, (uint32_t)k * 3u, (uint32_t)k * 5u, (uint32_t)k * 7u};
  __syncthreads();
  u32x4 acc0 = {}, acc1 = {};
  const bool timer = blockIdx.x == 0 && tid == 0;
  int64_t t[4];
  if (timer) clock_pair(t);
  for (int i = 0; i < iters; ++i) {
    // base <= 2047, so base + 256 k <= 3839 stays inside buf
    const int base = (tid + 64 * (i & 15)) & 2047;
    // three-input adds (v_add3_u32): two vector instructions per 16 bytes read
#pragma unroll
    for (int k = 0; k < 8; k += 4) {
      acc0 = acc0 + buf[base + 256 * k] + buf[base + 256 * (k + 1)];
      acc1 = acc1 + buf[base + 256 * (k + 2)] + buf[base + 256 * (k + 3)];
    }
  }
  const u32x4 acc = acc0 + acc1;
  if (timer) {
    clock_pair(t + 2);
#pragma unroll
    for (int k = 0; k < 4; ++k) clocks[k] = t[k];
  }
  sink[(size_t)blockIdx.x * RA_MB_LDS_THREADS + tid] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

constexpr int kStreamThreads = 256;
constexpr int kBlockWords = 4096 / 16;   // 16-byte words per 4 KiB block

constexpr int kStreamLoads = 4;            // 16-byte loads per lane in flight per round

// Block j of the pass: j itself, or order[j] clamped into the buffer.
template <bool kPaged>
__device__ __forceinline__ int64_t block_of(const int32_t *order, int64_t j, int64_t nblk) {
  if constexpr (kPaged)
    return min(max((int64_t)order[j], (int64_t)0), nblk - 1);
  else
    return j;
}

// Round r of a workgroup reads blocks r * gridDim.x * kStreamLoads + k * gridDim.x
// + blockIdx.x, k < kStreamLoads, one 16-byte word per lane of each: four loads
// per lane in flight. A paged pass requests the next round's block numbers
// after this round's data, so their latency hides under it, and waits for the
// data only (the loads return in order), never for the numbers.
template <bool kPaged>
__global__ __launch_bounds__(kStreamThreads) void stream_kernel(const u32x4 *src, int64_t nblk,
                                                                const int32_t *order,
                                                                uint32_t *sink) {
  const int tid = threadIdx.x;
  const int64_t step = gridDim.x, per_round = step * kStreamLoads;
  const int64_t full = nblk / per_round * per_round;   // blocks in whole rounds
  u32x4 acc[kStreamLoads];
#pragma unroll
  for (int k = 0; k < kStreamLoads; ++k) acc[k] = u32x4{0u, 0u, 0u, 0u};
  int64_t j0 = blockIdx.x;
  int64_t blk[kStreamLoads];
  if (j0 < full) {
#pragma unroll
    for (int k = 0; k < kStreamLoads; ++k) blk[k] = block_of<kPaged>(order, j0 + k * step, nblk);
  }
  for (; j0 < full; j0 += per_round) {
    u32x4 v[kStreamLoads];
#pragma unroll
    for (int k = 0; k < kStreamLoads; ++k)
      v[k] = __builtin_nontemporal_load(&src[blk[k] * kBlockWords + tid]);
    __builtin_amdgcn_sched_barrier(0);   // all four issued before any use
    // the next round's blocks (this round's again after the last one: in
    // range, and no branch between the loads and their use)
    const int64_t jn = j0 + per_round < full ? j0 + per_round : j0;
#pragma unroll
    for (int k = 0; k < kStreamLoads; ++k) blk[k] = block_of<kPaged>(order, jn + k * step, nblk);
#pragma unroll
    for (int k = 0; k < kStreamLoads; ++k) acc[k] ^= v[k];
  }
  for (int64_t j = full + blockIdx.x; j < nblk; j += step)
    acc[0] ^= src[block_of<kPaged>(order, j, nblk) * kBlockWords + tid];
#pragma unroll
  for (int k = 1; k < kStreamLoads; ++k) acc[0] ^= acc[k];
  sink[(size_t)blockIdx.x * kStreamThreads + tid] = acc[0][0] ^ acc[0][1] ^ acc[0][2] ^ acc[0][3];
}

// A fixed bijection of [0, 2^bits) (xor-shift and odd-multiply rounds, each
// invertible modulo 2^bits): block j of a pass reads block mix(j).
__device__ __forceinline__ int64_t mix_block(int64_t j, int bits) {
  const uint64_t mask = (bits >= 64) ? ~0ull : ((1ull << bits) - 1ull);
  const int sh = (bits + 1) / 2;
  uint64_t h = (uint64_t)j;
  h ^= h >> sh;
  h = (h * 0x9E3779B97F4A7C15ull) & mask;
  h ^= h >> sh;
  h = (h * 0xBF58476D1CE4E5B9ull) & mask;
  h ^= h >> sh;
  return (int64_t)h;
}

// Shuffled blocks of kBytes bytes: one load instruction of the workgroup takes
// 4096 / kBytes blocks (kBytes / 16 lanes each), four loads per lane in
// flight per round, no block numbers read from memory.
template <int kBytes>
__global__ __launch_bounds__(kStreamThreads) void block_read_kernel(const u32x4 *src, int64_t nblk,
                                                                    int bits, uint32_t *sink) {
  constexpr int kWords = kBytes / 16, kPer = 4096 / kBytes;
  const int tid = threadIdx.x, sub = tid / kWords, w = tid % kWords;
  u32x4 acc[kStreamLoads];
#pragma unroll
  for (int k = 0; k < kStreamLoads; ++k) acc[k] = u32x4{0u, 0u, 0u, 0u};
  const int64_t per_round = (int64_t)gridDim.x * kPer * kStreamLoads;
  // nblk is a power of two of at least kPer * kStreamLoads blocks and base a
  // multiple of that, so every j below is < nblk
  for (int64_t base = (int64_t)blockIdx.x * kPer * kStreamLoads; base < nblk; base += per_round) {
    u32x4 v[kStreamLoads];
#pragma unroll
    for (int k = 0; k < kStreamLoads; ++k) {
      const int64_t b = mix_block(base + k * kPer + sub, bits);
      v[k] = __builtin_nontemporal_load(&src[b * kWords + w]);
    }
    __builtin_amdgcn_sched_barrier(0);   // all four issued before any use
#pragma unroll
    for (int k = 0; k < kStreamLoads; ++k) acc[k] ^= v[k];
  }
#pragma unroll
  for (int k = 1; k < kStreamLoads; ++k) acc[0] ^= acc[k];
  sink[(size_t)blockIdx.x * kStreamThreads + tid] = acc[0][0] ^ acc[0][1] ^ acc[0][2] ^ acc[0][3];
}

// ---- reads that hit in the L2: direct global-to-LDS loads against loads into
// registers. Each wave moves 16 KB per round as 16 load instructions of 1 KB
// (16 bytes per lane) from a buffer small enough to stay in every XCD's L2.
constexpr int kL2Loads = 16;
constexpr int kL2Threads = 256;

__device__ __forceinline__ void mb_load_lds16(const u32x4 *g, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(g)
      : "memory");
}

// kLds: each wave's 16 loads of a round land in its own 16 KB of LDS (the
// next round overwrites them; nothing reads LDS); the wave waits until at
// most 8 loads are outstanding after each round. Otherwise the loads go to
// registers in two halves of 8, the second half of a round and the first of
// the next in flight while the other is folded into an accumulator.
template <bool kLds>
__global__ __launch_bounds__(kL2Threads) void l2_read_kernel(const u32x4 *src, int32_t nchunks,
                                                             int32_t iters, uint32_t *sink) {
  __shared__ __attribute__((aligned(1024))) u32x4 ring[kLds ? 4 * kL2Loads * 64 : 1];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  // chunk (1 KB) of load k of round i: (first + 64 i + 16 wave + k) mod nchunks,
  // nchunks a power of two
  const int first = (int)((blockIdx.x * 64u) & (uint32_t)(nchunks - 1));
  auto chunk = [&](int i, int k) __attribute__((always_inline)) {
    return src + (size_t)((first + 64 * i + 16 * wave + k) & (nchunks - 1)) * 64 + lane;
  };
  u32x4 acc = {0u, 0u, 0u, 0u};
  if constexpr (kLds) {
    const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)ring +
                          (uint32_t)wave * kL2Loads * 1024u;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
      for (int k = 0; k < kL2Loads; ++k) mb_load_lds16(chunk(i, k), base + 1024u * k);
      __builtin_amdgcn_s_waitcnt(0x0F78);   // vmcnt(8)
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);     // vmcnt(0): every load has landed
    __syncthreads();
    acc = ring[threadIdx.x];
  } else {
    constexpr int kHalf = kL2Loads / 2;
    u32x4 a[kHalf], b[kHalf];
#pragma unroll
    for (int k = 0; k < kHalf; ++k) a[k] = chunk(0, k)[0];
    for (int i = 0; i < iters; ++i) {
#pragma unroll
      for (int k = 0; k < kHalf; ++k) b[k] = chunk(i, kHalf + k)[0];
#pragma unroll
      for (int k = 0; k < kHalf; ++k) acc ^= a[k];
#pragma unroll
      for (int k = 0; k < kHalf; ++k) a[k] = chunk(i + 1, k)[0];
#pragma unroll
      for (int k = 0; k < kHalf; ++k) acc ^= b[k];
    }
#pragma unroll
    for (int k = 0; k < kHalf; ++k) acc ^= a[k];
  }
  sink[(size_t)blockIdx.x * kL2Threads + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

int launched() { return hipGetLastError() == hipSuccess ? 0 : 5; }

}  // namespace

extern "C" {

int ra_mb_mfma_bf16(const void *operands, int32_t blocks, int32_t iters, float *sink,
                    int64_t *clocks, hipStream_t stream) {
  if (!operands || !sink || !clocks) return 1;
  if (blocks <= 0 || iters <= 0) return 2;
  hipLaunchKernelGGL(mfma_kernel, dim3(blocks), dim3(RA_MB_MFMA_THREADS), 0, stream,
                     static_cast<const uint16_t *>(operands), iters, sink, clocks);
  return launched();
}

int ra_mb_lds_read(int32_t blocks, int32_t iters, uint32_t *sink, int64_t *clocks,
                   hipStream_t stream) {
  if (!sink || !clocks) return 1;
  if (blocks <= 0 || iters <= 0) return 2;
  hipLaunchKernelGGL(lds_kernel, dim3(blocks), dim3(RA_MB_LDS_THREADS), 0, stream, iters, sink,
                     clocks);
  return launched();
}

int ra_mb_stream_read(const void *src, int64_t bytes, const int32_t *order, int32_t blocks,
                      uint32_t *sink, hipStream_t stream) {
  if (!src || !sink) return 1;
  if (bytes <= 0 || bytes % 4096 != 0 || blocks <= 0) return 2;
  if (order)
    hipLaunchKernelGGL(stream_kernel<true>, dim3(blocks), dim3(kStreamThreads), 0, stream,
                       static_cast<const u32x4 *>(src), bytes / 4096, order, sink);
  else
    hipLaunchKernelGGL(stream_kernel<false>, dim3(blocks), dim3(kStreamThreads), 0, stream,
                       static_cast<const u32x4 *>(src), bytes / 4096, order, sink);
  return launched();
}

int ra_mb_block_read(const void *src, int64_t bytes, int32_t block_bytes, int32_t blocks,
                     uint32_t *sink, hipStream_t stream) {
  if (!src || !sink) return 1;
  if (block_bytes != 1024 && block_bytes != 2048 && block_bytes != 4096) return 2;
  if (bytes <= 0 || bytes % block_bytes != 0 || blocks <= 0) return 2;
  const int64_t nblk = bytes / block_bytes;
  if ((nblk & (nblk - 1)) != 0 || nblk < 16) return 2;
  int bits = 0;
  while ((int64_t(1) << bits) < nblk) ++bits;
  const u32x4 *s = static_cast<const u32x4 *>(src);
  if (block_bytes == 1024)
    hipLaunchKernelGGL(block_read_kernel<1024>, dim3(blocks), dim3(kStreamThreads), 0, stream, s,
                       nblk, bits, sink);
  else if (block_bytes == 2048)
    hipLaunchKernelGGL(block_read_kernel<2048>, dim3(blocks), dim3(kStreamThreads), 0, stream, s,
                       nblk, bits, sink);
  else
    hipLaunchKernelGGL(block_read_kernel<4096>, dim3(blocks), dim3(kStreamThreads), 0, stream, s,
                       nblk, bits, sink);
  return launched();
}

int ra_mb_l2_read(const void *src, int64_t bytes, int32_t to_lds, int32_t blocks, int32_t iters,
                  uint32_t *sink, hipStream_t stream) {
  if (!src || !sink) return 1;
  if (bytes < 64 * 1024 || bytes > (int64_t)1 << 24 || (bytes & (bytes - 1)) != 0) return 2;
  if (blocks <= 0 || iters <= 0 || iters > (1 << 24)) return 2;
  const u32x4 *s = static_cast<const u32x4 *>(src);
  const int32_t nchunks = (int32_t)(bytes / 1024);
  if (to_lds)
    hipLaunchKernelGGL(l2_read_kernel<true>, dim3(blocks), dim3(kL2Threads), 0, stream, s, nchunks,
                       iters, sink);
  else
    hipLaunchKernelGGL(l2_read_kernel<false>, dim3(blocks), dim3(kL2Threads), 0, stream, s,
                       nchunks, iters, sink);
  return launched();
}

}  // extern "C"
