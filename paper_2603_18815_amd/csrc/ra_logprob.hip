// Per-token log-probabilities under an LM head, fused: logits, log-sum-exp and
// the gather of the emitted token's logit, without writing the logits.
//
// For token n (hidden state h[n], emitted token t[n]) and the LM-head matrix
// W [V][D]: z_v = scale * <h[n], W[v]>, lse = ln sum_v exp z_v, and
// logp = z_t - lse.
//
// Partial kernel: one workgroup (4 waves) per (128-row vocabulary chunk,
// token block of 128, or 64 when N <= 64). Each wave computes the logits of
// its 32 vocabulary rows for the block's tokens on the matrix cores (4 or 2
// tiles of
// mfma_f32_32x32x16_bf16: A = W rows, B = h^T). The loop walks D in steps of
// 64 dims. W comes straight from memory, three steps ahead: a lane reads 64
// contiguous bytes of its row per step, the two lanes of a row 128 bytes. The
// block's h slice (tokens x 64 dims) is requested two steps ahead, staged once
// per step into LDS (double-buffered, rows padded to 144 B: conflict-free) and
// read by all four waves. The 64 dims of a step are split over the four products as lanes 0-31
// dims 8u + 0..7 and lanes 32-63 dims 32 + 8u + 0..7 (any split of the
// contraction is valid as long as A and B use the same one). The wave reduces
// its logits to a (max, sum of exp) pair per token in base 2, the four waves
// merge through LDS, and the workgroup writes one partial per (token, chunk);
// the workgroup whose chunk holds token n's target stores that logit. The
// grid is mapped so that the token blocks of one vocabulary chunk run on one
// XCD and re-read the chunk from that XCD's L2.
//
// From N = 512 on, the partials come from the 384 x 256 tiled kernel further
// down (384-row chunks) instead.
//
// Combine kernel: one workgroup per token merges its partials:
// M = max_c m_c, L = sum_c l_c 2^(m_c - M), lse = (M + log2 L) ln 2.
//
// Packed LM head: W [V][D] row-major makes every wave read 32 rows 128 bytes
// at a time, 8 KB apart. The packed copy stores the matrix in the order the
// products consume it, [D/64][tiles][4][64 lanes][8] (32-row tiles, V rounded
// up to whole 384-row chunks): each load instruction reads 1 KB contiguous,
// a wave's step is 4 KB contiguous, and the waves working on one 64-dim step
// at the same time read one narrow window of memory rather than thousands of
// separate runs. Same products in the same order: the results are bitwise
// those of the row-major matrix.
#include "ra_device.h"
#include "ra_internal.h"

namespace ra {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kLpWaves = 4;
constexpr int kLpThreads = kLpWaves * kWave;
constexpr int kVocabChunk = 32 * kLpWaves;    // vocabulary rows per workgroup
constexpr int kMaxTiles = 4;                  // 32-token tiles per workgroup (largest variant)
constexpr int kDimStep = 64;                  // dims per loop step (4 products)
constexpr int kXcds = 8;                      // XCDs of an MI355X
constexpr int kHPitch = kDimStep + 8;         // LDS row pitch of the h slice (elements)
constexpr int kTileMinN = 512;                // batches from this size use the 384 x 256 tiles
constexpr int kPackRows = 384;                // the packed copy covers V rounded up to this
// s_waitcnt immediates: vmcnt(0), export and LDS counters not waited on
constexpr int kWaitVm0 = 0x0F70;

struct LogprobArgs {
  const uint16_t *h;
  const uint16_t *hp;   // N >= kTileMinN: h in the tiled kernel's LDS stage order (workspace)
  const uint16_t *W;
  const int32_t *targets;
  float *ws_m;    // [N][chunks] running max, base-2 units
  float *ws_l;    // [N][chunks] sum of 2^(y - max)
  float *tgt;     // [N] logit of the target (natural units)
  int32_t N, V, D, chunks, token_blocks;
  float scale;        // logits = scale * <h, W_v>
  float scale_log2;   // scale * log2(e)
};

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Max / sum over lanes l and l ^ 32 (v_permlane32_swap gives each lane both).
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// kTiles 32-token tiles per workgroup: 2 for small batches (N <= 64), else 4.
template <int kTiles, bool kPacked>
__global__ __launch_bounds__(kLpThreads, 2) void logprob_partial_kernel(LogprobArgs a) {
  constexpr int kTokenBlock = 32 * kTiles;
  // XCD-aware placement: workgroup ids are dealt to the XCDs round-robin, so
  // ids id, id + 8, id + 16, ... share an XCD; those consecutive "slots" get
  // the token blocks of one vocabulary chunk.
  const int id = blockIdx.x;
  const int xcd = id % kXcds, slot = id / kXcds;
  const int chunk = (slot / a.token_blocks) * kXcds + xcd;
  const int tblock = slot - (slot / a.token_blocks) * a.token_blocks;
  if (chunk >= a.chunks) return;

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int col = lane & 31, half = lane >> 5;
  const int v0 = chunk * kVocabChunk + wave * 32;       // first vocabulary row of this wave
  const int t0 = tblock * kTokenBlock;                  // first token of the block

  // A row (vocabulary) this lane supplies, clamped into range for the loads
  // (packed: rows past V are stored as zeros); rows past V are masked after
  // the products.
  const uint16_t *wp =
      kPacked ? a.W + (size_t)(v0 / 32) * 4 * kWave * 8 + 8 * lane
              : a.W + (size_t)min(v0 + col, a.V - 1) * a.D + 32 * half;
  // h staging: thread i copies 16-byte chunks i + 256 j (j = 0..3) of the
  // block's 128 x 64 slice (token = chunk / 8, 8 dims per chunk); tokens past
  // N are clamped (their columns are never written back).
  constexpr int kHChunks = kTokenBlock * kDimStep / 8 / kLpThreads;   // 2 or 4
  __shared__ __attribute__((aligned(16))) uint16_t s_h[2][kTokenBlock * kHPitch];
  const uint16_t *hsrc[kHChunks];
  int hdst[kHChunks];
#pragma unroll
  for (int i = 0; i < kHChunks; ++i) {
    const int c = threadIdx.x + kLpThreads * i, tok = c >> 3, d8 = (c & 7) * 8;
    hsrc[i] = a.h + (size_t)min(t0 + tok, a.N - 1) * a.D + d8;
    hdst[i] = tok * kHPitch + d8;
  }
  // Two register sets for h (requested two steps ahead) and four for W
  // (three steps ahead); the loop body is four steps so that every set keeps
  // a fixed role and no operand is copied.
  u32x4 hx[kHChunks], hy[kHChunks];
  auto h_load = [&](u32x4 *dst, int s) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kHChunks; ++i) dst[i] = load_u32x4(hsrc[i] + s * kDimStep);
  };
  auto h_store = [&](int buf, const u32x4 *src) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kHChunks; ++i) store_u32x4(&s_h[buf][hdst[i]], src[i]);
  };
  // With one token block (kTiles == 2: N <= 64) no other workgroup reads this
  // chunk of W, and a packed W load takes 1 KB contiguous (whole cache lines):
  // those loads are marked nontemporal. Row-major loads take each line 32
  // bytes at a time over four instructions and stay ordinary.
  constexpr bool kStreamW = kPacked && kTiles == 2;
  // 32-row tiles of the packed copy: a 64-dim step of all of them is one block
  const size_t ntiles = (size_t)(((int64_t)a.V + kPackRows - 1) / kPackRows) * (kPackRows / 32);
  bf16x8 w0[4], w1[4], w2[4], w3[4];
  auto w_load = [&](bf16x8 *dst, int s) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
      dst[u] = kStreamW ? __builtin_bit_cast(bf16x8, load_stream_u32x4(wp + ((size_t)s * ntiles * 4 + u) * 8 * kWave))
                        : load_bf16x8(kPacked ? wp + ((size_t)s * ntiles * 4 + u) * 8 * kWave
                                              : wp + s * kDimStep + 8 * u);
  };
  const int nsteps = a.D / kDimStep;
  const int last = nsteps - 1;
  f32x16 acc[kTiles];
#pragma unroll
  for (int tt = 0; tt < kTiles; ++tt) acc[tt] = f32x16{};
  // Step s: request h(s + 2) into `hf` and W(s + 3) into `wf` (past the last
  // step the requests repeat it: branch-free, exact wait counts), run the
  // products of step s on `wu` and LDS buffer s & 1, then store h(s + 1)
  // (register set `hs`) into the other buffer.
  auto step = [&](int s, const bf16x8 *wu, bf16x8 *wf, u32x4 *hf, const u32x4 *hs)
      __attribute__((always_inline)) {
    h_load(hf, min(s + 2, last));
    w_load(wf, min(s + 3, last));
    const uint16_t *hb = &s_h[s & 1][col * kHPitch + 32 * half];
#pragma unroll
    for (int tt = 0; tt < kTiles; ++tt) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bf16x8 b = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4 *>(hb + 32 * tt * kHPitch + 8 * u));
        acc[tt] = mfma32x32x16(wu[u], b, acc[tt]);
      }
    }
    h_store((s + 1) & 1, hs);
    __syncthreads();
  };

  h_load(hx, 0);
  h_load(hy, min(1, last));
  w_load(w0, 0);
  w_load(w1, min(1, last));
  w_load(w2, min(2, last));
  h_store(0, hx);
  __syncthreads();
  // step s uses W set s % 4 and h register set (s + 1) % 2 for the store
  int s = 0;
  for (; s + 4 <= nsteps; s += 4) {
    step(s, w0, w3, hx, hy);
    step(s + 1, w1, w0, hy, hx);
    step(s + 2, w2, w1, hx, hy);
    step(s + 3, w3, w2, hy, hx);
  }
  if (s < nsteps) step(s, w0, w3, hx, hy);
  if (s + 1 < nsteps) step(s + 1, w1, w0, hy, hx);
  if (s + 2 < nsteps) step(s + 2, w2, w1, hx, hy);

  // Lane l holds, for token column t0 + 32 tt + col, the logits of vocabulary
  // rows v0 + 8 (r / 4) + 4 half + r % 4, r = 0..15.
  __shared__ float s_m[kLpWaves][kTokenBlock];
  __shared__ float s_l[kLpWaves][kTokenBlock];
#pragma unroll
  for (int tt = 0; tt < kTiles; ++tt) {
    const int t = t0 + 32 * tt + col;
    const int target = t < a.N ? a.targets[t] : -1;
    float y[16];
    float m = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int v = v0 + 8 * (r >> 2) + 4 * half + (r & 3);
      y[r] = v < a.V ? acc[tt][r] * a.scale_log2 : -INFINITY;
      m = fmaxf(m, y[r]);
      if (v == target) a.tgt[t] = acc[tt][r] * a.scale;
    }
    m = pair_max(m);
    const float m_use = m == -INFINITY ? 0.f : m;
    float sum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) sum += fast_exp2(y[r] - m_use);
    sum = pair_sum(sum);
    if (half == 0) {
      s_m[wave][32 * tt + col] = m;
      s_l[wave][32 * tt + col] = sum;
    }
  }
  __syncthreads();

  // Merge the four waves: one thread per token of the block.
  const int c = threadIdx.x;
  if (c < kTokenBlock && t0 + c < a.N) {
    float M = s_m[0][c];
#pragma unroll
    for (int w = 1; w < kLpWaves; ++w) M = fmaxf(M, s_m[w][c]);
    const float M_use = M == -INFINITY ? 0.f : M;
    float L = 0.f;
#pragma unroll
    for (int w = 0; w < kLpWaves; ++w) L += s_l[w][c] * fast_exp2(s_m[w][c] - M_use);
    const size_t part = (size_t)(t0 + c) * a.chunks + chunk;
    a.ws_m[part] = M;
    a.ws_l[part] = L;
  }
}

// ---- large batches: LDS-tiled products, 384 vocabulary rows x 256 tokens ----
//
// At N >= kTileMinN one workgroup of 8 waves (one per compute unit) owns a
// 384 x 256 tile of logits (vocabulary rows x tokens). Each compute unit then
// loads 40 KB of W and h per 384 x 256 x 32 multiply-adds, about 19 % fewer
// bytes per product than a 256 x 256 tile and less than half of what the 128 x 128
// tiles above load; those are bound by how fast the L2 delivers operands to
// the compute units, not by the matrix cores. The loop walks D in steps of 32
// dims through a ring of 3 LDS stages (24 KB of W and 16 KB of h each),
// refilled two steps ahead by direct global-to-LDS loads
// (global_load_lds_dwordx4, no register staging); the five refill loads of a
// wave and step are spread between its products. Wave w computes rows
// 96 (w % 4) .. + 95 (three 32-row tiles) against tokens 128 (w / 4) .. + 127
// (four 32-token tiles): 24 products per step from 14 LDS operand reads, 192
// accumulator registers.
//
// Stage layout: row r of a region holds its 32 dims as four 16-byte chunks,
// logical chunk c at slot c ^ ((r / 4) % 4), so that 16 lanes reading 16 rows
// at one logical chunk hit 16 distinct bank groups. A load instruction fills
// 16 rows: lane l fetches row 16 j + l / 4, the logical chunk stored at slot
// l % 4. The 32 dims of a step split over the two products as lanes 0-31 dims
// 8 u + 0..7 and lanes 32-63 dims 16 + 8 u + 0..7 (logical chunk 2 half + u).
constexpr int kTileRows = 256;        // tokens per workgroup
constexpr int kTileRowsA = 384;       // vocabulary rows per workgroup
constexpr int kTileWaves = 8;
constexpr int kTileThreads = kTileWaves * kWave;
constexpr int kTileDims = 32;         // dims per step
constexpr int kTileStages = 3;
constexpr int kTileElems = kTileRows * kTileDims;     // token region of a stage (16 KB)
constexpr int kTileElemsA = kTileRowsA * kTileDims;   // vocabulary region (24 KB)
constexpr int kLoadsA = kTileRowsA / 16 / kTileWaves;  // 3
constexpr int kLoadsB = kTileRows / 16 / kTileWaves;   // 2
// s_waitcnt vmcnt(5) (export and LDS counters not waited on): one later
// step's loads may stay in flight
constexpr int kWaitVm5 = 0x0F75;

// Direct global-to-LDS load of 16 bytes per lane: lane l's bytes land at LDS
// address `lds` + 16 l (lds wave-uniform). Written out rather than through the
// compiler builtin, which makes the compiler wait for every such load before
// any LDS read (it cannot tell the ring's stages apart); the kernel counts
// its own loads. M0 (the LDS base register) is restored before the statement
// ends.
__device__ __forceinline__ uint32_t lds_address(const uint16_t *p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void *)p;
}
__device__ __forceinline__ void load_lds16(const uint16_t *g, uint32_t lds) {
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

template <bool kPacked>
__global__ __launch_bounds__(kTileThreads, 1) void logprob_tile_kernel(LogprobArgs a) {
  const int id = blockIdx.x;
  const int xcd = id % kXcds, slot = id / kXcds;
  const int chunk = (slot / a.token_blocks) * kXcds + xcd;
  const int tblock = slot - (slot / a.token_blocks) * a.token_blocks;
  if (chunk >= a.chunks) return;

  __shared__ __attribute__((aligned(1024))) uint16_t sA[kTileStages][kTileElemsA];
  __shared__ __attribute__((aligned(1024))) uint16_t sB[kTileStages][kTileElems];
  __shared__ float s_m[4][kTileRows];
  __shared__ float s_l[4][kTileRows];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int v0 = chunk * kTileRowsA, t0 = tblock * kTileRows;

  // ---- loads: instructions kLoadsA * wave + k of the W region, kLoadsB *
  // wave + k of the h region ----
  const uint16_t *ga[kLoadsA], *gb[kLoadsB];
#pragma unroll
  for (int k = 0; k < kLoadsA; ++k) {
    const int r = 16 * (kLoadsA * wave + k) + lane / 4;
    const int lc = (lane % 4) ^ ((r >> 2) & 3);
    const int v = v0 + r;
    // packed: 16-byte unit ((s / 2 * tiles + tile) * 4 + lc) * 64 + 32 (s % 2) + v % 32
    // (the part that depends on the step s is added per step)
    ga[k] = kPacked ? a.W + ((size_t)(v / 32) * 4 + lc) * kWave * 8 + (v % 32) * 8
                    : a.W + (size_t)min(v, a.V - 1) * a.D + 8 * lc;
  }
  const int nsteps = a.D / kTileDims;
  // h comes from its staged copy, which holds each (token block, step) as the
  // 16 KB image of its LDS region: load instruction j reads 1 KB contiguous
#pragma unroll
  for (int k = 0; k < kLoadsB; ++k)
    gb[k] = a.hp + (size_t)tblock * nsteps * kTileElems + (size_t)(kLoadsB * wave + k) * 512 +
            lane * 8;
  const int last = nsteps - 1;
  const uint32_t blkA = (uint32_t)(kLoadsA * wave) * 1024u, blkB = (uint32_t)(kLoadsB * wave) * 1024u;
  // offsets (elements) of step s in W and h; steps past the last repeat it
  // (branch-free, so that every step issues the same number of loads)
  // elements per 64-dim step of the packed copy (all of its 32-row tiles)
  const size_t pstride =
      (size_t)(((int64_t)a.V + kPackRows - 1) / kPackRows) * (kPackRows / 32) * 4 * kWave * 8;
  auto w_off = [&](int s) __attribute__((always_inline)) {
    return kPacked ? (size_t)(s >> 1) * pstride + (s & 1) * 32 * 8 : (size_t)s * kTileDims;
  };
  auto load = [&](int st, int s, int d) __attribute__((always_inline)) {
    if (d < kLoadsA)
      load_lds16(ga[d] + w_off(s), lds_address(sA[st]) + blkA + 1024u * d);
    else
      load_lds16(gb[d - kLoadsA] + (size_t)s * kTileElems,
                 lds_address(sB[st]) + blkB + 1024u * (d - kLoadsA));
  };
  constexpr int kLoadsPerStep = kLoadsA + kLoadsB;
  // refill load d of a step goes after product kLoadAfter[d] of its 24
  constexpr int kLoadAfter[kLoadsPerStep] = {3, 8, 13, 18, 22};

  const int col = lane & 31, half = lane >> 5;
  const int wv = wave & 3, wt = wave >> 2;
  const int swz = (col >> 2) & 3;   // slot swizzle of every operand row (rows differ from col by multiples of 32)
  const int rowA = (96 * wv + col) * kTileDims, rowB = (128 * wt + col) * kTileDims;
  f32x16 acc[3][4];
#pragma unroll
  for (int i = 0; i < 3; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
  auto lds16 = [](const uint16_t *p) __attribute__((always_inline)) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
  };
  // Step s on stage st: wait until my loads for it have landed (the next
  // step's may still be in flight), barrier (everyone's have, and everyone is
  // done reading the stage used last step), then the products, with the
  // loads of step s + 2 into that freed stage between them.
  auto step = [&](int st, int s) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(kWaitVm5);
    __builtin_amdgcn_s_barrier();
    const uint16_t *A = sA[st], *B = sB[st];
    const int rs = min(s + kTileStages - 1, last), rst = (st + kTileStages - 1) % kTileStages;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = 8 * ((2 * half + u) ^ swz);
      bf16x8 av[3], bv[4];
#pragma unroll
      for (int i = 0; i < 3; ++i) av[i] = lds16(A + rowA + c + 32 * kTileDims * i);
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = lds16(B + rowB + c + 32 * kTileDims * j);
#pragma unroll
      for (int i = 0; i < 3; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = mfma32x32x16(av[i], bv[j], acc[i][j]);
          const int p = 12 * u + 4 * i + j;   // product index in the step, 0..23
#pragma unroll
          for (int d = 0; d < kLoadsPerStep; ++d)
            if (p == kLoadAfter[d]) {
              __builtin_amdgcn_sched_barrier(0);
              load(rst, rs, d);
              __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
  };
#pragma unroll
  for (int k = 0; k < kTileStages - 1; ++k)
#pragma unroll
    for (int d = 0; d < kLoadsPerStep; ++d) load(k, min(k, last), d);
  for (int s = 0; s < nsteps; s += kTileStages) {
#pragma unroll
    for (int k = 0; k < kTileStages; ++k)
      if (s + k < nsteps) step(k, s + k);
  }
  // the last loads (repeats of the last step) must land before the
  // workgroup's LDS is released
  __builtin_amdgcn_s_waitcnt(kWaitVm0);

  // ---- logits -> (max, sum) per token over this wave's 96 rows ----
  // Lane l holds, for token t0 + 128 wt + 32 j + col, the logits of rows
  // v0 + 96 wv + 32 i + 8 (r / 4) + 4 half + r % 4, r = 0..15.
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int tc = 128 * wt + 32 * j + col, t = t0 + tc;
    const int target = t < a.N ? a.targets[t] : -1;
    float y[3][16];
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = v0 + 96 * wv + 32 * i + 8 * (r >> 2) + 4 * half + (r & 3);
        y[i][r] = v < a.V ? acc[i][j][r] * a.scale_log2 : -INFINITY;
        m = fmaxf(m, y[i][r]);
        if (v == target) a.tgt[t] = acc[i][j][r] * a.scale;
      }
    m = pair_max(m);
    const float m_use = m == -INFINITY ? 0.f : m;
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) sum += fast_exp2(y[i][r] - m_use);
    sum = pair_sum(sum);
    if (half == 0) {
      s_m[wv][tc] = m;
      s_l[wv][tc] = sum;
    }
  }
  __syncthreads();
  // merge the four row groups: one thread per token of the tile
  const int c = threadIdx.x;
  if (c < kTileRows && t0 + c < a.N) {
    float M = s_m[0][c];
#pragma unroll
    for (int w = 1; w < 4; ++w) M = fmaxf(M, s_m[w][c]);
    const float M_use = M == -INFINITY ? 0.f : M;
    float L = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) L += s_l[w][c] * fast_exp2(s_m[w][c] - M_use);
    const size_t part = (size_t)(t0 + c) * a.chunks + chunk;
    a.ws_m[part] = M;
    a.ws_l[part] = L;
  }
}

// h staged for the tiled kernel: 16-byte unit u = ((tb * steps + s) * 256 + r) * 4
// + slot holds token 256 tb + r (zeros past N), dims 32 s + 8 (slot ^ ((r / 4) % 4))
// + 0..7 -- the LDS image of token block tb's step s.
__global__ __launch_bounds__(256) void logprob_stage_h_kernel(const uint16_t *__restrict__ h,
                                                              int32_t N, int32_t D, size_t units,
                                                              uint16_t *__restrict__ hp) {
  const size_t steps = (size_t)(D / kTileDims);
  for (size_t u = (size_t)blockIdx.x * blockDim.x + threadIdx.x; u < units;
       u += (size_t)gridDim.x * blockDim.x) {
    const int slot = (int)(u & 3);
    const size_t row = u >> 2;
    const int r = (int)(row % kTileRows);
    const size_t q = row / kTileRows, s = q % steps, tb = q / steps;
    const size_t t = tb * kTileRows + r;
    const int lc = slot ^ ((r >> 2) & 3);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (t < (size_t)N) v = load_u32x4(h + t * D + kTileDims * s + 8 * lc);
    store_u32x4(hp + 8 * u, v);
  }
}

// Packed copy of W: 16-byte unit i = ((s * tiles + tile) * 4 + u) * 64 + lane
// holds W[32 tile + lane % 32][64 s + 32 (lane / 32) + 8 u + 0..7] (zeros for
// rows past V; tiles = the copy's rows / 32).
__global__ __launch_bounds__(256) void logprob_pack_kernel(const uint16_t *__restrict__ W,
                                                           int32_t V, int32_t D, size_t units,
                                                           uint16_t *__restrict__ Wp) {
  const size_t steps = (size_t)(D / kDimStep);
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < units;
       i += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(i % kWave), u = (int)((i / kWave) % 4);
    const size_t ntiles = units / (4 * kWave * steps);
    const size_t tile = (i / (4 * kWave)) % ntiles, s = i / (4 * kWave * ntiles);
    const size_t row = 32 * tile + (lane & 31);
    const size_t dim = kDimStep * s + 32 * (lane >> 5) + 8 * u;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < (size_t)V) v = load_u32x4(W + row * D + dim);
    store_u32x4(Wp + 8 * i, v);
  }
}

__global__ __launch_bounds__(kLpThreads) void logprob_combine_kernel(LogprobArgs a, float *logp,
                                                                   float *lse) {
  // One workgroup per token: thread i folds chunks i, i + 256, ... in order;
  // the lanes of a wave are combined by a fixed butterfly and the four waves
  // in wave order, so the result does not depend on timing.
  __shared__ float s_red[2][kLpWaves];
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int t = blockIdx.x;
  const float *m = a.ws_m + (size_t)t * a.chunks;
  const float *l = a.ws_l + (size_t)t * a.chunks;
  float M = -INFINITY;
  for (int c = threadIdx.x; c < a.chunks; c += kLpThreads) M = fmaxf(M, m[c]);
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) M = fmaxf(M, __shfl_xor(M, o));
  if (lane == 0) s_red[0][wave] = M;
  __syncthreads();
  M = fmaxf(fmaxf(s_red[0][0], s_red[0][1]), fmaxf(s_red[0][2], s_red[0][3]));
  float L = 0.f;
  for (int c = threadIdx.x; c < a.chunks; c += kLpThreads) L += l[c] * fast_exp2(m[c] - M);
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) L += __shfl_xor(L, o);
  if (lane == 0) s_red[1][wave] = L;
  __syncthreads();
  if (threadIdx.x == 0) {
    L = ((s_red[1][0] + s_red[1][1]) + s_red[1][2]) + s_red[1][3];
    const float ls = (M + __log2f(L)) * kLn2;
    const int target = a.targets[t];
    logp[t] = target >= 0 && target < a.V ? a.tgt[t] - ls : __builtin_nanf("");
    if (lse) lse[t] = ls;
  }
}

}  // namespace

int32_t logprob_chunks(int32_t N, int32_t V) {
  const int rows = N >= kTileMinN ? kTileRowsA : kVocabChunk;
  return (int32_t)(((int64_t)V + rows - 1) / rows);
}

// The packed copy covers every row a workgroup reads: V rounded up to whole
// 384-row chunks (so to whole 128-row chunks too).
size_t logprob_packed_bytes(int32_t V, int32_t D) {
  return (size_t)(((int64_t)V + kPackRows - 1) / kPackRows) * kPackRows * D * sizeof(uint16_t);
}

hipError_t launch_logprob_pack(const uint16_t *W, int32_t V, int32_t D, uint16_t *Wp,
                               hipStream_t stream) {
  const size_t units = logprob_packed_bytes(V, D) / 16;
  const size_t want = (units + 255) / 256, blocks = want < 65536 ? want : 65536;
  hipLaunchKernelGGL(logprob_pack_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, W, V, D,
                     units, Wp);
  return hipGetLastError();
}

namespace {
// per-(token, chunk) partials and the target logits
size_t logprob_partial_bytes(int32_t N, int32_t V) {
  return ((size_t)N * logprob_chunks(N, V) * 2 + (size_t)N) * sizeof(float);
}
}  // namespace

// The partials, then (from N = kTileMinN) the staged copy of h at the next
// 256-byte boundary: N rounded up to whole 256-token blocks x D bf16.
size_t logprob_workspace_bytes(int32_t N, int32_t V, int32_t D) {
  const size_t partials = (logprob_partial_bytes(N, V) + 255) / 256 * 256;
  if (N < kTileMinN) return logprob_partial_bytes(N, V);
  return partials + (size_t)((N + kTileRows - 1) / kTileRows) * kTileRows * D * sizeof(uint16_t);
}

namespace {
int logprob_tiles(int32_t N) { return N <= 64 ? 2 : kMaxTiles; }
// tokens per workgroup
int logprob_token_block(int32_t N) { return N >= kTileMinN ? kTileRows : 32 * logprob_tiles(N); }
}  // namespace

int64_t logprob_grid(int32_t N, int32_t V) {
  const int64_t chunks_pad = (logprob_chunks(N, V) + kXcds - 1) / kXcds * kXcds;
  const int block = logprob_token_block(N);
  return chunks_pad * ((N + block - 1) / block);
}

hipError_t launch_logprob(const uint16_t *h, const uint16_t *W, const int32_t *targets, int32_t N,
                          int32_t V, int32_t D, float scale, float *logp, float *lse,
                          void *workspace, bool packed, hipStream_t stream) {
  LogprobArgs a;
  a.h = h;
  a.hp = nullptr;
  a.W = W;
  a.targets = targets;
  a.N = N;
  a.V = V;
  a.D = D;
  a.chunks = logprob_chunks(N, V);
  const int tiles = logprob_tiles(N);
  a.token_blocks = (N + logprob_token_block(N) - 1) / logprob_token_block(N);
  a.ws_m = static_cast<float *>(workspace);
  a.ws_l = a.ws_m + (size_t)N * a.chunks;
  a.tgt = a.ws_l + (size_t)N * a.chunks;
  a.scale = scale;
  a.scale_log2 = scale * kLog2e;
  const dim3 grid((unsigned)logprob_grid(N, V));
  if (N >= kTileMinN) {
    uint16_t *hp = reinterpret_cast<uint16_t *>(static_cast<char *>(workspace) +
                                                (logprob_partial_bytes(N, V) + 255) / 256 * 256);
    a.hp = hp;
    const size_t units = (size_t)a.token_blocks * kTileRows * D / 8;
    const size_t want = (units + 255) / 256, blocks = want < 65536 ? want : 65536;
    hipLaunchKernelGGL(logprob_stage_h_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, h, N,
                       D, units, hp);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (N >= kTileMinN && packed)
    hipLaunchKernelGGL(logprob_tile_kernel<true>, grid, dim3(kTileThreads), 0, stream, a);
  else if (N >= kTileMinN)
    hipLaunchKernelGGL(logprob_tile_kernel<false>, grid, dim3(kTileThreads), 0, stream, a);
  else if (tiles == 2 && packed)
    hipLaunchKernelGGL((logprob_partial_kernel<2, true>), grid, dim3(kLpThreads), 0, stream, a);
  else if (tiles == 2)
    hipLaunchKernelGGL((logprob_partial_kernel<2, false>), grid, dim3(kLpThreads), 0, stream, a);
  else if (packed)
    hipLaunchKernelGGL((logprob_partial_kernel<kMaxTiles, true>), grid, dim3(kLpThreads), 0,
                       stream, a);
  else
    hipLaunchKernelGGL((logprob_partial_kernel<kMaxTiles, false>), grid, dim3(kLpThreads), 0,
                       stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(logprob_combine_kernel, dim3((unsigned)N), dim3(kLpThreads), 0, stream, a,
                     logp, lse);
  return hipGetLastError();
}

}  // namespace ra
