// Append attention tile (causal chunked prefill against the paged cache),
// run by the planned persistent kernel for append calls and for mixed
// decode + append calls.
//
// One workgroup (8 waves, two per SIMD) owns a block of QB = 256 / G
// consecutive queries of one row and all G query heads of one KV head: 256
// "query rows" (query, head), 32 per wave, each wave's rows forming the 32
// columns of its 32x32 matrix tiles with their Q^T operands in registers.
// The key loop walks the row's pages 64 keys (4 pages) at a time. Each block
// of K and V is loaded once per workgroup into registers and stored to a ring
// of four LDS buffers, one barrier per block, and all eight waves consume it:
//   S^T[key][qrow] = K[key][:] · Q^T[:][qrow]        (bf16 mfma 32x32x16, fp32)
//   O^T[d][qrow]  += V^T[d][key] · P^T[key][qrow]    (P rounded to bf16)
// The work is software-pipelined over pairs of pages (32 keys): the step that
// takes the softmax of pair p also issues the P·V products of pair p - 1 and
// the score products of pair p + 1, none of which depends on that softmax, so
// the matrix cores are kept busy by the same wave while it exponentiates.
// Keys are ordered inside each pair of pages so that the 16 S values a lane
// receives are, in order, 8 consecutive slots of the first page and the same
// 8 slots of the second: exactly the P^T operands of the two P·V products it
// takes part in (no shuffles). Each query row stays in one lane column (two
// lanes), so the online-softmax state is lane-local. Weights are taken
// against a running max that moves only when they would grow too large
// (a per-wave check on the weight sums), so the common path has no max
// reduction and no cross-lane exchange. The causal mask (key position >
// ctx + i) is applied only on blocks that reach past the wave's first query
// position.
#pragma once

#include <type_traits>

#include "ra_device.h"
#include "ra_internal.h"

// Everything lives in ra::atile, apart from the decode-split names (ra::dsplit)
// that share a translation unit with it in the mixed kernel.
namespace ra {
namespace atile {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerGroup = kWaves * kRowsPerWave;   // 256
constexpr int kBlock = 64;                             // keys per staged block
constexpr int kBlockPages = kBlock / kPage;            // 4
constexpr int kPagesPerPass = kThreads / 256;          // pages one staging pass covers
constexpr int kPasses = kBlockPages / kPagesPerPass;   // 2
constexpr int kBlockElems = kBlock * kHeadDim;         // per pool, per buffer
constexpr float kSumLimit = 16384.f;                  // weight-sum bound between rescales

struct AppendArgs {
  const uint16_t *q;
  const uint16_t *k_pool;
  const uint16_t *v_pool;
  const int32_t *block_table;
  const int32_t *cu_q;
  const int32_t *ctx_lens;
  float *out;
  float *lse;
  int32_t hq, hkv, group, bt_stride, num_pages, total_q, max_q_len, max_kv_len, q_per_block;
  float scale_log2;   // softmax scale * log2(e) (* k_scale for fp8 pools)
  float v_scale;      // multiplies the output (fp8 pools; 1 for bf16)
  const float *cos_sin;   // rotary table [rope_rows][128] for q (kernels built for it)
  int32_t rope_rows;
};

// D(32x32, fp32) += A(32x16, bf16) * B(16x32, bf16). Lane l supplies A row
// (l % 32) and B column (l % 32), contraction slots 8 (l / 32) + 0..7; it
// receives D rows 8 (r / 4) + 4 (l / 32) + r % 4 of column l % 32, r = 0..15.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Max of x over lanes l and l ^ 32 (one v_permlane32_swap: each lane gets
// both values of its pair, in some order).
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ bf16x8 lds_bf16x8(const uint16_t *p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

// LDS layouts (per buffer). K: 64 key rows x 128 dims, rows padded to
// 272 B, so that 16 lanes reading the same chunk of 16 different rows (or 16
// chunks of one row) fall on distinct banks, and a lane's eight operand reads
// are one base address plus immediate offsets. V: [page][d][16 slots] (32 B
// rows); the two 8-slot halves of row d are swapped when bit 3 of d is set,
// for the same reason.
constexpr int kKPitch = kHeadDim + 8;                   // K row pitch (elements)
constexpr int kKBlockElems = kBlock * kKPitch;          // K buffer (elements)
__device__ __forceinline__ int k_lds(int row, int chunk) { return row * kKPitch + chunk * 8; }
__device__ __forceinline__ int v_lds(int page, int d, int half) {
  return (page * kHeadDim + d) * kPage + ((half ^ ((d >> 3) & 1)) * 8);
}

// LDS of one tile: a ring of four K and V blocks (block B in buffer B % 4).
constexpr int kBuffers = 4;
struct AppendLds {
  __attribute__((aligned(16))) uint16_t k[kBuffers * kKBlockElems];
  __attribute__((aligned(16))) uint16_t v[kBuffers * kBlockElems];
};

// Row b's chunk: its first query in q / out (cu0), its length T and the
// tokens cached before it (ctx), clamped so that no access leaves the
// caller's arrays. ctx < 0 marks a row whose chunk does not fit max_kv_len.
struct AppendRow {
  int cu0, T, ctx;
};
__device__ __forceinline__ AppendRow append_row(const AppendArgs &a, int b) {
  AppendRow r;
  r.cu0 = min(max(a.cu_q[b], 0), a.total_q);
  r.T = min(min(max(a.cu_q[b + 1] - r.cu0, 0), a.max_q_len), a.total_q - r.cu0);
  r.ctx = min(max(a.ctx_lens[b], 0), a.max_kv_len - r.T);
  return r;
}

// Key blocks that query block qblk of row b walks (0: nothing to compute).
__device__ __forceinline__ int append_tile_blocks(const AppendArgs &a, const AppendRow &r,
                                                  int qblk) {
  const int i0 = qblk * a.q_per_block;
  if (i0 >= r.T || r.ctx < 0) return 0;
  return (r.ctx + min(r.T, i0 + a.q_per_block) + kBlock - 1) / kBlock;
}

// One tile: query block qblk of row b, KV head g, by a workgroup of kThreads
// threads. Every thread of the workgroup calls it with the same arguments.
// kFp8: the pools hold E4M3 codes; the staging converts them exactly to bf16
// on their way into LDS, so everything after the staging is the bf16 tile.
// kRope: q is rotated at its position (table a.cos_sin) after it is loaded.
template <bool kPosScale, bool kFp8 = false, bool kRope = false>
__device__ __forceinline__ void append_tile(const AppendArgs &a, int qblk, int g, int b,
                                            AppendLds &lds) {
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int col = lane & 31, grp = lane >> 5;
  const int G = a.group, QB = a.q_per_block;

  const AppendRow row_ext = append_row(a, b);
  const int cu0 = row_ext.cu0, T = row_ext.T, ctx = row_ext.ctx;
  const int i0 = qblk * QB;
  if (i0 >= T || ctx < 0) return;
  const int i_end = min(T, i0 + QB);
  const int row_end = ctx + T;                 // keys present in the cache for this row
  const int kv_end = ctx + i_end;              // keys this workgroup attends to
  const int row_pages = (row_end + kPage - 1) / kPage;
  const int nblocks = (kv_end + kBlock - 1) / kBlock;
  const int32_t *bt = a.block_table + (size_t)b * a.bt_stride;
  const size_t head_stride = (size_t)kPage * kHeadDim;

  uint16_t *const sK = lds.k;
  uint16_t *const sV = lds.v;

  // ---- this lane's query row and Q^T operands (dims 16 kk + 8 grp + 0..7) ----
  const int r_wg = wave * kRowsPerWave + col;
  const int qi = r_wg / G, hh = r_wg - qi * G;
  const bool q_valid = r_wg < QB * G && i0 + qi < i_end;
  const int qpos = q_valid ? ctx + i0 + qi : -1;
  bf16x8 qop[8];
  if (q_valid) {
    const uint16_t *qp =
        a.q + ((size_t)(cu0 + i0 + qi) * a.hq + (size_t)g * G + hh) * kHeadDim + 8 * grp;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) qop[kk] = load_bf16x8(qp + 16 * kk);
  } else {
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) qop[kk] = bf16x8{};
  }
  if constexpr (kRope) {
    // q rotated at its position: the lane's dims 16 kk + 8 grp + 0..7 (kk < 4)
    // pair with dims 64 + the same, held in qop[kk + 4]
    const float *cs =
        a.cos_sin + (size_t)min(max(qpos, 0), a.rope_rows - 1) * kHeadDim + 8 * grp;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const f32x8 c = *reinterpret_cast<const f32x8 *>(cs + 16 * kk);
      const f32x8 sn = *reinterpret_cast<const f32x8 *>(cs + kHeadDim / 2 + 16 * kk);
      const bf16x8 lo = qop[kk], hi = qop[kk + 4];
      qop[kk] = rope8(lo, hi, c, sn, false);
      qop[kk + 4] = rope8(hi, lo, c, sn, true);
    }
  }
  // First query position of this wave (its rows are query-major).
  const int wave_q0 = ctx + i0 + (wave * kRowsPerWave) / G;

  // ---- staging: pass p moves pages 2p, 2p + 1 of the block; each thread one
  // 16-byte chunk of K and one of V. The page index is wave-uniform (waves
  // 0-3 stage the first page of a pass, 4-7 the second), so the block-table
  // read and the page base run on the scalar unit.
  const int st_page = __builtin_amdgcn_readfirstlane(tid >> 8), st_chunk = tid & 255;
  const int st_slot = st_chunk >> 4, st_kch = st_chunk & 15;   // K: slot, 16-B chunk
  const int st_d = st_chunk >> 1, st_half = st_chunk & 1;      // V: dim row, 8-slot half
  u32x4 kreg[kPasses], vreg[kPasses];
  // fp8 pools (2 KiB per page and head): one pass covers the block; thread
  // -> page tid / 128 (wave-uniform), K: slot and 16-dim chunk, V: one dim
  // row (all 16 slots).
  const int f_page = __builtin_amdgcn_readfirstlane(tid >> 7), f_idx = tid & 127;
  const int f_slot = f_idx >> 3, f_c16 = f_idx & 7;
  auto stage_load = [&](int blk) __attribute__((always_inline)) {
    if constexpr (kFp8) {
      const int pgi = blk * kBlockPages + f_page;
      const int id = clamp_page(pgi < row_pages ? bt[pgi] : bt[0], a.num_pages);
      const size_t base = ((size_t)id * a.hkv + g) * head_stride;   // bytes
      kreg[0] = *reinterpret_cast<const u32x4 *>(reinterpret_cast<const uint8_t *>(a.k_pool) +
                                                 base + f_slot * kHeadDim + f_c16 * 16);
      vreg[0] = *reinterpret_cast<const u32x4 *>(reinterpret_cast<const uint8_t *>(a.v_pool) +
                                                 base + f_idx * kPage);
      return;
    }
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int pgi = blk * kBlockPages + p * kPagesPerPass + st_page;
      const int id = clamp_page(pgi < row_pages ? bt[pgi] : bt[0], a.num_pages);
      const size_t base = ((size_t)id * a.hkv + g) * head_stride;
      kreg[p] = load_u32x4(a.k_pool + base + st_slot * kHeadDim + st_kch * 8);
      vreg[p] = load_u32x4(a.v_pool + base + st_d * kPage + st_half * 8);
    }
  };
  auto stage_store = [&](int blk, int buf) __attribute__((always_inline)) {
    if constexpr (kFp8) {
      const int pos0 = (blk * kBlockPages + f_page) * kPage;
      const bf16x8 k0 = fp8x8_to_bf16x8(u32x2{kreg[0][0], kreg[0][1]});
      const bf16x8 k1 = fp8x8_to_bf16x8(u32x2{kreg[0][2], kreg[0][3]});
      bf16x8 v0 = fp8x8_to_bf16x8(u32x2{vreg[0][0], vreg[0][1]});   // slots 0..7
      bf16x8 v1 = fp8x8_to_bf16x8(u32x2{vreg[0][2], vreg[0][3]});   // slots 8..15
      if (pos0 + kPage > row_end) {   // V slots past the row's end become zeros
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          v0[e] = pos0 + e < row_end ? v0[e] : (__bf16)0.f;
          v1[e] = pos0 + 8 + e < row_end ? v1[e] : (__bf16)0.f;
        }
      }
      uint16_t *kd = &sK[buf * kKBlockElems + k_lds(f_page * kPage + f_slot, 2 * f_c16)];
      *reinterpret_cast<bf16x8 *>(kd) = k0;
      *reinterpret_cast<bf16x8 *>(kd + 8) = k1;
      *reinterpret_cast<bf16x8 *>(&sV[buf * kBlockElems + v_lds(f_page, f_idx, 0)]) = v0;
      *reinterpret_cast<bf16x8 *>(&sV[buf * kBlockElems + v_lds(f_page, f_idx, 1)]) = v1;
      return;
    }
#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int j = p * kPagesPerPass + st_page;        // page in the block
      const int pos0 = (blk * kBlockPages + j) * kPage;
      // V slots at or past the row's end may hold anything (NaN included):
      // they are stored as zeros, so that a zero weight cannot meet a NaN in
      // the P·V product. K slots there need nothing: every key at or past
      // the row's end lies beyond the causal limit of every query, and its
      // score is replaced by -inf (a select, not an arithmetic mask).
      u32x4 vw = vreg[p];
      if (pos0 + kPage > row_end) {
        const int vpos = pos0 + st_half * 8;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo = vpos + 2 * e < row_end ? 0xffffu : 0u;
          const uint32_t hi = vpos + 2 * e + 1 < row_end ? 0xffff0000u : 0u;
          vw[e] &= lo | hi;
        }
      }
      *reinterpret_cast<u32x4 *>(&sK[buf * kKBlockElems + k_lds(j * kPage + st_slot, st_kch)]) =
          kreg[p];
      *reinterpret_cast<u32x4 *>(&sV[buf * kBlockElems + v_lds(j, st_d, st_half)]) = vw;
    }
  };

  // ---- operand addressing. A row i of an S tile holds key pi(i): bits 2 and
  // 3 of i swapped, so that lane l's value r is key 16 (r / 8) + 8 grp + r % 8.
  const int ka_key = (col & ~12) | ((col & 4) << 1) | ((col & 8) >> 1);
  // With a positive scale the scores stay raw and the scale is folded into
  // the exponent's FMA; otherwise scores are scaled first.
  const float c2 = a.scale_log2;
  const float cs = kPosScale ? c2 : 1.f;

  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;   // running max (scaled, base 2) and sum

  // S^T of pair pp of the block in LDS buffer buf: 32 keys x 32 query rows.
  auto scores = [&](int buf, int pp) __attribute__((always_inline)) {
    const uint16_t *kl = sK + buf * kKBlockElems;
    const int krow = 32 * pp + ka_key;
    f32x16 st = f32x16{};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk)
      st = mfma32x32x16(lds_bf16x8(&kl[k_lds(krow, 2 * kk + grp)]), qop[kk], st);
    return st;
  };

  // Software pipeline over pairs of pages (32 keys). Step p computes the
  // softmax of pair p while the matrix cores run P·V of pair p - 1 and the
  // scores of pair p + 1, none of which depends on it. Blocks of 64 keys
  // rotate through four LDS buffers: while block B is computed, block B - 1
  // is still read (V of its last pair), block B + 1 is complete (keys of the
  // look-ahead scores) and block B + 2 is being stored. Block -1 (the last
  // buffer) holds zero V operands (its second pair) for the first step's P·V,
  // whose weights are zero too.
  static_assert(kThreads * 8 == kBlockElems / 2, "one 16-byte store per thread");
  *reinterpret_cast<u32x4 *>(&sV[(kBuffers - 1) * kBlockElems + kBlockElems / 2 + 8 * tid]) =
      u32x4{};
  stage_load(0);
  stage_store(0, 0);
  if (nblocks > 1) {
    stage_load(1);
    stage_store(1, 1);
  }
  __syncthreads();
  f32x16 st = scores(0, 0);
  bf16x8 pb0 = bf16x8{}, pb1 = bf16x8{};   // weights of the previous pair (none yet)

  // P·V of pair pp of the block in buffer buf, weights pb0, pb1:
  // O^T[d][qrow] += V^T[d][key] P^T[key][qrow], page c of the pair, slots
  // 8 grp + 0..7, d = 32 dt + col
  auto pv = [&](int buf, int pp) __attribute__((always_inline)) {
    const uint16_t *vl = sV + buf * kBlockElems;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      o[dt] = mfma32x32x16(lds_bf16x8(&vl[v_lds(2 * pp, 32 * dt + col, grp)]), pb0, o[dt]);
      o[dt] = mfma32x32x16(lds_bf16x8(&vl[v_lds(2 * pp + 1, 32 * dt + col, grp)]), pb1, o[dt]);
    }
  };

  // One step: pair pp of the block starting at key key0. (vbuf, vpp): the
  // previous pair, whose P·V is issued now; (kbuf, kpp): the next pair, whose
  // scores are computed now. mask_tag: the block reaches past the wave's
  // first query (causal mask on).
  auto step = [&](int vbuf, int vpp, int kbuf, int kpp, int pp, int key0, auto mask_tag)
      __attribute__((always_inline)) {
    constexpr bool kMask = decltype(mask_tag)::value;
    pv(vbuf, vpp);   // the previous pair
    // scores of the next pair
    const f32x16 st_next = scores(kbuf, kpp);

    float sc[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) sc[r] = kPosScale ? st[r] : st[r] * c2;
    if constexpr (kMask) {
      // value r is key key0 + 32 pp + 8 grp + 16 (r / 8) + r % 8; masked past qpos
      const int rel = qpos - key0 - 32 * pp - 8 * grp;
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[r] = 16 * (r >> 3) + (r & 7) > rel ? -INFINITY : sc[r];
    }
    // Weights against the running max m_run. It is only moved (and O, l
    // rescaled) when some lane's weights sum past kSumLimit, or are not
    // finite (the first pair, while m_run is still -inf); the weights are
    // then recomputed against the new max. Between moves every weight
    // stays below kSumLimit, which fp32 and bf16 carry without loss, and
    // out = O / l does not depend on when the max moves.
    float psum;
    auto weights = [&]() __attribute__((always_inline)) {
      f32x8 p0, p1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p0[e] = fast_exp2(__builtin_fmaf(sc[e], cs, -m_run));
        p1[e] = fast_exp2(__builtin_fmaf(sc[8 + e], cs, -m_run));
      }
      pb0 = to_bf16x8(p0);
      pb1 = to_bf16x8(p1);
      const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
      float s0 = 0.f, s1 = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb0[2 * e], pb0[2 * e + 1]}, one, s0, false);
        s1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb1[2 * e], pb1[2 * e + 1]}, one, s1, false);
      }
      psum = s0 + s1;
    };
    weights();
    if (!__all(psum <= kSumLimit)) {
      float mx = fmaxf(fmaxf(sc[0], sc[1]), sc[2]);
#pragma unroll
      for (int r = 3; r < 15; r += 2) mx = fmaxf(fmaxf(mx, sc[r]), sc[r + 1]);
      mx = fmaxf(mx, sc[15]);
      mx = pair_max(mx);
      if (kPosScale) mx *= c2;
      float m_new = fmaxf(m_run, mx);
      if (m_new == -INFINITY) m_new = 0.f;   // nothing attended yet: any finite reference
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) o[dt] *= alpha;
      weights();
    }
    l_run += psum;
    st = st_next;
  };

  auto block = [&](int blk, auto mask_tag) __attribute__((always_inline)) {
    const int bcur = blk % kBuffers, bprev = (blk + kBuffers - 1) % kBuffers,
              bnext = (blk + 1) % kBuffers;
    if (blk + 2 < nblocks) stage_load(blk + 2);
    const int key0 = blk * kBlock;
    step(bprev, 1, bcur, 1, 0, key0, mask_tag);
    step(bcur, 0, bnext, 0, 1, key0, mask_tag);
    if (blk + 2 < nblocks) stage_store(blk + 2, (blk + 2) % kBuffers);
    __syncthreads();
  };
  // Blocks from mb on reach past the wave's first query and take the causal
  // mask; every wave passes the same barriers (one per block).
  const int mb = __builtin_amdgcn_readfirstlane(min(nblocks, (wave_q0 + 1) / kBlock));
  int blk = 0;
  for (; blk < mb; ++blk) block(blk, std::false_type{});
  for (; blk < nblocks; ++blk) block(blk, std::true_type{});
  pv((nblocks - 1) % kBuffers, 1);   // the last pair

  // ---- epilogue: normalise and store; lane holds d = 32 dt + 8 (r/4) + 4 grp + r%4 ----
  const float l = l_run + __shfl_xor(l_run, 32);
  if (qpos >= 0) {
    const size_t row = (size_t)(cu0 + i0 + qi) * a.hq + (size_t)g * G + hh;
    const float inv = (kFp8 ? a.v_scale : 1.f) / l;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = o[dt][4 * rq + e] * inv;
        *reinterpret_cast<f32x4 *>(&a.out[row * kHeadDim + 32 * dt + 8 * rq + 4 * grp]) = v;
      }
    if (a.lse && grp == 0) a.lse[row] = (m_run + __log2f(l)) * kLn2;
  }
}

// Kernel arguments of an append call (validated by the ABI layer).
inline AppendArgs make_append_args(const uint16_t *q, const int32_t *cu_q,
                                   const int32_t *ctx_lens, const PagedKV &kv, int32_t hq,
                                   int32_t total_q, int32_t max_q_len, int32_t max_kv_len,
                                   float scale, float *out, float *lse) {
  AppendArgs a;
  a.q = q;
  a.k_pool = kv.k_pool;
  a.v_pool = kv.v_pool;
  a.block_table = kv.block_table;
  a.cu_q = cu_q;
  a.ctx_lens = ctx_lens;
  a.out = out;
  a.lse = lse;
  a.hq = hq;
  a.hkv = kv.hkv;
  a.group = hq / kv.hkv;
  a.bt_stride = kv.bt_stride;
  a.num_pages = kv.num_pages;
  a.total_q = total_q;
  a.max_q_len = max_q_len;
  a.max_kv_len = max_kv_len;
  a.q_per_block = kRowsPerGroup / a.group;
  a.scale_log2 = scale * kLog2e * kv.k_scale;
  a.v_scale = kv.v_scale;
  a.cos_sin = nullptr;
  a.rope_rows = 0;
  return a;
}

}  // namespace atile
}  // namespace ra
