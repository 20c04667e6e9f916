// Append attention: causal chunked prefill of new observation tokens against
// each trajectory's paged cache.
//
// One workgroup (4 waves) owns a block of QB = 256 / G consecutive queries of
// one row and all G query heads of one KV head: 256 "query rows" (query,
// head), 64 per wave, as four 16-wide matrix columns per wave. The key loop
// walks the row's pages 64 keys (4 pages) at a time; each block of K and V is
// staged once in LDS (double buffered, one barrier per block) and consumed by
// all four waves from there:
//   S^T[key][qrow] = K[key][:] · Q^T[:][qrow]        (bf16 mfma 16x16x32, fp32)
//   O^T[d][qrow]  += V^T[d][key] · P^T[key][qrow]    (P rounded to bf16)
// Every K or V operand read from LDS feeds four matrix products (the wave's
// four columns). Keys are ordered inside each pair of pages so that a lane's
// S values are exactly the P^T operand it supplies next (no shuffles), and
// O^T keeps each query row in one lane column so that the online-softmax
// rescale is lane-local. The causal mask (key position > ctx + i) is applied
// only on blocks that reach past the wave's first query position.
#include "ra_device.h"
#include "ra_internal.h"

namespace ra {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;
constexpr int kCols = 4;                  // 16-wide matrix columns per wave
constexpr int kRowsPerWave = 16 * kCols;  // query rows per wave
constexpr int kRowsPerGroup = kWaves * kRowsPerWave;
constexpr int kBlock = 64;                // keys per staged block
constexpr int kBlockPages = kBlock / kPage;   // = kWaves: wave w stages page w
constexpr float kSlack = 8.f;             // lazy-rescale threshold (base-2 units)

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
  float scale_log2;
};

// K block in LDS: 64 key rows of 128 dims (256 B, no padding). The 16-byte
// chunk c of row R is stored at chunk c ^ swz(R): the 16 rows read together
// by one matrix operand load then fall on 16 distinct bank groups.
__device__ __forceinline__ int k_swz(int row) { return (row & 3) | (((row >> 3) & 3) << 2); }

// V block in LDS: [page][d][16 slots]; the two 8-slot halves of row d are
// swapped when bit 3 of d is set, for the same reason.
__device__ __forceinline__ int v_half(int d, int half) { return half ^ ((d >> 3) & 1); }

__global__ __launch_bounds__(kThreads, 1) void append_kernel(AppendArgs a) {
  const int qblk = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int col = lane & 15, kgrp = lane >> 4;
  const int G = a.group, QB = a.q_per_block;

  // Row extent, clamped so that no access leaves the caller's arrays.
  const int cu0 = min(max(a.cu_q[b], 0), a.total_q);
  const int T = min(min(max(a.cu_q[b + 1] - cu0, 0), a.max_q_len), a.total_q - cu0);
  const int i0 = qblk * QB;
  if (i0 >= T) return;
  const int ctx = min(max(a.ctx_lens[b], 0), a.max_kv_len - T);
  if (ctx < 0) return;
  const int i_end = min(T, i0 + QB);
  const int row_end = ctx + T;                 // keys present in the cache for this row
  const int kv_end = ctx + i_end;              // keys this workgroup attends to
  const int row_pages = (row_end + kPage - 1) / kPage;
  const int nblocks = (kv_end + kBlock - 1) / kBlock;
  const int32_t *bt = a.block_table + (size_t)b * a.bt_stride;
  const size_t head_stride = (size_t)kPage * kHeadDim;

  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kBlock * kHeadDim];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][kBlockPages * kHeadDim * kPage];

  // ---- this lane's query rows and Q^T operands ----
  int qpos[kCols];
  bf16x8 qop[kCols][4];
#pragma unroll
  for (int nt = 0; nt < kCols; ++nt) {
    const int r = wave * kRowsPerWave + nt * 16 + col;
    const int qi = r / G, hh = r - qi * G;
    const bool valid = r < QB * G && i0 + qi < i_end;
    qpos[nt] = valid ? ctx + i0 + qi : -1;
    if (valid) {
      const uint16_t *qp =
          a.q + ((size_t)(cu0 + i0 + qi) * a.hq + (size_t)g * G + hh) * kHeadDim + 8 * kgrp;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) qop[nt][kk] = load_bf16x8(qp + 32 * kk);
    } else {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) qop[nt][kk] = bf16x8{};
    }
  }
  // First query position of this wave (its rows are query-major).
  const int wave_q0 = ctx + i0 + (wave * kRowsPerWave) / G;

  // ---- staging: wave w copies page w of each block, K and V, straight
  // from HBM into LDS (global_load_lds, 16 bytes per lane, no registers).
  // The LDS destination of a lane is fixed (base + 16 * lane), so the swizzled
  // layout is produced by choosing which global chunk each lane fetches.
  // Slots past the row's end are not cleared here; their scores are always
  // masked (they lie beyond every query of the row) and their V entries are
  // replaced by zero when read (last block only).
  const int kr = lane >> 4, kpc = lane & 15;          // K: row in a 4-row chunk, phys. chunk
  const int vd = lane >> 1, vph = lane & 1;           // V: row in a 32-row chunk, phys. half
  auto stage = [&](int blk, int buf) {
    const int pgi = blk * kBlockPages + wave;
    const int id = clamp_page(pgi < row_pages ? bt[pgi] : bt[0], a.num_pages);
    const size_t base = ((size_t)id * a.hkv + g) * head_stride;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int row = wave * kPage + 4 * c + kr;      // row in the block
      const uint16_t *src = a.k_pool + base + (4 * c + kr) * kHeadDim + ((kpc ^ k_swz(row)) * 8);
      __builtin_amdgcn_global_load_lds(src, &sK[buf][(wave * kPage + 4 * c) * kHeadDim], 16, 0,
                                       0);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int d = 32 * c + vd;
      const uint16_t *src = a.v_pool + base + d * kPage + v_half(d, vph) * 8;
      __builtin_amdgcn_global_load_lds(src, &sV[buf][(wave * kHeadDim + 32 * c) * kPage], 16, 0,
                                       0);
    }
  };

  // ---- per-lane operand addressing inside a block ----
  // S tile t of pair pp, matrix row i = col holds key
  //   32 pp + 16 (col >> 3) + 8 ((col >> 2) & 1) + 4 t + (col & 3).
  const int ka_row = 16 * (col >> 3) + 8 * ((col >> 2) & 1) + (col & 3);  // + 32pp + 4t
  const int ka_swz = k_swz(ka_row);
  // S values / P^T / V^T operand of lane l: keys 32 pp + 16 (l >> 5) + 8 ((l >> 4) & 1) + e.
  const int sv_page = lane >> 5, sv_half = (lane >> 4) & 1;
  const int sv_key = 16 * sv_page + 8 * sv_half;                           // + 32pp + e
  const int va_half = v_half(col, sv_half);      // (16 mt + col) >> 3 has the bit of col

  f32x4 o[8][kCols];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
#pragma unroll
    for (int nt = 0; nt < kCols; ++nt) o[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[kCols], l_run[kCols];
#pragma unroll
  for (int nt = 0; nt < kCols; ++nt) {
    m_run[nt] = -INFINITY;
    l_run[nt] = 0.f;
  }

  stage(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int blk = 0; blk < nblocks; ++blk) {
    const int buf = blk & 1;
    if (blk + 1 < nblocks) stage(blk + 1, buf ^ 1);
    const uint16_t *k_lds = sK[buf];
    const uint16_t *v_lds = sV[buf];

    const int key0 = blk * kBlock;
    const bool need_mask = key0 + kBlock - 1 > wave_q0;
    const bool tail = key0 + kBlock > row_end;
    // The block is consumed one pair of pages (32 keys) at a time: scores,
    // online-softmax update, then the P·V product of that pair.
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      f32x4 st[2][kCols];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int nt = 0; nt < kCols; ++nt) st[t][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int row = 32 * pp + 4 * t + ka_row;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const bf16x8 ka = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4 *>(
                          &k_lds[row * kHeadDim + (((4 * kk + kgrp) ^ ka_swz) * 8)]));
#pragma unroll
          for (int nt = 0; nt < kCols; ++nt) st[t][nt] = mfma16x16x32(ka, qop[nt][kk], st[t][nt]);
        }
      }

      bf16x8 pb[kCols];
#pragma unroll
      for (int nt = 0; nt < kCols; ++nt) {
        float sc[8];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r) sc[4 * t + r] = st[t][nt][r] * a.scale_log2;
        if (need_mask) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int kpos = key0 + 32 * pp + sv_key + e;
            sc[e] = kpos > qpos[nt] ? -INFINITY : sc[e];
          }
        }
        float mx = sc[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sc[e]);
        mx = col_max4(mx);
        // Lazy rescaling: the running max only moves (and O, l are rescaled)
        // when a score exceeds it by more than 2^kSlack; otherwise the stale
        // max is kept and the weights may reach 2^kSlack, which fp32 and
        // bf16 carry without loss. out = O / l does not depend on the choice.
        const bool grow = mx > m_run[nt] + kSlack;
        if (__any(grow)) {
          const float m_new = grow ? mx : m_run[nt];
          const float alpha = grow ? fast_exp2(m_run[nt] - m_new) : 1.f;
          m_run[nt] = m_new;
          l_run[nt] *= alpha;
#pragma unroll
          for (int mt = 0; mt < 8; ++mt) o[mt][nt] *= alpha;
        }
        const float m_use = m_run[nt] == -INFINITY ? 0.f : m_run[nt];
        float psum = 0.f;
        f32x8 p;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          p[e] = fast_exp2(sc[e] - m_use);
          psum += p[e];
        }
        pb[nt] = to_bf16x8(p);
        l_run[nt] += psum;
      }

#pragma unroll
      for (int mt = 0; mt < 8; ++mt) {
        const int d = 16 * mt + col;
        bf16x8 va = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4 *>(
                        &v_lds[((2 * pp + sv_page) * kHeadDim + d) * kPage + va_half * 8]));
        if (tail) {
          // keys at or past the row's end: replace (not multiply) by zero
#pragma unroll
          for (int e = 0; e < 8; ++e)
            va[e] = key0 + 32 * pp + sv_key + e >= row_end ? (__bf16)0.f : va[e];
        }
#pragma unroll
        for (int nt = 0; nt < kCols; ++nt) o[mt][nt] = mfma16x16x32(va, pb[nt], o[mt][nt]);
      }
    }

    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  // ---- epilogue: normalise and store (lane holds d = 16 mt + 4 kgrp + 0..3) ----
#pragma unroll
  for (int nt = 0; nt < kCols; ++nt) {
    const float l = col_sum4(l_run[nt]);
    if (qpos[nt] < 0) continue;
    const int r = wave * kRowsPerWave + nt * 16 + col;
    const int qi = r / G, hh = r - qi * G;
    const size_t row = (size_t)(cu0 + i0 + qi) * a.hq + (size_t)g * G + hh;
    const float inv = 1.f / l;
#pragma unroll
    for (int mt = 0; mt < 8; ++mt)
      *reinterpret_cast<f32x4 *>(&a.out[row * kHeadDim + 16 * mt + 4 * kgrp]) = o[mt][nt] * inv;
    if (a.lse && kgrp == 0) a.lse[row] = (m_run[nt] + __log2f(l)) * kLn2;
  }
}

}  // namespace

hipError_t launch_append(const uint16_t *q, const int32_t *cu_q, const int32_t *ctx_lens,
                         const PagedKV &kv, int32_t B, int32_t hq, int32_t total_q,
                         int32_t max_q_len, int32_t max_kv_len, float scale, float *out,
                         float *lse, hipStream_t stream) {
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
  a.scale_log2 = scale * kLog2e;
  const int qblocks = (max_q_len + a.q_per_block - 1) / a.q_per_block;
  hipLaunchKernelGGL(append_kernel, dim3(qblocks, kv.hkv, B), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ra
