// Decode split (and combine) over paged KV caches, shared by the decode
// kernels and the mixed decode + append kernel.
//
// Split: one workgroup of kW waves (4 in the decode kernels, 8 in the mixed
// kernel) per (KV head g, split s, work item). The split covers up to split_tokens keys; each wave streams pairs of pages
// (32 keys) straight from HBM into registers with 16-byte loads and runs the
// dot products and the P·V update on the matrix cores:
//   S^T[key][col] = K[key][:] · Q^T[:][col]       (4 x mfma 16x16x32 per 16 keys)
//   O^T[d][col]  += V^T[d][key] · P^T[key][col]   (8 x mfma per 32 keys and tile)
// The matrix columns are query rows that read the same keys: the G = Hq / Hkv
// query heads of one row (plain decode), or the heads of up to 16 NT / G rows
// that share a prefix (shared-prefix decode), in NT tiles of 16 columns (zero
// padded), so every KV byte is read once for all of them. Softmax is the
// online (running max / running sum) form in fp32, in base 2 with log2(e)
// folded into the scale. P is fed to the matrix cores as bf16 hi + lo parts
// (two P·V products), which keeps the weights to about 16 mantissa bits; the
// extra products cost nothing in this HBM-bound kernel.
// The waves' partial states are merged through LDS and the split writes
// one (max, sum, unnormalised O) partial per column into its slot.
//
// Shared-prefix decode (the rollouts of one task share its prompt pages): the
// rows of a group attend keys [0, P) together, P being the group's shared
// prefix floored to 32 keys and capped at its shortest row, in prefix slots
// [0, prefix_slots); each row attends its own keys [P, L) in the slots after.
//
// Combine kernel: one workgroup per (row, query head) merges the slots in a
// fixed order (prefix, then suffix):
//   M = max_s m_s,  l = sum_s l_s 2^(m_s - M),  out = sum_s o_s 2^(m_s - M) / l.
// It reads the slots eight at a time, so that a row's loads are in flight
// together rather than one dependent round trip per slot.
#pragma once

#include "ra_device.h"
#include "ra_internal.h"

// Everything lives in ra::dsplit, apart from the append-tile names (ra::atile)
// that share a translation unit with it in the mixed kernel.
namespace ra {
namespace dsplit {

constexpr int kPairTokens = 2 * kPage;
constexpr int kOPitch = kHeadDim + 4;  // LDS pitch of one column's O row (floats)

struct DecodeArgs {
  const uint16_t *q;
  const uint16_t *k_pool;
  const uint16_t *v_pool;
  const int32_t *block_table;
  const int32_t *kv_lens;
  const int32_t *group_start;   // shared prefix: [num_groups + 1] row offsets; null otherwise
  const int32_t *prefix_len;    // shared prefix: [num_groups] tokens shared by the group
  float *ws_o;   // [B][Hq][slots][128]
  float *ws_m;   // [B][Hq][slots]   running max, base-2 units
  float *ws_l;   // [B][Hq][slots]   running sum
  int32_t B, hq, hkv, group, bt_stride, num_pages, max_kv_len, split_tokens;
  int32_t slots;          // partial slots per (row, query head)
  int32_t prefix_slots;   // slots [0, prefix_slots) hold prefix splits (0: plain decode)
  int32_t zdiv;           // shared prefix: work items per group along grid z
  int32_t rows_per_chunk; // shared prefix: rows of a group one prefix workgroup covers
  float scale_log2;       // softmax scale * log2(e) (* k_scale for fp8 pools)
  float v_scale;          // multiplies the output (1 for bf16 pools)
};

__device__ __forceinline__ int row_len(const DecodeArgs &a, int b) {
  return min(max(a.kv_lens[b], 0), a.max_kv_len);
}

// Rows [gs, ge) of group grp and its shared prefix P (a multiple of 32 keys,
// at most the group's shortest row).
struct GroupRows {
  int gs, ge, P;
};
__device__ __forceinline__ GroupRows group_rows(const DecodeArgs &a, int grp) {
  GroupRows r;
  r.gs = min(max(a.group_start[grp], 0), a.B);
  r.ge = min(max(a.group_start[grp + 1], r.gs), a.B);
  // (also capped at what the prefix slots hold, so that a prefix_len above
  // the host's bound cannot make the merge read past the prefix slots)
  int p = min(min(max(a.prefix_len[grp], 0), a.max_kv_len), a.prefix_slots * a.split_tokens);
  for (int b = r.gs; b < r.ge; ++b) p = min(p, row_len(a, b));
  r.P = p / (2 * kPage) * (2 * kPage);
  return r;
}

// kPrefix: a prefix workgroup of a shared-prefix group (columns = heads of
// up to rows_per_chunk rows); otherwise one row (plain decode, or a row's
// suffix in shared-prefix decode). NT: 16-column tiles.
// LDS of one split: the per-wave partial states before their merge.
template <int NT, int kW>
struct DecodeLds {
  float m[kW][16 * NT];
  float l[kW][16 * NT];
  float o[kW][16 * NT][kOPitch];
};

// One split of KV head g (work item z: a row, or a group's row chunk), by a
// workgroup of kW waves that all call it with the same arguments. kFp8: the
// pools hold E4M3 codes, converted exactly to bf16 operands after the load.
template <int NT, bool kPrefix, int kW, bool kFp8 = false>
__device__ __forceinline__ void decode_split(const DecodeArgs &a, int g, int split, int z,
                                             DecodeLds<NT, kW> &lds) {
  // ---- what this workgroup computes: keys [t0, t1) of row krow's table for
  // the rows r0 .. r0 + nr - 1, into partial slot `slot`.
  int krow, r0, nr, t0, t1, slot;
  if (a.group_start == nullptr) {
    const int b = z, L = row_len(a, b);
    krow = r0 = b;
    nr = 1;
    t0 = split * a.split_tokens;
    t1 = min(L, t0 + a.split_tokens);
    slot = split;
  } else {
    const int grp = z / a.zdiv, sub = z - grp * a.zdiv;
    const GroupRows gr = group_rows(a, grp);
    if (kPrefix) {
      krow = gr.gs;
      r0 = gr.gs + sub * a.rows_per_chunk;
      nr = min(a.rows_per_chunk, gr.ge - r0);
      t0 = split * a.split_tokens;
      t1 = min(gr.P, t0 + a.split_tokens);
      slot = split;
    } else {
      const int b = gr.gs + sub;
      krow = r0 = b;
      nr = b < gr.ge ? 1 : 0;
      t0 = gr.P + split * a.split_tokens;
      t1 = nr ? min(row_len(a, b), t0 + a.split_tokens) : t0;
      slot = a.prefix_slots + split;
    }
  }
  if (nr <= 0 || t0 >= t1) return;
  const int lane = threadIdx.x & (kWave - 1);
  // wave-uniform (an SGPR), so that the pair loop and its block-table reads
  // run on the scalar unit instead of as vector loads that each wait for
  // every load issued before them
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int npairs = (t1 - t0 + kPairTokens - 1) / kPairTokens;
  const int row_pages = (t1 + kPage - 1) / kPage;   // pages of row krow in use up to t1
  const int32_t *bt = a.block_table + (size_t)krow * a.bt_stride;

  const int col = lane & 15;     // matrix column within a tile
  const int kgrp = lane >> 4;    // contraction slot group
  const int G = a.group;

  // Q^T operands: column 16 nt + col = (row r0 + c / G, head c % G), dims
  // 32 kk + 8 kgrp + 0..7 (bf16 pools), or 64 (kk / 2) + 16 kgrp + 8 (kk % 2)
  // + 0..7 (fp8 pools: a lane then reads 16 contiguous K bytes per 64 dims).
  // Any order of the contraction is valid as long as K follows the same one.
  bf16x8 qop[NT][4];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int c = 16 * nt + col, r = c / G;
    if (r < nr) {
      const uint16_t *qrow =
          a.q + ((size_t)(r0 + r) * a.hq + (size_t)g * G + (c - r * G)) * kHeadDim;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        qop[nt][kk] = kFp8 ? load_bf16x8(qrow + 64 * (kk >> 1) + 16 * kgrp + 8 * (kk & 1))
                           : load_bf16x8(qrow + 32 * kk + 8 * kgrp);
    } else {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) qop[nt][kk] = bf16x8{};
    }
  }

  // Key order inside a pair of pages (32 keys). S tile t (0/1), matrix row
  // i = 4q + r holds key (page q / 2, slot 8 (q % 2) + 4t + r). Hence the
  // S values of lane l are keys of page l / 32, slots 8 ((l / 16) % 2) + e,
  // e = 4t + r: eight consecutive slots, exactly the eight contraction
  // slots that lane supplies to the P·V product.
  const int ka_sel = col >> 3;                              // page of A row col
  const int ka_slot = 8 * ((col >> 2) & 1) + (col & 3);     // + 4t
  const int sv_sel = lane >> 5;                             // page of my S/V keys
  const int sv_slot = 8 * ((lane >> 4) & 1);                // + e

  f32x4 o[NT][8];
  float m_run[NT], l_run[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) o[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[nt] = -INFINITY;
    l_run[nt] = 0.f;
  }

  const size_t head_stride = (size_t)kPage * kHeadDim;   // elements per (page, head)
  for (int pr = wave; pr < npairs; pr += kW) {
    const int tok = t0 + pr * kPairTokens;                // position of the pair's first key
    const int pg = tok / kPage;
    const int id0 = clamp_page(bt[pg], a.num_pages);
    const int id1 = pg + 1 < row_pages ? clamp_page(bt[pg + 1], a.num_pages) : id0;

    // V loads: each instruction takes whole 128-byte lines (512 contiguous
    // bytes per page), read once, so they are marked nontemporal; that keeps
    // the streamed V from displacing the K lines, each of which two
    // instructions read half at a time (K stays an ordinary load). Prefix
    // items keep ordinary loads: the chunks of a group re-read their pages
    // from the cache.
    auto load_v = [](const void *p) __attribute__((always_inline)) {
      return kPrefix ? *reinterpret_cast<const u32x4 *>(p) : load_stream_u32x4(p);
    };
    bf16x8 ka[2][4];
    bf16x8 va[8];
    if constexpr (kFp8) {
      // one byte per element: K rows as 2 x 16 bytes per lane
      const uint8_t *kb = reinterpret_cast<const uint8_t *>(a.k_pool) +
                          ((size_t)(ka_sel ? id1 : id0) * a.hkv + g) * head_stride;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const u32x4 w = *reinterpret_cast<const u32x4 *>(kb + (ka_slot + 4 * t) * kHeadDim +
                                                             64 * h + 16 * kgrp);
          ka[t][2 * h] = fp8x8_to_bf16x8(u32x2{w[0], w[1]});
          ka[t][2 * h + 1] = fp8x8_to_bf16x8(u32x2{w[2], w[3]});
        }
      const uint8_t *vb = reinterpret_cast<const uint8_t *>(a.v_pool) +
                          ((size_t)(sv_sel ? id1 : id0) * a.hkv + g) * head_stride;
      // Whole 16-slot V rows, 16 bytes per lane: lane l loads row
      // d = 16 (2 j + h) + col of its page (h = l / 16 % 2), so lanes l and
      // l ^ 16 hold rows 2j and 2j + 1 of one page; one v_permlane16_swap per
      // dword then leaves each lane the slots it supplies (8 h + 0..7) of both.
      const int vh = (lane >> 4) & 1;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u32x4 w = load_v(vb + (16 * (2 * j + vh) + col) * kPage);
        const auto s0 = __builtin_amdgcn_permlane16_swap(w[0], w[2], false, false);
        const auto s1 = __builtin_amdgcn_permlane16_swap(w[1], w[3], false, false);
        va[2 * j] = fp8x8_to_bf16x8(u32x2{s0[0], s1[0]});
        va[2 * j + 1] = fp8x8_to_bf16x8(u32x2{s0[1], s1[1]});
      }
    } else {
      const uint16_t *kb =
          a.k_pool + ((size_t)(ka_sel ? id1 : id0) * a.hkv + g) * head_stride;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          ka[t][kk] = load_bf16x8(kb + (ka_slot + 4 * t) * kHeadDim + 32 * kk + 8 * kgrp);
      const uint16_t *vb =
          a.v_pool + ((size_t)(sv_sel ? id1 : id0) * a.hkv + g) * head_stride;
#pragma unroll
      for (int mt = 0; mt < 8; ++mt)
        va[mt] = __builtin_bit_cast(bf16x8, load_v(vb + (16 * mt + col) * kPage + sv_slot));
    }

    // Keys at or past t1 are not attended: their scores become -inf and
    // their V entries are replaced (not multiplied) by zero, so that
    // whatever those slots hold cannot reach the output.
    const bool tail = tok + kPairTokens > t1;
    const int first = tok + sv_sel * kPage + sv_slot;
    if (tail) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool dead = first + e >= t1;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) va[mt][e] = dead ? (__bf16)0.f : va[mt][e];
      }
    }

#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4 st[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        st[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) st[t] = mfma16x16x32(ka[t][kk], qop[nt][kk], st[t]);
      }
      float sc[8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[4 * t + r] = st[t][r] * a.scale_log2;
      if (tail) {
#pragma unroll
        for (int e = 0; e < 8; ++e) sc[e] = first + e >= t1 ? -INFINITY : sc[e];
      }

      float mx = sc[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sc[e]);
      mx = col_max4(mx);
      const float m_new = fmaxf(m_run[nt], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(m_run[nt] - m_use);
      f32x8 p;
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = fast_exp2(sc[e] - m_use);
        psum += p[e];
      }
      l_run[nt] = l_run[nt] * alpha + psum;
      m_run[nt] = m_new;
      const bf16x8 p_hi = to_bf16x8(p);
      const bf16x8 p_lo = to_bf16x8(p - to_f32x8(p_hi));
#pragma unroll
      for (int mt = 0; mt < 8; ++mt) {
        o[nt][mt] *= alpha;
        o[nt][mt] = mfma16x16x32(va[mt], p_hi, o[nt][mt]);
        o[nt][mt] = mfma16x16x32(va[mt], p_lo, o[nt][mt]);
      }
    }
  }

  // Merge the kW waves through LDS. Lane l holds O^T rows
  // d = 16 mt + 4 kgrp + r of column 16 nt + col.
  auto &s_m = lds.m;
  auto &s_l = lds.l;
  auto &s_o = lds.o;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float l_sum = col_sum4(l_run[nt]);
    if (kgrp == 0) {
      s_m[wave][16 * nt + col] = m_run[nt];
      s_l[wave][16 * nt + col] = l_sum;
    }
#pragma unroll
    for (int mt = 0; mt < 8; ++mt)
      *reinterpret_cast<f32x4 *>(&s_o[wave][16 * nt + col][16 * mt + 4 * kgrp]) = o[nt][mt];
  }
  __syncthreads();

  const int ncols = min(nr * G, 16 * NT);
  for (int idx = threadIdx.x; idx < ncols * kHeadDim; idx += kW * kWave) {
    const int c = idx / kHeadDim, d = idx % kHeadDim;
    float M = s_m[0][c];
#pragma unroll
    for (int w = 1; w < kW; ++w) M = fmaxf(M, s_m[w][c]);
    const float M_use = M == -INFINITY ? 0.f : M;
    float acc = 0.f, lsum = 0.f;
#pragma unroll
    for (int w = 0; w < kW; ++w) {
      const float f = fast_exp2(s_m[w][c] - M_use);
      acc += f * s_o[w][c][d];
      lsum += f * s_l[w][c];
    }
    const int r = c / G;
    const size_t part = ((size_t)(r0 + r) * a.hq + (size_t)g * G + (c - r * G)) * a.slots + slot;
    a.ws_o[part * kHeadDim + d] = acc;
    if (d == 0) {
      a.ws_m[part] = M;
      a.ws_l[part] = lsum;
    }
  }
}

// The combine kernel is defined once per translation unit that includes
// this header.
namespace {

__global__ __launch_bounds__(kHeadDim) void decode_combine_kernel(DecodeArgs a, float *out,
                                                                  float *lse) {
  const int h = blockIdx.x;
  int b, P = 0, np = 0;
  if (a.group_start == nullptr) {
    b = blockIdx.y;
  } else {
    const int grp = blockIdx.y / a.zdiv;
    const GroupRows gr = group_rows(a, grp);
    b = gr.gs + (blockIdx.y - grp * a.zdiv);
    if (b >= gr.ge) return;
    P = gr.P;
    np = (P + a.split_tokens - 1) / a.split_tokens;
  }
  const int d = threadIdx.x;
  const size_t bh = (size_t)b * a.hq + h;
  const int ns = (row_len(a, b) - P + a.split_tokens - 1) / a.split_tokens;
  if (np + ns == 0) {
    out[bh * kHeadDim + d] = 0.f;
    if (lse && d == 0) lse[bh] = -INFINITY;
    return;
  }
  const float *m = a.ws_m + bh * a.slots;
  const float *l = a.ws_l + bh * a.slots;
  const float *o = a.ws_o + bh * a.slots * kHeadDim + d;
  // slots in merge order: prefix splits [0, np), then suffix splits
  auto slot = [&](int s) { return s < np ? s : a.prefix_slots + (s - np); };
  const int n = np + ns;
  constexpr int kBatch = 8;
  float M = -INFINITY;
  for (int s0 = 0; s0 < n; s0 += kBatch) {
    float mv[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) mv[j] = s0 + j < n ? m[slot(s0 + j)] : -INFINITY;
#pragma unroll
    for (int j = 0; j < kBatch; ++j) M = fmaxf(M, mv[j]);
  }
  float acc = 0.f, lsum = 0.f;
  for (int s0 = 0; s0 < n; s0 += kBatch) {
    float f[kBatch], ov[kBatch], lv[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const bool ok = s0 + j < n;
      const int k = slot(ok ? s0 + j : s0);
      ov[j] = o[(size_t)k * kHeadDim];
      lv[j] = l[k];
      f[j] = ok ? fast_exp2(m[k] - M) : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      acc += f[j] * ov[j];
      lsum += f[j] * lv[j];
    }
  }
  out[bh * kHeadDim + d] = acc / lsum * a.v_scale;
  if (lse && d == 0) lse[bh] = (M + __log2f(lsum)) * kLn2;
}

}  // namespace

inline DecodeArgs make_decode_args(const uint16_t *q, const PagedKV &kv, const int32_t *kv_lens,
                                   int32_t B, int32_t hq, int32_t max_kv_len, float scale,
                                   void *workspace, int32_t slots, const DecodePlan &plan) {
  const size_t parts = (size_t)B * hq * slots;
  DecodeArgs a;
  a.q = q;
  a.k_pool = kv.k_pool;
  a.v_pool = kv.v_pool;
  a.block_table = kv.block_table;
  a.kv_lens = kv_lens;
  a.group_start = nullptr;
  a.prefix_len = nullptr;
  a.ws_o = static_cast<float *>(workspace);
  a.ws_m = a.ws_o + parts * kHeadDim;
  a.ws_l = a.ws_m + parts;
  a.B = B;
  a.hq = hq;
  a.hkv = kv.hkv;
  a.group = hq / kv.hkv;
  a.bt_stride = kv.bt_stride;
  a.num_pages = kv.num_pages;
  a.max_kv_len = max_kv_len;
  a.split_tokens = plan.split_tokens;
  a.slots = slots;
  a.prefix_slots = 0;
  a.zdiv = 1;
  a.rows_per_chunk = 1;
  a.scale_log2 = scale * kLog2e * kv.k_scale;
  a.v_scale = kv.v_scale;
  return a;
}

}  // namespace dsplit
}  // namespace ra
