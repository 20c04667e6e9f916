// Decode attention over paged KV caches: split-K over pages, then combine.
//
// Split kernel: one workgroup (4 waves) per (row b, KV head g, split s). The
// split covers up to split_tokens keys; each wave streams pairs of pages
// (32 keys) straight from HBM into registers with 16-byte loads and runs the
// dot products and the P·V update on the matrix cores:
//   S^T[key][qrow] = K[key][:] · Q^T[:][qrow]      (4 x mfma 16x16x32 per 16 keys)
//   O^T[d][qrow]  += V^T[d][key] · P^T[key][qrow]  (8 x mfma per 32 keys)
// The G = Hq / Hkv query heads of the group fill the 16 matrix columns (zero
// padded), so every KV byte is read once for the whole group. Softmax is the
// online (running max / running sum) form in fp32, in base 2 with log2(e)
// folded into the scale. P is fed to the matrix cores as bf16 hi + lo parts
// (two P·V products), which keeps the weights to about 16 mantissa bits; the
// extra products cost nothing in this HBM-bound kernel.
// The four waves' partial states are merged through LDS and the split writes
// one (max, sum, unnormalised O) partial per query head.
//
// Combine kernel: one workgroup per (row, query head) merges the splits:
//   M = max_s m_s,  l = sum_s l_s 2^(m_s - M),  out = sum_s o_s 2^(m_s - M) / l.
#include <stdlib.h>

#include "ra_device.h"
#include "ra_internal.h"

namespace ra {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;
constexpr int kPairTokens = 2 * kPage;
constexpr int kOPitch = kHeadDim + 4;  // LDS pitch of one column's O row (floats)

struct DecodeArgs {
  const uint16_t *q;
  const uint16_t *k_pool;
  const uint16_t *v_pool;
  const int32_t *block_table;
  const int32_t *kv_lens;
  float *ws_o;   // [B][Hq][max_splits][128]
  float *ws_m;   // [B][Hq][max_splits]   running max, base-2 units
  float *ws_l;   // [B][Hq][max_splits]   running sum
  int32_t hq, hkv, group, bt_stride, num_pages, max_kv_len, split_tokens, max_splits;
  float scale_log2;
};

__global__ __launch_bounds__(kThreads, 2) void decode_split_kernel(DecodeArgs a) {
  // KV head fastest: the Hkv workgroups of one (row, split) are dispatched
  // together, so the Hkv adjacent 4 KiB blocks of every page they read are
  // requested close in time (DRAM row locality).
  const int g = blockIdx.x, split = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int L = min(a.kv_lens[b], a.max_kv_len);
  const int t0 = split * a.split_tokens;
  if (t0 >= L) return;
  const int t1 = min(L, t0 + a.split_tokens);
  const int npairs = (t1 - t0 + kPairTokens - 1) / kPairTokens;
  const int row_pages = (t1 + kPage - 1) / kPage;   // pages of this row in use up to t1
  const int32_t *bt = a.block_table + (size_t)b * a.bt_stride;

  const int col = lane & 15;     // matrix column = query head within the group
  const int kgrp = lane >> 4;    // contraction slot group
  const int G = a.group;

  // Q^T operand: column col, dims 32*kk + 8*kgrp + 0..7.
  bf16x8 qop[4];
  if (col < G) {
    const uint16_t *qp = a.q + ((size_t)b * a.hq + (size_t)g * G + col) * kHeadDim + 8 * kgrp;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qop[kk] = load_bf16x8(qp + 32 * kk);
  } else {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qop[kk] = bf16x8{};
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

  f32x4 o[8];
#pragma unroll
  for (int mt = 0; mt < 8; ++mt) o[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const size_t head_stride = (size_t)kPage * kHeadDim;   // elements per (page, head)
  for (int pr = wave; pr < npairs; pr += kWaves) {
    const int tok = t0 + pr * kPairTokens;                // position of the pair's first key
    const int pg = tok / kPage;
    const int id0 = clamp_page(bt[pg], a.num_pages);
    const int id1 = pg + 1 < row_pages ? clamp_page(bt[pg + 1], a.num_pages) : id0;

    const uint16_t *kb =
        a.k_pool + ((size_t)(ka_sel ? id1 : id0) * a.hkv + g) * head_stride;
    bf16x8 ka[2][4];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        ka[t][kk] = load_bf16x8(kb + (ka_slot + 4 * t) * kHeadDim + 32 * kk + 8 * kgrp);
    const uint16_t *vb =
        a.v_pool + ((size_t)(sv_sel ? id1 : id0) * a.hkv + g) * head_stride;
    bf16x8 va[8];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) va[mt] = load_bf16x8(vb + (16 * mt + col) * kPage + sv_slot);

    f32x4 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) st[t] = mfma16x16x32(ka[t][kk], qop[kk], st[t]);
    }
    float sc[8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) sc[4 * t + r] = st[t][r] * a.scale_log2;

    if (tok + kPairTokens > t1) {
      // Keys at or past t1 are not attended: their scores become -inf and
      // their V entries are replaced (not multiplied) by zero, so that
      // whatever those slots hold cannot reach the output.
      const int first = tok + sv_sel * kPage + sv_slot;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool dead = first + e >= t1;
        sc[e] = dead ? -INFINITY : sc[e];
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) va[mt][e] = dead ? (__bf16)0.f : va[mt][e];
      }
    }

    float mx = sc[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sc[e]);
    mx = col_max4(mx);
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    f32x8 p;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      p[e] = fast_exp2(sc[e] - m_use);
      psum += p[e];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
    const bf16x8 p_hi = to_bf16x8(p);
    const bf16x8 p_lo = to_bf16x8(p - to_f32x8(p_hi));
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) {
      o[mt] *= alpha;
      o[mt] = mfma16x16x32(va[mt], p_hi, o[mt]);
      o[mt] = mfma16x16x32(va[mt], p_lo, o[mt]);
    }
  }
  l_run = col_sum4(l_run);

  // Merge the four waves through LDS. Lane l holds O^T rows
  // d = 16 mt + 4 kgrp + r of column col.
  __shared__ float s_m[kWaves][16];
  __shared__ float s_l[kWaves][16];
  __shared__ float s_o[kWaves][16][kOPitch];
  if (kgrp == 0) {
    s_m[wave][col] = m_run;
    s_l[wave][col] = l_run;
  }
#pragma unroll
  for (int mt = 0; mt < 8; ++mt)
    *reinterpret_cast<f32x4 *>(&s_o[wave][col][16 * mt + 4 * kgrp]) = o[mt];
  __syncthreads();

  const size_t row_base = (size_t)b * a.hq + (size_t)g * G;
  for (int idx = threadIdx.x; idx < G * kHeadDim; idx += kThreads) {
    const int c = idx / kHeadDim, d = idx % kHeadDim;
    float M = s_m[0][c];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, s_m[w][c]);
    const float M_use = M == -INFINITY ? 0.f : M;
    float acc = 0.f, lsum = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = fast_exp2(s_m[w][c] - M_use);
      acc += f * s_o[w][c][d];
      lsum += f * s_l[w][c];
    }
    const size_t part = (row_base + c) * a.max_splits + split;
    a.ws_o[part * kHeadDim + d] = acc;
    if (d == 0) {
      a.ws_m[part] = M;
      a.ws_l[part] = lsum;
    }
  }
}

__global__ __launch_bounds__(kHeadDim) void decode_combine_kernel(
    const float *__restrict__ ws_o, const float *__restrict__ ws_m, const float *__restrict__ ws_l,
    const int32_t *__restrict__ kv_lens, int hq, int max_kv_len, int split_tokens, int max_splits,
    float *__restrict__ out, float *__restrict__ lse) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int d = threadIdx.x;
  const size_t bh = (size_t)b * hq + h;
  const int L = min(max(kv_lens[b], 0), max_kv_len);
  const int ns = (L + split_tokens - 1) / split_tokens;
  if (ns == 0) {
    out[bh * kHeadDim + d] = 0.f;
    if (lse && d == 0) lse[bh] = -INFINITY;
    return;
  }
  const float *m = ws_m + bh * max_splits;
  const float *l = ws_l + bh * max_splits;
  const float *o = ws_o + bh * max_splits * kHeadDim + d;
  float M = m[0];
  for (int s = 1; s < ns; ++s) M = fmaxf(M, m[s]);
  float acc = 0.f, lsum = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float f = fast_exp2(m[s] - M);
    acc += f * o[(size_t)s * kHeadDim];
    lsum += f * l[s];
  }
  out[bh * kHeadDim + d] = acc / lsum;
  if (lse && d == 0) lse[bh] = (M + __log2f(lsum)) * kLn2;
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
  if (const char *env = getenv("RA_SPLIT_TOKENS")) {
    const long v = strtol(env, nullptr, 10);
    if (v >= 128) split = (v + 127) / 128 * 128;
  }
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

hipError_t launch_decode(const uint16_t *q, const PagedKV &kv, const int32_t *kv_lens, int32_t B,
                         int32_t hq, int32_t max_kv_len, float scale, float *out, float *lse,
                         void *workspace, const DecodePlan &plan, hipStream_t stream) {
  const size_t parts = (size_t)B * hq * plan.max_splits;
  DecodeArgs a;
  a.q = q;
  a.k_pool = kv.k_pool;
  a.v_pool = kv.v_pool;
  a.block_table = kv.block_table;
  a.kv_lens = kv_lens;
  a.ws_o = static_cast<float *>(workspace);
  a.ws_m = a.ws_o + parts * kHeadDim;
  a.ws_l = a.ws_m + parts;
  a.hq = hq;
  a.hkv = kv.hkv;
  a.group = hq / kv.hkv;
  a.bt_stride = kv.bt_stride;
  a.num_pages = kv.num_pages;
  a.max_kv_len = max_kv_len;
  a.split_tokens = plan.split_tokens;
  a.max_splits = plan.max_splits;
  a.scale_log2 = scale * kLog2e;
  hipLaunchKernelGGL(decode_split_kernel, dim3(kv.hkv, plan.max_splits, B), dim3(kThreads), 0,
                     stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_combine_kernel, dim3(hq, B), dim3(kHeadDim), 0, stream, a.ws_o,
                     a.ws_m, a.ws_l, kv_lens, hq, max_kv_len, plan.split_tokens, plan.max_splits,
                     out, lse);
  return hipGetLastError();
}

}  // namespace ra
