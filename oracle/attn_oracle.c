/*
 * fp64 CPU oracle for paged rollout attention.
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may call anything in this directory. It shares no code,
 * header, table or helper with the HIP library; it reads the same plain arrays.
 *
 * What it computes. The ProRL Agent paper (arXiv 2603.18815) runs every agent
 * step as one LLM completion over the whole conversation so far (Sec. 3.3.2),
 * routes all calls of a task to one backend so the cached prefix is reused
 * (Sec. 3.3.2, load balancing), and keeps earlier turns' token ids while only
 * new observations are tokenised and appended (Sec. 3.3.3). On the GPU this is
 * attention of new tokens against a per-trajectory cache of keys and values.
 * The paper gives no attention formula, so the oracle is the textbook
 * definition of scaled dot-product attention with grouped KV heads, written
 * out in fp64:
 *
 *   s_j  = scale * sum_d q[d] * k_j[d]
 *   m    = max_j s_j
 *   w_j  = exp(s_j - m),      Z = sum_j w_j
 *   out  = (sum_j w_j * v_j) / Z,  lse = m + ln Z
 *
 * Readings the paper leaves open (each is also listed in the design notes):
 *   - query head h reads KV head g = h / G with G = Hq / Hkv (contiguous groups);
 *   - a decode row attends its kv_len cached keys, the current token included;
 *   - append query i of a row sits at absolute position ctx + i and attends keys
 *     0 .. ctx + i inclusive (bottom-right causal alignment);
 *   - an empty key set gives out = 0 and lse = -inf;
 *   - bf16 inputs are widened exactly (bits << 16 -> fp32 -> fp64).
 *
 * Paged layout (the address formula the library's header defines), with P the
 * page size and D the head dimension; logical token j of row b lives in
 * physical page bt[b * bt_stride + j / P] at slot j % P:
 *   K element (page, g, slot, d) at (((page * Hkv + g) * P + slot) * D + d)
 *   V element (page, g, slot, d) at (((page * Hkv + g) * D + d) * P + slot)
 * i.e. K pages are token-major and V pages are dimension-major.
 *
 * P and D are parameters here (the GPU library fixes P = 16, D = 128) so that
 * tiny hand-checkable cases can be run.
 *
 * fp8 pools (a reading: the paper is silent on KV precision). Elements are
 * OCP FP8 E4M3 codes (1 sign, 4 exponent bits with bias 7, 3 mantissa bits;
 * exponent field 0 is subnormal, 2^-6 * m / 8; 0x7F and 0xFF are NaN; no
 * infinities; largest finite 448) with one scale per pool: the element's
 * value is decode(code) * k_scale (or v_scale). Writing a bf16 value x stores
 * encode(fp32(x) * fp32(1 / scale)), the product rounded to fp32, where
 * encode is the finite E4M3 value nearest to its argument (a tie goes to the
 * code with the even mantissa), +-inf and magnitudes beyond 448 saturate to
 * +-448, and NaN becomes 0x7F.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC (no -ffast-math), see oracle/build.py.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double bf16_to_f64(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* E4M3 code -> value, from the format's definition. */
static double e4m3_to_f64(uint8_t c) {
  const int s = c >> 7, e = (c >> 3) & 15, m = c & 7;
  if (e == 15 && m == 7) return NAN;
  const double v = e == 0 ? ldexp(m / 8.0, -6) : ldexp(1.0 + m / 8.0, e - 7);
  return s ? -v : v;
}

/* value -> E4M3 code: the nearest finite code by exhaustive search over the
 * 127 non-negative finite codes (ties to the even code), saturating. */
static uint8_t f64_to_e4m3(double x) {
  if (isnan(x)) return 0x7F;
  const uint8_t sign = signbit(x) ? 0x80 : 0;
  const double a = fabs(x);
  if (isinf(a)) return sign | 0x7E;
  int best = 0;
  double best_d = INFINITY;
  for (int c = 0; c < 0x7F; ++c) {
    const double d = fabs(e4m3_to_f64((uint8_t)c) - a);
    if (d < best_d || (d == best_d && (c & 1) == 0)) {
      best = c;
      best_d = d;
    }
  }
  return sign | (uint8_t)best;
}

/* Pool element kinds: bf16 bits, or E4M3 codes times the pool's scale. */
enum { KV_BF16 = 0, KV_FP8 = 1 };

static double kv_value(const void *pool, int kind, size_t i, double scale) {
  if (kind == KV_BF16) return bf16_to_f64(((const uint16_t *)pool)[i]);
  return e4m3_to_f64(((const uint8_t *)pool)[i]) * scale;
}

static size_t k_index(int64_t page, int g, int slot, int d, int Hkv, int P, int D) {
  return (((size_t)page * Hkv + g) * P + slot) * D + d;
}

static size_t v_index(int64_t page, int g, int slot, int d, int Hkv, int P, int D) {
  return (((size_t)page * Hkv + g) * D + d) * P + slot;
}

/* Physical page holding logical token j of row b. */
static int64_t page_of(const int32_t *bt, int64_t bt_stride, int b, int64_t j, int P) {
  return bt[(int64_t)b * bt_stride + j / P];
}

/*
 * Attention of one query vector q[0..D) (bf16 bits) over the first nkeys
 * logical tokens of row b, KV head g. Writes out[0..D) and *lse.
 * scores: caller scratch of at least nkeys doubles.
 */
static void attend_one(const uint16_t *q, const void *k_pool, const void *v_pool, int kind,
                       double k_scale, double v_scale, const int32_t *bt, int64_t bt_stride,
                       int b, int g, int64_t nkeys, int Hkv, int P, int D, double scale,
                       double *scores, double *out, double *lse) {
  for (int d = 0; d < D; ++d) out[d] = 0.0;
  if (nkeys <= 0) {
    *lse = -INFINITY;
    return;
  }
  double m = -INFINITY;
  for (int64_t j = 0; j < nkeys; ++j) {
    int64_t page = page_of(bt, bt_stride, b, j, P);
    int slot = (int)(j % P);
    double dot = 0.0;
    for (int d = 0; d < D; ++d)
      dot += bf16_to_f64(q[d]) *
             kv_value(k_pool, kind, k_index(page, g, slot, d, Hkv, P, D), k_scale);
    scores[j] = scale * dot;
    if (scores[j] > m) m = scores[j];
  }
  double z = 0.0;
  for (int64_t j = 0; j < nkeys; ++j) {
    int64_t page = page_of(bt, bt_stride, b, j, P);
    int slot = (int)(j % P);
    double w = exp(scores[j] - m);
    z += w;
    for (int d = 0; d < D; ++d)
      out[d] += w * kv_value(v_pool, kind, v_index(page, g, slot, d, Hkv, P, D), v_scale);
  }
  for (int d = 0; d < D; ++d) out[d] /= z;
  *lse = m + log(z);
}

/*
 * Decode: one query token per row.
 *   q        bf16 [B][Hq][D]
 *   kv_lens  [B]   keys attended by each row (current token included)
 *   out      f64 [B][Hq][D],  lse f64 [B][Hq] (may be NULL)
 * Returns 0, or -1 on bad shape arguments.
 */
static int decode_pools(const uint16_t *q, const void *k_pool, const void *v_pool, int kind,
                        double k_scale, double v_scale, const int32_t *block_table,
                        int64_t bt_stride, const int32_t *kv_lens, int B, int Hq, int Hkv, int P,
                        int D, double scale, double *out, double *lse) {
  if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || P <= 0 || D <= 0) return -1;
  const int G = Hq / Hkv;
  int64_t max_len = 0;
  for (int b = 0; b < B; ++b)
    if (kv_lens[b] > max_len) max_len = kv_lens[b];
  int failed = 0;
#pragma omp parallel
  {
    double *scores = (double *)malloc(sizeof(double) * (size_t)(max_len > 0 ? max_len : 1));
    if (!scores) {
#pragma omp atomic write
      failed = 1;
    }
#pragma omp for collapse(2) schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
      for (int h = 0; h < Hq; ++h) {
        if (!scores) continue;
        double lse_bh;
        attend_one(q + ((size_t)b * Hq + h) * D, k_pool, v_pool, kind, k_scale, v_scale,
                   block_table, bt_stride, b, h / G, kv_lens[b], Hkv, P, D, scale, scores,
                   out + ((size_t)b * Hq + h) * D, &lse_bh);
        if (lse) lse[(size_t)b * Hq + h] = lse_bh;
      }
    }
    free(scores);
  }
  return failed ? -2 : 0;
}

int oracle_decode_f64(const uint16_t *q, const uint16_t *k_pool, const uint16_t *v_pool,
                      const int32_t *block_table, int64_t bt_stride, const int32_t *kv_lens,
                      int B, int Hq, int Hkv, int P, int D, double scale, double *out,
                      double *lse) {
  return decode_pools(q, k_pool, v_pool, KV_BF16, 1.0, 1.0, block_table, bt_stride, kv_lens, B,
                      Hq, Hkv, P, D, scale, out, lse);
}

/* Decode over fp8 pools (E4M3 codes, values code * k_scale / code * v_scale). */
int oracle_decode_fp8_f64(const uint16_t *q, const uint8_t *k_pool, const uint8_t *v_pool,
                          double k_scale, double v_scale, const int32_t *block_table,
                          int64_t bt_stride, const int32_t *kv_lens, int B, int Hq, int Hkv,
                          int P, int D, double scale, double *out, double *lse) {
  return decode_pools(q, k_pool, v_pool, KV_FP8, k_scale, v_scale, block_table, bt_stride,
                      kv_lens, B, Hq, Hkv, P, D, scale, out, lse);
}

/*
 * Append (chunked causal prefill against the cache). Row b owns queries
 * cu_q[b] .. cu_q[b+1]-1; query i of the row (i from 0) attends logical keys
 * 0 .. ctx_lens[b] + i. The chunk's own keys and values are already in the pool
 * at positions ctx_lens[b] .. ctx_lens[b] + T_b - 1.
 *   q    bf16 [total_q][Hq][D]
 *   out  f64 [total_q][Hq][D], lse f64 [total_q][Hq] (may be NULL)
 */
static int append_pools(const uint16_t *q, const int32_t *cu_q, const int32_t *ctx_lens,
                        const void *k_pool, const void *v_pool, int kind, double k_scale,
                        double v_scale, const int32_t *block_table, int64_t bt_stride, int B,
                        int Hq, int Hkv, int P, int D, double scale, double *out, double *lse) {
  if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || P <= 0 || D <= 0) return -1;
  const int G = Hq / Hkv;
  int64_t total_q = B > 0 ? cu_q[B] : 0;
  int64_t max_keys = 1;
  for (int b = 0; b < B; ++b) {
    int64_t n = (int64_t)ctx_lens[b] + (cu_q[b + 1] - cu_q[b]);
    if (n > max_keys) max_keys = n;
  }
  int failed = 0;
#pragma omp parallel
  {
    double *scores = (double *)malloc(sizeof(double) * (size_t)max_keys);
    if (!scores) {
#pragma omp atomic write
      failed = 1;
    }
#pragma omp for collapse(2) schedule(dynamic, 1)
    for (int64_t t = 0; t < total_q; ++t) {
      for (int h = 0; h < Hq; ++h) {
        if (!scores) continue;
        int b = 0; /* row that owns packed query t */
        while (b + 1 <= B && cu_q[b + 1] <= t) ++b;
        int64_t i = t - cu_q[b];
        int64_t nkeys = (int64_t)ctx_lens[b] + i + 1;
        double lse_th;
        attend_one(q + ((size_t)t * Hq + h) * D, k_pool, v_pool, kind, k_scale, v_scale,
                   block_table, bt_stride, b, h / G, nkeys, Hkv, P, D, scale, scores,
                   out + ((size_t)t * Hq + h) * D, &lse_th);
        if (lse) lse[(size_t)t * Hq + h] = lse_th;
      }
    }
    free(scores);
  }
  return failed ? -2 : 0;
}

int oracle_append_f64(const uint16_t *q, const int32_t *cu_q, const int32_t *ctx_lens,
                      const uint16_t *k_pool, const uint16_t *v_pool, const int32_t *block_table,
                      int64_t bt_stride, int B, int Hq, int Hkv, int P, int D, double scale,
                      double *out, double *lse) {
  return append_pools(q, cu_q, ctx_lens, k_pool, v_pool, KV_BF16, 1.0, 1.0, block_table,
                      bt_stride, B, Hq, Hkv, P, D, scale, out, lse);
}

/* Append over fp8 pools (E4M3 codes, values code * k_scale / code * v_scale). */
int oracle_append_fp8_f64(const uint16_t *q, const int32_t *cu_q, const int32_t *ctx_lens,
                          const uint8_t *k_pool, const uint8_t *v_pool, double k_scale,
                          double v_scale, const int32_t *block_table, int64_t bt_stride, int B,
                          int Hq, int Hkv, int P, int D, double scale, double *out,
                          double *lse) {
  return append_pools(q, cu_q, ctx_lens, k_pool, v_pool, KV_FP8, k_scale, v_scale, block_table,
                      bt_stride, B, Hq, Hkv, P, D, scale, out, lse);
}

/*
 * Page write: for each row b and new token t of that row, logical position
 * pos = start_pos[b] + t receives k_new / v_new row cu_new[b] + t for every KV
 * head. A bit copy; no other pool element changes.
 *   k_new, v_new  bf16 [total_new][Hkv][D]
 */
int oracle_page_write(const uint16_t *k_new, const uint16_t *v_new, const int32_t *cu_new,
                      const int32_t *start_pos, const int32_t *block_table, int64_t bt_stride,
                      int B, int Hkv, int P, int D, uint16_t *k_pool, uint16_t *v_pool) {
  if (B < 0 || Hkv <= 0 || P <= 0 || D <= 0) return -1;
  for (int b = 0; b < B; ++b) {
    for (int64_t t = 0; t < (int64_t)cu_new[b + 1] - cu_new[b]; ++t) {
      int64_t pos = (int64_t)start_pos[b] + t;
      int64_t page = page_of(block_table, bt_stride, b, pos, P);
      int slot = (int)(pos % P);
      size_t src_tok = (size_t)cu_new[b] + (size_t)t;
      for (int g = 0; g < Hkv; ++g) {
        for (int d = 0; d < D; ++d) {
          size_t src = (src_tok * Hkv + g) * D + d;
          k_pool[k_index(page, g, slot, d, Hkv, P, D)] = k_new[src];
          v_pool[v_index(page, g, slot, d, Hkv, P, D)] = v_new[src];
        }
      }
    }
  }
  return 0;
}

/*
 * Gather: logical tokens 0 .. lens[b]-1 of every row, copied out of the pages
 * into packed token-major arrays k_out, v_out bf16 [total][Hkv][D], row b
 * starting at cu_out[b].
 */
int oracle_page_gather(const uint16_t *k_pool, const uint16_t *v_pool, const int32_t *block_table,
                       int64_t bt_stride, const int32_t *lens, const int32_t *cu_out, int B,
                       int Hkv, int P, int D, uint16_t *k_out, uint16_t *v_out) {
  if (B < 0 || Hkv <= 0 || P <= 0 || D <= 0) return -1;
  for (int b = 0; b < B; ++b) {
    for (int64_t j = 0; j < lens[b]; ++j) {
      int64_t page = page_of(block_table, bt_stride, b, j, P);
      int slot = (int)(j % P);
      size_t dst_tok = (size_t)cu_out[b] + (size_t)j;
      for (int g = 0; g < Hkv; ++g) {
        for (int d = 0; d < D; ++d) {
          size_t dst = (dst_tok * Hkv + g) * D + d;
          k_out[dst] = k_pool[k_index(page, g, slot, d, Hkv, P, D)];
          v_out[dst] = v_pool[v_index(page, g, slot, d, Hkv, P, D)];
        }
      }
    }
  }
  return 0;
}

/* E4M3 codec on arrays (for the pins). */
void oracle_e4m3_decode(const uint8_t *codes, int64_t n, double *out) {
  for (int64_t i = 0; i < n; ++i) out[i] = e4m3_to_f64(codes[i]);
}

void oracle_e4m3_encode(const double *x, int64_t n, uint8_t *out) {
  for (int64_t i = 0; i < n; ++i) out[i] = f64_to_e4m3(x[i]);
}

/* The stored code of bf16 value x in a pool with scale s: encode(fp32(x) * fp32(1 / s)). */
static uint8_t quantize(uint16_t x, float inv_scale) {
  uint32_t u = (uint32_t)x << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  const float v = f * inv_scale;   /* one fp32 product, rounded to nearest even */
  return f64_to_e4m3((double)v);
}

/*
 * Page write into fp8 pools: as oracle_page_write, each element stored as
 * quantize(x) with the pool's scale (k_scale for K, v_scale for V).
 */
int oracle_page_write_fp8(const uint16_t *k_new, const uint16_t *v_new, const int32_t *cu_new,
                          const int32_t *start_pos, const int32_t *block_table, int64_t bt_stride,
                          int B, int Hkv, int P, int D, float k_scale, float v_scale,
                          uint8_t *k_pool, uint8_t *v_pool) {
  if (B < 0 || Hkv <= 0 || P <= 0 || D <= 0 || !(k_scale > 0.f) || !(v_scale > 0.f)) return -1;
  const float k_inv = 1.0f / k_scale, v_inv = 1.0f / v_scale;
  for (int b = 0; b < B; ++b) {
    for (int64_t t = 0; t < (int64_t)cu_new[b + 1] - cu_new[b]; ++t) {
      int64_t pos = (int64_t)start_pos[b] + t;
      int64_t page = page_of(block_table, bt_stride, b, pos, P);
      int slot = (int)(pos % P);
      size_t src_tok = (size_t)cu_new[b] + (size_t)t;
      for (int g = 0; g < Hkv; ++g) {
        for (int d = 0; d < D; ++d) {
          size_t src = (src_tok * Hkv + g) * D + d;
          k_pool[k_index(page, g, slot, d, Hkv, P, D)] = quantize(k_new[src], k_inv);
          v_pool[v_index(page, g, slot, d, Hkv, P, D)] = quantize(v_new[src], v_inv);
        }
      }
    }
  }
  return 0;
}

/* Gather from fp8 pools: as oracle_page_gather, the stored codes copied out. */
int oracle_page_gather_u8(const uint8_t *k_pool, const uint8_t *v_pool,
                          const int32_t *block_table, int64_t bt_stride, const int32_t *lens,
                          const int32_t *cu_out, int B, int Hkv, int P, int D, uint8_t *k_out,
                          uint8_t *v_out) {
  if (B < 0 || Hkv <= 0 || P <= 0 || D <= 0) return -1;
  for (int b = 0; b < B; ++b) {
    for (int64_t j = 0; j < lens[b]; ++j) {
      int64_t page = page_of(block_table, bt_stride, b, j, P);
      int slot = (int)(j % P);
      size_t dst_tok = (size_t)cu_out[b] + (size_t)j;
      for (int g = 0; g < Hkv; ++g) {
        for (int d = 0; d < D; ++d) {
          size_t dst = (dst_tok * Hkv + g) * D + d;
          k_out[dst] = k_pool[k_index(page, g, slot, d, Hkv, P, D)];
          v_out[dst] = v_pool[v_index(page, g, slot, d, Hkv, P, D)];
        }
      }
    }
  }
  return 0;
}

/* Threads an OpenMP parallel region of the oracle uses (for reporting). */
/*
 * Rotary position embedding of token rows (a reading: the paper does not
 * describe model internals; models of its kind rotate each query and key by
 * its position). Row x (128 dims) at position p, table row cs = cos_sin[p]
 * holding c_i = cs[i] and s_i = cs[64 + i] for i < 64:
 *   y_i = fp32(x_i c_i) - fp32(x_{i+64} s_i),  y_{i+64} = fp32(x_{i+64} c_i) + fp32(x_i s_i),
 * each product and sum rounded to fp32 (the build disables contraction), the
 * result rounded to bf16 (nearest even). The rounding to bf16 decides the
 * stored value, so it is taken in the precision the library states for it.
 * x, out: bf16 [n_rows][heads][128]; pos: [n_rows]; cos_sin: fp32 [rope_rows][128].
 * Returns -1 (nothing written) if a position lies outside the table.
 */
static uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);   /* quiet NaN */
  const uint32_t lsb = (u >> 16) & 1u;
  return (uint16_t)((u + 0x7fffu + lsb) >> 16);
}

int oracle_rope_bf16(const uint16_t *x, int64_t n_rows, int heads, const int32_t *pos,
                     const float *cos_sin, int64_t rope_rows, uint16_t *out) {
  const int D = 128, H = 64;
  for (int64_t r = 0; r < n_rows; ++r)
    if (pos[r] < 0 || pos[r] >= rope_rows) return -1;
  for (int64_t r = 0; r < n_rows; ++r) {
    const float *cs = cos_sin + (size_t)pos[r] * D;
    for (int h = 0; h < heads; ++h) {
      const uint16_t *xr = x + ((size_t)r * heads + h) * D;
      uint16_t *yr = out + ((size_t)r * heads + h) * D;
      for (int i = 0; i < H; ++i) {
        const float lo = (float)bf16_to_f64(xr[i]), hi = (float)bf16_to_f64(xr[i + H]);
        const float c = cs[i], s = cs[H + i];
        const float a = lo * c, b = hi * s, a2 = hi * c, b2 = lo * s;
        const float y_lo = a - b, y_hi = a2 + b2;
        yr[i] = f32_to_bf16_rne(y_lo);
        yr[i + H] = f32_to_bf16_rne(y_hi);
      }
    }
  }
  return 0;
}

int oracle_num_threads(void) { return omp_get_max_threads(); }

/* Threads of the parallel loops that follow (timing only; results do not
 * depend on it: each output element is computed by one thread). */
void oracle_set_num_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
}
