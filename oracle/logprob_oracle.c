/*
 * fp64 CPU oracle for per-token log-probabilities under an LM head.
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may call anything in this directory. It shares no code,
 * header, table or helper with the HIP library; it reads the same plain arrays.
 *
 * What it computes. The ProRL Agent paper (arXiv 2603.18815) passes token ids,
 * not text, between the rollout workers and the LLM backend, and every
 * generated token comes back with its log-probability (Sec. 3.3.3,
 * token-in/token-out), which RL training later uses. For a hidden state h
 * (the model's last layer output for one position), the LM-head matrix W (one
 * row per vocabulary entry) and the token t that was emitted, that is the
 * log-softmax of the logits at t, written out here in fp64:
 *
 *   z_v   = scale * sum_k h[k] * W[v][k]          (v = 0 .. V-1)
 *   M     = max_v z_v
 *   lse   = M + ln sum_v exp(z_v - M)
 *   logp  = z_t - lse
 *
 * Readings the paper leaves open (also listed in the design notes):
 *   - scale multiplies the logits (1 / temperature; 1 gives the raw model
 *     distribution);
 *   - a token id outside [0, V) has no log-probability: logp = NaN (lse is
 *     still returned);
 *   - bf16 inputs are widened exactly (bits << 16 -> fp32 -> fp64).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static double lp_bf16(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* h: [N][D] bf16 bits, W: [V][D] bf16 bits, targets: [N].
 * Writes logp[N] and lse[N]. Returns 0, or -1 on a bad size. */
int oracle_token_logprob_f64(const uint16_t *h, const uint16_t *W, const int32_t *targets,
                             int64_t N, int64_t V, int64_t D, double scale, double *logp,
                             double *lse) {
  if (N < 0 || V < 0 || D < 0) return -1;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t n = 0; n < N; ++n) {
    const uint16_t *hn = h + n * D;
    double M = -INFINITY, zt = NAN;
    /* first pass: the max logit (and the target's logit) */
    for (int64_t v = 0; v < V; ++v) {
      const uint16_t *wv = W + v * D;
      double z = 0.0;
      for (int64_t k = 0; k < D; ++k) z += lp_bf16(hn[k]) * lp_bf16(wv[k]);
      z *= scale;
      if (z > M) M = z;
      if (v == targets[n]) zt = z;
    }
    /* second pass: the sum of exp(z - M) */
    double s = 0.0;
    for (int64_t v = 0; v < V; ++v) {
      const uint16_t *wv = W + v * D;
      double z = 0.0;
      for (int64_t k = 0; k < D; ++k) z += lp_bf16(hn[k]) * lp_bf16(wv[k]);
      s += exp(z * scale - M);
    }
    lse[n] = V > 0 ? M + log(s) : -INFINITY;
    logp[n] = (targets[n] >= 0 && targets[n] < V) ? zt - lse[n] : NAN;
  }
  return 0;
}
