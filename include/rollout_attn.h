/*
 * rollout_attn.h — C ABI of the MI355X (gfx950) rollout-attention library.
 *
 * The library implements the GPU work that dominates multi-turn agent rollouts
 * as described in "ProRL Agent: Rollout-as-a-Service for RL Training of
 * Multi-Turn LLM Agents" (arXiv 2603.18815):
 *   - every agent step is one LLM completion over the whole conversation
 *     history (Sec. 3.3.2), i.e. a decode step of one new token per trajectory
 *     against that trajectory's cached keys and values;
 *   - all calls of one task go to one backend so that its cached prefix is
 *     reused (Sec. 3.3.2, load balancing), so each trajectory keeps a
 *     persistent paged KV cache across turns;
 *   - earlier turns keep their token ids and only new observations are
 *     tokenised and appended (Sec. 3.3.3), i.e. a causal chunked prefill of the
 *     observation tokens against the existing cache ("append").
 * The paper states no attention formula; the library computes standard
 * scaled dot-product softmax attention with grouped KV heads (query head h
 * reads KV head h / (Hq / Hkv)), bf16 inputs, fp32 accumulation and fp32
 * outputs.
 *
 * Conventions for every entry point
 *   - All array arguments are DEVICE pointers unless marked "host". The caller
 *     owns every buffer (pools, tables, outputs, workspace); the library
 *     allocates nothing and keeps no pointer after it returns.
 *   - Work is enqueued asynchronously on `stream` (0 = the null stream). Buffers
 *     must stay alive until the stream has executed the enqueued kernels.
 *     Concurrent calls on different streams are safe if their outputs and
 *     workspaces do not overlap.
 *   - Every function returns an ra_status. Arguments the host can check are
 *     checked before any HIP call. Nothing aborts. A softmax or logit `scale`
 *     must be finite (any sign; 0 weighs every key equally), else
 *     RA_ERR_SHAPE.
 *   - Zero work (B == 0, total_q == 0, total_new == 0) returns RA_OK without
 *     launching anything.
 *   - Device-resident metadata (lengths, block tables, cu_* offsets) is a
 *     precondition and is not read by the host: lengths >= 0, every position
 *     used lies below bt_stride * page_size, page ids lie in [0, num_pages),
 *     cu_* arrays are non-decreasing with cu[0] = 0. As a guard against
 *     memory faults the kernels clamp page ids into [0, num_pages) and
 *     lengths to the host-provided maxima; violating inputs give undefined
 *     numbers, never an out-of-bounds access.
 *   - Results are deterministic: the same inputs give bitwise the same
 *     outputs, independent of which physical pages the block table names.
 *   - Every entry point may be captured into a HIP graph: it allocates
 *     nothing, never synchronizes, issues no memset or copy (work counters
 *     are cleared by its own kernels), so each replay computes what an
 *     eager call would. Replays of one graph must not overlap in time if
 *     they share a workspace.
 *
 * Paged KV layout (ABI versions 2 to 6). Page size P = 16 tokens, head dim D = 128.
 * Logical token j of row b lives in physical page bt[b * bt_stride + j / P]
 * at slot j % P. Within a page each KV head owns one contiguous block:
 *   K pool  [num_pages][Hkv][P][D]   element (page, g, slot, d) at
 *           ((page * Hkv + g) * P + slot) * D + d           (token-major)
 *   V pool  [num_pages][Hkv][D][P]   element (page, g, slot, d) at
 *           ((page * Hkv + g) * D + d) * P + slot           (dim-major)
 * V is stored dimension-major so that the matrix-core operand for P·V (keys
 * along the contraction dimension) is a contiguous read.
 * Element types (kv_dtype):
 *   RA_KV_BF16      bf16 (4 KiB per page and head);
 *   RA_KV_FP8_E4M3  OCP FP8 E4M3 codes (2 KiB per page and head) with one
 *                   scale per pool: an element's value is decode(code) *
 *                   k_scale (K) or * v_scale (V). The paper is silent on KV
 *                   precision; this halves the bytes decode streams. A bf16
 *                   value x is stored as encode(fp32(x) * fp32(1 / scale)):
 *                   round to nearest even, magnitudes beyond 448 (and
 *                   infinities) saturate to +-448, NaN becomes 0x7F.
 *   fp8 pools are supported by every entry point: kv_page_write (and the
 *   write of rollout_attn_append_write) quantizes, kv_page_gather copies the
 *   codes out, the attention entry points convert the codes exactly to bf16
 *   operands. A mixed call takes one element type for both sides
 *   (RA_ERR_UNSUPPORTED otherwise).
 */
#ifndef ROLLOUT_ATTN_H
#define ROLLOUT_ATTN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RA_ABI_VERSION 6
#define RA_PAGE_SIZE 16
#define RA_HEAD_DIM 128

typedef enum {
  RA_OK = 0,
  RA_ERR_NULL = 1,        /* a required pointer is NULL */
  RA_ERR_SHAPE = 2,       /* inconsistent sizes (negative, Hq % Hkv != 0, ...) */
  RA_ERR_UNSUPPORTED = 3, /* valid but not built: page_size != 16, head_dim != 128,
                             a decode group size Hq / Hkv above 32, an
                             unknown kv_dtype,
                             pools of two element types in one mixed call */
  RA_ERR_WORKSPACE = 4,   /* workspace smaller than the *_workspace_size value */
  RA_ERR_HIP = 5          /* a HIP launch failed (no device, bad stream, ...) */
} ra_status;

typedef enum { RA_KV_BF16 = 0, RA_KV_FP8_E4M3 = 1 } ra_kv_dtype;

/* Caller-owned paged KV cache (device memory), see the layout above. */
typedef struct {
  void *k_pool;               /* [num_pages][num_kv_heads][page_size][head_dim] */
  void *v_pool;               /* [num_pages][num_kv_heads][head_dim][page_size] */
  const int32_t *block_table; /* int32 [B][bt_stride]; row b of the call's batch */
  int32_t num_pages;
  int32_t bt_stride;          /* entries per block-table row (>= 1) */
  int32_t num_kv_heads;       /* Hkv */
  int32_t page_size;          /* must be 16 */
  int32_t head_dim;           /* must be 128 */
  int32_t kv_dtype;           /* ra_kv_dtype of both pools */
  float k_scale, v_scale;     /* fp8 pools: finite, > 0 and with a finite fp32
                                 reciprocal (RA_ERR_SHAPE otherwise); ignored for
                                 bf16 pools */
} ra_paged_kv;

/* ABI version of the loaded library (RA_ABI_VERSION). */
int ra_abi_version(void);

/* Static, human-readable name of a status code. */
const char *ra_status_string(int status);

/*
 * Decode: one query token per trajectory against its cached keys
 * (Sec. 3.3.2: each agent step is a completion over the full history).
 * For row b and query head h with g = h / (Hq / Hkv):
 *   out[b][h] = softmax_j(scale * <q[b][h], K_j>) · V_j over j in [0, kv_lens[b])
 *   lse[b][h] = ln sum_j exp(scale * <q[b][h], K_j>)
 * kv_lens counts the token being decoded (write it with kv_page_write first).
 * Rows with kv_lens[b] <= 0 give out = 0 and lse = -inf.
 *
 *   q           bf16 [B][Hq][128]
 *   kv          pools and block table ([B][bt_stride])
 *   kv_lens     int32 [B]
 *   max_kv_len  host: an upper bound of kv_lens (plans the split over pages);
 *               must satisfy max_kv_len <= bt_stride * 16
 *   out         fp32 [B][Hq][128]
 *   lse         fp32 [B][Hq] or NULL
 *   workspace   device scratch of at least
 *               rollout_attn_decode_workspace_size(B, Hq, Hkv, max_kv_len) bytes
 *               (split partial results; contents on entry are ignored)
 * Errors: RA_ERR_NULL, RA_ERR_SHAPE (B < 0, Hq % Hkv, max_kv_len > bt_stride*16),
 *         RA_ERR_UNSUPPORTED, RA_ERR_WORKSPACE, RA_ERR_HIP.
 */
size_t rollout_attn_decode_workspace_size(int32_t B, int32_t Hq, int32_t Hkv,
                                          int32_t max_kv_len);
int rollout_attn_decode(const void *q, const ra_paged_kv *kv, const int32_t *kv_lens, int32_t B,
                        int32_t Hq, int32_t max_kv_len, float scale, float *out, float *lse,
                        void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Decode that allocates nothing, for callers that cannot allocate device
 * memory or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc. Arguments, results and errors are
 * those of rollout_attn_decode without the workspace; the split partial
 * results go to a scratch array of RA_NOALLOC_SCRATCH_BYTES that the library
 * holds in each GPU's memory until the process ends. A call whose
 * rollout_attn_decode_workspace_size(B, Hq, Hkv, max_kv_len) exceeds
 * RA_NOALLOC_SCRATCH_BYTES returns RA_ERR_WORKSPACE before any HIP call (64
 * MiB holds, e.g., 64 rows of 32 query heads at up to 32768 keys). Every call
 * on one GPU uses that GPU's one array and leaves its contents behind: calls
 * that overlap in time on one GPU (different streams, or threads whose calls
 * are in flight together) race and give wrong results; issue them on one
 * stream.
 */
#define RA_NOALLOC_SCRATCH_BYTES (64u << 20)
int rollout_attn_decode_noalloc(const void *q, const ra_paged_kv *kv, const int32_t *kv_lens,
                                int32_t B, int32_t Hq, int32_t max_kv_len, float scale,
                                float *out, float *lse, hipStream_t stream);

/*
 * Shared-prefix decode: decode for groups of rows whose caches begin with the
 * same physical pages, e.g. the rollouts of one task, which share its prompt
 * (Sec. 4 generates several rollouts per task instance; Sec. 3.3.2 keeps all
 * calls of a task on one backend so that its cached prefix is reused). The
 * result is that of rollout_attn_decode on the same rows (up to rounding: the
 * keys are split differently); the shared keys are read once for up to
 * 16 / (Hq / Hkv) rows of a group (one row per read for groups of more than
 * 16 query heads) instead of once per row, and the reads of one group's
 * chunks of rows are scheduled together so that the later ones mostly hit
 * the cache.
 * For group i, rows group_start[i] .. group_start[i+1]-1 attend their first P_i
 * keys together, P_i = min(prefix_len[i], shortest kv_lens of the group)
 * rounded down to a multiple of 32, read through the block table of the
 * group's first row; each row attends its keys P_i .. kv_lens[b]-1 alone.
 *
 *   q, kv, kv_lens, out, lse, scale: as rollout_attn_decode
 *   group_start     int32 [num_groups + 1], group_start[0] = 0, non-decreasing,
 *                   group_start[num_groups] = B (every row in one group)
 *   prefix_len      int32 [num_groups]: positions [0, prefix_len[i]) of every
 *                   row of group i map to the same pages as the group's first
 *                   row (a precondition: not checked; violating it gives wrong
 *                   numbers, never an out-of-bounds access)
 *   max_group_rows  host: an upper bound of the rows of a group, <= B
 *   max_prefix_len  host: an upper bound of prefix_len, <= max_kv_len
 *   workspace       device scratch of at least
 *                   rollout_attn_decode_shared_prefix_workspace_size(B, Hq, Hkv,
 *                   max_kv_len, max_prefix_len) bytes (contents on entry ignored)
 * Errors: as rollout_attn_decode; RA_ERR_SHAPE also for num_groups == 0 or
 *         max_group_rows == 0 with B > 0, max_group_rows > B, num_groups > B,
 *         max_prefix_len > max_kv_len; RA_ERR_UNSUPPORTED when the launch grid
 *         needs more than 65535 planes: num_groups * max_group_rows row planes
 *         plus ceil(num_groups * chunks * prefix splits / splits) prefix planes,
 *         chunks = ceil(max_group_rows / rows per chunk).
 */
size_t rollout_attn_decode_shared_prefix_workspace_size(int32_t B, int32_t Hq, int32_t Hkv,
                                                        int32_t max_kv_len,
                                                        int32_t max_prefix_len);
int rollout_attn_decode_shared_prefix(const void *q, const ra_paged_kv *kv,
                                      const int32_t *kv_lens, const int32_t *group_start,
                                      const int32_t *prefix_len, int32_t B, int32_t Hq,
                                      int32_t num_groups, int32_t max_group_rows,
                                      int32_t max_prefix_len, int32_t max_kv_len, float scale,
                                      float *out, float *lse, void *workspace,
                                      size_t workspace_bytes, hipStream_t stream);

/*
 * Append: causal chunked prefill of newly appended observation tokens against
 * each trajectory's cache (Sec. 3.3.3: earlier turns keep their tokens, new
 * observations are tokenised and appended). Row b owns packed queries
 * cu_q[b] .. cu_q[b+1]-1; its i-th query sits at absolute position
 * ctx_lens[b] + i and attends keys 0 .. ctx_lens[b] + i (inclusive):
 *   out[t][h] = softmax_j(scale * <q[t][h], K_j>) · V_j,  lse likewise.
 * The chunk's own keys and values must already be in the pool at positions
 * ctx_lens[b] .. ctx_lens[b] + T_b - 1 (kv_page_write with start_pos = ctx_lens
 * on the same stream first).
 *
 *   q           bf16 [total_q][Hq][128]
 *   cu_q        int32 [B+1], cu_q[0] = 0, cu_q[B] = total_q
 *   ctx_lens    int32 [B]
 *   max_q_len   host: an upper bound of T_b = cu_q[b+1] - cu_q[b]
 *   max_kv_len  host: an upper bound of ctx_lens[b] + T_b; <= bt_stride * 16
 *   out         fp32 [total_q][Hq][128]
 *   lse         fp32 [total_q][Hq] or NULL
 *   workspace   device scratch of at least
 *               rollout_attn_append_workspace_size(B, Hq, Hkv, max_q_len) bytes
 *               (the call's work list and counter, rewritten by every call;
 *               contents on entry are ignored). Calls that share a workspace
 *               must not overlap.
 * The work is planned on the device (a one-workgroup kernel orders the rows
 * longest first and queues each KV head's tiles for one XCD) and run by one
 * persistent workgroup per CU.
 * Errors as for decode; RA_ERR_UNSUPPORTED also for more than 256 KV heads.
 */
size_t rollout_attn_append_workspace_size(int32_t B, int32_t Hq, int32_t Hkv,
                                          int32_t max_q_len);
int rollout_attn_append(const void *q, const int32_t *cu_q, const int32_t *ctx_lens,
                        const ra_paged_kv *kv, int32_t B, int32_t Hq, int32_t total_q,
                        int32_t max_q_len, int32_t max_kv_len, float scale, float *out,
                        float *lse, void *workspace, size_t workspace_bytes,
                        hipStream_t stream);

/*
 * Append with the page write fused in: writes the chunk's keys and values into
 * the pages and computes the append attention in one launch (plus the
 * planning kernel). Equivalent, bitwise, to kv_page_write(k_new, v_new, cu_q,
 * start_pos = ctx_lens) followed by rollout_attn_append on the same stream
 * (Sec. 3.3.3: each new observation is appended to the retained tokens and
 * attended in the same step). The write runs inside the planning kernel's
 * launch (its other workgroups write while one plans), so the call is two
 * launches instead of the three of the separate calls; the attention kernel
 * then reads the chunk from the pages.
 *
 *   q, cu_q, ctx_lens, kv, B, Hq, total_q, max_q_len, max_kv_len, scale, out,
 *   lse, workspace: as rollout_attn_append (same workspace size)
 *   k_new, v_new  bf16 [total_q][Hkv][128]: the chunk tokens' keys and values,
 *                 packed like q; token i of row b goes to position
 *                 ctx_lens[b] + i
 * fp8 pools: the chunk is quantized as by kv_page_write (encode(fp32(x) *
 * fp32(1 / scale)), see the layout above) and attended as stored.
 * Precondition (not checked): no row of the call reads, below its ctx, a page
 * slot that another row of the call writes.
 * Errors: as rollout_attn_append.
 */
int rollout_attn_append_write(const void *q, const void *k_new, const void *v_new,
                              const int32_t *cu_q, const int32_t *ctx_lens, const ra_paged_kv *kv,
                              int32_t B, int32_t Hq, int32_t total_q, int32_t max_q_len,
                              int32_t max_kv_len, float scale, float *out, float *lse,
                              void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Rotary position embedding on write. Models of the paper's kind (e.g. Qwen3)
 * rotate each query and key by its position before attention; the paper does
 * not describe model internals, so the rotation is an option of the write
 * path: the key is rotated as it is written into its page, and in the fused
 * call the chunk's queries are rotated as they are loaded.
 *
 * Rotation of a 128-dim head row x at position p with the table cos_sin
 * (fp32 [rope_rows][128]; row p holds c_i = cos(p w_i) in columns 0..63 and
 * s_i = sin(p w_i) in columns 64..127, computed by the caller for its model's
 * frequencies w_i), for i in [0, 64):
 *   y_i      = fp32(x_i c_i) - fp32(x_{i+64} s_i)
 *   y_{i+64} = fp32(x_{i+64} c_i) + fp32(x_i s_i)
 * each product and each sum rounded to fp32 (no fused multiply-add), then y
 * rounded to bf16 (nearest even). The rotated bf16 row is what is written
 * (bit copy, or E4M3 quantization for fp8 pools, exactly as kv_page_write
 * writes a bf16 row) and what the attention uses.
 *
 * kv_page_write_rope: kv_page_write with the keys rotated at their positions
 *   start_pos[b] + t (values unrotated). Needs max_pos <= rope_rows.
 * rollout_attn_append_write_rope: rollout_attn_append_write with the chunk's
 *   keys rotated at ctx_lens[b] + i as they are written and its queries
 *   rotated at the same positions; equal, bitwise, to kv_page_write_rope
 *   followed by rollout_attn_append on the rotated queries. Needs
 *   max_kv_len <= rope_rows.
 * Errors: as the unrotated calls; RA_ERR_NULL (cos_sin NULL); RA_ERR_SHAPE
 * (rope_rows <= 0 or too few rows).
 */
int kv_page_write_rope(const void *k_new, const void *v_new, const int32_t *cu_new,
                       const int32_t *start_pos, const ra_paged_kv *kv, int32_t B,
                       int32_t total_new, int32_t max_new, int32_t max_pos, const float *cos_sin,
                       int32_t rope_rows, hipStream_t stream);
int rollout_attn_append_write_rope(const void *q, const void *k_new, const void *v_new,
                                   const int32_t *cu_q, const int32_t *ctx_lens,
                                   const ra_paged_kv *kv, int32_t B, int32_t Hq, int32_t total_q,
                                   int32_t max_q_len, int32_t max_kv_len, float scale,
                                   const float *cos_sin, int32_t rope_rows, float *out, float *lse,
                                   void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Mixed step: the attention of one rollout step in which some trajectories
 * decode a token while others have just had tool observations appended
 * (Sec. 3.3.1: many rollout workers drive their agent loops concurrently, each
 * firing LLM calls; Sec. 3.3.3: observations are appended to the retained
 * tokens). Computes, in one persistent launch over the GPU (plus the one-
 * workgroup planning kernel before it and the decode combine after it):
 *   - for the decode rows, exactly what rollout_attn_decode computes
 *     (up to rounding: each split is summed by twice as many waves);
 *   - for the append rows, bitwise what rollout_attn_append computes.
 * Append tiles are taken longest first and the decode splits are spread
 * among them, so that decode's HBM traffic can overlap append's matrix work.
 * The two sides may use different block tables (and pools); either side may
 * be empty (B_decode == 0, or B_append == 0 / total_q == 0 / max_q_len == 0),
 * in which case its pointers are not used and may be NULL.
 *
 *   decode side:  q_decode, kv_decode, kv_lens, B_decode, max_kv_len_decode,
 *                 out_decode, lse_decode: as q, kv, kv_lens, B, max_kv_len,
 *                 out, lse of rollout_attn_decode
 *   append side:  q_append, cu_q, ctx_lens, kv_append, B_append, total_q,
 *                 max_q_len, max_kv_len_append, out_append, lse_append: as q,
 *                 cu_q, ctx_lens, kv, B, total_q, max_q_len, max_kv_len, out,
 *                 lse of rollout_attn_append (the chunks' K/V already written)
 *   Hq, scale     shared by both sides
 *   workspace     device scratch of at least rollout_attn_mixed_workspace_size(
 *                 B_decode, B_append, Hq, Hkv_decode, Hkv_append,
 *                 max_kv_len_decode, max_q_len) bytes: work lists, a work
 *                 counter and decode partials, all rewritten by every call
 *                 (contents on entry are ignored). Calls that share a
 *                 workspace must not overlap.
 * Errors: as rollout_attn_decode / rollout_attn_append for each non-empty
 *         side; RA_ERR_UNSUPPORTED also for more than 256 KV heads or more
 *         than 2^31 - 2^16 work entries.
 */
size_t rollout_attn_mixed_workspace_size(int32_t B_decode, int32_t B_append, int32_t Hq,
                                         int32_t Hkv_decode, int32_t Hkv_append,
                                         int32_t max_kv_len_decode, int32_t max_q_len);
int rollout_attn_mixed(const void *q_decode, const ra_paged_kv *kv_decode,
                       const int32_t *kv_lens, int32_t B_decode, int32_t max_kv_len_decode,
                       float *out_decode, float *lse_decode, const void *q_append,
                       const int32_t *cu_q, const int32_t *ctx_lens, const ra_paged_kv *kv_append,
                       int32_t B_append, int32_t total_q, int32_t max_q_len,
                       int32_t max_kv_len_append, float *out_append, float *lse_append,
                       int32_t Hq, float scale, void *workspace, size_t workspace_bytes,
                       hipStream_t stream);

/*
 * Token log-probabilities under an LM head: for each position n, the
 * log-probability of the emitted token targets[n] (Sec. 3.3.3: token-in /
 * token-out returns every generated token with its log-probability), fused
 * into one pass over the LM-head matrix without writing the logits:
 *   z_v = scale * <h[n], W[v]>,  lse[n] = ln sum_v exp z_v,
 *   logprob[n] = z_{targets[n]} - lse[n]   (NaN if targets[n] is not in [0, V))
 * bf16 inputs, fp32 products and outputs.
 *
 *   h          bf16 [N][D] hidden states (row n: the position's last-layer output)
 *   W          bf16 [V][D] LM-head matrix, one row per vocabulary entry
 *   targets    int32 [N]
 *   scale      multiplies the logits (1 / temperature; 1 for the raw model)
 *   logprob    fp32 [N]
 *   lse        fp32 [N] or NULL
 *   workspace  device scratch of at least token_logprob_workspace_size(N, V, D)
 *              bytes (per-chunk partials and, from N = 512 on, a copy of h in
 *              the order the large-batch kernel loads it: N rounded up to 256
 *              rows x D bf16; contents on entry ignored)
 * Errors: RA_ERR_NULL; RA_ERR_SHAPE (N < 0, V <= 0, D <= 0);
 *         RA_ERR_UNSUPPORTED (D not a multiple of 64); RA_ERR_WORKSPACE;
 *         RA_ERR_HIP. N == 0 returns RA_OK without launching anything.
 */
size_t token_logprob_workspace_size(int32_t N, int32_t V, int32_t D);
int token_logprob(const void *h, const void *W, const int32_t *targets, int32_t N, int32_t V,
                  int32_t D, float scale, float *logprob, float *lse, void *workspace,
                  size_t workspace_bytes, hipStream_t stream);

/*
 * The same log-probabilities from a packed copy of the LM-head matrix. The
 * matrix is constant for a policy version, so it can be repacked once into
 * the order the kernel's matrix products consume it; each wave then reads
 * 4 KB contiguous per 64-dim step instead of 32 rows 128 bytes at a time,
 * and the waves on one step read one narrow window of memory.
 * Results are bitwise those of token_logprob on the unpacked matrix.
 *
 * Packed layout: bf16, 16-byte units; with T = ceil(V / 384) * 12 tiles of
 * 32 rows (V rounded up to a multiple of 384), unit
 *   i = ((s * T + tile) * 4 + u) * 64 + lane
 * holds W[32 * tile + lane % 32][64 * s + 32 * (lane / 32) + 8 * u + 0..7],
 * zeros for rows at or past V. ABI versions 4 and 5 stored the units tile by
 * tile, i = ((tile * (D / 64) + s) * 4 + u) * 64 + lane, and version 4 rounded
 * V up to 256 rows: a copy made by an older library must be packed again.
 *
 * token_logprob_packed_weight_size: bytes of the packed copy (0 if V <= 0,
 *   D <= 0 or D is not a multiple of 64).
 * token_logprob_pack_weight: writes the packed copy of W (bf16 [V][D]) into
 *   W_packed (device, packed_bytes >= the size above). Errors: RA_ERR_SHAPE
 *   (V <= 0, D <= 0), RA_ERR_NULL, RA_ERR_UNSUPPORTED (D % 64 != 0),
 *   RA_ERR_WORKSPACE (packed_bytes too small), RA_ERR_HIP.
 * token_logprob_packed: token_logprob with W_packed in place of W; the same
 *   arguments, errors and workspace size.
 */
size_t token_logprob_packed_weight_size(int32_t V, int32_t D);
int token_logprob_pack_weight(const void *W, int32_t V, int32_t D, void *W_packed,
                              size_t packed_bytes, hipStream_t stream);
int token_logprob_packed(const void *h, const void *W_packed, const int32_t *targets, int32_t N,
                         int32_t V, int32_t D, float scale, float *logprob, float *lse,
                         void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Page write: append new tokens' keys and values to each trajectory's cache
 * (Sec. 3.3.3: the tokens of earlier turns are kept as they are and only the
 * new observation tokens are tokenised and added after them; Sec. 3.3.2: each
 * agent step's completion extends the same history, so every decoded token is
 * added too). The cache that later steps reuse (Sec. 3.3.2, load balancing
 * keeps a task on one backend for this) is therefore only ever extended at
 * its end, one chunk or one token per row and call.
 * The write is a bit copy into bf16 pools and a quantization into fp8 pools
 * (each element stored as encode(fp32(x) * fp32(1 / scale)), see the layout
 * above). Row b's new tokens are packed rows cu_new[b] .. cu_new[b+1]-1 of
 * k_new / v_new; token t of the row goes to logical position start_pos[b] + t,
 * i.e. page bt[b][(start_pos[b] + t) / 16], slot (start_pos[b] + t) % 16. No
 * other pool byte changes. Rows of one call must not write the same slot.
 *
 *   k_new, v_new  bf16 [total_new][Hkv][128] (token-major), read only
 *   cu_new        int32 [B+1], non-decreasing, cu_new[0] = 0
 *   start_pos     int32 [B]
 *   kv            pools written in place (caller-owned), block table read
 *   B, total_new  host: rows and packed tokens of the call
 *   max_new       host: an upper bound of cu_new[b+1] - cu_new[b]
 *   max_pos       host: an upper bound of start_pos[b] + new tokens of row b;
 *                 <= bt_stride * 16
 * Errors: RA_ERR_NULL (a NULL pointer), RA_ERR_SHAPE (negative sizes,
 *         max_pos > bt_stride * 16, max_new > max_pos, bad fp8 scales),
 *         RA_ERR_UNSUPPORTED (page_size != 16, head_dim != 128, B > 65535),
 *         RA_ERR_HIP. B == 0, total_new == 0 or max_new == 0 launch nothing.
 */
int kv_page_write(const void *k_new, const void *v_new, const int32_t *cu_new,
                  const int32_t *start_pos, const ra_paged_kv *kv, int32_t B, int32_t total_new,
                  int32_t max_new, int32_t max_pos, hipStream_t stream);

/*
 * Page gather (test and export helper): read back, in logical order, the
 * cached history of each trajectory that the attention entry points attend to
 * (Sec. 3.3.2: a task's later calls reuse its cached prefix; Sec. 3.3.3: that
 * prefix is the retained token sequence with the observations appended). It
 * copies logical tokens 0 .. lens[b]-1 of every row out of the pages (token j
 * from page bt[b][j / 16], slot j % 16) into packed token-major arrays; row b
 * starts at packed row cu_out[b]. A bit copy of the stored elements (E4M3
 * codes for fp8 pools); it checks a write and exports a trajectory's cache.
 *
 *   kv       pools and block table, read only
 *   lens     int32 [B]; max_len host upper bound of lens (<= bt_stride * 16)
 *   cu_out   int32 [B+1], non-decreasing, cu_out[0] = 0, cu_out[B] <= total
 *   k_out, v_out  [total][Hkv][128] of the pools' element type (caller-owned,
 *            written)
 * Errors: RA_ERR_NULL, RA_ERR_SHAPE (negative sizes, max_len > bt_stride *
 *         16), RA_ERR_UNSUPPORTED (B > 65535, unsupported page layout),
 *         RA_ERR_HIP. B == 0, total == 0 or max_len == 0 launch nothing.
 */
int kv_page_gather(const ra_paged_kv *kv, const int32_t *lens, const int32_t *cu_out, int32_t B,
                   int32_t total, int32_t max_len, void *k_out, void *v_out,
                   hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* ROLLOUT_ATTN_H */
