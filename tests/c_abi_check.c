/*
 * A plain C99 caller of the library: compiles against include/rollout_attn.h
 * alone, links librollout_attn.so, and calls every entry point once with
 * arguments the host-side validation rejects (or zero work), so no GPU is
 * needed. Prints one line per failed check; exits non-zero if any failed.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "rollout_attn.h"

static int failures = 0;

static void expect(const char *what, int got, int want) {
  if (got != want) {
    printf("FAIL %s: got %d (%s), want %d (%s)\n", what, got, ra_status_string(got), want,
           ra_status_string(want));
    ++failures;
  }
}

int main(void) {
  /* never dereferenced: every call below is rejected (or does nothing) on the host */
  void *fake = (void *)(uintptr_t)0x1000;
  const int32_t *ifake = (const int32_t *)fake;
  float *ffake = (float *)fake;
  char ws[16];

  ra_paged_kv kv;
  memset(&kv, 0, sizeof kv);
  kv.k_pool = fake;
  kv.v_pool = fake;
  kv.block_table = ifake;
  kv.num_pages = 10;
  kv.bt_stride = 4;
  kv.num_kv_heads = 2;
  kv.page_size = RA_PAGE_SIZE;
  kv.head_dim = RA_HEAD_DIM;
  kv.kv_dtype = RA_KV_BF16;
  kv.k_scale = kv.v_scale = 1.0f;

  expect("abi version", ra_abi_version(), RA_ABI_VERSION);
  if (strcmp(ra_status_string(RA_ERR_WORKSPACE), "RA_ERR_WORKSPACE") != 0) {
    printf("FAIL status string\n");
    ++failures;
  }

  expect("decode workspace > 0", rollout_attn_decode_workspace_size(2, 4, 2, 64) > 0, 1);
  expect("decode: NULL q",
         rollout_attn_decode(NULL, &kv, ifake, 2, 4, 64, 0.1f, ffake, NULL, ws, sizeof ws, 0),
         RA_ERR_NULL);
  expect("decode: small workspace",
         rollout_attn_decode(fake, &kv, ifake, 2, 4, 64, 0.1f, ffake, NULL, ws, sizeof ws, 0),
         RA_ERR_WORKSPACE);
  expect("decode: no rows",
         rollout_attn_decode(fake, &kv, ifake, 0, 4, 64, 0.1f, ffake, NULL, ws, sizeof ws, 0),
         RA_OK);
  expect("decode_noalloc: NULL out",
         rollout_attn_decode_noalloc(fake, &kv, ifake, 2, 4, 64, 0.1f, NULL, NULL, 0),
         RA_ERR_NULL);
  {
    /* 256 rows x 64 heads of up to 65536 keys need more partials than the scratch holds */
    ra_paged_kv big = kv;
    big.num_kv_heads = 8;
    big.bt_stride = 4096;
    expect("decode_noalloc: plan beyond the scratch",
           rollout_attn_decode_noalloc(fake, &big, ifake, 256, 64, 65536, 0.1f, ffake, NULL, 0),
           RA_ERR_WORKSPACE);
    if (rollout_attn_decode_workspace_size(256, 64, 8, 65536) <= RA_NOALLOC_SCRATCH_BYTES) {
      printf("FAIL decode_noalloc: the rejected plan fits the scratch\n");
      ++failures;
    }
  }
  expect("shared-prefix decode: NULL group_start",
         rollout_attn_decode_shared_prefix(fake, &kv, ifake, NULL, ifake, 16, 4, 2, 8, 32, 64,
                                           0.1f, ffake, NULL, ws, sizeof ws, 0),
         RA_ERR_NULL);
  expect("shared-prefix workspace > 0",
         rollout_attn_decode_shared_prefix_workspace_size(16, 4, 2, 64, 32) > 0, 1);
  expect("append workspace > 0", rollout_attn_append_workspace_size(2, 4, 2, 5) > 0, 1);
  expect("append: Hq not a multiple of Hkv",
         rollout_attn_append(fake, ifake, ifake, &kv, 2, 5, 10, 5, 64, 0.1f, ffake, NULL, ws,
                             sizeof ws, 0),
         RA_ERR_SHAPE);
  expect("append_write: NULL k_new",
         rollout_attn_append_write(fake, NULL, fake, ifake, ifake, &kv, 2, 4, 10, 5, 64, 0.1f,
                                   ffake, NULL, ws, sizeof ws, 0),
         RA_ERR_NULL);
  expect("mixed workspace > 0", rollout_attn_mixed_workspace_size(2, 2, 4, 2, 2, 64, 5) > 0, 1);
  expect("mixed: NULL q_append",
         rollout_attn_mixed(fake, &kv, ifake, 2, 64, ffake, NULL, NULL, ifake, ifake, &kv, 2,
                            10, 5, 64, ffake, NULL, 4, 0.1f, ws, sizeof ws, 0),
         RA_ERR_NULL);
  expect("logprob workspace", (int)(token_logprob_workspace_size(8, 100, 128) > 0), 1);
  expect("logprob: D not a multiple of 64",
         token_logprob(fake, fake, ifake, 8, 100, 96, 1.0f, ffake, NULL, ws, sizeof ws, 0),
         RA_ERR_UNSUPPORTED);
  expect("packed weight size",
         (int)(token_logprob_packed_weight_size(100, 128) == (size_t)384 * 128 * 2), 1);
  expect("pack weight: small buffer",
         token_logprob_pack_weight(fake, 100, 128, fake, 16, 0), RA_ERR_WORKSPACE);
  expect("logprob packed: NULL W",
         token_logprob_packed(fake, NULL, ifake, 8, 100, 128, 1.0f, ffake, NULL, ws, sizeof ws,
                              0),
         RA_ERR_NULL);
  expect("page write: max_pos past the table",
         kv_page_write(fake, fake, ifake, ifake, &kv, 2, 4, 2, 65, 0), RA_ERR_SHAPE);
  expect("page write rope: NULL table",
         kv_page_write_rope(fake, fake, ifake, ifake, &kv, 2, 4, 2, 32, NULL, 64, 0),
         RA_ERR_NULL);
  expect("page write rope: table shorter than max_pos",
         kv_page_write_rope(fake, fake, ifake, ifake, &kv, 2, 4, 2, 32, ffake, 31, 0),
         RA_ERR_SHAPE);
  expect("append_write rope: no table rows",
         rollout_attn_append_write_rope(fake, fake, fake, ifake, ifake, &kv, 2, 4, 10, 5, 64,
                                        0.1f, ffake, 0, ffake, NULL, ws, sizeof ws, 0),
         RA_ERR_SHAPE);
  expect("append_write rope: small workspace",
         rollout_attn_append_write_rope(fake, fake, fake, ifake, ifake, &kv, 2, 4, 10, 5, 64,
                                        0.1f, ffake, 64, ffake, NULL, ws, sizeof ws, 0),
         RA_ERR_WORKSPACE);
  expect("page gather: NULL k_out",
         kv_page_gather(&kv, ifake, ifake, 2, 8, 4, NULL, fake, 0), RA_ERR_NULL);
  kv.kv_dtype = RA_KV_FP8_E4M3;
  kv.k_scale = 0.0f;
  expect("fp8 pool with a zero scale",
         rollout_attn_decode(fake, &kv, ifake, 2, 4, 64, 0.1f, ffake, NULL, ws, sizeof ws, 0),
         RA_ERR_SHAPE);

  printf("%s (%d failed)\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
