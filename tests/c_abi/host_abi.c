/* A plain C11 consumer of include/bsr.h: host-only context (no GPU), caller
 * arena, chunk keys, single and bulk store insertion, probe, removal, the
 * file tier, admission configuration and the error paths.  Prints one line
 * per result for the Python side to compare with the oracle; exits non-zero
 * on the first violated expectation. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "bsr.h"

#define CHECK(cond)                                                                         \
  do {                                                                                      \
    if (!(cond)) {                                                                          \
      fprintf(stderr, "FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond, bsr_last_error()); \
      return 1;                                                                             \
    }                                                                                       \
  } while (0)

enum { C = 16, N_CHUNKS = 6, N_TOKENS = C * N_CHUNKS + 5 };

static void fill(uint8_t* p, size_t n, uint32_t seed) {
  uint32_t x = seed * 2654435761u + 1u;
  for (size_t i = 0; i < n; ++i) {
    x ^= x << 13;
    x ^= x >> 17;
    x ^= x << 5;
    p[i] = (uint8_t)x;
  }
}

int main(int argc, char** argv) {
  const char* dir = argc > 1 ? argv[1] : NULL;
  CHECK(bsr_abi_version() == BSR_ABI_VERSION);
  CHECK(bsr_struct_size(BSR_STRUCT_CONFIG) == sizeof(bsr_config));
  CHECK(bsr_struct_size(BSR_STRUCT_ADMISSION) == sizeof(bsr_admission));

  bsr_layout L;
  memset(&L, 0, sizeof L);
  L.chunk_tokens = C;
  L.n_groups = 2;
  L.groups[0] = (bsr_group_desc){8, 2, 40, BSR_KIND_CONTIG, 0};
  L.groups[1] = (bsr_group_desc){32, 1, 36, BSR_KIND_PLANAR, 32};
  const uint64_t pay0 = 2u * C * 40u, pay1 = 1u * C * 36u;
  const uint64_t slot = bsr_slot_bytes(&L);
  CHECK(slot == ((pay0 + 255) / 256 * 256) + ((pay1 + 255) / 256 * 256));
  printf("slot %llu\n", (unsigned long long)slot);

  int32_t tokens[N_TOKENS];
  for (int i = 0; i < N_TOKENS; ++i) tokens[i] = (int32_t)(i * 7919 % 129280) - 3;
  const uint64_t salt = 0x9e3779b97f4a7c15ull;
  uint64_t keys[N_CHUNKS];
  CHECK(bsr_chunk_keys(salt, tokens, N_TOKENS, C, keys) == BSR_OK);
  for (int i = 0; i < N_CHUNKS; ++i) printf("key %d %016llx\n", i, (unsigned long long)keys[i]);

  bsr_config cfg;
  memset(&cfg, 0, sizeof cfg);
  cfg.window_chunks = 2;
  cfg.hip_device = -1;
  bsr_ctx* ctx = NULL;
  CHECK(bsr_ctx_create(&L, &cfg, &ctx) == BSR_OK && ctx);
  const uint64_t stride = (slot + 4095) / 4096 * 4096;
  uint8_t* arena = (uint8_t*)aligned_alloc(4096, stride * (N_CHUNKS + 2));
  CHECK(arena);
  CHECK(bsr_store_adopt(ctx, arena, stride * (N_CHUNKS + 2)) == BSR_OK);

  /* chunk payloads: chunk i, group g from seed 16 i + g */
  static uint8_t p0[N_CHUNKS][2 * C * 40], p1[N_CHUNKS][C * 36];
  const void* ptrs[N_CHUNKS * 2];
  for (int i = 0; i < N_CHUNKS; ++i) {
    fill(p0[i], sizeof p0[i], 16u * i);
    fill(p1[i], sizeof p1[i], 16u * i + 1u);
    ptrs[2 * i] = p0[i];
    ptrs[2 * i + 1] = p1[i];
  }
  /* chunk 0 alone, chunks 1..4 in bulk; chunk 5 is never stored */
  CHECK(bsr_store_put_chunk(ctx, keys[0], ptrs) == BSR_OK);
  CHECK(bsr_store_put_chunks(ctx, 4, keys + 1, ptrs + 2) == BSR_OK);
  void* a1 = NULL;
  void* a4 = NULL;
  uint64_t nb = 0, tag = 0;
  CHECK(bsr_store_payload(ctx, keys[1], 0, &a1, &nb, &tag) == BSR_OK && nb == pay0);
  CHECK(bsr_store_payload(ctx, keys[4], 0, &a4, NULL, NULL) == BSR_OK);
  CHECK((uint8_t*)a4 - (uint8_t*)a1 == (ptrdiff_t)(3 * stride));  /* bulk chunks sit back to back */
  CHECK(memcmp(a1, p0[1], pay0) == 0);
  for (int i = 0; i < N_CHUNKS - 1; ++i)
    for (uint32_t g = 0; g < 2; ++g) {
      CHECK(bsr_store_payload(ctx, keys[i], g, NULL, NULL, &tag) == BSR_OK);
      printf("tag %d %u %016llx\n", i, g, (unsigned long long)tag);
    }

  uint32_t n_hit = 99;
  uint8_t bitmap[1] = {0xff};
  uint64_t kout[N_CHUNKS];
  CHECK(bsr_probe(ctx, 7, salt, tokens, N_TOKENS, &n_hit, bitmap, kout) == BSR_OK);
  CHECK(n_hit == 5 && bitmap[0] == 0x1f && memcmp(kout, keys, sizeof keys) == 0);
  CHECK(bsr_store_remove(ctx, keys[2], 1) == BSR_OK);
  CHECK(bsr_probe(ctx, 8, salt, tokens, N_TOKENS, &n_hit, bitmap, NULL) == BSR_OK);
  CHECK(n_hit == 2 && bitmap[0] == 0x1b);
  printf("probe %u %02x\n", n_hit, bitmap[0]);
  CHECK(bsr_store_remove(ctx, keys[2], 1) == BSR_E_NOTFOUND);

  /* protocol and device errors on a host-only context */
  CHECK(bsr_restore_window(ctx, 8, 0, 1) == BSR_E_DEVICE);
  CHECK(bsr_commit(ctx, 8, NULL, NULL) == BSR_E_DEVICE);
  CHECK(bsr_set_timing(ctx, BSR_FLAG_TIME_INSTALL | BSR_FLAG_TIME_STAGE) == BSR_OK);
  CHECK(bsr_set_timing(ctx, 0) == BSR_OK);
  CHECK(bsr_set_timing(ctx, BSR_FLAG_SDMA_COPIES) == BSR_E_ARG);  /* not a timing flag */
  CHECK(bsr_set_timing(NULL, 0) == BSR_E_ARG);
  uint32_t w_first = 7, w_n = 7;
  CHECK(bsr_next_window(ctx, 8, &w_first, &w_n) == BSR_E_STATE);  /* nothing is bound */
  CHECK(bsr_next_window(ctx, 8, NULL, &w_n) == BSR_E_ARG);
  CHECK(bsr_next_window(NULL, 8, &w_first, &w_n) == BSR_E_ARG);
  uint8_t tiers[N_CHUNKS];
  CHECK(bsr_plan_tiers(ctx, 8, tiers, N_CHUNKS) == BSR_OK);
  CHECK(tiers[0] == BSR_TIER_PINNED && tiers[2] == BSR_TIER_NONE);
  bsr_admission adm;
  CHECK(bsr_admission_get(ctx, &adm) == BSR_OK && adm.max_bound_requests == 1 && adm.n_bound == 0);
  bsr_stats st;
  CHECK(bsr_request_stats(ctx, 8, &st) == BSR_E_NOTFOUND);
  CHECK(bsr_stats_get(ctx, &st) == BSR_OK && st.window_chunks == 2);

  /* the file tier, when a directory is given */
  if (dir) {
    CHECK(bsr_file_tier_open(ctx, dir, 2, 0, 0) == BSR_OK);
    CHECK(bsr_file_tier_put_chunk(ctx, keys[5], ptrs + 10) == BSR_OK);
    uint64_t n_files = 0;
    CHECK(bsr_file_tier_count(ctx, &n_files) == BSR_OK && n_files == 2);
    CHECK(bsr_tier_set_available(ctx, BSR_TIER_PINNED, 0) == BSR_OK);
    CHECK(bsr_probe(ctx, 9, salt, tokens, N_TOKENS, &n_hit, bitmap, NULL) == BSR_OK);
    CHECK(n_hit == 0 && bitmap[0] == 0x20);
    CHECK(bsr_file_tier_remove(ctx, keys[5], -1) == BSR_OK);
    CHECK(bsr_file_tier_count(ctx, &n_files) == BSR_OK && n_files == 0);
  }
  CHECK(bsr_request_end(ctx, 7) == BSR_OK);
  CHECK(bsr_ctx_destroy(ctx) == BSR_OK);

  /* configuration errors */
  cfg.max_bound_requests = 2;  /* more than one slot needs a budget */
  CHECK(bsr_ctx_create(&L, &cfg, &ctx) == BSR_E_ARG && ctx == NULL);
  cfg.max_bound_requests = 0;
  cfg.staging_budget_bytes = 5 * 2 * slot;
  CHECK(bsr_ctx_create(&L, &cfg, &ctx) == BSR_OK);
  CHECK(bsr_admission_get(ctx, &adm) == BSR_OK && adm.max_bound_requests == 5);
  CHECK(bsr_ctx_destroy(ctx) == BSR_OK);
  /* a context without allocations: one session slot on a GPU only */
  ctx = (bsr_ctx*)1;
  CHECK(bsr_ctx_create_static(&L, &cfg, &ctx) == BSR_E_ARG && ctx == NULL); /* budget set */
  cfg.staging_budget_bytes = 0;
  ctx = (bsr_ctx*)1;
  CHECK(bsr_ctx_create_static(&L, &cfg, &ctx) == BSR_E_ARG && ctx == NULL); /* hip_device = -1 */
  L.groups[1].split_bytes = 36; /* split must be < record */
  CHECK(bsr_slot_bytes(&L) == 0);
  free(arena);
  printf("ok\n");
  return 0;
}
