/*
 * Host-side checks of libkvc, built with AddressSanitizer and
 * UndefinedBehaviorSanitizer on the host code (tests/test_host_sanitizers.py).
 *
 * It drives every entry point's validation and the host work behind it
 * (layout checks, plan image construction, staging copy lists) over seeded
 * random layouts and the edge cases of the row and position limits.  The
 * "device" addresses are fake, so it runs only where there is no GPU: a
 * valid call then stops at the device check with KVC_ERR_DEVICE.  With a
 * GPU present it exits with 77 (skip) before calling the library.
 *
 * Exit status: 0 all checks passed, 1 a check failed, 77 skipped; a
 * sanitizer report aborts with its own status.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "kvc.h"

#define EXPECT(cond)                                                        \
  do {                                                                      \
    if (!(cond)) {                                                          \
      fprintf(stderr, "line %d: check failed: %s (last error: %s)\n",       \
              __LINE__, #cond, kvc_last_error());                           \
      return 1;                                                             \
    }                                                                       \
  } while (0)

static uint64_t g_state = 0x9e3779b97f4a7c15ull;

/* xorshift64* (Vigna), a seeded stream of test parameters */
static uint64_t next_u64(void) {
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return g_state * 2685821657736338717ull;
}

static int64_t uniform(int64_t lo, int64_t hi) { /* [lo, hi] */
  return lo + (int64_t)(next_u64() % (uint64_t)(hi - lo + 1));
}

/* fake, 256-byte aligned addresses far apart: never dereferenced */
static void* fake(int i) { return (void*)(uintptr_t)((uint64_t)(i + 1) << 46); }

/* a failed call leaves a message naming the entry point */
static int error_names(const char* entry) {
  const char* m = kvc_last_error();
  return m && strstr(m, entry) != NULL;
}

static int random_layout_round(int it) {
  const int32_t n_chunks = (int32_t)(it % 7 == 0 ? uniform(0, 3000) : uniform(0, 40));
  int32_t* len = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n_chunks > 0 ? n_chunks : 1));
  int64_t* old = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_chunks > 0 ? n_chunks : 1));
  uint8_t* zero = (uint8_t*)malloc((size_t)(n_chunks > 0 ? n_chunks : 1));
  double inv_freq[64];
  for (int32_t i = 0; i < n_chunks; ++i) {
    len[i] = (int32_t)(next_u64() % 8 == 0 ? 0 : uniform(1, it % 5 == 0 ? 40000 : 600));
    old[i] = uniform(-100000, 100000);
    zero[i] = (uint8_t)(next_u64() % 5 == 0);
  }
  for (int j = 0; j < 64; ++j) inv_freq[j] = 1.0 / (double)(j + 1);
  const int32_t hkv = (int32_t)uniform(1, 16);
  kvc_layout L;
  memset(&L, 0, sizeof(L));
  L.n_chunks = n_chunks;
  L.chunk_len = n_chunks > 0 ? len : NULL;
  L.chunk_old_pos0 = next_u64() % 2 ? old : NULL;
  L.n_query = uniform(0, 300);
  L.n_kv_heads = hkv;
  L.n_q_heads = hkv * (int32_t)uniform(1, 8);
  L.head_dim = 128;
  L.rope_theta = 500000.0;
  L.inv_freq = next_u64() % 3 == 0 ? inv_freq : NULL;
  L.zero_kv = next_u64() % 2 ? zero : NULL;

  int rc = 1;
  int64_t n_r = 0;
  for (int32_t i = 0; i < n_chunks; ++i) n_r += len[i];
  size_t pb = 0, wb = 0;
  if (kvc_plan_bytes(&L, &pb) != KVC_OK || pb == 0) goto done;
  if (kvc_blend_workspace(&L, &wb) != KVC_OK) goto done;
  /* a short plan buffer is refused; a full one builds the plan image and
     stops at the device check */
  kvc_plan plan;
  memset(&plan, 0, sizeof(plan));
  if (kvc_plan_upload(&L, fake(0), pb - 1, NULL, &plan, NULL) != KVC_ERR_WORKSPACE) goto done;
  if (kvc_plan_upload(&L, fake(0), pb, NULL, &plan, NULL) != KVC_ERR_DEVICE) goto done;
  if (!error_names("kvc_plan_upload")) goto done;
  if (plan.device != NULL) goto done; /* not filled on failure */
  /* host staging: the image is built into it (then the device check) */
  {
    void* staging = malloc(pb);
    const kvc_status st = kvc_plan_upload(&L, fake(0), pb, staging, &plan, NULL);
    free(staging);
    if (st != KVC_ERR_DEVICE) goto done;
  }
  /* a descriptor as the upload would fill it; one of another layout or too
     small a buffer is refused before the device check */
  plan.device = fake(0);
  plan.bytes = pb;
  if (kvc_layout_id(&L, &plan.layout_id) != KVC_OK || plan.layout_id == 0) goto done;
  if (kvc_rope_shift(&L, &plan, fake(1), fake(2), NULL) != (n_r > 0 ? KVC_ERR_DEVICE : KVC_OK)) goto done;
  if (n_r > 0) {
    kvc_plan stale = plan;
    stale.layout_id ^= 2;
    if (kvc_rope_shift(&L, &stale, fake(1), fake(2), NULL) != KVC_ERR_INVALID_ARG) goto done;
    stale = plan;
    stale.bytes = pb - 1;
    if (kvc_rope_shift(&L, &stale, fake(1), fake(2), NULL) != KVC_ERR_WORKSPACE) goto done;
  }
  {
    const double ratio = (double)uniform(0, 100) / 100.0;
    const int64_t k = kvc_recompute_count(ratio, n_r);
    if (k < 0 || k > n_r) goto done;
    const int64_t n_sel = k + L.n_query;
    const kvc_status want = (n_r > 0 || n_sel > 0) ? KVC_ERR_DEVICE : KVC_OK;
    if (kvc_blend_prefill_layer(&L, &plan, 1, ratio, fake(1), fake(2), fake(3), fake(4), fake(5), fake(6),
                                (int32_t*)fake(7), n_sel, fake(8), (float*)fake(9), fake(10), wb, NULL) != want)
      goto done;
    if (kvc_blend_prefill_layer(&L, &plan, 1, ratio, fake(1), fake(2), fake(3), fake(4), fake(5), fake(6),
                                (int32_t*)fake(7), n_sel + 1, fake(8), (float*)fake(9), fake(10), wb,
                                NULL) != KVC_ERR_INVALID_ARG)
      goto done;
    if (kvc_select_tokens(&L, &plan, ratio, fake(1), fake(2), fake(4), (int32_t*)fake(7), n_sel, fake(10), wb,
                          NULL) != want)
      goto done;
  }
  {
    /* staging: one pointer per chunk and layer, separators without one */
    enum { kLayers = 3 };
    const size_t nc = (size_t)(n_chunks > 0 ? n_chunks : 1);
    const void** kch = (const void**)calloc(nc * kLayers, sizeof(void*));
    const void** vch = (const void**)calloc(nc * kLayers, sizeof(void*));
    void* kc[kLayers];
    void* vc[kLayers];
    for (int l = 0; l < kLayers; ++l) {
      kc[l] = fake(20 + l);
      vc[l] = fake(30 + l);
      for (int32_t i = 0; i < n_chunks; ++i) {
        const int sep = L.zero_kv && zero[i];
        kch[(size_t)l * nc + (size_t)i] = sep ? NULL : fake(40 + l);
        vch[(size_t)l * nc + (size_t)i] = sep ? NULL : fake(50 + l);
      }
    }
    const kvc_status st = kvc_stage_layers(&L, &plan, kLayers, kch, vch, kc, vc, NULL, NULL);
    free(kch);
    free(vch);
    if (st != (n_r > 0 ? KVC_ERR_DEVICE : KVC_OK)) goto done;
  }
  rc = 0;
done:
  if (rc) fprintf(stderr, "random layout %d (n_chunks %d, n_reused %lld): %s\n", it, n_chunks, (long long)n_r,
                  kvc_last_error());
  free(len);
  free(old);
  free(zero);
  return rc;
}

int main(void) {
  int n_dev = 0;
  if (hipGetDeviceCount(&n_dev) == hipSuccess && n_dev > 0) {
    puts("skip: a GPU is present (these checks pass fake device addresses)");
    return 77;
  }
  EXPECT(kvc_abi_version() == KVC_ABI_VERSION);

  for (int it = 0; it < 600; ++it)
    if (random_layout_round(it)) return 1;

  /* row limits: 2^31 - 128 rows in total */
  const int64_t max_rows = ((int64_t)1 << 31) - 128;
  {
    int32_t len[2] = {1 << 30, (1 << 30) - 256};
    kvc_layout L;
    memset(&L, 0, sizeof(L));
    L.n_chunks = 2;
    L.chunk_len = len;
    L.n_query = 128;
    L.n_q_heads = 32;
    L.n_kv_heads = 8;
    L.head_dim = 128;
    L.rope_theta = 500000.0;
    size_t pb = 0;
    kvc_plan plan;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_OK);
    EXPECT(kvc_plan_upload(&L, fake(0), pb, NULL, &plan, NULL) == KVC_ERR_DEVICE);
    EXPECT(kvc_plan_upload(&L, fake(0), pb, NULL, NULL, NULL) == KVC_ERR_INVALID_ARG);
    L.n_query = 129;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_ERR_INVALID_ARG && error_names("kvc_plan_bytes"));
    int32_t one[1] = {(int32_t)max_rows};
    L.n_chunks = 1;
    L.chunk_len = one;
    L.n_query = 0;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_OK);
    EXPECT(kvc_plan_upload(&L, fake(0), pb, NULL, &plan, NULL) == KVC_ERR_DEVICE);
    one[0] = (int32_t)(max_rows + 1);
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_ERR_INVALID_ARG);
    int32_t big[3] = {2147483647, 2147483647, 2147483647};
    L.n_chunks = 3;
    L.chunk_len = big;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_ERR_INVALID_ARG);
    /* cached positions within +-2^53 */
    int32_t two[2] = {5, 7};
    int64_t old[2] = {(int64_t)1 << 53, -((int64_t)1 << 53)};
    L.n_chunks = 2;
    L.chunk_len = two;
    L.chunk_old_pos0 = old;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_OK);
    EXPECT(kvc_plan_upload(&L, fake(0), pb, NULL, &plan, NULL) == KVC_ERR_DEVICE);
    old[1] = INT64_MIN;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_ERR_INVALID_ARG);
    old[1] = 0;
    old[0] = INT64_MAX;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_ERR_INVALID_ARG);
    /* non-finite frequency table or theta */
    double f[64];
    for (int j = 0; j < 64; ++j) f[j] = 1.0;
    old[0] = 0;
    L.inv_freq = f;
    L.rope_theta = 0.0;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_OK);
    f[63] = 1.0 / 0.0;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_ERR_INVALID_ARG);
    L.inv_freq = NULL;
    L.rope_theta = -1.0;
    EXPECT(kvc_plan_bytes(&L, &pb) == KVC_ERR_INVALID_ARG);
  }

  /* k = floor(ratio * n) over the whole row range */
  for (int64_t n = 0; n <= max_rows; n = n * 3 + 1)
    for (int r = 0; r <= 100; ++r) {
      const int64_t k = kvc_recompute_count(r / 100.0, n);
      EXPECT(k >= 0 && k <= n);
    }
  EXPECT(kvc_recompute_count(1.5, 10) == -1 && kvc_recompute_count(0.0 / 0.0, 10) == -1);

  /* workspaces and the kernels' own argument checks at the limits */
  size_t b = 0;
  EXPECT(kvc_select_topk_workspace(max_rows, &b) == KVC_OK && b > 0);
  EXPECT(kvc_select_topk_workspace(max_rows + 1, &b) == KVC_ERR_INVALID_ARG);
  for (int64_t n = 0; n <= max_rows; n = n * 5 + 1) {
    EXPECT(kvc_attention_workspace(n, 32, 8, 128, &b) == KVC_OK);
    EXPECT(kvc_attention_workspace(n, 64, 64, 128, &b) == KVC_OK);
  }
  EXPECT(kvc_attention_workspace(max_rows + 1, 32, 8, 128, &b) == KVC_ERR_INVALID_ARG);
  EXPECT(kvc_kv_deviation(max_rows, 8, 128, fake(0), fake(1), (double*)fake(2), NULL) == KVC_ERR_DEVICE);
  EXPECT(kvc_kv_deviation(max_rows + 1, 8, 128, fake(0), fake(1), (double*)fake(2), NULL) == KVC_ERR_INVALID_ARG);
  EXPECT(kvc_select_topk_workspace(max_rows, &b) == KVC_OK);
  EXPECT(kvc_select_topk((const double*)fake(0), max_rows, max_rows / 2, (int32_t*)fake(1), fake(2), b - 1,
                         NULL) == KVC_ERR_WORKSPACE);
  EXPECT(kvc_select_topk((const double*)fake(0), max_rows, max_rows / 2, (int32_t*)fake(1), fake(2), b,
                         NULL) == KVC_ERR_DEVICE);
  /* one attention launch holds about 2 n_sel Hq work-items, at most 2^32 - 1 */
  EXPECT(kvc_sparse_query_attention(fake(0), max_rows, NULL, (const int32_t*)fake(1), max_rows, fake(2), fake(3),
                                    max_rows, 32, 8, 128, 0.0f, fake(4), NULL, NULL, 0, NULL) == KVC_ERR_INVALID_ARG);
  EXPECT(kvc_sparse_query_attention(fake(0), max_rows, NULL, (const int32_t*)fake(1), ((int64_t)1 << 26) - 64,
                                    fake(2), fake(3), max_rows, 32, 8, 128, 0.0f, fake(4), NULL, NULL, 0,
                                    NULL) == KVC_ERR_DEVICE);
  EXPECT(kvc_sparse_query_attention(fake(0), max_rows, NULL, (const int32_t*)fake(1), (int64_t)1 << 26, fake(2),
                                    fake(3), max_rows, 32, 8, 128, 0.0f, fake(4), NULL, NULL, 0,
                                    NULL) == KVC_ERR_INVALID_ARG);
  EXPECT(kvc_sparse_query_attention(fake(0), max_rows, NULL, (const int32_t*)fake(1), (int64_t)1 << 30, fake(2),
                                    fake(3), max_rows, 1, 1, 128, 0.0f, fake(4), NULL, NULL, 0, NULL) == KVC_ERR_DEVICE);
  EXPECT(kvc_sparse_query_attention(fake(0), 10, NULL, (const int32_t*)fake(1), 10, fake(2), fake(3),
                                    max_rows + 1, 32, 8, 128, 0.0f, fake(4), NULL, NULL, 0,
                                    NULL) == KVC_ERR_INVALID_ARG);
  EXPECT(kvc_rms_norm(fake(0), max_rows, NULL, max_rows, 4096, fake(1), 1e-5f, fake(2), NULL, NULL) ==
         KVC_ERR_DEVICE);
  EXPECT(kvc_swiglu(fake(0), 1000, 14336, fake(1), NULL) == KVC_ERR_DEVICE);
  EXPECT(kvc_swiglu(fake(0), max_rows, 1 << 24, fake(1), NULL) == KVC_ERR_INVALID_ARG);
  EXPECT(kvc_qkv_rope(fake(0), 1000, 32, 8, 8, 128, NULL, 500000.0, NULL, fake(1), fake(2), fake(3), NULL) ==
         KVC_ERR_DEVICE);

  /* projections: one launch holds 512 work-items per 256 x 256 output tile,
     at most 2^32 - 1; sizes up to the row and 2^24 limits do not overflow */
  EXPECT(kvc_projection(max_rows, 1024, 4096, fake(0), max_rows, NULL, fake(1), NULL, fake(2), NULL) ==
         KVC_ERR_INVALID_ARG);
  EXPECT(kvc_projection(max_rows, (int64_t)1 << 24, (int64_t)1 << 24, fake(0), max_rows, NULL, fake(1), fake(3),
                        fake(2), NULL) == KVC_ERR_INVALID_ARG);
  EXPECT(kvc_projection((int64_t)1 << 20, 4096, 14336, fake(0), (int64_t)1 << 20, NULL, fake(1), fake(3), fake(2),
                        NULL) == KVC_ERR_DEVICE);
  EXPECT(kvc_projection(256, (int64_t)1 << 24, 4096, fake(0), 7, (const int32_t*)fake(4), fake(1), NULL, fake(2),
                        NULL) == KVC_ERR_DEVICE);
  EXPECT(kvc_projection(256, 8, (int64_t)1 << 24, fake(0), 256, NULL, fake(1), fake(2), fake(2), NULL) ==
         KVC_ERR_DEVICE);
  EXPECT(kvc_projection(256, 8, ((int64_t)1 << 24) + 64, fake(0), 256, NULL, fake(1), NULL, fake(2), NULL) ==
         KVC_ERR_UNSUPPORTED);

  puts("host checks ok");
  return 0;
}
