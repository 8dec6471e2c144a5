/*
 * A plain C client of libkvc: one check layer of the selective-recompute
 * prefill through the C ABI alone, with the HIP runtime for device memory and
 * the stream (no Python, no torch).  tests/test_gpu_c_abi.py writes the input
 * file, runs this program and checks its output file against the oracle.
 *
 * Input (little-endian): int32 n_chunks; int32 chunk_len[n_chunks];
 * int64 n_query; int32 n_q_heads, n_kv_heads; float64 rope_theta, ratio;
 * then bf16 bits: k_src, v_cache, k_fresh, v_fresh [N, Hkv, 128] and
 * q [N, Hq, 128].
 * Output: int32 sel[n_sel]; bf16 out[n_sel, Hq, 128]; float32 lse[n_sel, Hq];
 * bf16 k_cache, v_cache [N, Hkv, 128].
 * Exit status: 0 done, 1 usage or file error, 2 a kvc_* call failed (its
 * message on stderr), 3 a HIP call failed.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "kvc.h"

#define HIP(call)                                                              \
  do {                                                                         \
    hipError_t e_ = (call);                                                    \
    if (e_ != hipSuccess) {                                                    \
      fprintf(stderr, "HIP error %d at %s\n", (int)e_, #call);                 \
      exit(3);                                                                 \
    }                                                                          \
  } while (0)

#define KVC(call)                                                              \
  do {                                                                         \
    kvc_status s_ = (call);                                                    \
    if (s_ != KVC_OK) {                                                        \
      fprintf(stderr, "kvc status %d: %s\n", (int)s_, kvc_last_error());       \
      exit(2);                                                                 \
    }                                                                          \
  } while (0)

static void read_exact(FILE* f, void* p, size_t n) {
  if (n && fread(p, 1, n, f) != n) {
    fprintf(stderr, "short input file\n");
    exit(1);
  }
}

static void* to_device(FILE* f, size_t n) {
  void* h = malloc(n ? n : 1);
  void* d = NULL;
  if (!h) exit(1);
  read_exact(f, h, n);
  HIP(hipMalloc(&d, n ? n : 16));
  HIP(hipMemcpy(d, h, n, hipMemcpyHostToDevice));
  free(h);
  return d;
}

static void to_file(FILE* f, const void* d, size_t n) {
  void* h = malloc(n ? n : 1);
  if (!h) exit(1);
  HIP(hipMemcpy(h, d, n, hipMemcpyDeviceToHost));
  if (n && fwrite(h, 1, n, f) != n) exit(1);
  free(h);
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s input output\n", argv[0]);
    return 1;
  }
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 1;
  int32_t n_chunks;
  read_exact(in, &n_chunks, sizeof n_chunks);
  if (n_chunks < 0 || n_chunks > 100000) return 1;
  int32_t* chunk_len = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n_chunks ? n_chunks : 1));
  if (!chunk_len) return 1;
  read_exact(in, chunk_len, sizeof(int32_t) * (size_t)n_chunks);
  int64_t n_query;
  int32_t hq, hkv;
  double theta, ratio;
  read_exact(in, &n_query, sizeof n_query);
  read_exact(in, &hq, sizeof hq);
  read_exact(in, &hkv, sizeof hkv);
  read_exact(in, &theta, sizeof theta);
  read_exact(in, &ratio, sizeof ratio);

  kvc_layout L = {0};
  L.n_chunks = n_chunks;
  L.chunk_len = chunk_len;
  L.n_query = n_query;
  L.n_q_heads = hq;
  L.n_kv_heads = hkv;
  L.head_dim = 128;
  L.rope_theta = theta;
  int64_t n_reused = 0;
  for (int32_t i = 0; i < n_chunks; ++i) n_reused += chunk_len[i];
  const int64_t n_rows = n_reused + n_query;
  const size_t kv_bytes = (size_t)n_rows * (size_t)hkv * 128 * 2;
  const size_t q_bytes = (size_t)n_rows * (size_t)hq * 128 * 2;

  void* k_src = to_device(in, kv_bytes);
  void* v_cache = to_device(in, kv_bytes);
  void* k_fresh = to_device(in, kv_bytes);
  void* v_fresh = to_device(in, kv_bytes);
  void* q = to_device(in, q_bytes);
  fclose(in);

  hipStream_t stream;
  HIP(hipStreamCreate(&stream));
  size_t plan_bytes = 0, ws_bytes = 0, attn_ws = 0;
  KVC(kvc_plan_bytes(&L, &plan_bytes));
  void *plan_dev = NULL, *staging = NULL, *ws = NULL, *k_cache = NULL, *out = NULL, *lse = NULL, *sel = NULL;
  HIP(hipMalloc(&plan_dev, plan_bytes));
  /* pinned staging: the upload is only enqueued; the staging memory stays
     untouched until the stream has been synchronised below */
  HIP(hipHostMalloc(&staging, plan_bytes, hipHostMallocDefault));
  kvc_plan plan;
  KVC(kvc_plan_upload(&L, plan_dev, plan_bytes, staging, &plan, stream));
  /* a ratio outside [0, 1] gives -1 here; the layer call then reports it */
  const int64_t k = kvc_recompute_count(ratio, n_reused);
  const int64_t n_sel = (k < 0 ? 0 : k) + n_query;
  KVC(kvc_blend_workspace(&L, &ws_bytes));
  KVC(kvc_attention_workspace(n_sel, hq, hkv, 128, &attn_ws));
  HIP(hipMalloc(&ws, ws_bytes + attn_ws));
  HIP(hipMalloc(&k_cache, kv_bytes));
  HIP(hipMalloc(&out, (size_t)(n_sel ? n_sel : 1) * (size_t)hq * 128 * 2));
  HIP(hipMalloc(&lse, (size_t)(n_sel ? n_sel : 1) * (size_t)hq * 4));
  HIP(hipMalloc(&sel, (size_t)(n_sel ? n_sel : 1) * 4));
  KVC(kvc_blend_prefill_layer(&L, &plan, 1, ratio, k_src, k_cache, v_cache, q, k_fresh, v_fresh,
                              (int32_t*)sel, n_sel, out, (float*)lse, ws, ws_bytes + attn_ws, stream));
  HIP(hipStreamSynchronize(stream));

  FILE* o = fopen(argv[2], "wb");
  if (!o) return 1;
  to_file(o, sel, (size_t)n_sel * 4);
  to_file(o, out, (size_t)n_sel * (size_t)hq * 128 * 2);
  to_file(o, lse, (size_t)n_sel * (size_t)hq * 4);
  to_file(o, k_cache, kv_bytes);
  to_file(o, v_cache, kv_bytes);
  fclose(o);
  HIP(hipStreamDestroy(stream));
  void* bufs[] = {k_src, v_cache, k_fresh, v_fresh, q, plan_dev, ws, k_cache, out, lse, sel};
  for (size_t i = 0; i < sizeof bufs / sizeof bufs[0]; ++i) HIP(hipFree(bufs[i]));
  HIP(hipHostFree(staging));
  free(chunk_len);
  return 0;
}
