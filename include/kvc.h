/*
 * kvc.h -- C ABI of libkvc, the MI355X (gfx950) selective-recompute prefill.
 *
 * The method (arXiv 2609.09768, "Fine-Tuning a KV Cache Concatenation-Aware
 * Model or Recomputing KV Caches? Why Not Both?"): a long prompt is built from
 * chunks whose per-layer KV caches were computed ahead of time, each on its
 * own.  Per layer, the chunk caches are concatenated and their keys moved to
 * the positions they take in the new context (Section 3.4); at a check layer
 * the keys of every token are recomputed and the tokens whose keys deviate
 * most from the cache are selected for recomputation (CacheBlend, Section 3.2,
 * 15 % of the tokens); only the selected tokens' queries are evaluated, with
 * attention that is causal by original position (Section 4 setup;
 * Limitations, item 1) against the whole blended cache.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensors are bfloat16, contiguous, token-major: K/V caches [rows, Hkv, D],
 *   queries and outputs [rows, Hq, D].  Device pointers must be 16-byte
 *   aligned.  Row r of the concatenated context sits at position r.
 * - Only head_dim D == 128 is supported (KVC_ERR_UNSUPPORTED otherwise).
 * - Row counts (n_rows, n_kv, n_sel, N, ...) are at most 2^31 - 128
 *   (KVC_ERR_INVALID_ARG above): row indices are int32.  Element and byte
 *   offsets are 64-bit, so a tensor may exceed 2^31 elements.
 * - The caller owns every buffer.  Entry points never allocate device memory;
 *   scratch comes in through a workspace argument whose size the matching
 *   *_workspace / *_bytes query returns.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Compute entry points only enqueue work on it and return without waiting.
 *   kvc_plan_upload without a staging buffer is the one exception: it waits
 *   for its own copy.
 * - Every argument is validated on the host before any HIP call; a bad one
 *   returns KVC_ERR_INVALID_ARG / _UNSUPPORTED / _WORKSPACE and enqueues
 *   nothing.  A HIP failure (including "no device") returns KVC_ERR_DEVICE.
 *   kvc_last_error() then describes the failure (thread-local).
 * - Inputs must be finite; NaN/Inf are not checked on the device.
 * - Within one call, an output or workspace buffer must share no byte with
 *   any other buffer argument (KVC_ERR_INVALID_ARG); read-only inputs may
 *   overlap each other.  The exceptions are the in-place forms an entry
 *   point names (k_dst == k_src, k_cache == k_src).
 * - Calls that share output or workspace buffers must be ordered on one
 *   stream by the caller.
 */
#ifndef KVC_H
#define KVC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVC_ABI_VERSION 4

typedef enum {
  KVC_OK = 0,
  KVC_ERR_INVALID_ARG = 1, /* null/misaligned pointer, inconsistent sizes, bad ratio */
  KVC_ERR_UNSUPPORTED = 2, /* valid but not implemented (e.g. head_dim != 128) */
  KVC_ERR_WORKSPACE = 3,   /* workspace or plan buffer too small */
  KVC_ERR_DEVICE = 4       /* HIP runtime / launch failure, or no GPU */
} kvc_status;

/*
 * Shape of one prefill request (host memory; read during the call only).
 * Rows [0, n_reused) hold the reused chunks in order, n_reused = sum of
 * chunk_len; rows [n_reused, N = n_reused + n_query) hold the final query
 * chunk (instruction + question), which is always recomputed.
 * Chunk i starts at row row0_i = sum_{j<i} chunk_len[j].  Its cached keys
 * were position-encoded starting at chunk_old_pos0[i] (NULL: all 0, i.e. each
 * chunk computed on its own from position 0, Section 1), so the adjustment
 * shifts them by delta_i = row0_i - chunk_old_pos0[i].
 * RoPE is the half-split (Llama) form with frequencies
 * f_j = rope_theta^(-2j/D), j < D/2, or the caller's table inv_freq[D/2]
 * (for models that rescale them, e.g. YaRN in Section 4.1).
 * zero_kv[i] != 0 marks a chunk whose cached K and V are all zero: the
 * special tokens between documents, whose cache entries the paper sets to
 * zero (Section 3.1, Section 4 setup).  Only kvc_stage_layer treats such
 * chunks differently (it writes their zeros instead of copying a cache);
 * every other entry point handles them like any chunk.
 */
typedef struct kvc_layout {
  int32_t n_chunks;              /* >= 0 */
  const int32_t* chunk_len;      /* [n_chunks], each >= 0; NULL only if n_chunks == 0 */
  const int64_t* chunk_old_pos0; /* [n_chunks] or NULL; each in [-2^53, 2^53] */
  int64_t n_query;               /* >= 0 */
  int32_t n_q_heads;             /* Hq >= 1, multiple of n_kv_heads */
  int32_t n_kv_heads;            /* Hkv >= 1 */
  int32_t head_dim;              /* D, must be 128 */
  double rope_theta;             /* > 0, used when inv_freq is NULL */
  const double* inv_freq;        /* [D/2] finite, or NULL */
  const uint8_t* zero_kv;        /* [n_chunks] or NULL (no zero chunks) */
} kvc_layout;

/* KVC_ABI_VERSION of the loaded library. */
int32_t kvc_abi_version(void);

/* Message for the last non-OK status returned on this thread ("" if none).
 * The pointer stays valid until the next kvc_* call on the same thread. */
const char* kvc_last_error(void);

/*
 * Number of reused tokens recomputed at ratio `ratio` (Section 3.2: a fixed
 * rate, 15 % in the paper): floor(ratio * n_reused), the product taken in
 * IEEE float64.  Returns -1 if ratio is NaN or outside [0, 1] or n_reused < 0.
 */
int64_t kvc_recompute_count(double ratio, int64_t n_reused);

/*
 * Position-adjustment plan (Section 3.4: chunk caches merged, then moved to
 * their new positions).  A plan is a device buffer holding, per chunk, the
 * rotation cos/sin of delta_i * f_j (computed in float64 on the host) and the
 * list of row tiles the adjustment kernel walks.  One plan serves every layer
 * of a request.  kvc_plan_upload describes the uploaded plan in a kvc_plan
 * (host memory, owned by the caller), which the entry points that adjust keys
 * take instead of a bare pointer: each compares the descriptor's layout_id
 * with the id of the layout it is given, before any launch, and rejects a
 * plan built for another layout with KVC_ERR_INVALID_ARG.
 */
typedef struct kvc_plan {
  const void* device;  /* the device buffer holding the plan */
  size_t bytes;        /* its size in bytes */
  uint64_t layout_id;  /* kvc_layout_id() of the layout the plan was built for */
} kvc_plan;

/*
 * kvc_layout_id: identity of everything a plan depends on (chunk lengths,
 * cached positions, kv heads, head size, frequencies, zero_kv flags, where a
 * NULL zero_kv equals an all-zero one).  Never 0.
 * kvc_plan_bytes: size of the plan for layout L.
 * kvc_plan_upload: builds the plan on the host and copies it to plan_dev
 * (device, 16-byte aligned, >= kvc_plan_bytes bytes) on `stream`, then fills
 * *plan_out (only on success).  host_staging NULL: the plan is built in the
 * library's own host memory and the call waits for the copy.  host_staging
 * non-NULL: host memory of at least kvc_plan_bytes bytes (allocated pinned,
 * e.g. with hipHostMalloc, for the copy to be asynchronous) into which the
 * plan is built; the copy is enqueued and the call returns without waiting,
 * and the caller keeps the staging memory unchanged until the copy has run
 * (e.g. until an event recorded on `stream` after the call has completed).
 */
kvc_status kvc_layout_id(const kvc_layout* L, uint64_t* id);
kvc_status kvc_plan_bytes(const kvc_layout* L, size_t* bytes);
kvc_status kvc_plan_upload(const kvc_layout* L, void* plan_dev, size_t plan_bytes, void* host_staging,
                           kvc_plan* plan_out, void* stream);

/*
 * Step a1: RoPE re-positioning of the reused chunks' cached keys
 * (Section 1; Section 2, PIE; Section 3.4; fp32-or-better adjustment,
 * Section 4 setup).
 * For every row r < n_reused of chunk i and kv head h, each pair
 * (x[j], x[j+D/2]) of k_src[r,h,:] is rotated by delta_i * f_j:
 *   y[j] = x[j] cos - x[j+D/2] sin,  y[j+D/2] = x[j+D/2] cos + x[j] sin,
 * computed in float64 and rounded once to bfloat16 (nearest, ties to even),
 * written to k_dst[r,h,:].  Rows >= n_reused are not touched.
 * k_src, k_dst: device bf16 [>= n_reused, Hkv, D]; k_dst may equal k_src
 * (in place; then chunks with delta 0 are skipped, they would not change).
 * Partial overlap of k_src and k_dst is not allowed.
 * plan: the descriptor kvc_plan_upload filled for this layout
 * (KVC_ERR_INVALID_ARG for a plan of another layout, KVC_ERR_WORKSPACE if
 * its buffer is smaller than kvc_plan_bytes).  k_dst must not overlap the
 * plan buffer.
 */
kvc_status kvc_rope_shift(const kvc_layout* L, const kvc_plan* plan, const void* k_src,
                          void* k_dst, void* stream);

/*
 * Step a2: per-token key deviation at the check layer (Section 2, CacheBlend;
 * Section 3.2, squared differences of the key entries as in LMCache):
 *   dev_out[r] = sum_{h < Hkv, e < D} (k_fresh[r,h,e] - k_cached[r,h,e])^2,
 * the exact real sum rounded once to float64 (nearest, ties to even) for
 * every finite input, so rows whose exact sums are equal get equal values.
 * Rows are summed in float64 double-double arithmetic, whose result is
 * returned when a per-row check proves it correctly rounded (always, for
 * inputs within 2^44 of each other and not far below the deviation); any
 * other row is summed again exactly in integer arithmetic.
 * k_cached (the adjusted cache), k_fresh: device bf16 [n_rows, Hkv, D].
 * dev_out: device float64 [n_rows].  n_rows == 0 is a no-op.
 */
kvc_status kvc_kv_deviation(int64_t n_rows, int32_t n_kv_heads, int32_t head_dim,
                            const void* k_cached, const void* k_fresh, double* dev_out,
                            void* stream);

/*
 * Step a3: top-k selection (Section 3.2: the tokens with the largest key
 * deviation, a fixed fraction of them).
 * idx_out[0..k) = the rows of the k largest dev values, ties broken by the
 * lower row, in ascending row order (int32).  -0.0 equals +0.0; NaN is not
 * allowed.  0 <= k <= n <= 2^31 - 128.  ws: device scratch of at least
 * kvc_select_topk_workspace(n) bytes, 16-byte aligned; it needs no
 * initialisation and holds nothing useful afterwards.
 */
kvc_status kvc_select_topk_workspace(int64_t n, size_t* bytes);
kvc_status kvc_select_topk(const double* dev, int64_t n, int64_t k, int32_t* idx_out,
                           void* ws, size_t ws_bytes, void* stream);

/*
 * Step a4 (scatter half): blend the recomputed K/V of the selected tokens
 * into the cache (Section 3.2 / Section 4 setup: selected tokens' K/V are
 * recomputed; everything else is reused).
 * For i < n_sel: k_cache[sel[i]] = k_fresh[s], v_cache[sel[i]] = v_fresh[s],
 * with s = i if fresh_is_compact, else s = sel[i].
 * sel: device int32 [n_sel]; entries outside [0, n_rows), or whose source row
 * is outside [0, n_fresh_rows), are skipped.  k_fresh/v_fresh: device bf16
 * [n_fresh_rows, Hkv, D]; k_cache/v_cache: device bf16 [n_rows, Hkv, D].
 * Duplicate sel entries race (undefined which source wins).
 */
kvc_status kvc_scatter_rows(const int32_t* sel, int64_t n_sel, int32_t fresh_is_compact,
                            const void* k_fresh, const void* v_fresh, int64_t n_fresh_rows,
                            void* k_cache, void* v_cache, int64_t n_rows,
                            int32_t n_kv_heads, int32_t head_dim, void* stream);

/*
 * Steps a4 (gather half) + a5: causal GQA attention of sparse queries
 * (Section 4 setup: selected queries against the full cache with a custom
 * mask; Limitations, item 1: the mask is causal by original position).
 * For i < n_sel, query head h, kv head g = h / (Hq / Hkv), p_i = q_pos[i]:
 *   s_j = scale * <Q[i,h], K[j,g]> for j = 0..p_i,
 *   out[i,h] = sum_j softmax(s)_j V[j,g],  lse[i,h] = ln sum_j exp(s_j).
 * Q[i] is row q_rows[i] of q (gather) or row i if q_rows is NULL.
 * q: device bf16 [n_q_rows, Hq, D]; q_rows: device int32 [n_sel] or NULL;
 * q_pos: device int32 [n_sel]; k, v: device bf16 [n_kv, Hkv, D];
 * out: device bf16 [n_sel, Hq, D]; lse: device float32 [n_sel, Hq] or NULL.
 * One launch holds about 2 n_sel Hq work-items, and HIP allows fewer than
 * 2^32: a larger n_sel x Hq (above about 2^31) is KVC_ERR_INVALID_ARG.
 * softmax_scale 0 means 1/sqrt(D).  Positions are clamped to n_kv - 1; a
 * query with q_pos < 0 or an out-of-range q_rows entry gets out = 0 and
 * lse = -inf.  Any order of positions is correct; ascending positions (what
 * the selection produces) run fastest.  QK^T and PV run on bf16 MFMA with
 * float32 accumulation and softmax.
 * ws is optional: with ws = NULL (or ws_bytes below the query's size) every
 * query block's keys are handled by one workgroup.  A selection too small
 * to keep the GPU evenly busy (fewer than two workgroups per CU) gets a
 * nonzero size from kvc_attention_workspace; given at least that much
 * (16-byte aligned), each block's key tiles are split over up to 8
 * workgroups (one per CU below one workgroup per CU, two splits between
 * one and two per CU; each split keeping at least 4 tiles of the longest
 * block), which write float32 partial outputs
 * and LSEs into ws, and a second launch merges them in a fixed order.  The
 * result is deterministic for a given shape and ws choice and differs from
 * the unsplit one by rounding only.
 */
kvc_status kvc_attention_workspace(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads,
                                   int32_t head_dim, size_t* bytes);
kvc_status kvc_sparse_query_attention(const void* q, int64_t n_q_rows, const int32_t* q_rows,
                                      const int32_t* q_pos, int64_t n_sel, const void* k,
                                      const void* v, int64_t n_kv, int32_t n_q_heads,
                                      int32_t n_kv_heads, int32_t head_dim, float softmax_scale,
                                      void* out, float* lse, void* ws, size_t ws_bytes,
                                      void* stream);

/*
 * Step a6: one layer of the selective-recompute prefill (Section 3.4 layer
 * pipeline, Section 4 setup), entirely on `stream`:
 *   1. a1: k_cache[0, n_reused) = adjusted k_src (kvc_rope_shift);
 *   2. check layer only: a2 deviation of the adjusted keys against
 *      k_fresh[0, n_reused), a3 top-k with k = kvc_recompute_count(ratio,
 *      n_reused), sel = top-k rows followed by the query rows
 *      n_reused .. N-1 (if k == n_reused every row is selected and the
 *      deviation is skipped: full recomputation = causal attention);
 *   3. a4: the selected rows of k_cache/v_cache take the recomputed K/V;
 *   4. a5: out = attention of the selected queries at positions sel.
 * Check layer (is_check_layer != 0): q_fresh/k_fresh/v_fresh hold all N rows
 * ([N, H, D]) and sel is written.  Reuse layer: they hold the n_sel selected
 * rows in the order of sel, which is read (from an earlier check layer).
 * n_sel must equal kvc_recompute_count(ratio, n_reused) + n_query.
 * k_src: device bf16 [>= n_reused, Hkv, D], cached keys at their old
 * positions, or NULL when rows [0, n_reused) of k_cache already hold the
 * adjusted keys (after kvc_stage_layer): step 1 is then skipped and plan
 * may be NULL (a non-NULL plan is still checked against L); k_cache: device
 * bf16 [N, Hkv, D] (may equal k_src);
 * v_cache: device bf16 [N, Hkv, D], updated in place; out: [n_sel, Hq, D];
 * lse: [n_sel, Hq] float32 or NULL; ws: >= kvc_blend_workspace(L) bytes,
 * and kvc_attention_workspace(n_sel, Hq, Hkv, D) bytes more to let the
 * attention split its key ranges (see kvc_sparse_query_attention).
 */
kvc_status kvc_blend_workspace(const kvc_layout* L, size_t* bytes);
kvc_status kvc_blend_prefill_layer(const kvc_layout* L, const kvc_plan* plan, int32_t is_check_layer,
                                   double ratio, const void* k_src, void* k_cache, void* v_cache,
                                   const void* q_fresh, const void* k_fresh, const void* v_fresh,
                                   int32_t* sel, int64_t n_sel, void* out, float* lse, void* ws,
                                   size_t ws_bytes, void* stream);

/*
 * kvc_blend_prefill_layer for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same arguments and results without the workspace.  The
 * layer's scratch (the check layer's deviations and selection state, and
 * the attention's key-range split partials when they fit beside them) is a
 * static device array of KVC_STATIC_SCRATCH_BYTES in the library, one per
 * GPU, held until the process ends; no call allocates or frees memory.  A
 * check layer needing more than that (kvc_blend_workspace(L) above it: more
 * than about 2 million reused rows) returns KVC_ERR_WORKSPACE; the split is
 * used only when its partials fit, so the results equal those of
 * kvc_blend_prefill_layer given kvc_blend_workspace(L) bytes, plus
 * kvc_attention_workspace bytes when the sum fits.  Nothing in the array
 * needs to start at zero.  Every call on one GPU uses that GPU's array:
 * calls that overlap on one GPU race, so order them on one stream.  The first
 * call on a device looks up the array's address there.
 */
#define KVC_STATIC_SCRATCH_BYTES (16u << 20)
kvc_status kvc_blend_prefill_layer_noalloc(const kvc_layout* L, const kvc_plan* plan, int32_t is_check_layer,
                                           double ratio, const void* k_src, void* k_cache, void* v_cache,
                                           const void* q_fresh, const void* k_fresh, const void* v_fresh,
                                           int32_t* sel, int64_t n_sel, void* out, float* lse, void* stream);

/*
 * The check layer's selection on its own (steps 1-2 of
 * kvc_blend_prefill_layer with is_check_layer = 1): a1 adjusts k_src into
 * k_cache (skipped if k_src is NULL), a2 takes the deviation of the adjusted
 * keys against k_fresh[0, n_reused), a3 writes to sel the top-k rows followed
 * by the query rows n_reused .. N-1.  Nothing else is touched.  This lets a
 * caller project keys for every token but queries and values for the
 * selected tokens only (Section 3.2 compares keys alone), and then finish
 * the layer with kvc_blend_prefill_layer(is_check_layer = 0, k_src = NULL)
 * on those compact rows.  Arguments as for kvc_blend_prefill_layer; k_fresh
 * is device bf16 [>= n_reused, Hkv, D] and ws needs kvc_blend_workspace(L)
 * bytes.
 */
kvc_status kvc_select_tokens(const kvc_layout* L, const kvc_plan* plan, double ratio, const void* k_src,
                             void* k_cache, const void* k_fresh, int32_t* sel, int64_t n_sel,
                             void* ws, size_t ws_bytes, void* stream);

/*
 * Decoder-layer steps around the attention of the selected tokens.  The
 * paper's models (Section 4.1, Llama-3.1-8B-Instruct and Qwen2.5-7B-Instruct)
 * are pre-norm decoder layers; with selective recompute only the selected
 * tokens pass through a layer (Section 3.4, Section 4 setup).  The
 * projections between these steps are kvc_projection below.
 *
 * kvc_rms_norm: RMS normalisation of rows (the norms before the attention
 * and before the feed-forward block):
 *   out[i,:] = x[r,:] / sqrt(mean_c x[r,c]^2 + eps) * gamma,
 * r = rows[i] (gather) or i if rows is NULL, in float32 and rounded once to
 * bfloat16 (nearest even).  With res_out non-NULL, res_out[i,:] = x[r,:]
 * (the gathered residual rows, for the residual additions that follow).
 * x: device bf16 [n_x_rows, hidden]; rows: device int32 [n] or NULL (then
 * n <= n_x_rows); gamma: device bf16 [hidden]; out, res_out: device bf16
 * [n, hidden].  hidden: a multiple of 8 in [8, 16384]; eps >= 0 (an
 * all-zero row with eps = 0 gives NaN, as the formula does).  A rows entry
 * outside [0, n_x_rows) gives zero rows in out and res_out.  out and res_out
 * must not overlap x, gamma or each other (rejected when they do).
 */
kvc_status kvc_rms_norm(const void* x, int64_t n_x_rows, const int32_t* rows, int64_t n,
                        int32_t hidden, const void* gamma, float eps, void* out, void* res_out,
                        void* stream);

/*
 * kvc_qkv_rope: splits the fused Q/K/V projection output and applies RoPE
 * to the queries and keys at each token's position.  Row i of y holds
 * n_q_heads query heads, then n_k_heads key heads, then n_v_heads value
 * heads, each D wide.  Query and key head pairs (x[j], x[j+D/2]) are rotated
 * by p_i * f_j (half-split RoPE, as for the cached keys) in float64 and
 * rounded once to bfloat16; value heads are copied.  p_i = pos[i], or i if
 * pos is NULL.  f_j = rope_theta^(-2j/D), or inv_freq[j] (host [D/2]) if
 * given.  y: device bf16 [n, (n_q+n_k+n_v) * D]; q: [n, n_q_heads, D],
 * k: [n, n_k_heads, D], v: [n, n_v_heads, D], device bf16 (a part with no
 * heads may be NULL).  Head counts >= 0 with a total in [1, 1024].  q, k, v
 * must not overlap y or each other (rejected when they do).
 * Projecting keys alone for every row (n_q = n_v = 0) gives the check
 * layer's k_fresh; queries and values for the selected rows
 * (n_k = 0, pos = sel) give the rest.
 */
kvc_status kvc_qkv_rope(const void* y, int64_t n, int32_t n_q_heads, int32_t n_k_heads,
                        int32_t n_v_heads, int32_t head_dim, const int32_t* pos, double rope_theta,
                        const double* inv_freq, void* q, void* k, void* v, void* stream);

/*
 * kvc_swiglu: gated SiLU of the feed-forward block.
 *   out[i,c] = silu(gu[i,c]) * gu[i, inter + c],  silu(g) = g / (1 + e^-g),
 * in float32 (hardware exponential and reciprocal, a few float32 ulps) and
 * rounded once to bfloat16.  gate_up: device bf16 [n, 2 * inter] (gate
 * first); out: device bf16 [n, inter], not overlapping gate_up; inter a
 * multiple of 8 in [8, 2^24].
 */
kvc_status kvc_swiglu(const void* gate_up, int64_t n, int64_t inter, void* out, void* stream);

/*
 * kvc_projection: the projections of the layer (fused Q/K/V, O, gate/up,
 * down) on the selected rows (Section 3.4, Section 4 setup: only the
 * selected tokens pass through a layer):
 *   c[i, j] = sum_e a[r_i, e] * w[j, e]  (+ residual[i, j]),
 * r_i = a_rows[i] (a gather) or i, with exact bf16 products summed in
 * float32 on the matrix cores, the residual added in float32, rounded once
 * to bfloat16 (nearest even).  a: device bf16 [n_a_rows, k] row-major;
 * a_rows: device int32 [m] or NULL (then m <= n_a_rows); an entry outside
 * [0, n_a_rows) gives a zero product row (c = residual there).  w: device
 * bf16 [n, k], the weight in the [out, in] layout of a linear layer;
 * residual: device bf16 [m, n] or NULL; c: device bf16 [m, n], which may be
 * the residual buffer itself (added in place) but must not overlap a, w or
 * a_rows.  k: a multiple of 64 in [64, 2^24] (KVC_ERR_UNSUPPORTED
 * otherwise); n: a multiple of 8 in [0, 2^24]; m <= 2^31 - 128 and about
 * m n <= 2^39 (one launch).  The O and down projections add the residual
 * stream here.
 */
kvc_status kvc_projection(int64_t m, int64_t n, int64_t k, const void* a, int64_t n_a_rows, const int32_t* a_rows,
                          const void* w, const void* residual, void* c, void* stream);

/*
 * Layer-wise pipeline, transfer stage (Section 3.4: per layer, the chunk
 * caches are transferred to the GPU, merged into one cache and moved to
 * their new positions on a stream of their own, so that the next layer's
 * transfer overlaps this layer's computation).  Enqueues on `stream`:
 *   1. for each chunk i with zero_kv[i] == 0, a copy of its cached K and V,
 *      k_chunks[i] and v_chunks[i] ([chunk_len[i], Hkv, D] bf16, host memory
 *      -- pinned for the copy to be asynchronous -- or device memory), into
 *      rows [row0_i, row0_i + chunk_len[i]) of k_cache and v_cache; a chunk
 *      whose source directly follows the previous chunk's in memory is
 *      copied with it, so a caller holding the chunks back to back pays one
 *      copy per tensor;
 *   2. one kernel that writes zeros (+0.0) into the K and V rows of the
 *      zero_kv chunks and adjusts the keys of every other chunk in place,
 *      exactly as kvc_rope_shift(L, plan, k_cache, k_cache).  (Adjusting a
 *      zero key instead, as the plain entry points do, may give -0.0.)
 * Rows [n_reused, N) are not touched.  A zero_kv chunk may have NULL chunk
 * pointers; if it has sources, they are copied like any chunk's (and its
 * rows then zero-filled), which lets a caller that holds a layer's chunks
 * in one buffer laid out like the rows pay one copy per tensor even across
 * separators.  The other chunks' pointers must not be NULL.  k_chunks / v_chunks
 * are host arrays [n_chunks] (NULL only if n_chunks == 0); k_cache, v_cache:
 * device bf16 [>= n_reused, Hkv, D], 16-byte aligned; plan as for
 * kvc_rope_shift.  The sources must stay valid until the copies run.
 */
kvc_status kvc_stage_layer(const kvc_layout* L, const kvc_plan* plan, const void* const* k_chunks,
                           const void* const* v_chunks, void* k_cache, void* v_cache, void* stream);

/*
 * Layer-wise pipeline (Section 3.4): stages n_layers layers of one request
 * on `stream`, in layer order (kvc_stage_layer for each), and records
 * events[l] right after layer l, so that the computation of layer l on
 * another stream can wait for exactly its own caches (hipStreamWaitEvent)
 * while later layers are still being transferred.  The events are the
 * caller's (hipEvent_t passed as void*, created beforehand, e.g. with
 * hipEventDisableTiming); events or any entry may be NULL (no record).
 * k_chunks / v_chunks: host arrays [n_layers * n_chunks] (layer l's chunk i
 * at l * n_chunks + i); k_cache / v_cache: host arrays [n_layers] of device
 * pointers.  Everything else as kvc_stage_layer.  Returns after enqueuing;
 * on an error the layers before the failing one are already enqueued.
 */
kvc_status kvc_stage_layers(const kvc_layout* L, const kvc_plan* plan, int32_t n_layers,
                            const void* const* k_chunks, const void* const* v_chunks,
                            void* const* k_cache, void* const* v_cache, void* const* events,
                            void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVC_H */
