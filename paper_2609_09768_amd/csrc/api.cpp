// C ABI of libkvc: host-side validation, plan building and kernel launches.
// Every argument is checked before the first HIP call; nothing here waits
// on the device except kvc_plan_upload's own copy when it has no staging
// buffer.
#include "../../include/kvc.h"
#include "kvc_internal.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <initializer_list>
#include <string>
#include <vector>

namespace {

thread_local std::string g_err;

kvc_status fail(kvc_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

kvc_status ok() {
  g_err.clear();
  return KVC_OK;
}

kvc_status hip_fail(const char* where, hipError_t e) {
  return fail(KVC_ERR_DEVICE, "%s: HIP error %d (%s)", where, (int)e, hipGetErrorString(e));
}

// A usable device must exist before anything is enqueued.
kvc_status need_device(const char* where) {
  int n = 0;
  const hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess) return hip_fail(where, e);
  if (n <= 0) return fail(KVC_ERR_DEVICE, "%s: no HIP device", where);
  return KVC_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// [a, a + na) and [b, b + nb) share a byte (either may be NULL: no overlap).
bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const char* x = static_cast<const char*>(a);
  const char* y = static_cast<const char*>(b);
  return x < y + nb && y < x + na;
}

// A buffer argument of a call: its first byte, its length, its name.
struct Span {
  const void* p;
  size_t n;
  const char* name;
};

// Every output (or workspace) must share no byte with another output or
// with any input; inputs may overlap each other (they are only read).
kvc_status check_disjoint(const char* where, std::initializer_list<Span> outs, std::initializer_list<Span> ins) {
  for (auto o = outs.begin(); o != outs.end(); ++o) {
    for (auto o2 = o + 1; o2 != outs.end(); ++o2)
      if (overlap(o->p, o->n, o2->p, o2->n)) return fail(KVC_ERR_INVALID_ARG, "%s: %s overlaps %s", where, o->name, o2->name);
    for (const Span& i : ins)
      if (overlap(o->p, o->n, i.p, i.n)) return fail(KVC_ERR_INVALID_ARG, "%s: %s overlaps %s", where, o->name, i.name);
  }
  return KVC_OK;
}

// The same rule for many buffers at once (sorted sweep, O(m log m)): no
// output span may share a byte with any other span.
struct TaggedSpan {
  uintptr_t begin, end;  // [begin, end)
  bool output;
  int layer;
  const char* name;
};
kvc_status check_disjoint_many(const char* where, std::vector<TaggedSpan>& v) {
  std::sort(v.begin(), v.end(), [](const TaggedSpan& a, const TaggedSpan& b) { return a.begin < b.begin; });
  const TaggedSpan* last_out = nullptr;  // the output, and any span, reaching furthest so far
  const TaggedSpan* last_any = nullptr;
  for (const TaggedSpan& x : v) {
    const TaggedSpan* hit = nullptr;
    if (x.output && last_any && x.begin < last_any->end) hit = last_any;
    else if (!x.output && last_out && x.begin < last_out->end) hit = last_out;
    if (hit)
      return fail(KVC_ERR_INVALID_ARG, "%s: layer %d %s overlaps layer %d %s", where, x.layer, x.name, hit->layer,
                  hit->name);
    if (!last_any || x.end > last_any->end) last_any = &x;
    if (x.output && (!last_out || x.end > last_out->end)) last_out = &x;
  }
  return KVC_OK;
}

// Row indices are int32, and the attention rounds a key count up to whole
// 64-row tiles in int32, so row counts stop 128 short of 2^31.
constexpr int64_t kMaxRows = (int64_t(1) << 31) - 128;
// Cached positions stay within the integers float64 holds exactly, so each
// chunk's shift row0 - old_pos0 neither overflows nor rounds.
constexpr int64_t kMaxPos = int64_t(1) << 53;

struct LayoutInfo {
  int64_t n_reused = 0;
  int64_t n_rows = 0;
  int n_tiles = 0;
};

kvc_status check_heads(const char* where, int32_t hq, int32_t hkv, int32_t d) {
  if (hkv < 1 || hkv > 64) return fail(KVC_ERR_INVALID_ARG, "%s: n_kv_heads=%d must be in [1, 64]", where, hkv);
  if (hq < 1 || hq % hkv != 0)
    return fail(KVC_ERR_INVALID_ARG, "%s: n_q_heads=%d must be a positive multiple of n_kv_heads=%d", where, hq, hkv);
  if (hq > 1024) return fail(KVC_ERR_INVALID_ARG, "%s: n_q_heads=%d too large", where, hq);
  if (d != kvc::kHeadDim) return fail(KVC_ERR_UNSUPPORTED, "%s: head_dim=%d (only 128 is supported)", where, d);
  return KVC_OK;
}

kvc_status check_layout(const char* where, const kvc_layout* L, LayoutInfo* info) {
  if (!L) return fail(KVC_ERR_INVALID_ARG, "%s: layout is NULL", where);
  if (L->n_chunks < 0) return fail(KVC_ERR_INVALID_ARG, "%s: n_chunks=%d < 0", where, L->n_chunks);
  if (L->n_chunks > 0 && !L->chunk_len) return fail(KVC_ERR_INVALID_ARG, "%s: chunk_len is NULL", where);
  if (L->n_query < 0) return fail(KVC_ERR_INVALID_ARG, "%s: n_query=%lld < 0", where, (long long)L->n_query);
  kvc_status st = check_heads(where, L->n_q_heads, L->n_kv_heads, L->head_dim);
  if (st != KVC_OK) return st;
  if (L->inv_freq) {
    for (int j = 0; j < L->head_dim / 2; ++j)
      if (!std::isfinite(L->inv_freq[j])) return fail(KVC_ERR_INVALID_ARG, "%s: inv_freq[%d] not finite", where, j);
  } else if (!(L->rope_theta > 0.0) || !std::isfinite(L->rope_theta)) {
    return fail(KVC_ERR_INVALID_ARG, "%s: rope_theta must be finite and > 0", where);
  }
  int64_t n_r = 0;
  for (int32_t i = 0; i < L->n_chunks; ++i) {
    if (L->chunk_len[i] < 0) return fail(KVC_ERR_INVALID_ARG, "%s: chunk_len[%d]=%d < 0", where, i, L->chunk_len[i]);
    if (L->chunk_old_pos0 && (L->chunk_old_pos0[i] > kMaxPos || L->chunk_old_pos0[i] < -kMaxPos))
      return fail(KVC_ERR_INVALID_ARG, "%s: chunk_old_pos0[%d] outside [-2^53, 2^53]", where, i);
    n_r += L->chunk_len[i];
    if (n_r > kMaxRows) return fail(KVC_ERR_INVALID_ARG, "%s: too many rows", where);
  }
  const int tile_rows = kvc::shift_tile_rows(n_r, L->n_kv_heads);
  int64_t tiles = 0;
  for (int32_t i = 0; i < L->n_chunks; ++i) tiles += (L->chunk_len[i] + tile_rows - 1) / tile_rows;
  if (n_r + L->n_query > kMaxRows) return fail(KVC_ERR_INVALID_ARG, "%s: too many rows", where);
  if (tiles > (int64_t(1) << 30)) return fail(KVC_ERR_INVALID_ARG, "%s: too many tiles", where);
  if (info) {
    info->n_reused = n_r;
    info->n_rows = n_r + L->n_query;
    info->n_tiles = (int)tiles;
  }
  return KVC_OK;
}

uint64_t fnv(uint64_t h, const void* p, size_t n) {
  const unsigned char* c = static_cast<const unsigned char*>(p);
  for (size_t i = 0; i < n; ++i) h = (h ^ c[i]) * 1099511628211ull;
  return h;
}

// Identity of everything the plan depends on.
uint64_t layout_hash(const kvc_layout* L) {
  uint64_t h = 1469598103934665603ull;
  h = fnv(h, &L->n_chunks, sizeof(L->n_chunks));
  h = fnv(h, &L->n_kv_heads, sizeof(L->n_kv_heads));
  h = fnv(h, &L->head_dim, sizeof(L->head_dim));
  if (L->n_chunks > 0) h = fnv(h, L->chunk_len, sizeof(int32_t) * (size_t)L->n_chunks);
  // values, not representations: a NULL chunk_old_pos0 equals all zeros, a
  // NULL zero_kv equals all-zero flags, and the frequencies are the table
  // in effect (theta's or the caller's)
  for (int32_t i = 0; i < L->n_chunks; ++i) {
    const int64_t old = L->chunk_old_pos0 ? L->chunk_old_pos0[i] : 0;
    const unsigned char z = L->zero_kv && L->zero_kv[i] != 0;
    h = fnv(h, &old, sizeof(old));
    h = fnv(h, &z, 1);
  }
  for (int j = 0; j < L->head_dim / 2; ++j) {
    const double f = L->inv_freq ? L->inv_freq[j] : std::pow(L->rope_theta, -(2.0 * j) / L->head_dim);
    h = fnv(h, &f, sizeof(f));
  }
  return h | 1ull;  // never 0, so a zeroed buffer never matches
}

size_t plan_bytes(const kvc_layout* L, const LayoutInfo& li) {
  return kvc::plan_tile_offset(L->n_chunks) + kvc::align256(sizeof(kvc::ShiftTile) * (size_t)(li.n_tiles > 0 ? li.n_tiles : 1));
}

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// A plan descriptor fit for layout L: built for it, buffer large enough.
kvc_status check_plan(const char* W, const kvc_layout* L, const LayoutInfo& li, const kvc_plan* plan) {
  if (!plan) return fail(KVC_ERR_INVALID_ARG, "%s: plan is NULL", W);
  if (!plan->device || !aligned16(plan->device))
    return fail(KVC_ERR_INVALID_ARG, "%s: plan->device is NULL or not 16-byte aligned", W);
  const uint64_t id = layout_hash(L);
  if (plan->layout_id != id)
    return fail(KVC_ERR_INVALID_ARG, "%s: the plan was built for another layout (id %016llx, this layout %016llx)", W,
                (unsigned long long)plan->layout_id, (unsigned long long)id);
  const size_t need = plan_bytes(L, li);
  if (plan->bytes < need) return fail(KVC_ERR_WORKSPACE, "%s: plan buffer %zu bytes, need %zu", W, plan->bytes, need);
  return KVC_OK;
}

// The plan buffer as an input span of a call (empty when absent).
Span plan_span(const kvc_plan* plan) {
  return {plan ? plan->device : nullptr, plan ? plan->bytes : 0, "plan"};
}

// Checks shared by kvc_blend_prefill_layer and kvc_select_tokens: layout,
// ratio against n_sel, and the buffers of the adjustment (a1) and, on the
// check layer, of the deviation and selection (a2, a3).  *k_out = k.
// static_ws: the layer's scratch is the library's static array (checked
// for size only; its address is taken after validation).
kvc_status check_select(const char* W, const kvc_layout* L, LayoutInfo* li, const kvc_plan* plan, bool check,
                        double ratio, const void* k_src, const void* k_cache, const void* k_fresh,
                        const int32_t* sel, int64_t n_sel, const void* ws, size_t ws_bytes, bool static_ws,
                        int64_t* k_out) {
  kvc_status st = check_layout(W, L, li);
  if (st != KVC_OK) return st;
  const int64_t k = kvc_recompute_count(ratio, li->n_reused);
  if (k < 0) return fail(KVC_ERR_INVALID_ARG, "%s: ratio=%g not in [0, 1]", W, ratio);
  if (n_sel != k + L->n_query)
    return fail(KVC_ERR_INVALID_ARG, "%s: n_sel=%lld, expected floor(ratio*n_reused)+n_query=%lld", W,
                (long long)n_sel, (long long)(k + L->n_query));
  if (kvc::attention_work_items(n_sel, L->n_q_heads, L->n_kv_heads) > (int64_t)UINT32_MAX)
    return fail(KVC_ERR_INVALID_ARG, "%s: n_sel x n_q_heads too large for one launch", W);
  // k_src NULL: the reused keys in k_cache are already adjusted (staged)
  const bool shift = li->n_reused > 0 && k_src;
  if ((shift || n_sel > 0) && (!k_cache || !aligned16(k_cache)))
    return fail(KVC_ERR_INVALID_ARG, "%s: k_cache NULL or misaligned", W);
  if (shift && !aligned16(k_src)) return fail(KVC_ERR_INVALID_ARG, "%s: k_src misaligned", W);
  if (shift || plan) {
    st = check_plan(W, L, *li, plan);
    if (st != KVC_OK) return st;
  }
  if (shift && k_src != k_cache) {
    const size_t bytes = (size_t)li->n_reused * L->n_kv_heads * L->head_dim * 2;
    const char* a = static_cast<const char*>(k_src);
    const char* b = static_cast<const char*>(k_cache);
    if (a < b + bytes && b < a + bytes)
      return fail(KVC_ERR_INVALID_ARG, "%s: k_src and k_cache partially overlap", W);
  }
  if (n_sel > 0 && (!sel || (reinterpret_cast<uintptr_t>(sel) & 3u)))
    return fail(KVC_ERR_INVALID_ARG, "%s: sel NULL or misaligned", W);
  if (check && k > 0 && k < li->n_reused) {
    size_t need_ws = 0;
    kvc_blend_workspace(L, &need_ws);
    if (!k_fresh || !aligned16(k_fresh)) return fail(KVC_ERR_INVALID_ARG, "%s: k_fresh NULL or misaligned", W);
    if (static_ws) {
      if (need_ws > kvc::kStaticScratchBytes)
        return fail(KVC_ERR_WORKSPACE, "%s: this check layer needs %zu bytes of scratch (%lld reused rows); "
                    "the static scratch holds %zu", W, need_ws, (long long)li->n_reused, kvc::kStaticScratchBytes);
    } else {
      if (!ws || !aligned16(ws)) return fail(KVC_ERR_INVALID_ARG, "%s: ws NULL or not 16-byte aligned", W);
      if (ws_bytes < need_ws) return fail(KVC_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", W, ws_bytes, need_ws);
    }
  }
  *k_out = k;
  return KVC_OK;
}

// a1 (k_src non-NULL), then on the check layer a2 + a3: the launches shared
// by kvc_blend_prefill_layer and kvc_select_tokens (arguments already checked).
hipError_t shift_and_select(const kvc_layout* L, const LayoutInfo& li, const kvc_plan* plan, bool check,
                            int64_t k, const void* k_src, void* k_cache, const void* k_fresh,
                            int32_t* sel, void* ws, hipStream_t s) {
  const int hkv = L->n_kv_heads;
  hipError_t e;
  if (li.n_reused > 0 && k_src) {
    e = kvc::launch_rope_shift(plan->device, plan->layout_id, L->n_chunks, li.n_tiles, hkv, static_cast<const uint16_t*>(k_src),
                               static_cast<uint16_t*>(k_cache), nullptr, s);
    if (e != hipSuccess) return e;
  }
  if (!check || k + L->n_query == 0) return hipSuccess;
  if (k > 0 && k < li.n_reused) {
    double* dev = static_cast<double*>(ws);
    void* tws = static_cast<char*>(ws) + kvc::align256(sizeof(double) * (size_t)li.n_reused);
    e = kvc::launch_kv_deviation(li.n_reused, hkv, static_cast<const uint16_t*>(k_cache),
                                 static_cast<const uint16_t*>(k_fresh), dev, s);
    if (e != hipSuccess) return e;
    return kvc::launch_select_topk(dev, li.n_reused, k, L->n_query, sel, tws, s);
  }
  // k == 0: only the query rows; k == n_reused: every row (causal attention)
  return kvc::launch_select_topk(nullptr, li.n_reused, k, L->n_query, sel, nullptr, s);
}

}  // namespace

extern "C" {

int32_t kvc_abi_version(void) { return KVC_ABI_VERSION; }

const char* kvc_last_error(void) { return g_err.c_str(); }

int64_t kvc_recompute_count(double ratio, int64_t n_reused) {
  if (!(ratio >= 0.0 && ratio <= 1.0) || n_reused < 0) return -1;
  return (int64_t)std::floor(ratio * (double)n_reused);
}

kvc_status kvc_plan_bytes(const kvc_layout* L, size_t* bytes) {
  LayoutInfo li;
  kvc_status st = check_layout("kvc_plan_bytes", L, &li);
  if (st != KVC_OK) return st;
  if (!bytes) return fail(KVC_ERR_INVALID_ARG, "kvc_plan_bytes: bytes is NULL");
  *bytes = plan_bytes(L, li);
  return ok();
}

kvc_status kvc_layout_id(const kvc_layout* L, uint64_t* id) {
  kvc_status st = check_layout("kvc_layout_id", L, nullptr);
  if (st != KVC_OK) return st;
  if (!id) return fail(KVC_ERR_INVALID_ARG, "kvc_layout_id: id is NULL");
  *id = layout_hash(L);
  return ok();
}

kvc_status kvc_plan_upload(const kvc_layout* L, void* plan, size_t plan_bytes_in, void* host_staging,
                           kvc_plan* plan_out, void* stream) {
  const char* W = "kvc_plan_upload";
  LayoutInfo li;
  kvc_status st = check_layout(W, L, &li);
  if (st != KVC_OK) return st;
  if (!plan || !aligned16(plan)) return fail(KVC_ERR_INVALID_ARG, "%s: plan is NULL or not 16-byte aligned", W);
  if (!plan_out) return fail(KVC_ERR_INVALID_ARG, "%s: plan_out is NULL", W);
  const size_t need = plan_bytes(L, li);
  if (plan_bytes_in < need)
    return fail(KVC_ERR_WORKSPACE, "%s: plan buffer %zu bytes, need %zu", W, plan_bytes_in, need);

  // host image of the plan (built before the device check, so host-only
  // tests exercise it too)
  const int tile_rows = kvc::shift_tile_rows(li.n_reused, L->n_kv_heads);
  std::vector<unsigned char> own;
  unsigned char* img = static_cast<unsigned char*>(host_staging);
  if (!img) {
    own.assign(need, 0);
    img = own.data();
  } else {
    std::memset(img, 0, need);
  }
  kvc::PlanHeader hdr;
  std::memset(&hdr, 0, sizeof(hdr));
  hdr.layout_hash = layout_hash(L);
  hdr.n_chunks = L->n_chunks;
  hdr.n_tiles = li.n_tiles;
  hdr.n_reused = li.n_reused;
  hdr.rot_offset = (int64_t)kvc::plan_rot_offset();
  hdr.tile_offset = (int64_t)kvc::plan_tile_offset(L->n_chunks);
  std::memcpy(img, &hdr, sizeof(hdr));

  const int D = L->head_dim;
  std::vector<double> f(D / 2);
  for (int j = 0; j < D / 2; ++j)
    f[j] = L->inv_freq ? L->inv_freq[j] : std::pow(L->rope_theta, -(2.0 * j) / D);
  double* rot = reinterpret_cast<double*>(img + hdr.rot_offset);
  kvc::ShiftTile* tiles = reinterpret_cast<kvc::ShiftTile*>(img + hdr.tile_offset);
  int64_t row0 = 0;
  int nt = 0;
  for (int32_t i = 0; i < L->n_chunks; ++i) {
    const int64_t delta = row0 - (L->chunk_old_pos0 ? L->chunk_old_pos0[i] : 0);
    for (int j = 0; j < D / 2; ++j) {
      const double a = (double)delta * f[j];
      rot[((size_t)i * kvc::kHalf + j) * 2 + 0] = std::cos(a);
      rot[((size_t)i * kvc::kHalf + j) * 2 + 1] = std::sin(a);
    }
    for (int64_t r = 0; r < L->chunk_len[i]; r += tile_rows) {
      kvc::ShiftTile t;
      t.chunk = i;
      t.row_begin = (int32_t)(row0 + r);
      t.row_end = (int32_t)(row0 + std::min<int64_t>(r + tile_rows, L->chunk_len[i]));
      t.flags = (delta == 0 ? kvc::kTileDeltaZero : 0u) | (L->zero_kv && L->zero_kv[i] != 0 ? kvc::kTileZeroKv : 0u);
      tiles[nt++] = t;
    }
    row0 += L->chunk_len[i];
  }
  st = need_device(W);
  if (st != KVC_OK) return st;
  hipError_t e = hipMemcpyAsync(plan, img, need, hipMemcpyHostToDevice, as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  if (!host_staging) {
    // the image lives in this call's memory: wait until it has been read
    e = hipStreamSynchronize(as_stream(stream));
    if (e != hipSuccess) return hip_fail(W, e);
  }
  plan_out->device = plan;
  plan_out->bytes = plan_bytes_in;
  plan_out->layout_id = hdr.layout_hash;
  return ok();
}

kvc_status kvc_rope_shift(const kvc_layout* L, const kvc_plan* plan, const void* k_src, void* k_dst,
                          void* stream) {
  const char* W = "kvc_rope_shift";
  LayoutInfo li;
  kvc_status st = check_layout(W, L, &li);
  if (st != KVC_OK) return st;
  if (li.n_reused == 0) return ok();
  st = check_plan(W, L, li, plan);
  if (st != KVC_OK) return st;
  if (!k_src || !k_dst || !aligned16(k_src) || !aligned16(k_dst))
    return fail(KVC_ERR_INVALID_ARG, "%s: k_src/k_dst NULL or not 16-byte aligned", W);
  const size_t bytes = (size_t)li.n_reused * L->n_kv_heads * L->head_dim * 2;
  if (k_src != k_dst) {
    const char* a = static_cast<const char*>(k_src);
    const char* b = static_cast<const char*>(k_dst);
    if (a < b + bytes && b < a + bytes)
      return fail(KVC_ERR_INVALID_ARG, "%s: k_src and k_dst partially overlap", W);
  }
  st = check_disjoint(W, {{k_dst, bytes, "k_dst"}}, {plan_span(plan)});
  if (st != KVC_OK) return st;
  st = need_device(W);
  if (st != KVC_OK) return st;
  hipError_t e = kvc::launch_rope_shift(plan->device, plan->layout_id, L->n_chunks, li.n_tiles, L->n_kv_heads,
                                        static_cast<const uint16_t*>(k_src),
                                        static_cast<uint16_t*>(k_dst), nullptr, as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_kv_deviation(int64_t n_rows, int32_t n_kv_heads, int32_t head_dim,
                            const void* k_cached, const void* k_fresh, double* dev_out,
                            void* stream) {
  const char* W = "kvc_kv_deviation";
  if (n_rows < 0 || n_rows > kMaxRows) return fail(KVC_ERR_INVALID_ARG, "%s: n_rows=%lld out of range", W, (long long)n_rows);
  kvc_status st = check_heads(W, n_kv_heads, n_kv_heads, head_dim);
  if (st != KVC_OK) return st;
  if (n_rows == 0) return ok();
  if (!k_cached || !k_fresh || !dev_out || !aligned16(k_cached) || !aligned16(k_fresh) ||
      (reinterpret_cast<uintptr_t>(dev_out) & 7u))
    return fail(KVC_ERR_INVALID_ARG, "%s: NULL or misaligned pointer", W);
  const size_t kb = (size_t)n_rows * n_kv_heads * head_dim * 2;
  st = check_disjoint(W, {{dev_out, (size_t)n_rows * 8, "dev_out"}}, {{k_cached, kb, "k_cached"}, {k_fresh, kb, "k_fresh"}});
  if (st != KVC_OK) return st;
  st = need_device(W);
  if (st != KVC_OK) return st;
  hipError_t e = kvc::launch_kv_deviation(n_rows, n_kv_heads, static_cast<const uint16_t*>(k_cached),
                                          static_cast<const uint16_t*>(k_fresh), dev_out,
                                          as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_select_topk_workspace(int64_t n, size_t* bytes) {
  if (n < 0 || n > kMaxRows) return fail(KVC_ERR_INVALID_ARG, "kvc_select_topk_workspace: n=%lld out of range", (long long)n);
  if (!bytes) return fail(KVC_ERR_INVALID_ARG, "kvc_select_topk_workspace: bytes is NULL");
  *bytes = kvc::topk_ws_bytes(n);
  return ok();
}

static kvc_status select_topk_impl(const char* W, const double* dev, int64_t n, int64_t k,
                                   int64_t n_append, int32_t* idx_out, void* ws, size_t ws_bytes,
                                   hipStream_t s) {
  if (n < 0 || n > kMaxRows) return fail(KVC_ERR_INVALID_ARG, "%s: n=%lld out of range", W, (long long)n);
  if (k < 0 || k > n) return fail(KVC_ERR_INVALID_ARG, "%s: k=%lld not in [0, n=%lld]", W, (long long)k, (long long)n);
  if (k + n_append == 0) return ok();
  if (!idx_out || (reinterpret_cast<uintptr_t>(idx_out) & 3u))
    return fail(KVC_ERR_INVALID_ARG, "%s: idx_out NULL or misaligned", W);
  if (k > 0 && k < n) {
    if (!dev || (reinterpret_cast<uintptr_t>(dev) & 7u)) return fail(KVC_ERR_INVALID_ARG, "%s: dev NULL or misaligned", W);
    if (!ws || !aligned16(ws)) return fail(KVC_ERR_INVALID_ARG, "%s: ws NULL or not 16-byte aligned", W);
    if (ws_bytes < kvc::topk_ws_bytes(n))
      return fail(KVC_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", W, ws_bytes, kvc::topk_ws_bytes(n));
  }
  const bool radix = k > 0 && k < n;
  kvc_status st = check_disjoint(W, {{idx_out, (size_t)(k + n_append) * 4, "idx_out"}, {radix ? ws : nullptr, ws_bytes, "ws"}},
                                 {{radix ? dev : nullptr, (size_t)n * 8, "dev"}});
  if (st != KVC_OK) return st;
  st = need_device(W);
  if (st != KVC_OK) return st;
  hipError_t e = kvc::launch_select_topk(dev, n, k, n_append, idx_out, ws, s);
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_select_topk(const double* dev, int64_t n, int64_t k, int32_t* idx_out, void* ws,
                           size_t ws_bytes, void* stream) {
  return select_topk_impl("kvc_select_topk", dev, n, k, 0, idx_out, ws, ws_bytes, as_stream(stream));
}

kvc_status kvc_scatter_rows(const int32_t* sel, int64_t n_sel, int32_t fresh_is_compact,
                            const void* k_fresh, const void* v_fresh, int64_t n_fresh_rows,
                            void* k_cache, void* v_cache, int64_t n_rows, int32_t n_kv_heads,
                            int32_t head_dim, void* stream) {
  const char* W = "kvc_scatter_rows";
  if (n_sel < 0 || n_fresh_rows < 0 || n_rows < 0 || n_sel > kMaxRows || n_rows > kMaxRows || n_fresh_rows > kMaxRows)
    return fail(KVC_ERR_INVALID_ARG, "%s: negative or too large size", W);
  kvc_status st = check_heads(W, n_kv_heads, n_kv_heads, head_dim);
  if (st != KVC_OK) return st;
  if (n_sel == 0) return ok();
  if (!sel || (reinterpret_cast<uintptr_t>(sel) & 3u) || !k_fresh || !v_fresh || !k_cache || !v_cache ||
      !aligned16(k_fresh) || !aligned16(v_fresh) || !aligned16(k_cache) || !aligned16(v_cache))
    return fail(KVC_ERR_INVALID_ARG, "%s: NULL or misaligned pointer", W);
  {
    const size_t rb = (size_t)n_kv_heads * head_dim * 2;
    st = check_disjoint(W, {{k_cache, (size_t)n_rows * rb, "k_cache"}, {v_cache, (size_t)n_rows * rb, "v_cache"}},
                        {{sel, (size_t)n_sel * 4, "sel"}, {k_fresh, (size_t)n_fresh_rows * rb, "k_fresh"},
                         {v_fresh, (size_t)n_fresh_rows * rb, "v_fresh"}});
    if (st != KVC_OK) return st;
  }
  st = need_device(W);
  if (st != KVC_OK) return st;
  hipError_t e = kvc::launch_scatter_rows(sel, n_sel, fresh_is_compact != 0,
                                          static_cast<const uint16_t*>(k_fresh),
                                          static_cast<const uint16_t*>(v_fresh), n_fresh_rows,
                                          static_cast<uint16_t*>(k_cache),
                                          static_cast<uint16_t*>(v_cache), n_rows, n_kv_heads,
                                          as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_attention_workspace(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads,
                                   int32_t head_dim, size_t* bytes) {
  const char* W = "kvc_attention_workspace";
  if (n_sel < 0 || n_sel > kMaxRows) return fail(KVC_ERR_INVALID_ARG, "%s: n_sel out of range", W);
  kvc_status st = check_heads(W, n_q_heads, n_kv_heads, head_dim);
  if (st != KVC_OK) return st;
  if (!bytes) return fail(KVC_ERR_INVALID_ARG, "%s: bytes is NULL", W);
  *bytes = kvc::attention_ws_bytes(n_sel, n_q_heads, n_kv_heads);
  return ok();
}

static kvc_status attention_impl(const char* W, const void* q, int64_t n_q_rows,
                                 const int32_t* q_rows, const int32_t* q_pos, int64_t n_sel,
                                 const void* k, const void* v, int64_t n_kv, int32_t n_q_heads,
                                 int32_t n_kv_heads, int32_t head_dim, float softmax_scale,
                                 void* out, float* lse, void* ws, size_t ws_bytes, hipStream_t s) {
  if (n_sel < 0 || n_sel > kMaxRows || n_q_rows < 0 || n_q_rows > kMaxRows || n_kv < 0 || n_kv > kMaxRows)
    return fail(KVC_ERR_INVALID_ARG, "%s: size out of range", W);
  kvc_status st = check_heads(W, n_q_heads, n_kv_heads, head_dim);
  if (st != KVC_OK) return st;
  if (!(softmax_scale >= 0.0f) || !std::isfinite(softmax_scale))
    return fail(KVC_ERR_INVALID_ARG, "%s: softmax_scale must be finite and >= 0", W);
  if (!q_rows && n_q_rows < n_sel)
    return fail(KVC_ERR_INVALID_ARG, "%s: compact queries need n_q_rows >= n_sel", W);
  if (kvc::attention_work_items(n_sel, n_q_heads, n_kv_heads) > (int64_t)UINT32_MAX)
    return fail(KVC_ERR_INVALID_ARG, "%s: n_sel x n_q_heads too large for one launch", W);
  if (n_sel == 0) return ok();
  if (!q || !q_pos || !k || !v || !out || !aligned16(q) || !aligned16(k) || !aligned16(v) ||
      !aligned16(out) || (reinterpret_cast<uintptr_t>(q_pos) & 3u) ||
      (q_rows && (reinterpret_cast<uintptr_t>(q_rows) & 3u)) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)))
    return fail(KVC_ERR_INVALID_ARG, "%s: NULL or misaligned pointer", W);
  if (ws && ws_bytes > 0 && !aligned16(ws)) return fail(KVC_ERR_INVALID_ARG, "%s: ws not 16-byte aligned", W);
  {
    const size_t qr = (size_t)n_q_heads * head_dim * 2, kr = (size_t)n_kv_heads * head_dim * 2;
    st = check_disjoint(W,
                        {{out, (size_t)n_sel * qr, "out"}, {lse, (size_t)n_sel * n_q_heads * 4, "lse"},
                         {ws, ws_bytes, "ws"}},
                        {{q, (size_t)n_q_rows * qr, "q"}, {q_rows, (size_t)n_sel * 4, "q_rows"},
                         {q_pos, (size_t)n_sel * 4, "q_pos"}, {k, (size_t)n_kv * kr, "k"}, {v, (size_t)n_kv * kr, "v"}});
    if (st != KVC_OK) return st;
  }
  st = need_device(W);
  if (st != KVC_OK) return st;
  const float scale = softmax_scale > 0.0f ? softmax_scale : 1.0f / std::sqrt((float)head_dim);
  hipError_t e = kvc::launch_attention(static_cast<const uint16_t*>(q), n_q_rows, q_rows, q_pos, n_sel,
                                       static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v),
                                       n_kv, n_q_heads, n_kv_heads, scale, static_cast<uint16_t*>(out),
                                       lse, ws, ws_bytes, s);
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_sparse_query_attention(const void* q, int64_t n_q_rows, const int32_t* q_rows,
                                      const int32_t* q_pos, int64_t n_sel, const void* k,
                                      const void* v, int64_t n_kv, int32_t n_q_heads,
                                      int32_t n_kv_heads, int32_t head_dim, float softmax_scale,
                                      void* out, float* lse, void* ws, size_t ws_bytes,
                                      void* stream) {
  return attention_impl("kvc_sparse_query_attention", q, n_q_rows, q_rows, q_pos, n_sel, k, v, n_kv,
                        n_q_heads, n_kv_heads, head_dim, softmax_scale, out, lse, ws, ws_bytes,
                        as_stream(stream));
}

kvc_status kvc_blend_workspace(const kvc_layout* L, size_t* bytes) {
  LayoutInfo li;
  kvc_status st = check_layout("kvc_blend_workspace", L, &li);
  if (st != KVC_OK) return st;
  if (!bytes) return fail(KVC_ERR_INVALID_ARG, "kvc_blend_workspace: bytes is NULL");
  // deviation vector, then the top-k scratch
  *bytes = kvc::align256(sizeof(double) * (size_t)(li.n_reused > 0 ? li.n_reused : 1)) +
           kvc::topk_ws_bytes(li.n_reused);
  return ok();
}

}  // extern "C"

namespace {

// kvc_blend_prefill_layer, and with static_ws its variant that takes its
// scratch from the library's static array (ws and ws_bytes ignored).
kvc_status blend_layer(const char* W, const kvc_layout* L, const kvc_plan* plan, int32_t is_check_layer,
                       double ratio, const void* k_src, void* k_cache, void* v_cache, const void* q_fresh,
                       const void* k_fresh, const void* v_fresh, int32_t* sel, int64_t n_sel, void* out,
                       float* lse, void* ws, size_t ws_bytes, bool static_ws, void* stream) {
  if (static_ws) {
    ws = nullptr;
    ws_bytes = 0;
  }
  LayoutInfo li;
  int64_t k = 0;
  const bool check = is_check_layer != 0;
  kvc_status st = check_select(W, L, &li, plan, check, ratio, k_src, k_cache, k_fresh, sel, n_sel, ws,
                               ws_bytes, static_ws, &k);
  if (st != KVC_OK) return st;
  if (n_sel > 0 && (!v_cache || !q_fresh || !k_fresh || !v_fresh || !out || !aligned16(v_cache) ||
                    !aligned16(q_fresh) || !aligned16(k_fresh) || !aligned16(v_fresh) ||
                    !aligned16(out) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3u))))
    return fail(KVC_ERR_INVALID_ARG, "%s: NULL or misaligned tensor pointer", W);
  const bool shift = li.n_reused > 0 && k_src;
  {
    // k_src may be k_cache itself (adjusted in place); partial overlap was refused above
    const size_t kr = (size_t)L->n_kv_heads * L->head_dim * 2, qr = (size_t)L->n_q_heads * L->head_dim * 2;
    const size_t fresh_rows = (size_t)(check ? li.n_rows : n_sel);
    const bool sel_used = n_sel > 0;
    st = check_disjoint(W,
                        {{k_cache, (size_t)li.n_rows * kr, "k_cache"},
                         {sel_used ? v_cache : nullptr, (size_t)li.n_rows * kr, "v_cache"},
                         {sel_used ? sel : nullptr, (size_t)n_sel * 4, "sel"},
                         {sel_used ? out : nullptr, (size_t)n_sel * qr, "out"},
                         {sel_used ? lse : nullptr, (size_t)n_sel * L->n_q_heads * 4, "lse"},
                         {ws, ws_bytes, "ws"}},
                        {{k_src != k_cache ? k_src : nullptr, (size_t)li.n_reused * kr, "k_src"}, plan_span(plan),
                         {sel_used ? q_fresh : nullptr, fresh_rows * qr, "q_fresh"},
                         {sel_used || check ? k_fresh : nullptr, fresh_rows * kr, "k_fresh"},
                         {sel_used ? v_fresh : nullptr, fresh_rows * kr, "v_fresh"}});
    if (st != KVC_OK) return st;
  }
  if (n_sel == 0 && !shift) return ok();
  st = need_device(W);
  if (st != KVC_OK) return st;
  const hipStream_t s = as_stream(stream);
  const int hkv = L->n_kv_heads;
  if (static_ws) {
    // the layer's own part, plus the attention's split partials if they fit
    void* p = nullptr;
    const hipError_t e = kvc::static_scratch(&p);
    if (e != hipSuccess) return hip_fail(W, e);
    size_t need_ws = 0;
    kvc_blend_workspace(L, &need_ws);
    const size_t attn = kvc::attention_ws_bytes(n_sel, L->n_q_heads, hkv);
    ws = p;
    ws_bytes = need_ws + attn <= kvc::kStaticScratchBytes ? need_ws + attn : need_ws;
  }

  // a1 (+ a2, a3 on the check layer)
  hipError_t e = shift_and_select(L, li, plan, check, k, k_src, k_cache, k_fresh, sel, ws, s);
  if (e != hipSuccess) return hip_fail(W, e);
  if (n_sel == 0) return ok();
  // a4: recomputed K/V into the selected rows
  e = kvc::launch_scatter_rows(sel, n_sel, check ? 0 : 1, static_cast<const uint16_t*>(k_fresh),
                               static_cast<const uint16_t*>(v_fresh), check ? li.n_rows : n_sel,
                               static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache),
                               li.n_rows, hkv, s);
  if (e != hipSuccess) return hip_fail(W, e);
  // a4 gather + a5: attention of the selected queries at positions sel; the
  // workspace beyond the layer's own part, if large enough, lets a small
  // selection split its key range
  size_t need_ws = 0;
  kvc_blend_workspace(L, &need_ws);
  void* aws = nullptr;
  size_t aws_bytes = 0;
  if (ws && ws_bytes > need_ws) {
    aws = static_cast<char*>(ws) + need_ws;
    aws_bytes = ws_bytes - need_ws;
  }
  e = kvc::launch_attention(static_cast<const uint16_t*>(q_fresh), check ? li.n_rows : n_sel,
                            check ? sel : nullptr, sel, n_sel, static_cast<const uint16_t*>(k_cache),
                            static_cast<const uint16_t*>(v_cache), li.n_rows, L->n_q_heads, hkv,
                            1.0f / std::sqrt((float)L->head_dim), static_cast<uint16_t*>(out), lse, aws,
                            aws_bytes, s);
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

}  // namespace

extern "C" {

kvc_status kvc_blend_prefill_layer(const kvc_layout* L, const kvc_plan* plan, int32_t is_check_layer,
                                   double ratio, const void* k_src, void* k_cache, void* v_cache,
                                   const void* q_fresh, const void* k_fresh, const void* v_fresh,
                                   int32_t* sel, int64_t n_sel, void* out, float* lse, void* ws,
                                   size_t ws_bytes, void* stream) {
  return blend_layer("kvc_blend_prefill_layer", L, plan, is_check_layer, ratio, k_src, k_cache, v_cache, q_fresh,
                     k_fresh, v_fresh, sel, n_sel, out, lse, ws, ws_bytes, false, stream);
}

kvc_status kvc_blend_prefill_layer_noalloc(const kvc_layout* L, const kvc_plan* plan, int32_t is_check_layer,
                                           double ratio, const void* k_src, void* k_cache, void* v_cache,
                                           const void* q_fresh, const void* k_fresh, const void* v_fresh,
                                           int32_t* sel, int64_t n_sel, void* out, float* lse, void* stream) {
  return blend_layer("kvc_blend_prefill_layer_noalloc", L, plan, is_check_layer, ratio, k_src, k_cache, v_cache,
                     q_fresh, k_fresh, v_fresh, sel, n_sel, out, lse, nullptr, 0, true, stream);
}

kvc_status kvc_select_tokens(const kvc_layout* L, const kvc_plan* plan, double ratio, const void* k_src,
                             void* k_cache, const void* k_fresh, int32_t* sel, int64_t n_sel, void* ws,
                             size_t ws_bytes, void* stream) {
  const char* W = "kvc_select_tokens";
  LayoutInfo li;
  int64_t k = 0;
  kvc_status st = check_select(W, L, &li, plan, true, ratio, k_src, k_cache, k_fresh, sel, n_sel, ws,
                               ws_bytes, false, &k);
  if (st != KVC_OK) return st;
  {
    const size_t kr = (size_t)L->n_kv_heads * L->head_dim * 2;
    st = check_disjoint(W,
                        {{k_cache, (size_t)li.n_reused * kr, "k_cache"}, {sel, (size_t)n_sel * 4, "sel"},
                         {ws, ws_bytes, "ws"}},
                        {{k_src != k_cache ? k_src : nullptr, (size_t)li.n_reused * kr, "k_src"}, plan_span(plan),
                         {k_fresh, (size_t)li.n_reused * kr, "k_fresh"}});
    if (st != KVC_OK) return st;
  }
  if (n_sel == 0 && !(li.n_reused > 0 && k_src)) return ok();
  st = need_device(W);
  if (st != KVC_OK) return st;
  const hipError_t e = shift_and_select(L, li, plan, true, k, k_src, k_cache, k_fresh, sel, ws, as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_rms_norm(const void* x, int64_t n_x_rows, const int32_t* rows, int64_t n, int32_t hidden,
                        const void* gamma, float eps, void* out, void* res_out, void* stream) {
  const char* W = "kvc_rms_norm";
  if (n < 0 || n_x_rows < 0 || n > kMaxRows || n_x_rows > kMaxRows)
    return fail(KVC_ERR_INVALID_ARG, "%s: negative or too large row count", W);
  if (hidden < 8 || hidden > kvc::kMaxHidden || hidden % 8 != 0)
    return fail(KVC_ERR_INVALID_ARG, "%s: hidden=%d must be a multiple of 8 in [8, %d]", W, hidden, kvc::kMaxHidden);
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return fail(KVC_ERR_INVALID_ARG, "%s: eps must be finite and >= 0", W);
  if (!rows && n > n_x_rows) return fail(KVC_ERR_INVALID_ARG, "%s: n=%lld rows but x has %lld", W, (long long)n, (long long)n_x_rows);
  if (n == 0) return ok();
  if (!x || !gamma || !out || !aligned16(x) || !aligned16(gamma) || !aligned16(out) ||
      (res_out && !aligned16(res_out)) || (rows && (reinterpret_cast<uintptr_t>(rows) & 3u)))
    return fail(KVC_ERR_INVALID_ARG, "%s: NULL or misaligned pointer", W);
  const size_t xb = (size_t)n_x_rows * hidden * 2, ob = (size_t)n * hidden * 2;
  kvc_status st = check_disjoint(W, {{out, ob, "out"}, {res_out, ob, "res_out"}},
                                 {{x, xb, "x"}, {gamma, (size_t)hidden * 2, "gamma"}, {rows, (size_t)n * 4, "rows"}});
  if (st != KVC_OK) return st;
  st = need_device(W);
  if (st != KVC_OK) return st;
  const hipError_t e = kvc::launch_rms_norm(static_cast<const uint16_t*>(x), n_x_rows, rows, n, hidden,
                                            static_cast<const uint16_t*>(gamma), eps,
                                            static_cast<uint16_t*>(out), static_cast<uint16_t*>(res_out),
                                            as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_qkv_rope(const void* y, int64_t n, int32_t n_q_heads, int32_t n_k_heads, int32_t n_v_heads,
                        int32_t head_dim, const int32_t* pos, double rope_theta, const double* inv_freq,
                        void* q, void* k, void* v, void* stream) {
  const char* W = "kvc_qkv_rope";
  if (n < 0 || n > kMaxRows) return fail(KVC_ERR_INVALID_ARG, "%s: n=%lld out of range", W, (long long)n);
  if (n_q_heads < 0 || n_k_heads < 0 || n_v_heads < 0 || n_q_heads + n_k_heads + n_v_heads < 1 ||
      n_q_heads + n_k_heads + n_v_heads > 1024)
    return fail(KVC_ERR_INVALID_ARG, "%s: head counts %d/%d/%d (each >= 0, total in [1, 1024])", W,
                n_q_heads, n_k_heads, n_v_heads);
  if (head_dim != kvc::kHeadDim) return fail(KVC_ERR_UNSUPPORTED, "%s: head_dim=%d (only 128 is supported)", W, head_dim);
  double f[kvc::kHalf];
  if (inv_freq) {
    for (int j = 0; j < kvc::kHalf; ++j) {
      if (!std::isfinite(inv_freq[j])) return fail(KVC_ERR_INVALID_ARG, "%s: inv_freq[%d] not finite", W, j);
      f[j] = inv_freq[j];
    }
  } else {
    if (!(rope_theta > 0.0) || !std::isfinite(rope_theta))
      return fail(KVC_ERR_INVALID_ARG, "%s: rope_theta must be finite and > 0", W);
    for (int j = 0; j < kvc::kHalf; ++j) f[j] = std::pow(rope_theta, -(2.0 * j) / head_dim);
  }
  if (n == 0) return ok();
  if (!y || !aligned16(y) || (n_q_heads > 0 && (!q || !aligned16(q))) ||
      (n_k_heads > 0 && (!k || !aligned16(k))) || (n_v_heads > 0 && (!v || !aligned16(v))) ||
      (pos && (reinterpret_cast<uintptr_t>(pos) & 3u)))
    return fail(KVC_ERR_INVALID_ARG, "%s: NULL or misaligned pointer", W);
  const size_t yb = (size_t)n * (n_q_heads + n_k_heads + n_v_heads) * head_dim * 2;
  const size_t qb = (size_t)n * n_q_heads * head_dim * 2, kb = (size_t)n * n_k_heads * head_dim * 2,
               vb = (size_t)n * n_v_heads * head_dim * 2;
  kvc_status st = check_disjoint(W, {{q, qb, "q"}, {k, kb, "k"}, {v, vb, "v"}},
                                 {{y, yb, "y"}, {pos, (size_t)n * 4, "pos"}});
  if (st != KVC_OK) return st;
  st = need_device(W);
  if (st != KVC_OK) return st;
  const hipError_t e = kvc::launch_qkv_rope(static_cast<const uint16_t*>(y), n, n_q_heads, n_k_heads,
                                            n_v_heads, pos, f, static_cast<uint16_t*>(q),
                                            static_cast<uint16_t*>(k), static_cast<uint16_t*>(v),
                                            as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_swiglu(const void* gate_up, int64_t n, int64_t inter, void* out, void* stream) {
  const char* W = "kvc_swiglu";
  if (n < 0 || n > kMaxRows) return fail(KVC_ERR_INVALID_ARG, "%s: n=%lld out of range", W, (long long)n);
  if (inter < 8 || inter % 8 != 0 || inter > (int64_t(1) << 24))
    return fail(KVC_ERR_INVALID_ARG, "%s: inter=%lld must be a multiple of 8 in [8, 2^24]", W, (long long)inter);
  if (n == 0) return ok();
  if (!gate_up || !out || !aligned16(gate_up) || !aligned16(out))
    return fail(KVC_ERR_INVALID_ARG, "%s: NULL or misaligned pointer", W);
  kvc_status st0 = check_disjoint(W, {{out, (size_t)n * inter * 2, "out"}}, {{gate_up, (size_t)n * inter * 4, "gate_up"}});
  if (st0 != KVC_OK) return st0;
  kvc_status st = need_device(W);
  if (st != KVC_OK) return st;
  const hipError_t e = kvc::launch_swiglu(static_cast<const uint16_t*>(gate_up), n, inter,
                                          static_cast<uint16_t*>(out), as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_projection(int64_t m, int64_t n, int64_t k, const void* a, int64_t n_a_rows, const int32_t* a_rows,
                          const void* w, const void* residual, void* c, void* stream) {
  const char* W = "kvc_projection";
  if (m < 0 || m > kMaxRows || n_a_rows < 0 || n_a_rows > kMaxRows)
    return fail(KVC_ERR_INVALID_ARG, "%s: m=%lld or n_a_rows=%lld out of range", W, (long long)m, (long long)n_a_rows);
  if (n < 0 || n > (int64_t(1) << 24) || n % 8 != 0)
    return fail(KVC_ERR_INVALID_ARG, "%s: n=%lld must be a multiple of 8 in [0, 2^24]", W, (long long)n);
  if (k < 64 || k > (int64_t(1) << 24) || k % 64 != 0)
    return fail(KVC_ERR_UNSUPPORTED, "%s: k=%lld must be a multiple of 64 in [64, 2^24]", W, (long long)k);
  if (!a_rows && m > n_a_rows)
    return fail(KVC_ERR_INVALID_ARG, "%s: m=%lld rows but a has %lld", W, (long long)m, (long long)n_a_rows);
  if (m == 0 || n == 0) return ok();
  if (n_a_rows == 0) return fail(KVC_ERR_INVALID_ARG, "%s: a has no rows", W);
  if (kvc::gemm_work_items(m, n) > (int64_t)UINT32_MAX)
    return fail(KVC_ERR_INVALID_ARG, "%s: m x n too large for one launch", W);
  if (!a || !w || !c || !aligned16(a) || !aligned16(w) || !aligned16(c) || (residual && !aligned16(residual)) ||
      (a_rows && (reinterpret_cast<uintptr_t>(a_rows) & 3u)))
    return fail(KVC_ERR_INVALID_ARG, "%s: NULL or misaligned pointer", W);
  const size_t cb = (size_t)m * (size_t)n * 2;
  // c may be the residual itself (added in place); otherwise it overlaps no input
  kvc_status st = check_disjoint(W, {{c, cb, "c"}},
                                 {{a, (size_t)n_a_rows * (size_t)k * 2, "a"}, {w, (size_t)n * (size_t)k * 2, "w"},
                                  {a_rows, (size_t)m * 4, "a_rows"}, {residual != c ? residual : nullptr, cb, "residual"}});
  if (st != KVC_OK) return st;
  st = need_device(W);
  if (st != KVC_OK) return st;
  const hipError_t e = kvc::launch_gemm(m, n, k, static_cast<const uint16_t*>(a), n_a_rows, a_rows,
                                        static_cast<const uint16_t*>(w), static_cast<const uint16_t*>(residual),
                                        static_cast<uint16_t*>(c), as_stream(stream));
  if (e != hipSuccess) return hip_fail(W, e);
  return ok();
}

kvc_status kvc_stage_layers(const kvc_layout* L, const kvc_plan* plan, int32_t n_layers,
                            const void* const* k_chunks, const void* const* v_chunks,
                            void* const* k_cache, void* const* v_cache, void* const* events,
                            void* stream);

kvc_status kvc_stage_layer(const kvc_layout* L, const kvc_plan* plan, const void* const* k_chunks,
                           const void* const* v_chunks, void* k_cache, void* v_cache, void* stream) {
  void* kc[1] = {k_cache};
  void* vc[1] = {v_cache};
  const kvc_status st = kvc_stage_layers(L, plan, 1, k_chunks, v_chunks, kc, vc, nullptr, stream);
  if (st != KVC_OK) {
    // report under this entry point's name, without the layer index
    std::string m = g_err;
    for (const char* pre : {"kvc_stage_layers: ", "layer 0: "})
      if (m.compare(0, std::strlen(pre), pre) == 0) m = m.substr(std::strlen(pre));
    return fail(st, "kvc_stage_layer: %s", m.c_str());
  }
  return st;
}

kvc_status kvc_stage_layers(const kvc_layout* L, const kvc_plan* plan, int32_t n_layers,
                            const void* const* k_chunks, const void* const* v_chunks,
                            void* const* k_cache, void* const* v_cache, void* const* events,
                            void* stream) {
  const char* W = "kvc_stage_layers";
  LayoutInfo li;
  kvc_status st = check_layout(W, L, &li);
  if (st != KVC_OK) return st;
  if (n_layers < 0) return fail(KVC_ERR_INVALID_ARG, "%s: n_layers=%d < 0", W, n_layers);
  if (n_layers == 0 || li.n_reused == 0) return ok();
  st = check_plan(W, L, li, plan);
  if (st != KVC_OK) return st;
  if (!k_cache || !v_cache) return fail(KVC_ERR_INVALID_ARG, "%s: k_cache/v_cache array is NULL", W);
  if (!k_chunks || !v_chunks) return fail(KVC_ERR_INVALID_ARG, "%s: k_chunks/v_chunks is NULL", W);
  const size_t nc = (size_t)L->n_chunks;
  // every layer's arguments before the first HIP call
  for (int32_t l = 0; l < n_layers; ++l) {
    if (!k_cache[l] || !v_cache[l] || !aligned16(k_cache[l]) || !aligned16(v_cache[l]))
      return fail(KVC_ERR_INVALID_ARG, "%s: layer %d: k_cache/v_cache NULL or not 16-byte aligned", W, l);
    for (size_t i = 0; i < nc; ++i) {
      const bool zero = L->zero_kv && L->zero_kv[i];
      if (!zero && L->chunk_len[i] > 0 && (!k_chunks[l * nc + i] || !v_chunks[l * nc + i]))
        return fail(KVC_ERR_INVALID_ARG, "%s: layer %d: chunk %zu has no cache pointer", W, l, i);
    }
  }
  {
    // the layers' caches (outputs) share no byte with each other or with any
    // chunk source; sources may overlap each other
    const size_t rb = (size_t)L->n_kv_heads * L->head_dim * 2;
    std::vector<TaggedSpan> spans;
    spans.reserve((size_t)n_layers * (2 + 2 * nc) + 1);
    spans.push_back({reinterpret_cast<uintptr_t>(plan->device), reinterpret_cast<uintptr_t>(plan->device) + plan->bytes,
                     false, 0, "plan"});
    for (int32_t l = 0; l < n_layers; ++l) {
      const size_t cb = (size_t)li.n_reused * rb;
      spans.push_back({reinterpret_cast<uintptr_t>(k_cache[l]), reinterpret_cast<uintptr_t>(k_cache[l]) + cb, true, l, "k_cache"});
      spans.push_back({reinterpret_cast<uintptr_t>(v_cache[l]), reinterpret_cast<uintptr_t>(v_cache[l]) + cb, true, l, "v_cache"});
      for (size_t i = 0; i < nc; ++i) {
        const size_t bytes = (size_t)L->chunk_len[i] * rb;
        for (const void* c : {k_chunks[l * nc + i], v_chunks[l * nc + i]})
          if (c && bytes)
            spans.push_back({reinterpret_cast<uintptr_t>(c), reinterpret_cast<uintptr_t>(c) + bytes, false, l, "chunk source"});
      }
    }
    st = check_disjoint_many(W, spans);
    if (st != KVC_OK) return st;
  }
  st = need_device(W);
  if (st != KVC_OK) return st;
  const hipStream_t s = as_stream(stream);
  const size_t row_bytes = (size_t)L->n_kv_heads * L->head_dim * 2;
  for (int32_t l = 0; l < n_layers; ++l) {
    // copies, merging chunks whose sources are back to back; K and V apart
    for (int which = 0; which < 2; ++which) {
      const void* const* src = (which == 0 ? k_chunks : v_chunks) + (size_t)l * nc;
      char* dst = static_cast<char*>(which == 0 ? k_cache[l] : v_cache[l]);
      const char* run_src = nullptr;
      size_t run_dst = 0, run_bytes = 0, row0 = 0;
      for (size_t i = 0; i <= nc; ++i) {
        const bool end = i == nc;
        const size_t bytes = end ? 0 : (size_t)L->chunk_len[i] * row_bytes;
        const bool zero = !end && L->zero_kv && L->zero_kv[i];
        // a zero chunk given a source is copied like any chunk (its rows are
        // zero-filled afterwards); without one it ends the current run
        const char* c = (end || bytes == 0) ? nullptr : static_cast<const char*>(src[i]);
        const bool gap = zero && !c;
        const bool extend = c && run_bytes > 0 && c == run_src + run_bytes && row0 * row_bytes == run_dst + run_bytes;
        if (!extend && (end || gap || c) && run_bytes > 0) {
          const hipError_t e = hipMemcpyAsync(dst + run_dst, run_src, run_bytes, hipMemcpyDefault, s);
          if (e != hipSuccess) return hip_fail(W, e);
          run_bytes = 0;
        }
        if (c) {
          if (extend) {
            run_bytes += bytes;
          } else {
            run_src = c;
            run_dst = row0 * row_bytes;
            run_bytes = bytes;
          }
        }
        if (!end) row0 += (size_t)L->chunk_len[i];
      }
    }
    // zeros for the separator slots, keys adjusted in place
    hipError_t e = kvc::launch_rope_shift(plan->device, plan->layout_id, L->n_chunks, li.n_tiles, L->n_kv_heads,
                                          static_cast<const uint16_t*>(k_cache[l]),
                                          static_cast<uint16_t*>(k_cache[l]), static_cast<uint16_t*>(v_cache[l]), s);
    if (e != hipSuccess) return hip_fail(W, e);
    if (events && events[l]) {
      e = hipEventRecord(reinterpret_cast<hipEvent_t>(events[l]), s);
      if (e != hipSuccess) return hip_fail(W, e);
    }
  }
  return ok();
}

}  // extern "C"
