// Internal declarations shared by the C ABI (api.cpp) and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kvc {

constexpr int kHeadDim = 128;      // D: the only supported head size
constexpr int kHalf = kHeadDim / 2;
// Work tile of the adjustment kernel: up to 1024 16-byte units (8 pairs of
// one head row), four per thread of a 256-thread workgroup, all loaded
// before the first is rotated: 16 rows of 8 kv heads, 128 rows of one.
constexpr int kShiftTileUnits = 1024;
// Requests of fewer than 16,384 reused rows get tiles of at most 16 rows,
// so that they still spread over the CUs (4.1k rows of one kv head: 256
// tiles instead of 32).
inline int shift_tile_rows(int64_t n_reused, int n_kv_heads) {
  const int rows = kShiftTileUnits / (8 * n_kv_heads);  // >= 2 for n_kv_heads <= 64
  return n_reused < 16384 && rows > 16 ? 16 : rows;
}
constexpr int kMaxHidden = 16384;  // widest row the RMS normalisation keeps in registers
// Grid cap of the grid-stride kernels (and of each batch of shift tiles):
// 2^20 workgroups of up to 512 threads
// stay far below HIP's 2^32 work-items per launch and fill the GPU many times.
constexpr int64_t kMaxGrid = int64_t(1) << 20;

// ---- plan (device buffer written by kvc_plan_upload) ----------------------
// [PlanHeader][double2 rot[n_chunks][64]][ShiftTile tiles[n_tiles]], each
// part 256-byte aligned; the offsets follow from n_chunks alone, so the host
// passes them to the kernel with n_tiles and only the header's hash and the
// tile itself are read before the data.
struct PlanHeader {
  uint64_t layout_hash;  // checked by the kernel: a stale plan does nothing
  int32_t n_chunks;
  int32_t n_tiles;
  int64_t n_reused;
  int64_t rot_offset;    // bytes from plan start
  int64_t tile_offset;   // bytes from plan start
};
constexpr uint32_t kTileDeltaZero = 1;  // the chunk keeps its positions
constexpr uint32_t kTileZeroKv = 2;     // the chunk's cached K/V are all zero (separator slot)
struct ShiftTile {       // 16 bytes: one scalar load
  int32_t chunk;
  int32_t row_begin;
  int32_t row_end;
  uint32_t flags;        // kTileDeltaZero | kTileZeroKv
};
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline size_t plan_rot_offset() { return align256(sizeof(PlanHeader)); }
inline size_t plan_tile_offset(int n_chunks) {
  return plan_rot_offset() + align256(sizeof(double) * 2 * kHalf * (size_t)n_chunks);
}

// ---- top-k workspace --------------------------------------------------------
struct TopkState {
  unsigned long long prefix;  // bits of the threshold key found so far
  unsigned long long mask;    // which bits of prefix are fixed
  long long rem;              // how many of the rows matching prefix are still to take
  unsigned int done;          // blocks finished in the current pass
  unsigned int pad;
  unsigned int hist[256];
};
constexpr int kTopkRowsPerBlock = 2048;  // 256 threads x 8 rows
inline int64_t topk_blocks(int64_t n) { return (n + kTopkRowsPerBlock - 1) / kTopkRowsPerBlock; }
// State of the fused selection (one launch for all passes, grid barriers):
// three rotating byte histograms and the barrier's arrival counter.
struct TopkFused {
  unsigned int hist[3][256];
  unsigned int arrive;
  unsigned int pad[63];
};
inline size_t topk_ws_bytes(int64_t n) {
  const size_t state = sizeof(TopkState) > sizeof(TopkFused) ? sizeof(TopkState) : sizeof(TopkFused);
  return align256(state) + align256(size_t(2) * sizeof(unsigned int) * size_t(topk_blocks(n) > 0 ? topk_blocks(n) : 1));
}

// ---- launchers (return hipGetLastError() of their launches) ---------------
// v_zero non-NULL (staging): tiles of zero_kv chunks get zeros in k_dst and
// v_zero instead of a rotation.
hipError_t launch_rope_shift(const void* plan, uint64_t layout_hash, int n_chunks, int n_tiles, int n_kv_heads,
                             const uint16_t* k_src, uint16_t* k_dst, uint16_t* v_zero,
                             hipStream_t s);
hipError_t launch_kv_deviation(int64_t n_rows, int n_kv_heads, const uint16_t* k_cached,
                               const uint16_t* k_fresh, double* dev, hipStream_t s);
hipError_t launch_select_topk(const double* dev, int64_t n, int64_t k, int64_t n_append,
                              int32_t* idx_out, void* ws, hipStream_t s);
hipError_t launch_scatter_rows(const int32_t* sel, int64_t n_sel, int compact,
                               const uint16_t* k_fresh, const uint16_t* v_fresh,
                               int64_t n_fresh, uint16_t* k_cache, uint16_t* v_cache,
                               int64_t n_rows, int n_kv_heads, hipStream_t s);
// Attention; with ws of at least attention_ws_bytes(...) bytes a selection
// too small to fill the GPU runs with its key range split over several
// workgroups (partials in ws, then a combine launch).
hipError_t launch_attention(const uint16_t* q, int64_t n_q_rows, const int32_t* q_rows,
                            const int32_t* q_pos, int64_t n_sel, const uint16_t* k,
                            const uint16_t* v, int64_t n_kv, int n_q_heads, int n_kv_heads,
                            float scale, uint16_t* out, float* lse, void* ws, size_t ws_bytes,
                            hipStream_t s);
int attention_splits(int64_t n_sel, int n_q_heads, int n_kv_heads);
// Work-items of the attention launch (and of its merge launch) without a
// key-range split; a shape above 2^32 - 1 of them cannot be launched.
int64_t attention_work_items(int64_t n_sel, int n_q_heads, int n_kv_heads);
// Decoder-layer steps around the attention (layer_ops.hip).
hipError_t launch_rms_norm(const uint16_t* x, int64_t n_x_rows, const int32_t* rows, int64_t n,
                           int hidden, const uint16_t* gamma, float eps, uint16_t* out,
                           uint16_t* res_out, hipStream_t s);
hipError_t launch_qkv_rope(const uint16_t* y, int64_t n, int n_q, int n_k, int n_v,
                           const int32_t* pos, const double* freqs, uint16_t* q, uint16_t* k,
                           uint16_t* v, hipStream_t s);
hipError_t launch_swiglu(const uint16_t* gu, int64_t n, int64_t inter, uint16_t* out,
                         hipStream_t s);
size_t attention_ws_bytes(int64_t n_sel, int n_q_heads, int n_kv_heads);

// Projection GEMM of the selected rows (gemm.hip): c = a[rows] w^T (+ res).
hipError_t launch_gemm(int64_t m, int64_t n, int64_t k, const uint16_t* a, int64_t n_a_rows,
                       const int32_t* a_rows, const uint16_t* w, const uint16_t* res, uint16_t* c,
                       hipStream_t s);
// Work-items of that launch (HIP allows fewer than 2^32 per launch).
int64_t gemm_work_items(int64_t m, int64_t n);

// ---- static scratch (static_scratch.hip) -------------------------------------
// Size of the per-GPU device array behind kvc_blend_prefill_layer_noalloc
// (KVC_STATIC_SCRATCH_BYTES in kvc.h).
constexpr size_t kStaticScratchBytes = size_t(16) << 20;
// Device address of that array on the current device (looked up once per
// device with hipGetSymbolAddress, then cached).
hipError_t static_scratch(void** ptr);

}  // namespace kvc
