// Step a1: RoPE re-positioning of reused chunk keys (gfx950).
//
// Paper: per-chunk caches are merged and moved to their new positions
// (Section 3.4) in more than bfloat16 precision (Section 4 setup).  Each
// row of chunk i is rotated by delta_i * f_j per pair (x[j], x[j + 64]).
//
// Bandwidth-bound: 2 bytes read + 2 bytes written per element, streamed
// with non-temporal loads and stores.  One workgroup (8 waves) owns a tile
// of up to 64 rows of one chunk (512 head rows: longer tiles with fewer than
// 8 kv heads; 16 rows in requests of fewer than 16,384 reused rows, so that
// they still spread over the CUs), so the chunk's cos/sin live in registers:
// thread t always handles the pairs 8*(t%8) .. 8*(t%8)+7 (the 512-thread
// stride keeps t%8 fixed), loading 16 bytes from each half of the head
// vector.  Arithmetic is float64 with the table computed in float64 on the
// host; the result is rounded once to bfloat16, so it equals the correctly
// rounded rotation.
//
// The same kernel serves the transfer stage of the layer-wise pipeline
// (Section 3.4): given the V cache, it writes zeros into both caches for
// the tiles of separator chunks, whose cached K/V are zero (Section 3.1),
// and adjusts the other tiles' keys in place.
#include "kvc_internal.h"
#include "bf16_util.h"

namespace kvc {
namespace {

constexpr int kThreads = 512;  // 8 waves per 64-row tile (measured 10 % faster than 4)
constexpr int kUnroll = 1;  // fewer registers, more waves in flight (measured best)

__device__ __forceinline__ void rotate8(const uint4& a, const uint4& b, const double* c,
                                        const double* s, uint4& oa, uint4& ob) {
  uint32_t ra[8], rb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double x = (double)bf16x8_elem(a, e);
    const double y = (double)bf16x8_elem(b, e);
    ra[e] = f64_to_bf16_rne(fma(x, c[e], -(y * s[e])));
    rb[e] = f64_to_bf16_rne(fma(y, c[e], x * s[e]));
  }
  oa = make_uint4(ra[0] | (ra[1] << 16), ra[2] | (ra[3] << 16), ra[4] | (ra[5] << 16),
                  ra[6] | (ra[7] << 16));
  ob = make_uint4(rb[0] | (rb[1] << 16), rb[2] | (rb[3] << 16), rb[4] | (rb[5] << 16),
                  rb[6] | (rb[7] << 16));
}

// One tile of rows of one chunk (the whole workgroup).
__device__ __forceinline__ void shift_tile(const char* __restrict__ plan, const PlanHeader* hdr, int tile,
                                           int n_kv_heads, const uint16_t* src, uint16_t* dst,
                                           uint16_t* v_zero, int in_place) {
  const ShiftTile t = reinterpret_cast<const ShiftTile*>(plan + hdr->tile_offset)[tile];
  const int tid = threadIdx.x;
  const int64_t row_elems = (int64_t)n_kv_heads * kHeadDim;
  if (v_zero && t.zero_kv) {
    // separator slot while staging: its cache is zero, nothing to rotate
    const int64_t n16 = (int64_t)(t.row_end - t.row_begin) * row_elems / 8;
    uint4* kz = reinterpret_cast<uint4*>(dst + (int64_t)t.row_begin * row_elems);
    uint4* vz = reinterpret_cast<uint4*>(v_zero + (int64_t)t.row_begin * row_elems);
    for (int64_t i = tid; i < n16; i += kThreads) {
      kz[i] = make_uint4(0, 0, 0, 0);
      vz[i] = make_uint4(0, 0, 0, 0);
    }
    return;
  }
  if (in_place && t.delta_zero) return;

  const int jg = tid & 7;  // pairs 8*jg .. 8*jg+7
  const double2* rot =
      reinterpret_cast<const double2*>(plan + hdr->rot_offset) + (size_t)t.chunk * kHalf + jg * 8;
  double c[8], s[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double2 cs = rot[e];
    c[e] = cs.x;
    s[e] = cs.y;
  }

  const uint16_t* sb = src + (int64_t)t.row_begin * row_elems;
  uint16_t* db = dst + (int64_t)t.row_begin * row_elems;
  // unit u = (row, head, jg): 8 pairs = 16 bytes from each half
  const int units = (t.row_end - t.row_begin) * n_kv_heads * 8;
  for (int u0 = tid; u0 < units; u0 += kThreads * kUnroll) {
    uint4 a[kUnroll], b[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const int u = u0 + k * kThreads;
      if (u < units) {
        const int64_t off = (int64_t)(u >> 3) * kHeadDim + jg * 8;
        a[k] = load_nt(sb + off);
        b[k] = load_nt(sb + off + kHalf);
      }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const int u = u0 + k * kThreads;
      if (u < units) {
        const int64_t off = (int64_t)(u >> 3) * kHeadDim + jg * 8;
        uint4 oa, ob;
        rotate8(a[k], b[k], c, s, oa, ob);
        store_nt(db + off, oa);
        store_nt(db + off + kHalf, ob);
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void rope_shift_kernel(const char* __restrict__ plan,
                                                              uint64_t layout_hash, int n_kv_heads,
                                                              const uint16_t* src,  // may equal dst
                                                              uint16_t* dst,
                                                              uint16_t* v_zero,  // staging only
                                                              int in_place) {
  const PlanHeader* hdr = reinterpret_cast<const PlanHeader*>(plan);
  // the host already refused plans of another layout; this is a backstop
  // for a plan buffer overwritten since its descriptor was made
  if (hdr->layout_hash != layout_hash) return;
  for (int tile = blockIdx.x; tile < hdr->n_tiles; tile += gridDim.x)
    shift_tile(plan, hdr, tile, n_kv_heads, src, dst, v_zero, in_place);
}

}  // namespace

hipError_t launch_rope_shift(const void* plan, uint64_t layout_hash, int n_tiles, int n_kv_heads,
                             const uint16_t* k_src, uint16_t* k_dst, uint16_t* v_zero,
                             hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  const unsigned grid = (unsigned)std::min<int64_t>(n_tiles, kMaxGrid);
  hipLaunchKernelGGL(rope_shift_kernel, dim3(grid), dim3(kThreads), 0, s,
                     static_cast<const char*>(plan), layout_hash, n_kv_heads, k_src, k_dst, v_zero,
                     (int)(k_src == k_dst));
  return hipGetLastError();
}

}  // namespace kvc
