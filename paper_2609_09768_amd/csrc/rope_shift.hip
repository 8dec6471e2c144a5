// Step a1: RoPE re-positioning of reused chunk keys (gfx950).
//
// Paper: per-chunk caches are merged and moved to their new positions
// (Section 3.4) in more than bfloat16 precision (Section 4 setup).  Each
// row of chunk i is rotated by delta_i * f_j per pair (x[j], x[j + 64]).
//
// Bandwidth-bound: 2 bytes read + 2 bytes written per element, streamed
// with non-temporal loads and stores.  A unit is 8 pairs of one head row
// (16 bytes from each half of the head vector); a workgroup of 256 threads
// owns a tile of up to 1024 units of one chunk, four per thread, and issues
// all eight loads of a thread before the first rotation, so that many short
// workgroups keep enough bytes in flight (measured: the same traffic with
// 512-thread workgroups over 64-row tiles and one unit per thread in flight
// reached 4.9 TB/s on cold buffers, these tiles 5.9).  Thread t always
// handles the pairs 8*(t%8) .. 8*(t%8)+7 (the 256-thread stride keeps t%8
// fixed), so the chunk's cos/sin live in registers.
//
// Arithmetic is float64 with the table computed in float64 on the host:
// r = x cos - y sin as fma(x, cos, -(y sin)), then r is rounded once to
// bfloat16 (nearest, ties to even).  The rounding uses the hardware
// float64 -> float32 conversion and the packed float32 -> bfloat16
// conversion, both round to nearest even.  Rounding twice differs from
// rounding once only where the float32 value is exactly halfway between two
// bfloat16 values while r is not (then the second rounding's tie-break may
// go the wrong way); such a float32 is moved one unit towards r before the
// second rounding, which then goes to r's side.  float32 keeps 16 more bits
// than bfloat16, so every other float32 lies strictly on one side of the
// midpoint that r lies on, and the result is r correctly rounded, also in
// the subnormal range (gradual underflow) and to infinity past the largest
// bfloat16.  Such midpoints are rare (about 1 in 65,536 values), so the
// repair is one branch per four pairs that is almost never taken.
//
// The same kernel serves the transfer stage of the layer-wise pipeline
// (Section 3.4): given the V cache, it writes zeros into both caches for
// the tiles of separator chunks, whose cached K/V are zero (Section 3.1),
// and adjusts the other tiles' keys in place.
#include "kvc_internal.h"
#include "bf16_util.h"

namespace kvc {
namespace {

constexpr int kThreads = 256;
constexpr int kUnits = kShiftTileUnits / kThreads;  // units per thread, loaded together

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two float32 values to packed bfloat16, nearest with ties to even.
__device__ __forceinline__ uint32_t pack_bf16_rne(uint32_t a, uint32_t b) {
  const f32x2_t v = {__uint_as_float(a), __uint_as_float(b)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// float32 bits on a bfloat16 midpoint (low 16 bits 0x8000)
__device__ __forceinline__ bool on_midpoint(uint32_t f) { return (f & 0xFFFFu) == 0x8000u; }

// Move a float32 that sits on a bfloat16 midpoint one unit towards the
// float64 value r it was rounded from (nothing if it equals r).
__device__ __forceinline__ uint32_t off_midpoint(uint32_t f, double r) {
  if (!on_midpoint(f)) return f;
  const double d = (double)__uint_as_float(f);
  if (d == r) return f;
  return fabs(d) > fabs(r) ? f - 1u : f + 1u;  // magnitude down or up, sign kept
}

// Rotates the 8 pairs of a unit and rounds them, 4 pairs at a time: fewer
// live registers, so that with one tile per workgroup (no loop) the kernel
// fits 96 registers and five waves per SIMD instead of four (2-3 % faster
// on cold buffers).
__device__ __forceinline__ void rotate8(const uint4& a, const uint4& b, const double* c,
                                        const double* s, uint4& oa, uint4& ob) {
  uint32_t pa[4], pb[4];
#pragma unroll
  for (int g0 = 0; g0 < 8; g0 += 4) {
    double ra[4], rb[4];
    uint32_t fa[4], fb[4];
    int mid = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = g0 + i;
      const double x = (double)bf16x8_elem(a, e);
      const double y = (double)bf16x8_elem(b, e);
      ra[i] = fma(x, c[e], -(y * s[e]));
      rb[i] = fma(y, c[e], x * s[e]);
      fa[i] = __float_as_uint((float)ra[i]);
      fb[i] = __float_as_uint((float)rb[i]);
      mid |= (int)on_midpoint(fa[i]) | (int)on_midpoint(fb[i]);
    }
    if (__builtin_expect(mid, 0)) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        fa[i] = off_midpoint(fa[i], ra[i]);
        fb[i] = off_midpoint(fb[i], rb[i]);
      }
    }
    pa[g0 / 2] = pack_bf16_rne(fa[0], fa[1]);
    pa[g0 / 2 + 1] = pack_bf16_rne(fa[2], fa[3]);
    pb[g0 / 2] = pack_bf16_rne(fb[0], fb[1]);
    pb[g0 / 2 + 1] = pack_bf16_rne(fb[2], fb[3]);
  }
  oa = make_uint4(pa[0], pa[1], pa[2], pa[3]);
  ob = make_uint4(pb[0], pb[1], pb[2], pb[3]);
}

// One tile of rows of one chunk (the whole workgroup).
__device__ __forceinline__ void shift_tile(const ShiftTile& t, const double2* __restrict__ rot_table,
                                           int n_kv_heads, const uint16_t* src, uint16_t* dst,
                                           uint16_t* v_zero, int in_place) {
  const int tid = threadIdx.x;
  const int64_t row_elems = (int64_t)n_kv_heads * kHeadDim;
  if (v_zero && (t.flags & kTileZeroKv)) {
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
  if (in_place && (t.flags & kTileDeltaZero)) return;

  const int jg = tid & 7;  // pairs 8*jg .. 8*jg+7
  const uint16_t* sb = src + (int64_t)t.row_begin * row_elems;
  uint16_t* db = dst + (int64_t)t.row_begin * row_elems;
  // unit u = (row, head, jg): 8 pairs = 16 bytes from each half; the host
  // makes tiles of at most kShiftTileUnits units
  const int units = (t.row_end - t.row_begin) * n_kv_heads * 8;
  uint4 a[kUnits], b[kUnits];
  auto load = [&](int u0) {
#pragma unroll
    for (int k = 0; k < kUnits; ++k) {
      const int u = u0 + tid + k * kThreads;
      if (u < units) {
        const int64_t off = (int64_t)(u >> 3) * kHeadDim + jg * 8;
        a[k] = load_nt(sb + off);
        b[k] = load_nt(sb + off + kHalf);
      }
    }
  };
  double c[8], s[8];
  auto rotate_store = [&](int u0) {
#pragma unroll
    for (int k = 0; k < kUnits; ++k) {
      const int u = u0 + tid + k * kThreads;
      if (u < units) {
        const int64_t off = (int64_t)(u >> 3) * kHeadDim + jg * 8;
        uint4 oa, ob;
        rotate8(a[k], b[k], c, s, oa, ob);
        store_nt(db + off, oa);
        store_nt(db + off + kHalf, ob);
      }
    }
  };
  load(0);  // the data first, then the chunk's table, which hits in cache
  const double2* rot = rot_table + (size_t)t.chunk * kHalf + jg * 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double2 cs = rot[e];
    c[e] = cs.x;
    s[e] = cs.y;
  }
  rotate_store(0);
}

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(5, 8))) void rope_shift_kernel(const PlanHeader* __restrict__ hdr,
                                                              const ShiftTile* __restrict__ tiles,
                                                              uint64_t layout_hash, int n_kv_heads,
                                                              const uint16_t* src,  // may equal dst
                                                              uint16_t* dst,
                                                              uint16_t* v_zero,  // staging only
                                                              int in_place, const double2* __restrict__ rot_table) {
  // one tile per workgroup (the host launches tiles in batches of at most
  // kMaxGrid); one test of all its fields and the hash makes the loads
  // issue together, before any wait.  The host already refused plans of
  // another layout: the hash is a backstop for a plan buffer overwritten
  // since its descriptor was made (the tile then lies within the buffer but
  // is not used).
  const ShiftTile t = tiles[blockIdx.x];
  if ((hdr->layout_hash != layout_hash) | (t.row_end < t.row_begin) | (t.chunk < 0) |
      (t.flags > (kTileDeltaZero | kTileZeroKv)))
    return;
  shift_tile(t, rot_table, n_kv_heads, src, dst, v_zero, in_place);
}

}  // namespace

hipError_t launch_rope_shift(const void* plan, uint64_t layout_hash, int n_chunks, int n_tiles, int n_kv_heads,
                             const uint16_t* k_src, uint16_t* k_dst, uint16_t* v_zero,
                             hipStream_t s) {
  const char* base = static_cast<const char*>(plan);
  const ShiftTile* tiles = reinterpret_cast<const ShiftTile*>(base + plan_tile_offset(n_chunks));
  for (int64_t t0 = 0; t0 < n_tiles; t0 += kMaxGrid) {
    const unsigned grid = (unsigned)std::min<int64_t>(n_tiles - t0, kMaxGrid);
    hipLaunchKernelGGL(rope_shift_kernel, dim3(grid), dim3(kThreads), 0, s,
                       reinterpret_cast<const PlanHeader*>(base), tiles + t0, layout_hash, n_kv_heads, k_src,
                       k_dst, v_zero, (int)(k_src == k_dst),
                       reinterpret_cast<const double2*>(base + plan_rot_offset()));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace kvc
