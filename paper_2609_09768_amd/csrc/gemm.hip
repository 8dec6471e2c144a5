// Projections of the decoder layer on the selected tokens (gfx950).
//
// Paper: under selective recompute only the selected tokens pass through a
// layer (Section 3.4; Section 4 setup), so every projection of the layer
// (fused Q/K/V, O, gate/up, down) multiplies the selected rows' activations
// by a weight matrix:
//   c[i, j] = sum_e a[r_i, e] * w[j, e]  (+ residual[i, j]),
// with r_i = a_rows[i] (a gather of the selected rows) or i, and w in the
// [out, in] layout of the model's linear layers.  The residual addition of
// the O and down projections is fused into the store.
//
// A dense contraction, so it runs on the matrix cores:
// v_mfma_f32_16x16x32_bf16, float32 accumulation, rounded once to bf16 after
// the residual is added in float32.  (The 16x16 shape moves half the
// accumulator bytes per FLOP of the 32x32 one; on this power-limited chip
// it ran 8-13 % faster on the layer's shapes, with identical results.)
// - A workgroup (8 waves, two per SIMD) computes a 256 x 256 tile of c over
//   the whole K, in slices of 64: each slice of the 256 activation rows and
//   of the 256 weight rows goes from memory straight into LDS (global loads
//   with an LDS destination: per-lane 64-bit addresses, so the row gather
//   costs nothing; no registers, no VALU), double-buffered, one barrier per
//   slice.
// - LDS rows are 128 bytes (64 bf16 of K); the 16-byte piece p of row r is
//   stored at p ^ ((r >> 1) & 7), so the operand reads (16 lanes: 16
//   consecutive rows, one piece) fall in 16 distinct bank groups.
// - Each wave owns 64 output columns x 128 output rows (4 x 8 tiles of
//   16 x 16).  The MFMA computes each tile transposed (weight rows as the
//   first operand), so a lane ends with one output row and four consecutive
//   columns per tile: 8-byte stores, and 8-byte residual loads.  The
//   fragments of the second 32-wide K step of a slice are read from LDS
//   between the MFMAs of the first, fenced so the compiler keeps the
//   interleave.
// - Workgroup ids are dispatched round-robin over the 8 XCDs; they are
//   renumbered so that each XCD gets a contiguous range of tiles, walked in
//   groups of 4 row tiles, so workgroups that share activation or weight
//   slices tend to share an L2.
#include "kvc_internal.h"

namespace kvc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kBM = 256;            // output rows (activation rows) per workgroup
constexpr int kBN = 256;            // output columns (weight rows) per workgroup
constexpr int kBK = 64;             // K per slice
constexpr int kRowHalfs = kBK;      // bf16 per LDS row
constexpr int kSlice = kBM * kBK;   // bf16 per operand slice (32 KB)
constexpr int kGroupM = 4;          // row tiles per group of the tile walk
constexpr int kXcds = 8;
// s_waitcnt immediate (gfx9 encoding): vector-memory and LDS counts 0
constexpr int kWaitVm0 = 0 | (7 << 4);

struct GemmParams {
  const uint16_t* a;
  const int32_t* a_rows;
  long long n_a_rows;
  const uint16_t* w;
  const uint16_t* res;
  uint16_t* c;
  long long m, n, k;
  int tiles_m, tiles_n;
};

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& u) { return __builtin_bit_cast(bf16x8, u); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Workgroup id -> (row tile, column tile).  Ids go round-robin over the
// XCDs; v renumbers them so each XCD holds a contiguous range of v (a
// bijection on [0, T)), and v walks groups of kGroupM row tiles column by
// column.
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
  const int per = total / kXcds, rem = total % kXcds;
  const int x = bid % kXcds, slot = bid / kXcds;
  const int v = x * per + min(x, rem) + slot;
  const int group = v / (kGroupM * tiles_n);
  const int first = group * kGroupM;
  const int gm = min(kGroupM, tiles_m - first);
  const int in_group = v - group * kGroupM * tiles_n;
  tm = first + in_group % gm;
  tn = in_group / gm;
}

__global__ __launch_bounds__(kThreads) void gemm_kernel(const GemmParams P) {
  // one array per buffer, so the compiler's wait-count pass can tell the
  // loads into one buffer from the reads of the other
  __shared__ __attribute__((aligned(16))) uint16_t A0[kSlice], A1[kSlice];
  __shared__ __attribute__((aligned(16))) uint16_t W0[kSlice], W1[kSlice];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int tm, tn;
  tile_of((int)blockIdx.x, P.tiles_m, P.tiles_n, tm, tn);
  const long long m0 = (long long)tm * kBM, n0 = (long long)tn * kBN;
  const int wn = wave & 3;   // 64-column strip of the tile
  const int wm = wave >> 2;  // 128-row strip of the tile

  // Loads: wave w fills rows 32 w .. 32 w + 31 of both slices, 8 rows per
  // instruction; lane l writes 16 bytes at row 32 w + 8 j + l / 8, slot l % 8,
  // which holds piece (l % 8) ^ ((row >> 1) & 7) of that row.  Rows past m
  // or n read the last valid row (their results are not stored).
  const uint16_t* a_src[4];
  const uint16_t* w_src[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = 32 * wave + 8 * j + (lane >> 3);
    const int piece = (lane & 7) ^ ((row >> 1) & 7);
    long long am = m0 + row;
    if (am >= P.m) am = P.m - 1;
    long long ar = P.a_rows ? (long long)P.a_rows[am] : am;
    if (ar < 0 || ar >= P.n_a_rows) ar = 0;  // an invalid gather entry: its row is zeroed at the store
    a_src[j] = P.a + ar * P.k + 8 * piece;
    long long wr = n0 + row;
    if (wr >= P.n) wr = P.n - 1;
    w_src[j] = P.w + wr * P.k + 8 * piece;
  }
  auto load_slice = [&](int t, uint16_t* as_, uint16_t* ws_) __attribute__((always_inline)) {
    const long long koff = (long long)t * kBK;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int lrow = 32 * wave + 8 * j;
      __builtin_amdgcn_global_load_lds((const void*)(a_src[j] + koff), (lds_void*)(as_ + lrow * kRowHalfs), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(w_src[j] + koff), (lds_void*)(ws_ + lrow * kRowHalfs), 16, 0, 0);
    }
  };

  // Operand reads (16x16x32): lane l reads row l % 16 of a 16-row block,
  // K piece 4 ks + l / 16 (8 bf16), from its swizzled slot.
  const int rl = lane & 15, q = lane >> 4, sw = (rl >> 1) & 7;
  int rd[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) rd[ks] = rl * kRowHalfs + 8 * ((4 * ks + q) ^ sw);
  constexpr int NT = 4, MT = 8;  // 16 x 16 tiles per wave: 64 columns x 128 rows
  f32x4 acc[NT][MT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto frag = [&](const uint16_t* base, int row0, int ks) __attribute__((always_inline)) {
    return as_bf16x8(*reinterpret_cast<const uint4*>(base + row0 * kRowHalfs + rd[ks]));
  };

  // One step: wait for slice t (this wave's loads, then everyone's at the
  // barrier, which also means every wave is done with slice t - 1), start
  // the loads of slice t + 1 into the other buffer, multiply slice t: the
  // MFMAs of its first K step, each followed by one read of the second
  // step's fragments (12 of them over the first 24 MFMAs), then the MFMAs of
  // the second step.
  const int nk = (int)(P.k / kBK);
  auto step = [&](int t, const uint16_t* as, const uint16_t* ws, uint16_t* as_next, uint16_t* ws_next)
      __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
    if (t + 1 < nk) load_slice(t + 1, as_next, ws_next);
    bf16x8 fw[2][NT], fa[2][MT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) fw[0][nt] = frag(ws, wn * 64 + nt * 16, 0);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) fa[0][mt] = frag(as, wm * 128 + mt * 16, 0);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int i = 0; i < NT * MT; ++i) {
        const int nt = i / MT, mt = i % MT;
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[ks][nt], fa[ks][mt], acc[nt][mt], 0, 0, 0);
        if (ks == 0 && (i & 1) && i / 2 < NT + MT) {
          const int j = i / 2;
          if (j < NT) fw[1][j] = frag(ws, wn * 64 + j * 16, 1);
          else fa[1][j - NT] = frag(as, wm * 128 + (j - NT) * 16, 1);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  load_slice(0, A0, W0);
  for (int t = 0; t < nk; t += 2) {
    step(t, A0, W0, A1, W1);
    if (t + 1 < nk) step(t + 1, A1, W1, A0, W0);
  }

  // Store: tile (nt, mt) gives lane l output row m0 + wm 128 + mt 16 + l % 16
  // and columns n0 + wn 64 + nt 16 + 4 (l / 16) + 0..3.
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const long long m = m0 + wm * 128 + mt * 16 + rl;
    if (m >= P.m) continue;
    bool zero = false;
    if (P.a_rows) {
      const long long ar = P.a_rows[m];
      zero = ar < 0 || ar >= P.n_a_rows;
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const long long n = n0 + wn * 64 + nt * 16 + 4 * q;
      if (n >= P.n) continue;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = zero ? 0.f : acc[nt][mt][e];
      if (P.res) {
        const uint2 r2 = *reinterpret_cast<const uint2*>(P.res + m * P.n + n);
        v[0] += __uint_as_float(r2.x << 16);
        v[1] += __uint_as_float(r2.x & 0xFFFF0000u);
        v[2] += __uint_as_float(r2.y << 16);
        v[3] += __uint_as_float(r2.y & 0xFFFF0000u);
      }
      *reinterpret_cast<uint2*>(P.c + m * P.n + n) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
    }
  }
}

}  // namespace

int64_t gemm_work_items(int64_t m, int64_t n) {
  if (m <= 0 || n <= 0) return 0;
  return ((m + kBM - 1) / kBM) * ((n + kBN - 1) / kBN) * kThreads;
}

hipError_t launch_gemm(int64_t m, int64_t n, int64_t k, const uint16_t* a, int64_t n_a_rows,
                       const int32_t* a_rows, const uint16_t* w, const uint16_t* res, uint16_t* c,
                       hipStream_t s) {
  if (m <= 0 || n <= 0) return hipSuccess;
  GemmParams P;
  P.a = a;
  P.a_rows = a_rows;
  P.n_a_rows = n_a_rows;
  P.w = w;
  P.res = res;
  P.c = c;
  P.m = m;
  P.n = n;
  P.k = k;
  P.tiles_m = (int)((m + kBM - 1) / kBM);
  P.tiles_n = (int)((n + kBN - 1) / kBN);
  hipLaunchKernelGGL(gemm_kernel, dim3((unsigned)P.tiles_m * (unsigned)P.tiles_n), dim3(kThreads), 0, s, P);
  return hipGetLastError();
}

}  // namespace kvc
