// Decoder-layer steps around the attention of the selected tokens (gfx950).
//
// The models the paper evaluates (Section 4.1) are pre-norm decoder layers;
// under selective recompute only the selected tokens pass through a layer
// (Section 3.4; Section 4 setup), so these steps run on the selected rows:
//   * RMS normalisation, optionally gathering the rows it normalises;
//   * the split of the fused Q/K/V projection output into Q, K and V with
//     RoPE applied to Q and K at each token's position;
//   * the gated SiLU of the feed-forward block.
// The projections themselves are plain GEMMs left to a GEMM library.
//
// All three kernels are bound by HBM bandwidth: each reads its input once
// and writes its output once, in 16-byte vectors.  Outputs use ordinary
// stores, since the next GEMM reads them right away.
#include "kvc_internal.h"
#include "bf16_util.h"

namespace kvc {
namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats to two bfloat16 (round to nearest even), packed low-first.
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ float lo16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// ---- RMS normalisation ------------------------------------------------------
// One wave per row; lane l holds 16-byte chunks l, l + 64, ... of the row in
// registers (NC of them), so the row is read from HBM once.
constexpr int kNormWaves = 4;

template <int NC>
__global__ __launch_bounds__(64 * kNormWaves) void rms_norm_kernel(
    const uint16_t* __restrict__ x, int64_t n_x_rows, const int32_t* __restrict__ rows, int64_t n,
    int hidden, const uint16_t* __restrict__ gamma, float eps, uint16_t* __restrict__ out,
    uint16_t* __restrict__ res_out) {
  const int lane = threadIdx.x & 63;
  for (int64_t i = (int64_t)blockIdx.x * kNormWaves + (threadIdx.x >> 6); i < n;
       i += (int64_t)gridDim.x * kNormWaves) {
  const int64_t r = rows ? (int64_t)rows[i] : i;
  const bool valid = r >= 0 && r < n_x_rows;
  const int chunks = hidden >> 3;
  const uint4* src = reinterpret_cast<const uint4*>(x + (valid ? r : 0) * (int64_t)hidden);
  uint4 v[NC];
  float ss = 0.0f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int ch = lane + 64 * c;
    v[c] = (valid && ch < chunks) ? load_nt(src + ch) : make_uint4(0, 0, 0, 0);
    const uint32_t w[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = lo16(w[e]), b = hi16(w[e]);
      ss = fmaf(a, a, ss);
      ss = fmaf(b, b, ss);
    }
  }
  ss = wave_sum(ss);
  const float inv = valid ? 1.0f / sqrtf(ss / (float)hidden + eps) : 0.0f;
  uint4* dst = reinterpret_cast<uint4*>(out + i * (int64_t)hidden);
  uint4* res = res_out ? reinterpret_cast<uint4*>(res_out + i * (int64_t)hidden) : nullptr;
  const uint4* g4 = reinterpret_cast<const uint4*>(gamma);
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int ch = lane + 64 * c;
    if (ch >= chunks) break;
    const uint4 g = g4[ch];
    const uint32_t w[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
    const uint32_t gw[4] = {g.x, g.y, g.z, g.w};
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[e] = pack2(lo16(w[e]) * inv * lo16(gw[e]), hi16(w[e]) * inv * hi16(gw[e]));
    dst[ch] = make_uint4(o[0], o[1], o[2], o[3]);
    if (res) res[ch] = v[c];
  }
  }
}

// ---- Q/K/V split with RoPE --------------------------------------------------
// One wave per row.  Lane l reduces the angle p * f_l modulo 2 pi in
// float64 (with 2 pi rounded to float64, the reduced angle is off by
// turns * 2.4e-16 rad: below 1e-10 rad up to positions of about 2.6e6 at
// f_0 = 1, and 8e-8 rad at 2^31), takes its
// sine and cosine in float32 and hands them to the lanes that need them;
// for the rotated heads lane l owns pairs 8 (l % 8) .. 8 (l % 8) + 7 of
// heads l / 8, l / 8 + 8, ..., loading 16 bytes from each half of the head.
// The rotation is float32, rounded once to bfloat16: within half a
// bfloat16 ulp of the exact value plus a few float32 ulps of the pair's
// magnitude.  (The cached keys' position adjustment stays in float64; this
// is the model's own RoPE on fresh queries and keys.)  The V heads are
// copied first and each lane's rotated heads (up to six per batch: 48
// heads per wave) are requested before the angle work, so that with few
// heads per row the angle's latency overlaps the loads and with many heads
// enough loads are in flight.
constexpr int kRopeWaves = 4;
constexpr int kRopeBatch = 6;  // heads per lane loaded at once

struct QkvRopeArgs {
  const uint16_t* y;
  int64_t n;
  int n_q, n_k, n_v;
  const int32_t* pos;
  uint16_t* q;
  uint16_t* k;
  uint16_t* v;
  double f[kHalf];
};

__device__ __forceinline__ void rotate8_f32(const uint4& a, const uint4& b, const float* c,
                                            const float* s, uint4& oa, uint4& ob) {
  const uint32_t wa[4] = {a.x, a.y, a.z, a.w};
  const uint32_t wb[4] = {b.x, b.y, b.z, b.w};
  uint32_t ra[4], rb[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float x0 = lo16(wa[e]), x1 = hi16(wa[e]);
    const float y0 = lo16(wb[e]), y1 = hi16(wb[e]);
    const float c0 = c[2 * e], c1 = c[2 * e + 1], s0 = s[2 * e], s1 = s[2 * e + 1];
    ra[e] = pack2(fmaf(x0, c0, -(y0 * s0)), fmaf(x1, c1, -(y1 * s1)));
    rb[e] = pack2(fmaf(y0, c0, x0 * s0), fmaf(y1, c1, x1 * s1));
  }
  oa = make_uint4(ra[0], ra[1], ra[2], ra[3]);
  ob = make_uint4(rb[0], rb[1], rb[2], rb[3]);
}

__global__ __launch_bounds__(64 * kRopeWaves) void qkv_rope_kernel(const QkvRopeArgs A) {
  const int lane = threadIdx.x & 63;
  // one row per wave at a time; the row index is the same in every lane, so
  // the shuffles below always have the whole wave
  for (int64_t i = (int64_t)blockIdx.x * kRopeWaves + (threadIdx.x >> 6); i < A.n;
       i += (int64_t)gridDim.x * kRopeWaves) {
  const int n_rot = A.n_q + A.n_k;
  const int heads = n_rot + A.n_v;
  const uint16_t* yr = A.y + i * (int64_t)heads * kHeadDim;
  const int jg = lane & 7;

  // V heads: copied
  const int vch = A.n_v * (kHeadDim / 8);
  const uint4* vs = reinterpret_cast<const uint4*>(yr + n_rot * kHeadDim);
  uint4* vd = reinterpret_cast<uint4*>(A.v + i * A.n_v * kHeadDim);
  for (int c = lane; c < vch; c += 64) vd[c] = load_nt(vs + c);

  float c[8], s[8];
  bool have_cs = false;
  // rotated heads, kRopeBatch per lane at a time (48 heads in one batch)
  // the loop bound is the same for every lane: the shuffles below need the
  // whole wave
  for (int base = 0; base < n_rot; base += 8 * kRopeBatch) {
    const int h0 = base + (lane >> 3);
    uint4 a[kRopeBatch], b[kRopeBatch];
#pragma unroll
    for (int t = 0; t < kRopeBatch; ++t) {
      const int h = h0 + 8 * t;
      if (h < n_rot) {
        a[t] = load_nt(yr + h * kHeadDim + 8 * jg);
        b[t] = load_nt(yr + h * kHeadDim + kHalf + 8 * jg);
      }
    }
    if (!have_cs) {
      // angle work after the first loads are out, so their latencies overlap
      const double p = A.pos ? (double)A.pos[i] : (double)i;
      const double ang = p * A.f[lane];
      const double turns = rint(ang * 0.15915494309189535);  // 1 / (2 pi)
      const float r = (float)fma(-turns, 6.283185307179586, ang);
      float s_l, c_l;
      sincosf(r, &s_l, &c_l);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        c[e] = __shfl(c_l, 8 * jg + e, 64);
        s[e] = __shfl(s_l, 8 * jg + e, 64);
      }
      have_cs = true;
    }
#pragma unroll
    for (int t = 0; t < kRopeBatch; ++t) {
      const int h = h0 + 8 * t;
      if (h < n_rot) {
        uint16_t* dst = h < A.n_q ? A.q + (i * A.n_q + h) * kHeadDim
                                  : A.k + (i * A.n_k + (h - A.n_q)) * kHeadDim;
        uint4 oa, ob;
        rotate8_f32(a[t], b[t], c, s, oa, ob);
        *reinterpret_cast<uint4*>(dst + 8 * jg) = oa;
        *reinterpret_cast<uint4*>(dst + kHalf + 8 * jg) = ob;
      }
    }
  }
  }
}

// ---- gated SiLU -------------------------------------------------------------
// Thread per 8 outputs; a block covers 256 x 8 outputs of one row.
constexpr int kGluThreads = 256;

__global__ __launch_bounds__(kGluThreads) void swiglu_kernel(const uint16_t* __restrict__ gu,
                                                             int64_t inter, int blocks_per_row,
                                                             int64_t n_units, uint16_t* __restrict__ out) {
  for (int64_t b = blockIdx.x; b < n_units; b += gridDim.x) {
  const int64_t row = b / blocks_per_row;
  const int64_t u = (b % blocks_per_row) * kGluThreads + threadIdx.x;
  if (u * 8 >= inter) continue;
  const uint16_t* gr = gu + row * 2 * inter;
  const uint4 g = load_nt(gr + u * 8);
  const uint4 up = load_nt(gr + inter + u * 8);
  const uint32_t gw[4] = {g.x, g.y, g.z, g.w};
  const uint32_t uw[4] = {up.x, up.y, up.z, up.w};
  uint32_t o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float g0 = lo16(gw[e]), g1 = hi16(gw[e]);
    // silu(g) = g / (1 + e^-g); e^-g = inf for very negative g gives -0
    const float s0 = g0 * __builtin_amdgcn_rcpf(1.0f + __expf(-g0));
    const float s1 = g1 * __builtin_amdgcn_rcpf(1.0f + __expf(-g1));
    o[e] = pack2(s0 * lo16(uw[e]), s1 * hi16(uw[e]));
  }
  *reinterpret_cast<uint4*>(out + row * inter + u * 8) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

}  // namespace

hipError_t launch_rms_norm(const uint16_t* x, int64_t n_x_rows, const int32_t* rows, int64_t n,
                           int hidden, const uint16_t* gamma, float eps, uint16_t* out,
                           uint16_t* res_out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const dim3 grid((unsigned)std::min<int64_t>((n + kNormWaves - 1) / kNormWaves, kMaxGrid)), block(64 * kNormWaves);
  const int nc = (hidden / 8 + 63) / 64;
#define KVC_NORM(NC)                                                                        \
  hipLaunchKernelGGL(rms_norm_kernel<NC>, grid, block, 0, s, x, n_x_rows, rows, n, hidden, \
                     gamma, eps, out, res_out)
  if (nc <= 1) KVC_NORM(1);
  else if (nc <= 2) KVC_NORM(2);
  else if (nc <= 4) KVC_NORM(4);
  else if (nc <= 8) KVC_NORM(8);
  else if (nc <= 16) KVC_NORM(16);
  else KVC_NORM(32);
#undef KVC_NORM
  return hipGetLastError();
}

hipError_t launch_qkv_rope(const uint16_t* y, int64_t n, int n_q, int n_k, int n_v,
                           const int32_t* pos, const double* freqs, uint16_t* q, uint16_t* k,
                           uint16_t* v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  QkvRopeArgs A;
  A.y = y;
  A.n = n;
  A.n_q = n_q;
  A.n_k = n_k;
  A.n_v = n_v;
  A.pos = pos;
  A.q = q;
  A.k = k;
  A.v = v;
  for (int j = 0; j < kHalf; ++j) A.f[j] = freqs[j];
  hipLaunchKernelGGL(qkv_rope_kernel, dim3((unsigned)std::min<int64_t>((n + kRopeWaves - 1) / kRopeWaves, kMaxGrid)),
                     dim3(64 * kRopeWaves), 0, s, A);
  return hipGetLastError();
}

hipError_t launch_swiglu(const uint16_t* gu, int64_t n, int64_t inter, uint16_t* out,
                         hipStream_t s) {
  if (n <= 0 || inter <= 0) return hipSuccess;
  const int64_t bpr = (inter / 8 + kGluThreads - 1) / kGluThreads;
  const int64_t units = n * bpr;
  hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)std::min<int64_t>(units, kMaxGrid)), dim3(kGluThreads), 0, s,
                     gu, inter, (int)bpr, units, out);
  return hipGetLastError();
}

}  // namespace kvc
