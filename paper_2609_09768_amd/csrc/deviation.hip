// Step a2: per-token squared key deviation at the check layer (gfx950).
//
// Paper: CacheBlend ranks tokens by how much their cached keys differ from
// keys recomputed with full attention (Section 2), measured as squared
// differences of the key entries (Section 3.2).  Here
//   d[r] = sum_{h,e} (k_fresh[r,h,e] - k_cached[r,h,e])^2.
//
// Bandwidth-bound (2 x 2 bytes read per element).  One wave owns a row
// (rows of one or two kv heads: several rows per wave); each lane reads
// 16-byte pieces of both rows.  The sum is carried as a
// float64 double-double: the difference of two bfloat16 values is exact in
// float64 (exponents within 2^44), its square is split exactly with an FMA,
// and the running sum keeps its rounding error (TwoSum).  The final
// hi + lo is therefore the exactly rounded sum, so rows whose exact
// deviations tie produce equal values and the top-k tie rule applies to
// them, whatever the order of the terms.
#include "kvc_internal.h"
#include "bf16_util.h"

namespace kvc {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsPerIter = 2;

__device__ __forceinline__ void two_sum(double a, double b, double& s, double& e) {
  s = a + b;
  const double bb = s - a;
  e = (a - (s - bb)) + (b - bb);
}

__device__ __forceinline__ void accumulate8(const uint4& f, const uint4& c, double& hi,
                                            double& lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double t = (double)bf16x8_elem(f, e) - (double)bf16x8_elem(c, e);
    const double p = t * t;
    const double perr = fma(t, t, -p);
    double s, serr;
    two_sum(hi, p, s, serr);
    hi = s;
    lo += serr + perr;
  }
}

// CPL: 16-byte pieces per lane per row (row = Hkv * 16 pieces).
template <int CPL>
__global__ __launch_bounds__(kThreads) void kv_deviation_kernel(const uint16_t* __restrict__ kc,
                                                                const uint16_t* __restrict__ kf,
                                                                double* __restrict__ dev,
                                                                int64_t n_rows, int pieces) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * kThreads) >> 6;
  const uint4* C = reinterpret_cast<const uint4*>(kc);
  const uint4* F = reinterpret_cast<const uint4*>(kf);
  for (int64_t r0 = wave * kRowsPerIter; r0 < n_rows; r0 += n_waves * kRowsPerIter) {
    uint4 vf[kRowsPerIter][CPL], vc[kRowsPerIter][CPL];
#pragma unroll
    for (int rr = 0; rr < kRowsPerIter; ++rr) {
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        const int p = lane + 64 * i;
        const int64_t r = r0 + rr;
        if (r < n_rows && p < pieces) {
          vf[rr][i] = load_nt(F + r * pieces + p);
          vc[rr][i] = load_nt(C + r * pieces + p);
        } else {
          vf[rr][i] = make_uint4(0, 0, 0, 0);
          vc[rr][i] = make_uint4(0, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int rr = 0; rr < kRowsPerIter; ++rr) {
      double hi = 0.0, lo = 0.0;
#pragma unroll
      for (int i = 0; i < CPL; ++i) accumulate8(vf[rr][i], vc[rr][i], hi, lo);
      // butterfly over the wave: every lane ends with the same (hi, lo)
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        const double h2 = __shfl_xor(hi, m);
        const double l2 = __shfl_xor(lo, m);
        double s, e;
        two_sum(hi, h2, s, e);
        hi = s;
        lo = (lo + l2) + e;
      }
      const int64_t r = r0 + rr;
      if (lane == 0 && r < n_rows) dev[r] = hi + lo;
    }
  }
}

// Rows narrower than a wave (one or two kv heads: 16 or 32 pieces): LPR
// lanes per row, one piece per lane, 64 / LPR rows per wave at a time and
// kNarrowSteps such row groups loaded before any is summed, so the whole
// wave moves data (the wide kernel would leave 48 or 32 lanes idle).
constexpr int kNarrowSteps = 4;

template <int LPR>
__global__ __launch_bounds__(kThreads) void kv_deviation_narrow_kernel(const uint16_t* __restrict__ kc,
                                                                       const uint16_t* __restrict__ kf,
                                                                       double* __restrict__ dev,
                                                                       int64_t n_rows) {
  constexpr int kRpw = 64 / LPR;
  const int lane = threadIdx.x & 63;
  const int sub = lane / LPR, p = lane % LPR;
  const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * kThreads) >> 6;
  const uint4* C = reinterpret_cast<const uint4*>(kc);
  const uint4* F = reinterpret_cast<const uint4*>(kf);
  for (int64_t r0 = wave * kRpw * kNarrowSteps; r0 < n_rows; r0 += n_waves * kRpw * kNarrowSteps) {
    uint4 vf[kNarrowSteps], vc[kNarrowSteps];
#pragma unroll
    for (int st = 0; st < kNarrowSteps; ++st) {
      const int64_t r = r0 + st * kRpw + sub;
      if (r < n_rows) {
        vf[st] = load_nt(F + r * LPR + p);
        vc[st] = load_nt(C + r * LPR + p);
      } else {
        vf[st] = make_uint4(0, 0, 0, 0);
        vc[st] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int st = 0; st < kNarrowSteps; ++st) {
      double hi = 0.0, lo = 0.0;
      accumulate8(vf[st], vc[st], hi, lo);
      // butterfly inside the row's LPR lanes
#pragma unroll
      for (int m = LPR / 2; m >= 1; m >>= 1) {
        const double h2 = __shfl_xor(hi, m);
        const double l2 = __shfl_xor(lo, m);
        double sum, e;
        two_sum(hi, h2, sum, e);
        hi = sum;
        lo = (lo + l2) + e;
      }
      const int64_t r = r0 + st * kRpw + sub;
      if (p == 0 && r < n_rows) dev[r] = hi + lo;
    }
  }
}

template <int LPR>
hipError_t launch_narrow(int64_t n_rows, const uint16_t* kc, const uint16_t* kf, double* dev, hipStream_t s) {
  constexpr int64_t rows_per_wave = (64 / LPR) * kNarrowSteps;
  const int64_t waves_needed = (n_rows + rows_per_wave - 1) / rows_per_wave;
  int64_t blocks = (waves_needed + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(kv_deviation_narrow_kernel<LPR>, dim3((unsigned)blocks), dim3(kThreads), 0, s, kc, kf,
                     dev, n_rows);
  return hipGetLastError();
}

template <int CPL>
hipError_t launch_cpl(int64_t n_rows, int pieces, const uint16_t* kc, const uint16_t* kf,
                      double* dev, hipStream_t s) {
  const int64_t waves_needed = (n_rows + kRowsPerIter - 1) / kRowsPerIter;
  int64_t blocks = (waves_needed + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(kv_deviation_kernel<CPL>, dim3((unsigned)blocks), dim3(kThreads), 0, s, kc,
                     kf, dev, n_rows, pieces);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_kv_deviation(int64_t n_rows, int n_kv_heads, const uint16_t* k_cached,
                               const uint16_t* k_fresh, double* dev, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  const int pieces = n_kv_heads * (kHeadDim / 8);
  if (pieces == 16) return launch_narrow<16>(n_rows, k_cached, k_fresh, dev, s);
  if (pieces == 32) return launch_narrow<32>(n_rows, k_cached, k_fresh, dev, s);
  const int cpl = (pieces + 63) / 64;
  if (cpl <= 1) return launch_cpl<1>(n_rows, pieces, k_cached, k_fresh, dev, s);
  if (cpl <= 2) return launch_cpl<2>(n_rows, pieces, k_cached, k_fresh, dev, s);
  if (cpl <= 4) return launch_cpl<4>(n_rows, pieces, k_cached, k_fresh, dev, s);
  if (cpl <= 8) return launch_cpl<8>(n_rows, pieces, k_cached, k_fresh, dev, s);
  return launch_cpl<16>(n_rows, pieces, k_cached, k_fresh, dev, s);  // Hkv <= 64 (checked by the API)
}

}  // namespace kvc
