// Step a2: per-token squared key deviation at the check layer (gfx950).
//
// Paper: CacheBlend ranks tokens by how much their cached keys differ from
// keys recomputed with full attention (Section 2), measured as squared
// differences of the key entries (Section 3.2).  Here
//   d[r] = sum_{h,e} (k_fresh[r,h,e] - k_cached[r,h,e])^2,
// the exact real sum rounded once to float64 (nearest, ties to even), for
// every finite bfloat16 input.  Rows whose exact sums tie therefore get
// equal values whatever the order of their terms, and the top-k tie rule
// applies to them.
//
// Bandwidth-bound (2 x 2 bytes read per element).  Rows of one kv head are
// shared by 8 lanes, of 2 or 4 by 16, of 8 by 32 (several rows per wave),
// other rows by a whole wave; each lane reads 16-byte pieces of both rows.
//
// Fast path, every row.  The difference t of two bfloat16 values is exact in
// float64 when their exponents are at most 44 apart (or one is zero); its
// square is split exactly with an FMA (p + e = t^2) and the running sum is a
// double-double: hi keeps the rounded sum (TwoSum), lo adds up the exact
// errors serr + e in plain float64.  Every term is >= 0, so every partial
// sum is <= S (the exact row sum) up to a factor 1 + 2^-45, and the 2n + 63
// errors that lo adds up (n terms, 63 butterfly merges) are each <= 2^-53 S.
// y = RN(hi + lo) is returned when these checks pass:
//  * range: the largest and the smallest nonzero magnitude of the row's
//    inputs (packed 16-bit maxima of the bit patterns) are at most 2^44
//    apart, so every t is exact; and then either
//  * granularity: every input is a multiple of 2^q (q from the smallest
//    magnitude), so every error and every partial sum in lo is a multiple
//    of 2^(2q); if (2n + 63) 2^-53 S <= 2^(2q + 53) they are all exact, lo
//    is exactly the sum of the errors, hi + lo = S and y = RN(S), ties
//    included.  This holds for ordinary data (inputs within ~2^40 of the
//    row's deviation);
//  * or certificate: lo, a float64 sum of those errors with 2n + 126
//    roundings, is within E = (2n+126)(2n+63) 2^-106 S (x 1.001) of their
//    exact sum.  With r = hi + lo - y (exact, TwoSum), S = y + r + (error
//    of lo), and y = RN(S) when |r| + E is below half the smaller spacing
//    of float64 values next to y (false only for sums within about 2^-30
//    of that half spacing of a rounding boundary, or exactly on one).
//
// Exact path, rows that fail either check.  (f - c)^2 = f^2 - 2fc + c^2, and
// each product of two bfloat16 values is an integer below 2^17 times a power
// of two in [2^-266, 2^241]; the wave adds all of them into a 640-bit
// fixed-point accumulator in LDS (20 signed 64-bit digits of 32 bits, LDS
// atomics), then one lane propagates the carries and rounds the integer to
// float64 (nearest, ties to even, sticky bit from everything below).
#include "kvc_internal.h"
#include "bf16_util.h"

// Every floating-point operation here is written to round exactly where it
// is written: a product fused into a following sum (the compiler's default
// contraction) would break the error-free TwoSum and FMA splits.
#pragma clang fp contract(off)

namespace kvc {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsPerIter = 2;
constexpr int kDigits = 20;         // 32-bit digits of the exact accumulator
constexpr int kDigitBias = 330;     // accumulator bit b holds 2^(b - 330)

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void two_sum(double a, double b, double& s, double& e) {
  s = a + b;
  const double bb = s - a;
  e = (a - (s - bb)) + (b - bb);
}

// The same for a, b >= 0: the larger one first (Dekker's fast form), five
// operations instead of six.
__device__ __forceinline__ void two_sum_nonneg(double a, double b, double& s, double& e) {
  s = a + b;
  const double big = fmax(a, b), small = fmin(a, b);
  e = small - (s - big);
}

__device__ __forceinline__ u16x2 as_u16x2(uint32_t w) { return __builtin_bit_cast(u16x2, w); }
__device__ __forceinline__ uint32_t as_u32(u16x2 v) { return __builtin_bit_cast(uint32_t, v); }

// Fast-path accumulation of eight terms, plus the packed range statistics:
// mx = per-half maximum of the magnitude bits, mn = per-half maximum of
// (-magnitude mod 2^16), i.e. the minimum over nonzero magnitudes (zero maps
// to 0 and never wins).
__device__ __forceinline__ void accumulate8(const uint4& f, const uint4& c, double& hi,
                                            double& lo, uint32_t& mx, uint32_t& mn) {
  const uint32_t fw[4] = {f.x, f.y, f.z, f.w};
  const uint32_t cw[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const u16x2 af = as_u16x2(fw[w] & 0x7FFF7FFFu), ac = as_u16x2(cw[w] & 0x7FFF7FFFu);
    const u16x2 zero = {0, 0};
    u16x2 vmx = as_u16x2(mx), vmn = as_u16x2(mn);
    vmx = __builtin_elementwise_max(vmx, __builtin_elementwise_max(af, ac));
    vmn = __builtin_elementwise_max(vmn, __builtin_elementwise_max(zero - af, zero - ac));
    mx = as_u32(vmx);
    mn = as_u32(vmn);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double t = (double)bf16x8_elem(f, e) - (double)bf16x8_elem(c, e);
    const double p = t * t;
    const double perr = fma(t, t, -p);
    double s, serr;
    two_sum_nonneg(hi, p, s, serr);
    hi = s;
    lo += serr + perr;
  }
}

// Merge the partner lane's partial sum (hi, lo) (xor butterfly step).
__device__ __forceinline__ void merge(double& hi, double& lo, uint32_t& rng, int m) {
  const double h2 = __shfl_xor(hi, m);
  const double l2 = __shfl_xor(lo, m);
  const uint32_t r2 = (uint32_t)__shfl_xor((int)rng, m);
  double s, e;
  two_sum_nonneg(hi, h2, s, e);
  hi = s;
  lo = (lo + l2) + e;
  rng = as_u32(__builtin_elementwise_max(as_u16x2(rng), as_u16x2(r2)));
}

// Lane-local range statistics folded into one word: high half = largest
// magnitude bits, low half = -(smallest nonzero magnitude bits) mod 2^16.
__device__ __forceinline__ uint32_t fold_range(uint32_t mx, uint32_t mn) {
  const uint32_t a = max(mx & 0xFFFFu, mx >> 16);
  const uint32_t b = max(mn & 0xFFFFu, mn >> 16);
  return (a << 16) | b;
}

// The fast path's result is the exactly rounded sum: range, then either the
// granularity test or the certificate (see the file comment).  n_terms:
// terms in the row.  Writes y = RN(hi + lo).
__device__ __forceinline__ bool fast_result_exact(double hi, double lo, uint32_t rng, int n_terms,
                                                  double& y) {
  double r;
  two_sum(hi, lo, y, r);
  const uint32_t big = rng >> 16, neg_small = rng & 0xFFFFu;
  if (neg_small == 0) return true;  // every input zero
  // range: exponents (0 read as 1, bfloat16 subnormals) at most 44 apart
  const uint32_t small = (0x10000u - neg_small) & 0xFFFFu;
  const int eb = max((int)(big >> 7), 1), es = max((int)(small >> 7), 1);
  if (eb - es > 44) return false;
  const double n2 = 2.0 * n_terms;
  // granularity: every input is a multiple of 2^q, q = es - 134, so every
  // error summed into lo, and every partial sum of them, is a multiple of
  // 2^(2q); below 2^(2q + 53) in magnitude they are all exact in float64
  const double err_sum = (n2 + 63.0) * 0x1p-53 * 1.001 * y;
  if (err_sum <= __longlong_as_double((long long)(2 * es - 215 + 1023) << 52)) return true;
  const double bound = (n2 + 126.0) * err_sum * 0x1p-53;
  const unsigned long long yb = (unsigned long long)__double_as_longlong(y);
  const long long ye = (long long)((yb >> 52) & 0x7FF);
  const long long pow2 = (yb & 0xFFFFFFFFFFFFFull) == 0 ? 1 : 0;
  // half the spacing below y (the smaller one when y is a power of two)
  const double half = __longlong_as_double((ye - 53 - pow2) << 52);
  return fabs(r) + bound < half;
}

// ---- exact path -------------------------------------------------------------
// bfloat16 bits -> m * 2^q with m an integer in [0, 255], q in [-133, 121].
__device__ __forceinline__ void bf16_decode(uint32_t x, uint32_t& m, int& q, uint32_t& s) {
  const uint32_t e = (x >> 7) & 0xFFu;
  m = (x & 0x7Fu) | (e ? 0x80u : 0u);
  q = (int)(e ? e : 1u) - 134;
  s = (x >> 15) & 1u;
}

// acc += (neg ? -1 : 1) * v * 2^x  (v < 2^17; one or two digits)
__device__ __forceinline__ void acc_add(unsigned long long* acc, uint32_t v, int x, bool neg) {
  if (v == 0) return;
  const int b = x + kDigitBias;  // >= 64
  const int d = b >> 5;
  const unsigned long long w = (unsigned long long)v << (b & 31);
  unsigned long long lo = w & 0xFFFFFFFFull, hi = w >> 32;
  if (neg) {
    lo = 0ull - lo;
    hi = 0ull - hi;
  }
  atomicAdd(acc + d, lo);
  if (w >> 32) atomicAdd(acc + d + 1, hi);
}

// Adds f^2 - 2 f c + c^2 for the eight element pairs of (f, c).
__device__ __forceinline__ void exact_add8(unsigned long long* acc, const uint4& f, const uint4& c) {
  const uint32_t fw[4] = {f.x, f.y, f.z, f.w};
  const uint32_t cw[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t xf = (e & 1) ? fw[e >> 1] >> 16 : fw[e >> 1] & 0xFFFFu;
    const uint32_t xc = (e & 1) ? cw[e >> 1] >> 16 : cw[e >> 1] & 0xFFFFu;
    uint32_t mf, mc, sf, sc;
    int qf, qc;
    bf16_decode(xf, mf, qf, sf);
    bf16_decode(xc, mc, qc, sc);
    acc_add(acc, mf * mf, 2 * qf, false);
    acc_add(acc, mc * mc, 2 * qc, false);
    acc_add(acc, 2u * mf * mc, qf + qc, sf == sc);  // -2 f c
  }
}

// Carry propagation and rounding of the accumulator (one lane; the digits
// are normalised in place to [0, 2^32), so nothing is indexed in registers).
__device__ double exact_round(unsigned long long* acc) {
  long long carry = 0;
  int top = -1;
  for (int d = 0; d < kDigits; ++d) {
    const long long v = (long long)acc[d] + carry;
    acc[d] = v & 0xFFFFFFFFll;
    carry = v >> 32;
    if (v & 0xFFFFFFFFll) top = d;
  }
  if (top < 2) return 0.0;  // digits 0 and 1 never receive a term
  const uint32_t d0 = (uint32_t)acc[top], d1 = (uint32_t)acc[top - 1], d2 = (uint32_t)acc[top - 2];
  const int lz = __clz(d0);
  const unsigned long long h64 = ((unsigned long long)d0 << 32) | d1;
  const unsigned long long t = lz ? (h64 << lz) | (d2 >> (32 - lz)) : h64;
  bool sticky = (t & 0x3FFull) != 0 || (lz ? (uint32_t)(d2 << lz) != 0 : d2 != 0);
  for (int d = 0; d < top - 2; ++d) sticky |= acc[d] != 0;
  unsigned long long mant = t >> 11;
  const bool round = (t >> 10) & 1ull;
  if (round && (sticky || (mant & 1ull))) ++mant;
  return ldexp((double)mant, 32 * (top - 1) - lz + 11 - kDigitBias);
}

// The exact path for one row, run by the `lanes` lanes that share it (lane
// index `l` among them): the row is read again from memory, every lane adds
// its pieces' products into the row's LDS accumulator, lane 0 rounds.  The
// row is re-read rather than kept in registers through the fast path.
__device__ __forceinline__ double exact_row(unsigned long long* acc, const uint4* F, const uint4* C, int64_t r,
                                         int pieces, int l, int lanes) {
  for (int d = l; d < kDigits; d += lanes) acc[d] = 0ull;
  __threadfence_block();
  for (int i = l; i < pieces; i += lanes) exact_add8(acc, F[r * pieces + i], C[r * pieces + i]);
  __threadfence_block();
  double y = 0.0;
  if (l == 0) y = exact_round(acc);
  __threadfence_block();
  return y;
}

// CPL: 16-byte pieces per lane per row (row = Hkv * 16 pieces).
template <int CPL>
__global__ __launch_bounds__(kThreads) void kv_deviation_kernel(const uint16_t* __restrict__ kc,
                                                                const uint16_t* __restrict__ kf,
                                                                double* __restrict__ dev,
                                                                int64_t n_rows, int pieces) {
  __shared__ unsigned long long sacc[kThreads / 64][kDigits];
  const int lane = threadIdx.x & 63;
  unsigned long long* acc = sacc[threadIdx.x >> 6];
  const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * kThreads) >> 6;
  const uint4* C = reinterpret_cast<const uint4*>(kc);
  const uint4* F = reinterpret_cast<const uint4*>(kf);
  const int n_terms = pieces * 8;
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
      uint32_t mx = 0, mn = 0;
#pragma unroll
      for (int i = 0; i < CPL; ++i) accumulate8(vf[rr][i], vc[rr][i], hi, lo, mx, mn);
      // butterfly over the wave: every lane ends with the same values
      uint32_t rng = fold_range(mx, mn);
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) merge(hi, lo, rng, m);
      const int64_t r = r0 + rr;
      double y;
      if (r < n_rows && !fast_result_exact(hi, lo, rng, n_terms, y))  // wave-uniform
        y = exact_row(acc, F, C, r, pieces, lane, 64);
      if (lane == 0 && r < n_rows) dev[r] = y;
    }
  }
}

// Rows of up to eight kv heads (16 to 128 pieces): LPR lanes per row, PPL
// pieces per lane, 64 / LPR rows per wave at a time and STEPS such row
// groups loaded before any is summed.  Fewer lanes per row than the wide
// kernel's 64 means a shorter butterfly and fewer per-row checks for the
// same elements: with 8 kv heads, 32 lanes x 4 pieces (32 terms per lane,
// 5 merge steps) instead of 64 lanes x 2 pieces (16 terms, 6 steps).  (16
// lanes x 8 pieces keeps twice the loads in flight per lane, but at 107
// registers four waves per SIMD instead of six, and measured 3-4 % slower
// on cold buffers.)
template <int LPR, int PPL, int STEPS>
__global__ __launch_bounds__(kThreads) void kv_deviation_rows_kernel(const uint16_t* __restrict__ kc,
                                                                     const uint16_t* __restrict__ kf,
                                                                     double* __restrict__ dev,
                                                                     int64_t n_rows) {
  constexpr int kRpw = 64 / LPR;
  constexpr int kPieces = LPR * PPL;
  __shared__ unsigned long long sacc[kThreads / 64][kRpw][kDigits];
  const int lane = threadIdx.x & 63;
  const int sub = lane / LPR, p = lane % LPR;
  unsigned long long* acc = sacc[threadIdx.x >> 6][sub];
  const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * kThreads) >> 6;
  const uint4* C = reinterpret_cast<const uint4*>(kc);
  const uint4* F = reinterpret_cast<const uint4*>(kf);
  for (int64_t r0 = wave * kRpw * STEPS; r0 < n_rows; r0 += n_waves * kRpw * STEPS) {
    uint4 vf[STEPS][PPL], vc[STEPS][PPL];
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
      const int64_t r = r0 + st * kRpw + sub;
#pragma unroll
      for (int i = 0; i < PPL; ++i) {
        if (r < n_rows) {
          vf[st][i] = load_nt(F + r * kPieces + p + LPR * i);
          vc[st][i] = load_nt(C + r * kPieces + p + LPR * i);
        } else {
          vf[st][i] = make_uint4(0, 0, 0, 0);
          vc[st][i] = make_uint4(0, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
      double hi = 0.0, lo = 0.0;
      uint32_t mx = 0, mn = 0;
#pragma unroll
      for (int i = 0; i < PPL; ++i) accumulate8(vf[st][i], vc[st][i], hi, lo, mx, mn);
      // butterfly inside the row's LPR lanes
      uint32_t rng = fold_range(mx, mn);
#pragma unroll
      for (int m = LPR / 2; m >= 1; m >>= 1) merge(hi, lo, rng, m);
      const int64_t r = r0 + st * kRpw + sub;
      double y;
      if (r < n_rows && !fast_result_exact(hi, lo, rng, kPieces * 8, y))  // uniform within the row's lanes
        y = exact_row(acc, F, C, r, kPieces, p, LPR);
      if (p == 0 && r < n_rows) dev[r] = y;
    }
  }
}

template <int LPR, int PPL, int STEPS>
hipError_t launch_rows(int64_t n_rows, const uint16_t* kc, const uint16_t* kf, double* dev, hipStream_t s) {
  constexpr int64_t rows_per_wave = (64 / LPR) * STEPS;
  const int64_t waves_needed = (n_rows + rows_per_wave - 1) / rows_per_wave;
  int64_t blocks = (waves_needed + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL((kv_deviation_rows_kernel<LPR, PPL, STEPS>), dim3((unsigned)blocks), dim3(kThreads), 0, s,
                     kc, kf, dev, n_rows);
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
  if (pieces == 16) return launch_rows<8, 2, 2>(n_rows, k_cached, k_fresh, dev, s);  // 13 % faster than 16 x 1
  if (pieces == 32) return launch_rows<16, 2, 2>(n_rows, k_cached, k_fresh, dev, s);
  if (pieces == 64) return launch_rows<16, 4, 1>(n_rows, k_cached, k_fresh, dev, s);
  if (pieces == 128) return launch_rows<32, 4, 1>(n_rows, k_cached, k_fresh, dev, s);
  const int cpl = (pieces + 63) / 64;
  if (cpl <= 1) return launch_cpl<1>(n_rows, pieces, k_cached, k_fresh, dev, s);
  if (cpl <= 2) return launch_cpl<2>(n_rows, pieces, k_cached, k_fresh, dev, s);
  if (cpl <= 4) return launch_cpl<4>(n_rows, pieces, k_cached, k_fresh, dev, s);
  if (cpl <= 8) return launch_cpl<8>(n_rows, pieces, k_cached, k_fresh, dev, s);
  return launch_cpl<16>(n_rows, pieces, k_cached, k_fresh, dev, s);  // Hkv <= 64 (checked by the API)
}

}  // namespace kvc
