// bfloat16 helpers for the gfx950 kernels (device side only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvc {

// Element e (0..7) of eight packed bf16 values, as float (exact).
__device__ __forceinline__ float bf16x8_elem(const uint4& v, int e) {
  const uint32_t w = (e >> 1) == 0 ? v.x : (e >> 1) == 1 ? v.y : (e >> 1) == 2 ? v.z : v.w;
  return __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
}

// Round a float64 to bfloat16, nearest with ties to even, in one step (no
// float32 intermediate, hence no double rounding).  Finite inputs; results
// beyond the bfloat16 range become infinity.
__device__ __forceinline__ uint32_t f64_to_bf16_rne(double x) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(x);
  const uint32_t sign = (uint32_t)(b >> 48) & 0x8000u;
  const unsigned long long mag = b & 0x7FFFFFFFFFFFFFFFull;
  if (mag >= (897ull << 52)) {  // |x| >= 2^-126: normal bfloat16 range
    // keep 7 fraction bits (bits 51..45); round at bit 45, ties to even
    const unsigned long long r = mag + 0xFFFFFFFFFFFull + ((mag >> 45) & 1ull);
    const int e = (int)(r >> 52) - 1023 + 127;
    if (e >= 255) return sign | 0x7F80u;
    return sign | ((uint32_t)e << 7) | ((uint32_t)(r >> 45) & 0x7Fu);
  }
  // |x| < 2^-126: subnormal grid of spacing 2^-133 (128 encodes 2^-126)
  const double q = rint(fabs(x) * 0x1p133);
  return sign | (uint32_t)q;
}

}  // namespace kvc
