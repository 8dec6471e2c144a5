// bfloat16 helpers for the gfx950 kernels (device side only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvc {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Streaming 16-byte accesses: non-temporal, so data touched once does not
// displace reusable lines in L2 and the MALL.
__device__ __forceinline__ uint4 load_nt(const void* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void store_nt(void* p, const uint4& u) {
  const u32x4 v = {u.x, u.y, u.z, u.w};
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// Element e (0..7) of eight packed bf16 values, as float (exact).
__device__ __forceinline__ float bf16x8_elem(const uint4& v, int e) {
  const uint32_t w = (e >> 1) == 0 ? v.x : (e >> 1) == 1 ? v.y : (e >> 1) == 2 ? v.z : v.w;
  return __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
}

// Round a float64 to bfloat16, nearest with ties to even, in one step (no
// float32 intermediate, hence no double rounding), branch-free.  Finite
// inputs; magnitudes past the bfloat16 range become infinity, and results
// below 2^-126 in magnitude (bfloat16 subnormals) become signed zero.
__device__ __forceinline__ uint32_t f64_to_bf16_rne(double x) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(x);
  const uint32_t sign = (uint32_t)(b >> 48) & 0x8000u;
  const unsigned long long mag = b & 0x7FFFFFFFFFFFFFFFull;
  // keep 7 fraction bits (bits 51..45); round at bit 45, ties to even; a
  // carry out of the fraction moves into the exponent as it should
  const unsigned long long r = mag + 0xFFFFFFFFFFFull + ((mag >> 45) & 1ull);
  const uint32_t rh = (uint32_t)(r >> 45);        // float64 exponent << 7 | 7 fraction bits
  uint32_t v = rh - (896u << 7);                  // rebias 1023 -> 127
  v = mag >= (897ull << 52) ? v : 0u;             // below 2^-126
  v = rh >= (1151u << 7) ? 0x7F80u : v;           // bfloat16 exponent 255 and up
  return sign | v;
}

}  // namespace kvc
