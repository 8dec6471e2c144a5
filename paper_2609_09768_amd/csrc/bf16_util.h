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

}  // namespace kvc
