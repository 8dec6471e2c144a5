// Step a4 (scatter half): recomputed K/V of the selected tokens replace the
// cached rows (Section 3.2 / Section 4 setup: only selected tokens are
// recomputed, the rest is reused).  One wave copies one selected row of K
// and of V, 16 bytes per lane per access.  The gather half (selected
// queries) is fused into the attention kernel's query load.
#include "kvc_internal.h"

namespace kvc {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void scatter_rows_kernel(
    const int32_t* __restrict__ sel, long long n_sel, int compact, const uint4* __restrict__ kf,
    const uint4* __restrict__ vf, long long n_fresh, uint4* __restrict__ kc, uint4* __restrict__ vc,
    long long n_rows, int pieces) {
  const int lane = threadIdx.x & 63;
  const long long wave = ((long long)blockIdx.x * kThreads + threadIdx.x) >> 6;
  const long long n_waves = ((long long)gridDim.x * kThreads) >> 6;
  for (long long i = wave; i < n_sel; i += n_waves) {
    const long long dst = sel[i];
    const long long src = compact ? i : dst;
    if (dst < 0 || dst >= n_rows || src < 0 || src >= n_fresh) continue;
    for (int p = lane; p < pieces; p += 64) {
      const uint4 a = kf[src * pieces + p];
      const uint4 b = vf[src * pieces + p];
      kc[dst * pieces + p] = a;
      vc[dst * pieces + p] = b;
    }
  }
}

}  // namespace

hipError_t launch_scatter_rows(const int32_t* sel, int64_t n_sel, int compact,
                               const uint16_t* k_fresh, const uint16_t* v_fresh, int64_t n_fresh,
                               uint16_t* k_cache, uint16_t* v_cache, int64_t n_rows,
                               int n_kv_heads, hipStream_t s) {
  if (n_sel <= 0) return hipSuccess;
  const int pieces = n_kv_heads * (kHeadDim / 8);
  long long blocks = (n_sel + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(scatter_rows_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, sel,
                     (long long)n_sel, compact, reinterpret_cast<const uint4*>(k_fresh),
                     reinterpret_cast<const uint4*>(v_fresh), (long long)n_fresh,
                     reinterpret_cast<uint4*>(k_cache), reinterpret_cast<uint4*>(v_cache),
                     (long long)n_rows, pieces);
  return hipGetLastError();
}

}  // namespace kvc
