// Step a3: top-k row selection by deviation (gfx950).
//
// Paper: the tokens with the largest key deviation are recomputed, a fixed
// fraction of them (Section 3.2).  The selection here: the k largest d,
// ties to the lower row, returned in ascending row order.
//
// No sort.  Each float64 d maps to a 64-bit key whose unsigned order is the
// order of d.  A radix select finds the k-th largest key T one byte at a
// time (8 passes over the keys, most significant byte first): every
// workgroup histograms the byte of the keys that still match the prefix
// found so far, and the last workgroup to finish (atomic ticket) picks the
// byte, updates the prefix and the remaining rank, and clears the
// histogram for the next pass.  Then rows with key > T, plus the first
// `rem` rows with key == T in row order, are compacted in row order with
// a per-block count and a scan; this yields the ascending output
// directly.  n and k are known on the host, so nothing is read back.
#include "kvc_internal.h"

namespace kvc {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = kTopkRowsPerBlock / kThreads;  // 8 consecutive rows per thread

__device__ __forceinline__ unsigned long long order_key(double x) {
  unsigned long long b = (unsigned long long)__double_as_longlong(x);
  if ((b << 1) == 0ull) b = 0ull;  // -0.0 == +0.0
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

// Exclusive scan over the 256 threads of a block; returns the block total.
__device__ __forceinline__ unsigned int block_excl_scan(unsigned int v, unsigned int* sh,
                                                        unsigned int& total) {
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
#pragma unroll
  for (int off = 1; off < kThreads; off <<= 1) {
    const unsigned int add = (t >= off) ? sh[t - off] : 0u;
    __syncthreads();
    sh[t] += add;
    __syncthreads();
  }
  total = sh[kThreads - 1];
  const unsigned int incl = sh[t];
  __syncthreads();
  return incl - v;
}

__global__ __launch_bounds__(kThreads) void topk_init(TopkState* st, long long k) {
  const int t = threadIdx.x;
  st->hist[t] = 0u;
  if (t == 0) {
    st->prefix = 0ull;
    st->mask = 0ull;
    st->rem = k;
    st->done = 0u;
  }
}

__global__ __launch_bounds__(kThreads) void topk_radix_pass(const double* __restrict__ dev,
                                                            long long n, TopkState* st,
                                                            int shift) {
  __shared__ unsigned int h[kThreads];
  __shared__ unsigned int suf[kThreads];
  __shared__ int is_last;
  const int t = threadIdx.x;
  const unsigned long long prefix = st->prefix;
  const unsigned long long mask = st->mask;
  const long long rem = st->rem;
  h[t] = 0u;
  __syncthreads();
  for (long long i = (long long)blockIdx.x * kThreads + t; i < n; i += (long long)gridDim.x * kThreads) {
    const unsigned long long key = order_key(dev[i]);
    if ((key & mask) == prefix) atomicAdd(&h[(key >> shift) & 255ull], 1u);
  }
  __syncthreads();
  if (h[t]) atomicAdd(&st->hist[t], h[t]);
  __threadfence();
  __syncthreads();
  if (t == 0) is_last = (atomicAdd(&st->done, 1u) == gridDim.x - 1);
  __syncthreads();
  if (!is_last) return;
  __threadfence();
  const unsigned int cnt = __hip_atomic_load(&st->hist[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // suf[b] = number of matching keys whose byte is >= b
  suf[t] = cnt;
  __syncthreads();
#pragma unroll
  for (int off = 1; off < kThreads; off <<= 1) {
    const unsigned int add = (t + off < kThreads) ? suf[t + off] : 0u;
    __syncthreads();
    suf[t] += add;
    __syncthreads();
  }
  const long long above = (long long)(suf[t] - cnt);
  if (above < rem && rem <= (long long)suf[t]) {  // exactly one byte value qualifies
    st->prefix = prefix | ((unsigned long long)t << shift);
    st->mask = mask | (255ull << shift);
    st->rem = rem - above;
  }
  st->hist[t] = 0u;
  if (t == 0) st->done = 0u;
}

// Per block of 2048 rows: how many keys are above T and equal to T.
__global__ __launch_bounds__(kThreads) void topk_count(const double* __restrict__ dev, long long n,
                                                       const TopkState* st,
                                                       unsigned int* __restrict__ bc) {
  __shared__ unsigned int sh[kThreads];
  const unsigned long long T = st->prefix;
  const long long base = (long long)blockIdx.x * kTopkRowsPerBlock + (long long)threadIdx.x * kItems;
  unsigned int gt = 0u, eq = 0u;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const long long r = base + i;
    if (r < n) {
      const unsigned long long key = order_key(dev[r]);
      gt += key > T;
      eq += key == T;
    }
  }
  unsigned int tot_gt, tot_eq;
  block_excl_scan(gt, sh, tot_gt);
  block_excl_scan(eq, sh, tot_eq);
  if (threadIdx.x == 0) {
    bc[2 * blockIdx.x] = tot_gt;
    bc[2 * blockIdx.x + 1] = tot_eq;
  }
}

__global__ __launch_bounds__(kThreads) void topk_write(const double* __restrict__ dev, long long n,
                                                       const TopkState* st,
                                                       const unsigned int* __restrict__ bc,
                                                       long long k, int32_t* __restrict__ out) {
  __shared__ unsigned int sh[kThreads];
  __shared__ unsigned long long red[2];
  const int t = threadIdx.x;
  const unsigned long long T = st->prefix;
  const long long need_eq = st->rem;  // rows equal to T still to take, in row order

  // counts of all earlier blocks
  unsigned long long gtb = 0ull, eqb = 0ull;
  for (int b = t; b < (int)blockIdx.x; b += kThreads) {
    gtb += bc[2 * b];
    eqb += bc[2 * b + 1];
  }
  if (t == 0) { red[0] = 0ull; red[1] = 0ull; }
  __syncthreads();
  if (gtb) atomicAdd(&red[0], gtb);
  if (eqb) atomicAdd(&red[1], eqb);
  __syncthreads();
  const long long gt_before = (long long)red[0];
  const long long eq_before = (long long)red[1];
  const long long sel_before = gt_before + (eq_before < need_eq ? eq_before : need_eq);

  const long long base = (long long)blockIdx.x * kTopkRowsPerBlock + (long long)t * kItems;
  unsigned long long keys[kItems];
  unsigned int eq_t = 0u;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const long long r = base + i;
    keys[i] = (r < n) ? order_key(dev[r]) : 0ull;
    eq_t += (r < n) && keys[i] == T;
  }
  unsigned int tot;
  const unsigned int eq_excl = block_excl_scan(eq_t, sh, tot);
  bool take[kItems];
  unsigned int sel_t = 0u;
  long long rank = eq_before + eq_excl;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const long long r = base + i;
    const bool valid = r < n;
    const bool is_eq = valid && keys[i] == T;
    take[i] = valid && (keys[i] > T || (is_eq && rank < need_eq));
    rank += is_eq;
    sel_t += take[i];
  }
  const unsigned int sel_excl = block_excl_scan(sel_t, sh, tot);
  long long o = sel_before + sel_excl;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    if (take[i] && o < k) out[o++] = (int32_t)(base + i);  // o < k always; the guard keeps writes in bounds
  }
}

// out[i] = start + i for i < count
__global__ __launch_bounds__(kThreads) void iota_kernel(int32_t* __restrict__ out, long long count,
                                                        long long start) {
  for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < count;
       i += (long long)gridDim.x * kThreads)
    out[i] = (int32_t)(start + i);
}

hipError_t launch_iota(int32_t* out, long long count, long long start, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  long long blocks = (count + kThreads - 1) / kThreads;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(iota_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, out, count, start);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_select_topk(const double* dev, int64_t n, int64_t k, int64_t n_append,
                              int32_t* idx_out, void* ws, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (k == 0) return launch_iota(idx_out, n_append, n, s);
  if (k == n) return launch_iota(idx_out, n + n_append, 0, s);
  TopkState* st = static_cast<TopkState*>(ws);
  unsigned int* bc = reinterpret_cast<unsigned int*>(static_cast<char*>(ws) + align256(sizeof(TopkState)));
  const long long nblk = topk_blocks(n);
  long long pass_blocks = (n + kThreads * 8 - 1) / (kThreads * 8);
  if (pass_blocks > 1024) pass_blocks = 1024;
  hipLaunchKernelGGL(topk_init, dim3(1), dim3(kThreads), 0, s, st, (long long)k);
  for (int shift = 56; shift >= 0; shift -= 8)
    hipLaunchKernelGGL(topk_radix_pass, dim3((unsigned)pass_blocks), dim3(kThreads), 0, s, dev,
                       (long long)n, st, shift);
  hipLaunchKernelGGL(topk_count, dim3((unsigned)nblk), dim3(kThreads), 0, s, dev, (long long)n, st, bc);
  hipLaunchKernelGGL(topk_write, dim3((unsigned)nblk), dim3(kThreads), 0, s, dev, (long long)n, st,
                     bc, (long long)k, idx_out);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_iota(idx_out + k, n_append, n, s);
}

}  // namespace kvc
