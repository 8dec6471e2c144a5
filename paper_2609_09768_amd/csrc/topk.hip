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
//
// From 16,385 to 262,144 candidates the passes, count and write run in one
// launch with grid barriers (below).  Up to 16,384 candidates (contexts to
// about 16k tokens) one workgroup does all of it in one launch: each of its 1,024 threads keeps 16 consecutive
// rows' keys in registers (32 would spill), the 8 passes histogram into
// per-wave LDS bins, and two block scans write the output.  Small layers
// would otherwise spend most of their time in the 11 dependent launches of
// the general path.
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
                                                       long long k, long long n_append,
                                                       int32_t* __restrict__ out) {
  __shared__ unsigned int sh[kThreads];
  __shared__ unsigned long long red[2];
  const int t = threadIdx.x;
  // the appended rows n .. n + n_append - 1 after the selection (no launch of their own)
  for (long long i = (long long)blockIdx.x * kThreads + t; i < n_append; i += (long long)gridDim.x * kThreads)
    out[k + i] = (int32_t)(n + i);
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

// ---- single-workgroup path -------------------------------------------------
constexpr int kSmallThreads = 1024;
constexpr int kSmallWaves = kSmallThreads / 64;
constexpr int kSmallItems = 16;  // consecutive rows per thread, keys in registers
constexpr long long kSmallMax = (long long)kSmallThreads * kSmallItems;

// Exclusive scan over the block's 1,024 threads (wave scans + wave totals).
__device__ __forceinline__ unsigned int scan1024(unsigned int v, unsigned int* wsum,
                                                 unsigned int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned int u = __shfl_up(incl, off, 64);
    if (lane >= off) incl += u;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  unsigned int before = 0u, tot = 0u;
#pragma unroll
  for (int w = 0; w < kSmallWaves; ++w) {
    const unsigned int x = wsum[w];
    before += (w < wave) ? x : 0u;
    tot += x;
  }
  __syncthreads();  // wsum is reused by the next scan
  total = tot;
  return before + incl - v;
}

__global__ __launch_bounds__(kSmallThreads) void topk_small(const double* __restrict__ dev, long long n,
                                                            long long k, long long n_append,
                                                            int32_t* __restrict__ out) {
  __shared__ unsigned int wh[kSmallWaves][256];  // per-wave byte histograms
  __shared__ unsigned int cnt[256];
  __shared__ unsigned int wsum[kSmallWaves];
  __shared__ unsigned long long s_prefix, s_mask;
  __shared__ long long s_rem;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const long long base = (long long)t * kSmallItems;
  unsigned long long key[kSmallItems];
#pragma unroll
  for (int i = 0; i < kSmallItems; ++i) key[i] = (base + i < n) ? order_key(dev[base + i]) : 0ull;

  unsigned long long prefix = 0ull, mask = 0ull;
  long long rem = k;
  for (int shift = 56; shift >= 0; shift -= 8) {
    // a wave's own bins: cleared and filled by that wave alone, in order
    for (int b = lane; b < 256; b += 64) wh[wave][b] = 0u;
#pragma unroll
    for (int i = 0; i < kSmallItems; ++i)
      if (base + i < n && (key[i] & mask) == prefix) atomicAdd(&wh[wave][(key[i] >> shift) & 255ull], 1u);
    __syncthreads();
    if (t < 256) {
      unsigned int c = 0u;
#pragma unroll
      for (int w = 0; w < kSmallWaves; ++w) c += wh[w][t];
      cnt[t] = c;
    }
    __syncthreads();
    if (wave == 0) {
      // lane l holds bins 4l .. 4l+3; above = matching keys in higher bins
      unsigned int c4[4];
      unsigned int v = 0u;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c4[j] = cnt[4 * lane + j];
        v += c4[j];
      }
      unsigned int suf = v;  // sum over lanes >= lane
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const unsigned int u = __shfl_down(suf, off, 64);
        if (lane + off < 64) suf += u;
      }
      long long above = (long long)(suf - v);
#pragma unroll
      for (int j = 3; j >= 0; --j) {
        if (above < rem && rem <= above + (long long)c4[j]) {  // exactly one bin qualifies
          s_prefix = prefix | ((unsigned long long)(4 * lane + j) << shift);
          s_mask = mask | (255ull << shift);
          s_rem = rem - above;
        }
        above += c4[j];
      }
    }
    __syncthreads();
    prefix = s_prefix;
    mask = s_mask;
    rem = s_rem;
  }

  // prefix is now the k-th largest key T; rem = rows equal to T to take
  unsigned int eq_t = 0u;
#pragma unroll
  for (int i = 0; i < kSmallItems; ++i) eq_t += (base + i < n) && key[i] == prefix;
  unsigned int tot;
  long long rank = scan1024(eq_t, wsum, tot);
  unsigned int take = 0u, sel_t = 0u;
#pragma unroll
  for (int i = 0; i < kSmallItems; ++i) {
    const bool valid = base + i < n;
    const bool is_eq = valid && key[i] == prefix;
    const bool tk = valid && (key[i] > prefix || (is_eq && rank < rem));
    rank += is_eq;
    take |= (unsigned int)tk << i;
    sel_t += tk;
  }
  long long o = scan1024(sel_t, wsum, tot);
#pragma unroll
  for (int i = 0; i < kSmallItems; ++i)
    if ((take >> i & 1u) && o < k) out[o++] = (int32_t)(base + i);  // o < k always; kept in bounds
  for (long long i = t; i < n_append; i += kSmallThreads) out[k + i] = (int32_t)(n + i);
}


// ---- fused path: all passes in one launch ------------------------------------
// From 16,385 to kFusedMaxRows candidates: one workgroup per 2,048 rows (at
// most 128, so every workgroup is resident at once on the 256 CUs), each
// thread keeping its 8 consecutive rows' keys in registers.  The passes and
// the ordered write are separated by grid barriers (an arrival counter in
// the workspace); after each pass every workgroup reads the same byte
// histogram and picks the same byte, so no workgroup has to publish it.
// Pass p adds into histogram p % 3; after barrier p, workgroup 0 clears
// histogram (p + 2) % 3, which every workgroup finished reading before it
// arrived at barrier p and which nobody adds into before barrier p + 1.
// Two launches instead of eleven, and the keys are read once (124k: 42 us
// instead of 90).
constexpr int kFusedMaxBlocks = 128;
constexpr long long kFusedMaxRows = (long long)kFusedMaxBlocks * kTopkRowsPerBlock;
// A bound on every barrier wait (seconds), so that no wait is endless: it is
// reached only if some workgroup of the grid cannot run at all, which at
// most 128 workgroups of 256 threads on 256 CUs does not happen (the other
// kernels that may share the GPU, on other streams, all finish on their
// own); the selection would then be wrong.
constexpr int kSpinLimit = 1 << 22;

__global__ __launch_bounds__(kThreads) void topk_fused_init(TopkFused* st) {
  const int t = threadIdx.x;
  st->hist[0][t] = 0u;
  st->hist[1][t] = 0u;
  if (t == 0) st->arrive = 0u;
}

// Every workgroup of the grid arrives once per barrier id; returns when all
// have arrived at barrier id (or the spin bound is reached).  Everything the
// workgroups exchange (histogram adds and clears, block counts, the arrival
// counter) is a device-scope atomic, performed where all XCDs see it, so
// the barrier needs no cache writeback: each wave waits until its own
// atomics are done before the workgroup arrives, and a workgroup reads the
// exchanged values only after it has seen every arrival.
__device__ __forceinline__ void grid_barrier(TopkFused* st, unsigned int id) {
  __builtin_amdgcn_s_waitcnt(0);  // this wave's adds and stores are done
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(&st->arrive, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned int target = (id + 1u) * gridDim.x;
    for (int it = 0; it < kSpinLimit; ++it) {
      if (__hip_atomic_load(&st->arrive, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target) break;
      __builtin_amdgcn_s_sleep(2);
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kThreads) void topk_fused(const double* __restrict__ dev, long long n, long long k,
                                                       long long n_append, TopkFused* st,
                                                       unsigned int* __restrict__ bc, int32_t* __restrict__ out) {
  __shared__ unsigned int h[kThreads];
  __shared__ unsigned int sh[kThreads];
  __shared__ unsigned long long s_prefix, s_mask, red[2];
  __shared__ long long s_rem;
  const int t = threadIdx.x;
  const long long base = (long long)blockIdx.x * kTopkRowsPerBlock + (long long)t * kItems;
  unsigned long long key[kItems];
  unsigned int valid = 0u;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const bool v = base + i < n;
    key[i] = v ? order_key(dev[base + i]) : 0ull;
    valid |= (unsigned int)v << i;
  }
  unsigned long long prefix = 0ull, mask = 0ull;
  long long rem = k;
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
    unsigned int* gh = st->hist[pass % 3];
    h[t] = 0u;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kItems; ++i)
      if ((valid >> i & 1u) && (key[i] & mask) == prefix) atomicAdd(&h[(key[i] >> shift) & 255ull], 1u);
    __syncthreads();
    if (h[t]) atomicAdd(&gh[t], h[t]);
    grid_barrier(st, (unsigned int)pass);
    const unsigned int cnt = __hip_atomic_load(&gh[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (blockIdx.x == 0 && pass + 2 < 8)
      __hip_atomic_store(&st->hist[(pass + 2) % 3][t], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // suf[b] = matching keys whose byte is >= b
    sh[t] = cnt;
    __syncthreads();
#pragma unroll
    for (int off = 1; off < kThreads; off <<= 1) {
      const unsigned int add = (t + off < kThreads) ? sh[t + off] : 0u;
      __syncthreads();
      sh[t] += add;
      __syncthreads();
    }
    const long long above = (long long)(sh[t] - cnt);
    if (above < rem && rem <= (long long)sh[t]) {  // exactly one byte value qualifies
      s_prefix = prefix | ((unsigned long long)t << shift);
      s_mask = mask | (255ull << shift);
      s_rem = rem - above;
    }
    __syncthreads();
    prefix = s_prefix;
    mask = s_mask;
    rem = s_rem;
    __syncthreads();  // sh and the shared prefix are rewritten by the next pass
  }
  // prefix is the k-th largest key T; rem = rows equal to T still to take.
  // Per workgroup: rows above T and rows equal to T, then the ordered write.
  const unsigned long long T = prefix;
  unsigned int gt_t = 0u, eq_t = 0u;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const bool v = valid >> i & 1u;
    gt_t += v && key[i] > T;
    eq_t += v && key[i] == T;
  }
  unsigned int tot_gt, tot_eq;
  block_excl_scan(gt_t, sh, tot_gt);
  const unsigned int eq_excl = block_excl_scan(eq_t, sh, tot_eq);
  if (t == 0) {
    __hip_atomic_store(&bc[2 * blockIdx.x], tot_gt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&bc[2 * blockIdx.x + 1], tot_eq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    red[0] = 0ull;
    red[1] = 0ull;
  }
  grid_barrier(st, 8u);
  unsigned long long gtb = 0ull, eqb = 0ull;
  for (int b = t; b < (int)blockIdx.x; b += kThreads) {
    gtb += __hip_atomic_load(&bc[2 * b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    eqb += __hip_atomic_load(&bc[2 * b + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (gtb) atomicAdd(&red[0], gtb);
  if (eqb) atomicAdd(&red[1], eqb);
  __syncthreads();
  const long long gt_before = (long long)red[0];
  const long long eq_before = (long long)red[1];
  const long long sel_before = gt_before + (eq_before < rem ? eq_before : rem);
  unsigned int take = 0u, sel_t = 0u;
  long long rank = eq_before + eq_excl;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const bool v = valid >> i & 1u;
    const bool is_eq = v && key[i] == T;
    const bool tk = v && (key[i] > T || (is_eq && rank < rem));
    rank += is_eq;
    take |= (unsigned int)tk << i;
    sel_t += tk;
  }
  unsigned int tot;
  long long o = sel_before + block_excl_scan(sel_t, sh, tot);
#pragma unroll
  for (int i = 0; i < kItems; ++i)
    if ((take >> i & 1u) && o < k) out[o++] = (int32_t)(base + i);  // o < k always; kept in bounds
  for (long long i = (long long)blockIdx.x * kThreads + t; i < n_append; i += (long long)gridDim.x * kThreads)
    out[k + i] = (int32_t)(n + i);
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
  if (k == 0) return launch_iota(idx_out, n_append, n, s);
  if (k == n) return launch_iota(idx_out, n + n_append, 0, s);
  if (n <= kSmallMax) {
    hipLaunchKernelGGL(topk_small, dim3(1), dim3(kSmallThreads), 0, s, dev, (long long)n, (long long)k,
                       (long long)n_append, idx_out);
    return hipGetLastError();
  }
  const size_t state = sizeof(TopkState) > sizeof(TopkFused) ? sizeof(TopkState) : sizeof(TopkFused);
  unsigned int* bc = reinterpret_cast<unsigned int*>(static_cast<char*>(ws) + align256(state));
  const long long nblk = topk_blocks(n);
  if (n <= kFusedMaxRows) {
    TopkFused* fs = static_cast<TopkFused*>(ws);
    hipLaunchKernelGGL(topk_fused_init, dim3(1), dim3(kThreads), 0, s, fs);
    hipLaunchKernelGGL(topk_fused, dim3((unsigned)nblk), dim3(kThreads), 0, s, dev, (long long)n, (long long)k,
                       (long long)n_append, fs, bc, idx_out);
    return hipGetLastError();
  }
  TopkState* st = static_cast<TopkState*>(ws);
  long long pass_blocks = (n + kThreads * 8 - 1) / (kThreads * 8);
  if (pass_blocks > 1024) pass_blocks = 1024;
  hipLaunchKernelGGL(topk_init, dim3(1), dim3(kThreads), 0, s, st, (long long)k);
  for (int shift = 56; shift >= 0; shift -= 8)
    hipLaunchKernelGGL(topk_radix_pass, dim3((unsigned)pass_blocks), dim3(kThreads), 0, s, dev,
                       (long long)n, st, shift);
  hipLaunchKernelGGL(topk_count, dim3((unsigned)nblk), dim3(kThreads), 0, s, dev, (long long)n, st, bc);
  hipLaunchKernelGGL(topk_write, dim3((unsigned)nblk), dim3(kThreads), 0, s, dev, (long long)n, st,
                     bc, (long long)k, (long long)n_append, idx_out);
  return hipGetLastError();
}

}  // namespace kvc
