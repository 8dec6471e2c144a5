// Steps a4 (gather) + a5: causal GQA attention of sparse queries (gfx950).
//
// Paper: the selected tokens' queries attend to the whole blended cache
// with a mask that is causal by original position (Section 4 setup;
// Limitations, item 1, which asks for a fast attention over selected query
// indices).  For query i at position p_i and head h (kv head g = h / G):
//   O = softmax_j(scale * <q, k_j>) v_j over j <= p_i.
//
// A dense contraction, so it runs on the matrix cores:
// v_mfma_f32_32x32x16_bf16 (32x32 tile, K = 16, 8 bf16 per lane).
// - A workgroup (8 waves, two per SIMD) owns 32*8/hpw selected queries x
//   hpw query heads of one kv head (hpw = 4 for Llama's G = 4), so all
//   eight waves share every K/V tile staged in LDS.  Each wave owns 32
//   queries of one head.
// - Scores are computed transposed, S^T = K Q^T: in the accumulator each
//   lane holds one query and 16 keys, so the softmax max/sum are in-lane
//   plus one exchange with lane^32.
// - The accumulator of S^T is reused directly as the B operand of
//   O^T = V^T P^T.  V stays row-major in LDS; its V^T operand comes from
//   transposing LDS reads (ds_read_b64_tr_b16) whose per-lane addresses
//   follow the key order the accumulator implies inside each 16-key step
//   (bits 2 and 3 of the key index swapped), so no data moves between
//   lanes.
// - Online softmax in the exp2 domain (scale * log2 e folded into one FMA),
//   float32 accumulation; P is rounded to bf16 for the PV product and the
//   row sums add those same bf16 weights (v_dot2), so O is an exact
//   weighted average of V.  A tile's weights are taken against the lane's
//   current offset without waiting for the tile max: the lane's tile sum of
//   weights bounds them, and only a sum above 2^16 (or an overflow) sends
//   the wave into a rare branch that moves the offset of the queries
//   concerned to the tile max, scales O and takes the tile's weights again.
// - K/V tiles go from HBM straight into LDS (buffer loads with an LDS
//   destination, no registers, out-of-range rows arriving as zeros) into
//   four slots, three tiles ahead, with bank-spreading swizzles.
// - Software pipeline (one barrier per 64-key tile) in two phases of 16
//   MFMAs each: the QK^T MFMAs of tile t+1 beside the exponentials of the
//   second half of tile t, then the PV MFMAs of tile t beside the
//   exponentials of the first half of tile t+1.  Every MFMA is followed by
//   the LDS reads of a later operand and three VALU instructions, fenced so
//   the compiler keeps the interleave and both pipes stay fed.
// - Key tiles entirely below the smallest position of a wave skip the mask.
// - Workgroups run longest query block first, and consecutive workgroup
//   ids (which the dispatcher spreads over the 8 XCDs) take consecutive kv
//   heads, so with 8 kv heads each XCD's L2 serves one head's K/V.
// - A selection too small for two workgroups per CU can split every query
//   block's key tiles over several workgroups (when the caller provides the
//   workspace for their float32 partial outputs and LSEs); a second kernel
//   merges the partials of each query head in split order.

#include "kvc_internal.h"

#include <limits.h>

#include <type_traits>

namespace kvc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) v4s lds_v4s;

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kBN = 64;     // keys per tile
constexpr int kSlots = 4;                // LDS tile slots: tiles stream in three steps ahead
constexpr int kKGroup = 4 * kHeadDim + 32;    // bf16 per four K rows in LDS (1088 B: 64 B apart)
constexpr int kKSlot = (kBN / 4) * kKGroup;   // bf16 per K tile
constexpr int kVSlot = kBN * kHeadDim;        // bf16 per V tile (rows 256 B apart)
// s_waitcnt immediates (gfx9 encoding: vmcnt bits 3:0 and 15:14, expcnt
// 6:4, lgkmcnt 11:8): vector-memory count at most 4 or 0, LDS count 0.
// the four tile-load instructions of a step go after these MFMAs (bit i:
// MFMA i) of phase 1, then of phase 2 (after every fourth MFMA of phase 1
// measured best)
constexpr unsigned kLoadMask1 = 0x8888u;
constexpr unsigned kLoadMask2 = 0x0000u;
constexpr int kWaitVm4 = 4 | (7 << 4);
constexpr int kWaitVm0 = 0 | (7 << 4);
constexpr float kSumLimit = 65536.0f;     // bound on a lane's tile sum of weights (32 of them)

struct AttnParams {
  const uint16_t* q;
  long long n_q_rows;
  const int32_t* q_rows;
  const int32_t* q_pos;
  long long n_sel;
  const uint16_t* k;
  const uint16_t* v;
  long long n_kv;
  int n_q_heads;
  int n_kv_heads;
  int group;      // G = Hq / Hkv
  int hpw;        // query heads per workgroup (4, 2 or 1)
  int qpw;        // queries per workgroup = 32 * kWaves / hpw
  int n_hgroups;  // G / hpw
  int n_qblocks;
  float scale_log2;  // softmax scale * log2(e)
  uint16_t* out;
  float* lse;
  // split of each query block's key tiles over n_split workgroups: with
  // n_split > 1 every workgroup writes its normalised partial output and
  // its log2-domain LSE here, and attn_combine_kernel merges them
  int n_split;
  float* part_o;    // [n_split][n_sel][Hq][D]
  float* part_lse;  // [n_split][n_sel][Hq]
};

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& u) {
  return __builtin_bit_cast(bf16x8, u);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__global__ __launch_bounds__(kThreads) void sparse_attn_kernel(const AttnParams P) {
  // one array per slot, so alias analysis can tell a slot being loaded
  // from the slots being read
  __shared__ __attribute__((aligned(16))) uint16_t K0[kKSlot], K1[kKSlot], K2[kKSlot], K3[kKSlot];
  __shared__ __attribute__((aligned(16))) uint16_t V0[kVSlot], V1[kVSlot], V2[kVSlot], V3[kVSlot];
  uint16_t* const Ks[kSlots] = {K0, K1, K2, K3};
  uint16_t* const Vs[kSlots] = {V0, V1, V2, V3};
  __shared__ int s_pmax;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave-uniform, so tile LDS addresses and loop bounds stay in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ql = lane & 31;
  const int half = lane >> 5;

  const int hk_total = P.n_kv_heads * P.n_hgroups;
  const int hk = (int)(blockIdx.x % (unsigned)hk_total);
  const unsigned rest = blockIdx.x / (unsigned)hk_total;
  const int split = (int)(rest % (unsigned)P.n_split);
  const int qb = P.n_qblocks - 1 - (int)(rest / (unsigned)P.n_split);
  const int g = hk % P.n_kv_heads;
  const int hgroup = hk / P.n_kv_heads;
  const int hw = wave % P.hpw;
  const int qs = wave / P.hpw;
  const int h = g * P.group + hgroup * P.hpw + hw;
  const long long q0 = (long long)qb * P.qpw;
  const long long n_kv = P.n_kv;

  if (tid == 0) s_pmax = -1;
  __syncthreads();
  if (tid < P.qpw) {
    const long long qi = q0 + tid;
    if (qi < P.n_sel) {
      long long p = P.q_pos[qi];
      if (p > n_kv - 1) p = n_kv - 1;
      if (p >= 0) atomicMax(&s_pmax, (int)p);
    }
  }

  // this lane's query (one per lane pair l, l^32)
  const long long qi = q0 + (long long)qs * 32 + ql;
  const bool in_range = qi < P.n_sel;
  int p = -1;
  long long row = -1;
  if (in_range) {
    long long pp = P.q_pos[qi];
    row = P.q_rows ? (long long)P.q_rows[qi] : qi;
    if (row < 0 || row >= P.n_q_rows) { row = -1; pp = -1; }
    if (pp > n_kv - 1) pp = n_kv - 1;
    p = (int)(pp < 0 ? -1 : pp);
  }
  uint4 qraw[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) qraw[ks] = make_uint4(0, 0, 0, 0);
  if (row >= 0) {
    const uint16_t* qp = P.q + (row * P.n_q_heads + h) * (long long)kHeadDim + half * 8;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qraw[ks] = *reinterpret_cast<const uint4*>(qp + ks * 16);
  }
  // Consume the query registers here so the loads complete before the key
  // loop; otherwise the wait-count pass treats them as possibly in flight in
  // every iteration and waits for the next tile's prefetch before the MFMAs.
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    uint32_t a = qraw[ks].x, b = qraw[ks].y, c = qraw[ks].z, d = qraw[ks].w;
    asm volatile("" : "+v"(a), "+v"(b), "+v"(c), "+v"(d));
    qraw[ks] = make_uint4(a, b, c, d);
  }
  bf16x8 qreg[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) qreg[ks] = as_bf16x8(qraw[ks]);
  // smallest position among the wave's live queries (tiles at or below it need no mask)
  int pw_min = in_range ? p : INT_MAX;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) pw_min = min(pw_min, __shfl_xor(pw_min, m));
  pw_min = __builtin_amdgcn_readfirstlane(pw_min);  // equal in every lane: the mask test is scalar
  __syncthreads();
  const int pmax = s_pmax;
  // this workgroup's share of the block's key tiles (all of them unless split)
  const int n_all = (pmax + kBN) / kBN;  // pmax = -1 -> 0 tiles
  const int t0 = (int)((long long)n_all * split / P.n_split);
  const int n_tiles = (int)((long long)n_all * (split + 1) / P.n_split) - t0;

  // Tiles go straight from HBM to LDS (buffer loads with an LDS destination:
  // lane l of an instruction writes 16 bytes at the wave's LDS address +
  // 16 l), so staging them costs no registers and no VALU.  The scalar base
  // of the buffer resource moves by one tile per step and the per-lane
  // offsets stay fixed; rows at or past n_kv fall outside the resource and
  // arrive as zeros.  Wave w loads rows 8w .. 8w+7 of the K and of the V
  // tile, four rows per instruction.  LDS layouts, in 16-byte pieces
  // p = 0..15 of a 256-byte row:
  //   K: groups of four rows 1088 bytes apart, row r of a group at 256 r,
  //      piece p stored at p ^ (r & 3), so the QK^T operand reads (16 rows,
  //      one piece) fall in 16 distinct bank groups;
  //   V: rows 256 bytes apart, piece p stored at p ^ 4 (r & 3), so the
  //      transposing PV operand reads (4 rows x 4 pieces per half wave)
  //      fall in 16 distinct bank groups.
  const long long row_bytes = (long long)P.n_kv_heads * kHeadDim * 2;
  const char* kbase = reinterpret_cast<const char*>(P.k);
  const char* vbase = reinterpret_cast<const char*>(P.v);
  int koff[2], voff[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = 8 * wave + 4 * j + (lane >> 4);  // tile row this lane fills
    const int slot = lane & 15;                     // its piece position in LDS
    koff[j] = (int)(r * row_bytes) + g * kHeadDim * 2 + 16 * (slot ^ (r & 3));
    voff[j] = (int)(r * row_bytes) + g * kHeadDim * 2 + 16 * (slot ^ (4 * (r & 3)));
  }
  // load part q (0..3) of tile t: K rows (q = 0, 1) or V rows (q = 2, 3)
  // Rows in key tile i: kBN below n_full, the tail at n_full (the tiles a
  // workgroup loads never start past its last visible key, so never past
  // n_kv); int32 compares keep the count in scalar instructions.
  const int n_full = (int)(n_kv / kBN);
  const int n_tail = (int)(n_kv % kBN);
  auto load_part = [&](int t, uint16_t* ks_, uint16_t* vs_, int q) __attribute__((always_inline)) {
    const int tile = t0 + t;
    const long long r0 = (long long)tile * kBN;
    const int rows = tile < n_full ? kBN : (tile == n_full ? n_tail : 0);
    const int nbytes = rows * (int)row_bytes;
    const int j = q & 1;
    if (q < 2) {
      const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)(kbase + r0 * row_bytes), (short)0, nbytes, 0x00020000);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(ks_ + (2 * wave + j) * kKGroup), 16, koff[j], 0, 0, 0);
    } else {
      const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)(vbase + r0 * row_bytes), (short)0, nbytes, 0x00020000);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(vs_ + (8 * wave + 4 * j) * kHeadDim), 16, voff[j], 0, 0, 0);
    }
  };
  auto load_tile = [&](int t, uint16_t* ks_, uint16_t* vs_) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 4; ++q) load_part(t, ks_, vs_, q);
  };
  // QK^T operand (A = K rows kb*32 + lane%32, dims 16 ks + 8 half .. +8):
  // the swizzled piece is 2 (ks ^ e1) + (half ^ (lane & 1)), e1 = bit 1 of
  // the lane, so even and odd ks use two bases with immediate offsets.
  const int k_a0 = (ql >> 2) * kKGroup + (lane & 3) * kHeadDim + 8 * (half ^ (lane & 1));
  const int k_e1 = 16 * ((lane >> 1) & 1);
  const int k_rd[2] = {k_a0 + k_e1, k_a0 - k_e1};
  // PV operand (A = V^T: dims 32 dt + lane%32, keys of step kk in the order
  // the S^T accumulator gives them, 8 (e/4) + 4 half + e%4 for e = 0..7),
  // read with ds_read_b64_tr_b16: in each 16-lane group, lane j receives
  // element j%4 of the 4-element pieces addressed by lanes j/4 + 4r,
  // r = 0..3.  Lane i of group (half, gd) addresses key 4 half + i/4 and
  // dims 32 dt + 16 gd + 4 (i%4), so lane j gets four consecutive keys of
  // dim 32 dt + 16 gd + j.
  int v_rd[4];
  {
    const int i = lane & 15, gd = (lane >> 4) & 1, sr = i >> 2;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
      v_rd[dt] = (4 * half + sr) * kHeadDim + 32 * (dt ^ sr) + 16 * gd + 4 * (i & 3);
  }
  auto k_frag = [&](const uint16_t* ks_, int i) __attribute__((always_inline)) {
    const int kb = i >> 3, ks = i & 7;
    return *reinterpret_cast<const uint4*>(ks_ + k_rd[ks & 1] + kb * 8 * kKGroup + 16 * ks);
  };
  auto v_frag = [&](const uint16_t* vs_, int i) __attribute__((always_inline)) {
    const int kk = i >> 2, dt = i & 3;
    const uint16_t* b = vs_ + v_rd[dt] + kk * 16 * kHeadDim;
    const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(b));
    const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(b + 8 * kHeadDim));
    const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
    return make_uint4(l2.x, l2.y, h2.x, h2.y);
  };
  // S^T = K Q^T for the 64 keys of a K tile
  auto qk = [&](const uint16_t* ks_, f32x16* s) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int kb = i >> 3, ks = i & 7;
      s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(k_frag(ks_, i)), qreg[ks], ks == 0 ? f32x16{} : s[kb], 0, 0, 0);
    }
  };

  // Running max (log2 domain) of the lane's query, and the offset the
  // exponentials subtract (0 while the query has seen no key).
  float m_run = -INFINITY;
  float m_use = 0.f;
  float l_run = 0.f;        // this lane's partial sum (its 16 keys of each 32)
  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.f;
  const float c2 = P.scale_log2;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  auto mask = [&](int t, f32x16* s) __attribute__((always_inline)) {
    const int key0 = (t0 + t) * kBN;
    if (key0 + kBN - 1 > pw_min) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + kb * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
          s[kb][r] = key > p ? -INFINITY : s[kb][r];
        }
    }
  };
  // max over a tile of the lane's query (log2 domain); lanes l and l^32 hold
  // the two halves of the same query's keys
  auto tile_max = [&](const f32x16* s) __attribute__((always_inline)) {
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * c2;
  };
  // Weights of half a tile (keys 32*hf .. 32*hf+31, accumulator s[hf]) as
  // the bf16 B operands of two 16-key PV steps; the tile sum adds those same
  // bf16 weights.
  auto exp_half = [&](const f32x16* s, auto hfc, bf16x8* pb2, float& lt) __attribute__((always_inline)) {
    constexpr int hf = decltype(hfc)::value;
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[hf][k2 * 8 + 2 * e], c2, -m_use));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[hf][k2 * 8 + 2 * e + 1], c2, -m_use));
        const f32x2 pv2 = {p0, p1};
        const bf16x2 pw = __builtin_convertvector(pv2, bf16x2);
        lt = __builtin_amdgcn_fdot2_f32_bf16(pw, ones, lt, false);
        w[e] = __builtin_bit_cast(uint32_t, pw);
      }
      pb2[k2] = as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
    }
  };
  using H0 = std::integral_constant<int, 0>;
  using H1 = std::integral_constant<int, 1>;
  // The weights of a tile are taken against the current offset without
  // first looking at the tile max; the lane's tile sum then bounds them.  A
  // sum above kSumLimit (weights too large, or an overflow) sends the wave
  // into this rare branch: the queries concerned move their running
  // max up to the tile max, scale O and their sum, and every weight of the
  // tile is taken again.  Other queries keep their offset and get the same
  // weights again, so a query's result does not depend on the other
  // queries of its wave.
  auto redo = [&](const f32x16* s, bf16x8* pl, bf16x8* ph, float& lt, bool bad) __attribute__((always_inline)) {
    const float mt = tile_max(s);
    const auto sw = __builtin_amdgcn_permlane32_swap((uint32_t)bad, (uint32_t)bad, false, false);
    const bool bad_q = (sw[0] | sw[1]) != 0u;
    const float m_new = bad_q ? fmaxf(m_run, mt) : m_run;
    const float alpha = m_new > m_run ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;
    l_run *= alpha;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
    m_run = m_new;
    m_use = (m_run == -INFINITY) ? 0.f : m_run;
    lt = 0.f;
    exp_half(s, H0{}, pl, lt);
    exp_half(s, H1{}, ph, lt);
  };
  // O^T += V^T P^T for a V^T tile, 16 keys per step (steps 0, 1 from the
  // tile's first half, 2, 3 from its second)
  auto pv = [&](const bf16x8* pl, const bf16x8* ph, const uint16_t* vs_) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int kk = i >> 2, dt = i & 3;
      o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(v_frag(vs_, i)), kk < 2 ? pl[kk] : ph[kk - 2], o[dt], 0, 0, 0);
    }
  };
  // The two phases of a pipeline step.  Each issues 16 MFMAs of one product
  // and, between them, the 48 VALU instructions that turn half a tile of
  // scores into weights: every MFMA is followed by the LDS read for the MFMA
  // two places later and by three VALU instructions (one weight pair per
  // two MFMAs: exponent FMAs, exponentials, bf16 pack, sum) that run two
  // places ahead, so the first of them cover the latency of the first LDS
  // reads.  The groups are fenced so the compiler keeps this order.
  auto exp_part = [&](const f32x16* se, int hf, int i, float& p0, float& x1, uint32_t (&w)[2][4], float& lt)
      __attribute__((always_inline)) {
    const int j = i >> 1, k2 = j >> 2, e = j & 3;
    if ((i & 1) == 0) {
      p0 = __builtin_amdgcn_exp2f(fmaf(se[hf][k2 * 8 + 2 * e], c2, -m_use));
      x1 = fmaf(se[hf][k2 * 8 + 2 * e + 1], c2, -m_use);
    } else {
      const float p1 = __builtin_amdgcn_exp2f(x1);
      const f32x2 pv2 = {p0, p1};
      const bf16x2 pw = __builtin_convertvector(pv2, bf16x2);
      lt = __builtin_amdgcn_fdot2_f32_bf16(pw, ones, lt, false);
      w[k2][e] = __builtin_bit_cast(uint32_t, pw);
    }
  };
  // phase 1: S^T of the next tile (K tile ks_) beside the weights of the
  // second half of the current tile (scores se); its last two slots read
  // the first two V^T fragments of phase 2 (tile vt_) into fv.
  auto phase1 = [&](const uint16_t* ks_, f32x16* sq, const f32x16* se, bf16x8* ph, float& lt,
                    const uint16_t* vt_, uint4 (&fv)[2], auto&& after) __attribute__((always_inline)) {
    uint4 fr[3];
    float p0 = 0.f, x1 = 0.f;
    uint32_t w[2][4];
    fr[0] = k_frag(ks_, 0);
    fr[1] = k_frag(ks_, 1);
    __builtin_amdgcn_sched_barrier(0);
    exp_part(se, 1, 0, p0, x1, w, lt);
    exp_part(se, 1, 1, p0, x1, w, lt);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i + 2 < 16) fr[(i + 2) % 3] = k_frag(ks_, i + 2);
      else fv[i - 14] = v_frag(vt_, i - 14);
      const int kb = i >> 3, ks = i & 7;
      sq[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(fr[i % 3]), qreg[ks], ks == 0 ? f32x16{} : sq[kb], 0, 0, 0);
      if (i + 2 < 16) exp_part(se, 1, i + 2, p0, x1, w, lt);
      after(i);
      __builtin_amdgcn_sched_barrier(0);
    }
    ph[0] = as_bf16x8(make_uint4(w[0][0], w[0][1], w[0][2], w[0][3]));
    ph[1] = as_bf16x8(make_uint4(w[1][0], w[1][1], w[1][2], w[1][3]));
  };
  // phase 2: O^T += V^T P^T for the current tile (V^T tile vt_, weights pl,
  // ph; first two fragments already in fv) beside the weights of the first
  // half of the next tile (scores se)
  auto phase2 = [&](const uint16_t* vt_, const uint4 (&fv)[2], const bf16x8* pl, const bf16x8* ph,
                    const f32x16* se, bf16x8* pn, float& lt, auto&& after) __attribute__((always_inline)) {
    uint4 fr[3];
    float p0 = 0.f, x1 = 0.f;
    uint32_t w[2][4];
    fr[0] = fv[0];
    fr[1] = fv[1];
    exp_part(se, 0, 0, p0, x1, w, lt);
    exp_part(se, 0, 1, p0, x1, w, lt);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i + 2 < 16) fr[(i + 2) % 3] = v_frag(vt_, i + 2);
      const int kk = i >> 2, dt = i & 3;
      o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(fr[i % 3]), kk < 2 ? pl[kk] : ph[kk - 2], o[dt], 0, 0, 0);
      if (i + 2 < 16) exp_part(se, 0, i + 2, p0, x1, w, lt);
      after(i);
      __builtin_amdgcn_sched_barrier(0);
    }
    pn[0] = as_bf16x8(make_uint4(w[0][0], w[0][1], w[0][2], w[0][3]));
    pn[1] = as_bf16x8(make_uint4(w[1][0], w[1][1], w[1][2], w[1][3]));
  };

  // Software pipeline over key tiles: four LDS slots, tiles arriving three
  // steps ahead, one barrier per tile.  Entering step t, the scores of tile
  // t are in s[t%2] and the weights of its first half in pbl[t%2].  Step t:
  //   phase 1: QK^T MFMAs of tile t+1 beside the exponentials of the second
  //     half of tile t, with the four load instructions of tile t+3 (into
  //     slot (t+3)%4, whose tile t-1 was last read in step t-1 before the
  //     previous barrier) spread over it: issued together after the
  //     barrier, the eight waves' loads made a burst of LDS writes that
  //     delayed the first operand reads;
  //   bound check of tile t (rare branch), mask of tile t+1 (branch, only
  //     on tiles reaching past the wave's smallest position);
  //   phase 2: PV MFMAs of tile t beside the exponentials of the first half
  //     of tile t+1;
  //   wait for this wave's loads of tile t+2 (issued one step earlier;
  //     only the four of tile t+3 stay in flight), then the barrier, after
  //     which every wave's part of tile t+2 is in LDS.
  // The loop is unrolled four times so slots (t%4) and score registers
  // (t%2) are static.  The wait is explicit and the barrier has no fence:
  // a fence would also wait for the loads of tile t+3.
  f32x16 s[2][2];
  bf16x8 pbl[2][2], pbh[2];
  float lt[2] = {0.f, 0.f};
  auto check = [&](auto parc) __attribute__((always_inline)) {
    constexpr int PA = decltype(parc)::value;
    const bool bad = !(lt[PA] <= kSumLimit);
    if (__any(bad)) redo(s[PA], pbl[PA], pbh, lt[PA], bad);
    l_run += lt[PA];
  };
  auto step = [&](auto slotc, auto parc, int t) __attribute__((always_inline)) {
    constexpr int B0 = decltype(slotc)::value;
    constexpr int B1 = (B0 + 1) % kSlots;
    constexpr int B3 = (B0 + 3) % kSlots;
    constexpr int PA = decltype(parc)::value;
    // loads of tile t+3, spread over phase 1 (the last tile may load again; harmless)
    const int tl = min(t + 3, n_tiles - 1);
    uint4 fv[2];
    phase1(Ks[B1], s[1 - PA], s[PA], pbh, lt[PA], Vs[B0], fv, [&](int i) __attribute__((always_inline)) {
      if (kLoadMask1 >> i & 1) load_part(tl, Ks[B3], Vs[B3], __builtin_popcount(kLoadMask1 & ((1u << i) - 1)));
    });
    check(parc);
    mask(t + 1, s[1 - PA]);
    lt[1 - PA] = 0.f;
    phase2(Vs[B0], fv, pbl[PA], pbh, s[1 - PA], pbl[1 - PA], lt[1 - PA], [&](int i) __attribute__((always_inline)) {
      if (kLoadMask2 >> i & 1) load_part(tl, Ks[B3], Vs[B3], __builtin_popcount(kLoadMask1) + __builtin_popcount(kLoadMask2 & ((1u << i) - 1)));
    });
    __builtin_amdgcn_s_waitcnt(kWaitVm4);
    __builtin_amdgcn_s_barrier();
  };
  auto last = [&](auto slotc, auto parc, int t) __attribute__((always_inline)) {
    constexpr int B0 = decltype(slotc)::value;
    constexpr int PA = decltype(parc)::value;
    exp_half(s[PA], H1{}, pbh, lt[PA]);
    check(parc);
    pv(pbl[PA], pbh, Vs[B0]);
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;

  if (n_tiles > 0) {
    load_tile(0, Ks[0], Vs[0]);
    load_tile(min(1, n_tiles - 1), Ks[1], Vs[1]);
    load_tile(min(2, n_tiles - 1), Ks[2], Vs[2]);
  }
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __builtin_amdgcn_s_barrier();
  if (n_tiles > 0) {
    qk(Ks[0], s[0]);
    mask(0, s[0]);
    m_run = tile_max(s[0]);
    m_use = (m_run == -INFINITY) ? 0.f : m_run;
    exp_half(s[0], H0{}, pbl[0], lt[0]);
    int t = 0;
    for (; t + 4 < n_tiles; t += 4) {
      step(I0{}, I0{}, t);
      step(I1{}, I1{}, t + 1);
      step(I2{}, I0{}, t + 2);
      step(I3{}, I1{}, t + 3);
    }
    // t is a multiple of 4 here; at most three full steps remain
    if (t + 1 < n_tiles) { step(I0{}, I0{}, t); ++t; }
    if (t + 1 < n_tiles) { step(I1{}, I1{}, t); ++t; }
    if (t + 1 < n_tiles) { step(I2{}, I0{}, t); ++t; }
    switch (t % 4) {
      case 0: last(I0{}, I0{}, t); break;
      case 1: last(I1{}, I1{}, t); break;
      case 2: last(I2{}, I0{}, t); break;
      default: last(I3{}, I1{}, t); break;
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!in_range) return;
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (P.n_split > 1) {
    const long long pi = ((long long)split * P.n_sel + qi) * P.n_q_heads + h;
    float* po = P.part_o + pi * kHeadDim + half * 4;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr)
        *reinterpret_cast<float4*>(po + dt * 32 + rr * 8) =
            make_float4(o[dt][rr * 4] * inv, o[dt][rr * 4 + 1] * inv, o[dt][rr * 4 + 2] * inv, o[dt][rr * 4 + 3] * inv);
    if (half == 0) P.part_lse[pi] = (l_tot > 0.f) ? m_run + log2f(l_tot) : -INFINITY;
    return;
  }
  uint16_t* op = P.out + (qi * P.n_q_heads + h) * (long long)kHeadDim + half * 4;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const uint32_t w0 = pack_bf16x2(o[dt][rr * 4 + 0] * inv, o[dt][rr * 4 + 1] * inv);
      const uint32_t w1 = pack_bf16x2(o[dt][rr * 4 + 2] * inv, o[dt][rr * 4 + 3] * inv);
      *reinterpret_cast<uint2*>(op + dt * 32 + rr * 8) = make_uint2(w0, w1);
    }
  if (P.lse && half == 0)
    P.lse[qi * P.n_q_heads + h] = (l_tot > 0.f) ? (m_run + log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
}

// Merge of the split partials of one (query, head) pair per wave, two
// channels per lane: weights 2^(lse_s - max) in split order, so the result
// is deterministic; a pair with no visible key gets 0 and LSE -inf.
__global__ __launch_bounds__(256) void attn_combine_kernel(const float* __restrict__ part_o,
                                                           const float* __restrict__ part_lse, int n_split,
                                                           long long n_pairs, uint16_t* __restrict__ out,
                                                           float* __restrict__ lse) {
  const long long pair = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (pair >= n_pairs) return;
  const int lane = threadIdx.x & 63;
  float m = -INFINITY;
  for (int sp = 0; sp < n_split; ++sp) m = fmaxf(m, part_lse[sp * n_pairs + pair]);
  float a0 = 0.f, a1 = 0.f, wsum = 0.f;
  if (m > -INFINITY) {
    for (int sp = 0; sp < n_split; ++sp) {
      const float l = part_lse[sp * n_pairs + pair];
      if (l == -INFINITY) continue;
      const float w = __builtin_amdgcn_exp2f(l - m);
      const float2 v = *reinterpret_cast<const float2*>(part_o + (sp * n_pairs + pair) * kHeadDim + 2 * lane);
      wsum += w;
      a0 = fmaf(w, v.x, a0);
      a1 = fmaf(w, v.y, a1);
    }
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  reinterpret_cast<uint32_t*>(out + pair * kHeadDim)[lane] = pack_bf16x2(a0 * inv, a1 * inv);
  if (lse && lane == 0) lse[pair] = wsum > 0.f ? (m + log2f(wsum)) * 0.69314718055994531f : -INFINITY;
}

// Splitting aims at one workgroup per CU with at least 4 key tiles each
// (below one workgroup per CU; between one and two per CU, two splits):
// measured against two per CU and 8 tiles, 4.1k at 15 % takes 56 instead of
// 76 us, 32k at 5 % 541 instead of 561 us, Tiny 22.6 instead of 25.3 us
// (more splits cost more partial writes and merging than they balance).
constexpr int kTargetWorkgroups = 256;
constexpr int kMaxSplit = 8;
constexpr int kMinTilesPerSplit = 4;

struct Grid {
  int hpw, qpw, n_hgroups, n_qblocks;
  long long n_wg;
};
Grid grid_of(int64_t n_sel, int n_q_heads, int n_kv_heads) {
  Grid g;
  const int group = n_q_heads / n_kv_heads;
  g.hpw = (group % 4 == 0) ? 4 : (group % 2 == 0) ? 2 : 1;
  g.qpw = 32 * (kWaves / g.hpw);
  g.n_hgroups = group / g.hpw;
  g.n_qblocks = (int)((n_sel + g.qpw - 1) / g.qpw);
  g.n_wg = (long long)g.n_qblocks * n_kv_heads * g.n_hgroups;
  return g;
}

}  // namespace

int attention_splits(int64_t n_sel, int n_q_heads, int n_kv_heads) {
  if (n_sel <= 0) return 1;
  const Grid g = grid_of(n_sel, n_q_heads, n_kv_heads);
  if (g.n_wg >= 2 * kTargetWorkgroups) return 1;
  // one to two workgroups per CU: with positions spread over the context
  // the longest query blocks alone would set the time (about twice the
  // average load), so halve every block's key range
  if (g.n_wg >= kTargetWorkgroups) return 2;
  const long long s = (kTargetWorkgroups + g.n_wg - 1) / g.n_wg;
  return (int)(s < kMaxSplit ? s : kMaxSplit);
}

int64_t attention_work_items(int64_t n_sel, int n_q_heads, int n_kv_heads) {
  if (n_sel <= 0) return 0;
  return grid_of(n_sel, n_q_heads, n_kv_heads).n_wg * kThreads;
}

size_t attention_ws_bytes(int64_t n_sel, int n_q_heads, int n_kv_heads) {
  const int sp = attention_splits(n_sel, n_q_heads, n_kv_heads);
  if (sp <= 1) return 0;
  return (size_t)sp * (size_t)n_sel * (size_t)n_q_heads * (kHeadDim + 1) * sizeof(float);
}

hipError_t launch_attention(const uint16_t* q, int64_t n_q_rows, const int32_t* q_rows,
                            const int32_t* q_pos, int64_t n_sel, const uint16_t* k,
                            const uint16_t* v, int64_t n_kv, int n_q_heads, int n_kv_heads,
                            float scale, uint16_t* out, float* lse, void* ws, size_t ws_bytes,
                            hipStream_t s) {
  if (n_sel <= 0) return hipSuccess;
  AttnParams P;
  P.q = q;
  P.n_q_rows = n_q_rows;
  P.q_rows = q_rows;
  P.q_pos = q_pos;
  P.n_sel = n_sel;
  P.k = k;
  P.v = v;
  P.n_kv = n_kv;
  P.n_q_heads = n_q_heads;
  P.n_kv_heads = n_kv_heads;
  const Grid g = grid_of(n_sel, n_q_heads, n_kv_heads);
  P.group = n_q_heads / n_kv_heads;
  P.hpw = g.hpw;
  P.qpw = g.qpw;
  P.n_hgroups = g.n_hgroups;
  P.n_qblocks = g.n_qblocks;
  P.scale_log2 = scale * 1.4426950408889634f;
  P.out = out;
  P.lse = lse;
  // split the key tiles only with the workspace for the partials, and only
  // as far as every split keeps kMinTilesPerSplit tiles of the longest block
  int sp = 1;
  const size_t need = attention_ws_bytes(n_sel, n_q_heads, n_kv_heads);
  if (ws && need > 0 && ws_bytes >= need) {
    const long long tiles = (n_kv + kBN - 1) / kBN;
    const long long cap = tiles / kMinTilesPerSplit;
    sp = attention_splits(n_sel, n_q_heads, n_kv_heads);
    if (sp > cap) sp = (int)(cap > 1 ? cap : 1);
  }
  P.n_split = sp;
  P.part_o = sp > 1 ? static_cast<float*>(ws) : nullptr;
  P.part_lse = sp > 1 ? P.part_o + (size_t)sp * n_sel * n_q_heads * kHeadDim : nullptr;
  hipLaunchKernelGGL(sparse_attn_kernel, dim3((unsigned)(g.n_wg * sp)), dim3(kThreads), 0, s, P);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || sp == 1) return e;
  const long long pairs = n_sel * (long long)n_q_heads;
  hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)((pairs + 3) / 4)), dim3(256), 0, s, P.part_o,
                     P.part_lse, sp, pairs, out, lse);
  return hipGetLastError();
}

}  // namespace kvc
