// Internal declarations shared by the host plan code and the HIP kernels of
// the nested-Winograd library.  Not part of the public ABI (see include/nwg.h).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "../../include/nwg.h"
#include "plan.h"

namespace nwg {

// ---------------------------------------------------------------------------
// Base F(2,3) (eq. 2.3), applied to values spaced by a stride.
//   B^T rows: q0 = x0 - x2, q1 = x1 + x2, q2 = x2 - x1, q3 = x1 - x3
//   G   rows: g0 = w0, g1 = (w0+w1+w2)/2, g2 = (w0-w1+w2)/2, g3 = w2
//   A^T rows: y0 = v0 + v1 + v2, y1 = v1 - v2 - v3
// ---------------------------------------------------------------------------

// Work-group i of G -> logical block: the dispatcher deals work-groups
// round-robin over the 8 XCDs (i % 8); this numbering gives each XCD a
// contiguous run of logical blocks, so blocks that share operand tiles
// share one L2.
__device__ __forceinline__ long long xcd_remap(long long i, long long G) {
  const long long q = G / 8, rem = G % 8;
  const long long xcd = i % 8, slot = i / 8;
  return xcd < rem ? xcd * (q + 1) + slot : rem * (q + 1) + (xcd - rem) * q + slot;
}

// Position of the k-th set bit (k from 0) of the 128-bit mask (w1:w0).
__device__ __forceinline__ int select_bit(unsigned long long w0, unsigned long long w1, int k) {
  const int c0 = __popcll(w0);
  unsigned long long w = k < c0 ? w0 : w1;
  int pos = k < c0 ? 0 : 64;
  k = k < c0 ? k : k - c0;
#pragma unroll
  for (int sh = 32; sh >= 1; sh >>= 1) {
    const unsigned long long low = w & ((1ULL << sh) - 1);
    const int c = __popcll(low);
    if (k >= c) {
      k -= c;
      w >>= sh;
      pos += sh;
    } else {
      w = low;
    }
  }
  return pos;
}

// Live bits of the four axis prefixes 4 b .. 4 b + 3 (level-2 digit q2 =
// 0..3 under the block b of the digits above it: b = 5 q4 + q3 on the mixed
// nest at depth 4, 4 q4 + q3 on four F(2,3) levels, q3 at depth 3): a
// nibble, which never straddles two 32-bit words of the mask.
__device__ __forceinline__ unsigned prefix_nibble(unsigned long long m0, unsigned long long m1,
                                                  int b) {
  const int i = 4 * b;
  const unsigned long long w = i < 64 ? m0 : m1;
  const unsigned h = (i & 63) < 32 ? (unsigned)w : (unsigned)(w >> 32);
  return (h >> (i & 31)) & 0xfu;
}

// The live groups (q2r, q2c) of a branch from its row and column nibbles,
// as a 16-bit mask, bit 4 q2r + q2c.
__device__ __forceinline__ unsigned nibble_live(unsigned nr, unsigned nc) {
  unsigned live = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) live |= ((nr >> q) & 1u) ? nc << (4 * q) : 0u;
  return live;
}

// Stores of the live quads only, without a branch per quad (branches
// around the 64 stores of an unrolled branch transform make the compiler
// spill): every quad goes through a raw buffer resource that spans the
// wave's branches, and the lanes of a dead quad (its group dead, or its
// level-1 row digit q1r = 3 when q3 is set) pass an offset past the range,
// which the hardware drops with no memory traffic.
constexpr unsigned kDrop = 0x80000000u;     // above every span (host checks)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t span_rsrc(float4* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ void drop_store(__amdgpu_buffer_rsrc_t r, unsigned off, float4 v) {
  typedef unsigned u4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, v), r, (int)off, 0, 0);
}

// soff: a wave-uniform byte offset added to off (kDrop + soff stays past
// every span: the host keeps spans and soff below 2^30)
__device__ __forceinline__ void drop_store1(__amdgpu_buffer_rsrc_t r, unsigned off, float v,
                                            unsigned soff = 0) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)off, (int)soff, 0);
}

// Entry i of a plan's group list (GroupMap): the group the contraction
// computes as its i-th.
__device__ __forceinline__ long long live_group(const GroupMap& m, long long i) {
  if (m.np == 0) return i;
  const int ir = (int)(i / m.np), ic = (int)(i - (long long)ir * m.np);
  int pr = select_bit(m.mask0, m.mask1, ir), pc = select_bit(m.mask0, m.mask1, ic);
  long long g = 0;
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    if (d < m.nd) {
      g += (long long)(pr % m.rad[d]) * m.wr[d] + (long long)(pc % m.rad[d]) * m.wc[d];
      pr /= m.rad[d];
      pc /= m.rad[d];
    }
  }
  return g;
}

// Wait until at most N vector-memory loads of this wavefront are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// ---------------------------------------------------------------------------
// Two-term bf16 split (precision NWG_PRECISION_BF16_SPLIT): v ~ hi + lo with
// hi = bf16(v) and lo = bf16(v - hi), both rounded to nearest even; packed
// in one 32-bit word, hi in the low half.  hi + lo carries 16 significant
// bits of v.  Finite inputs (a NaN or infinity gives an unspecified pair).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t bf16_rne_bits(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ uint32_t split_pair(float v) {
  const uint32_t hi = bf16_rne_bits(v);
  const uint32_t lo = bf16_rne_bits(v - __uint_as_float(hi << 16));
  return hi | (lo << 16);
}
// a Winograd-domain quad as stored: fp32 values, or their split pairs
template <bool SPLIT>
__device__ __forceinline__ float4 store_quad(float a, float b, float c, float d) {
  if constexpr (SPLIT)
    return make_float4(__uint_as_float(split_pair(a)), __uint_as_float(split_pair(b)),
                       __uint_as_float(split_pair(c)), __uint_as_float(split_pair(d)));
  else
    return make_float4(a, b, c, d);
}

constexpr int kBase = 4;   // l
constexpr int kOut = 2;    // m
constexpr int kTaps = 3;   // r of the base

// Taps of row q of B^T: offsets in units of the level stride, and signs.
__host__ __device__ constexpr int bt_tap0(int q) { return q == 0 ? 0 : 1; }
__host__ __device__ constexpr int bt_tap1(int q) { return q == 3 ? 3 : 2; }
__host__ __device__ constexpr float bt_sign0(int q) { return q == 2 ? -1.0f : 1.0f; }
__host__ __device__ constexpr float bt_sign1(int q) { return (q == 0 || q == 3) ? -1.0f : 1.0f; }

// One level of B^T at stride S on a vector v: out[q][u] = sum_a BT[q][a] v[u + S a].
template <int S, int LEN>
__device__ __forceinline__ void bt_level(const float* v, float (*out)[LEN]) {
#pragma unroll
  for (int u = 0; u < LEN; ++u) {
    out[0][u] = v[u] - v[u + 2 * S];
    out[1][u] = v[u + S] + v[u + 2 * S];
    out[2][u] = v[u + 2 * S] - v[u + S];
    out[3][u] = v[u + S] - v[u + 3 * S];
  }
}

// Two inner levels of the nested input transform on a length-10 vector:
// level 2 (stride 2) then level 1 (stride 1); out index = q2*4 + q1.
// Q3: level-1 digit 3 is not needed (its output is set to 0), nor v[9].
template <bool Q3 = false>
__device__ __forceinline__ void bt_inner2(const float (&v)[10], float (&out)[16]) {
  float z[4][Q3 ? 3 : 4];
  bt_level<2, Q3 ? 3 : 4>(v, z);
#pragma unroll
  for (int q2 = 0; q2 < 4; ++q2) {
    out[q2 * 4 + 0] = z[q2][0] - z[q2][2];
    out[q2 * 4 + 1] = z[q2][1] + z[q2][2];
    out[q2 * 4 + 2] = z[q2][2] - z[q2][1];
    if constexpr (Q3)
      out[q2 * 4 + 3] = 0.0f;
    else
      out[q2 * 4 + 3] = z[q2][1] - z[q2][3];
  }
}

__device__ __forceinline__ void bt_one(const float (&v)[4], float (&out)[4]) {
  out[0] = v[0] - v[2];
  out[1] = v[1] + v[2];
  out[2] = v[2] - v[1];
  out[3] = v[1] - v[3];
}

__device__ __forceinline__ void g_one(float w0, float w1, float w2, float (&out)[4]) {
  out[0] = w0;
  out[1] = 0.5f * (w0 + w1 + w2);
  out[2] = 0.5f * (w0 - w1 + w2);
  out[3] = w2;
}

// G coefficient G[q][k].
__host__ __device__ constexpr float g_coef(int q, int k) {
  return q == 0 ? (k == 0 ? 1.0f : 0.0f)
       : q == 3 ? (k == 2 ? 1.0f : 0.0f)
       : q == 1 ? 0.5f
       : (k == 1 ? -0.5f : 0.5f);
}

// A^T coefficient A^T[i][q].
__host__ __device__ constexpr float at_coef(int i, int q) {
  return i == 0 ? (q == 3 ? 0.0f : 1.0f)
                : (q == 0 ? 0.0f : (q == 1 ? 1.0f : -1.0f));
}

// ---- helpers shared by the F(2,3) kernels ----------------------------------

// inner G transform (level 2 over k2, level 1 over k1) of a 9-vector
// indexed k2*3 + k1 -> 16 values indexed q2*4 + q1
__device__ __forceinline__ void g_inner2(const float (&v)[9], float (&out)[16]) {
  float h[4][3];
#pragma unroll
  for (int k1 = 0; k1 < 3; ++k1) {
    float o[4];
    g_one(v[0 * 3 + k1], v[1 * 3 + k1], v[2 * 3 + k1], o);
#pragma unroll
    for (int q = 0; q < 4; ++q) h[q][k1] = o[q];
  }
#pragma unroll
  for (int q2 = 0; q2 < 4; ++q2) {
    float o[4];
    g_one(h[q2][0], h[q2][1], h[q2][2], o);
#pragma unroll
    for (int q1 = 0; q1 < 4; ++q1) out[q2 * 4 + q1] = o[q1];
  }
}

// Level 2 for one branch: 16 quads (q2r, q2c) -> 4x4 partial tile
// po[rr][cc], rr = i1r + 2*i2r, cc = i1c + 2*i2c.  zb points at the branch's
// first quad for this (n, t); gstride is the distance between groups.
// live: bit q2r * 4 + q2c set for the groups whose Z is read (the others
// are zero and not read).
__device__ __forceinline__ void level2_reduce(const float4* __restrict__ zb, size_t gstride,
                                              float (&po)[4][4], unsigned live = 0xffffu) {
  float4 v[4][4];
#pragma unroll
  for (int q2r = 0; q2r < 4; ++q2r)
#pragma unroll
    for (int q2c = 0; q2c < 4; ++q2c)
      v[q2r][q2c] = (live >> (q2r * 4 + q2c)) & 1u ? zb[(size_t)(q2r * 4 + q2c) * gstride]
                                                    : make_float4(0.f, 0.f, 0.f, 0.f);
  // along columns: h[q2r][i2c] (float4 over (i1r, i1c))
  float4 h[4][2];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    h[q][0] = v[q][0] + v[q][1] + v[q][2];
    h[q][1] = v[q][1] - v[q][2] - v[q][3];
  }
#pragma unroll
  for (int i2c = 0; i2c < 2; ++i2c) {
    const float4 e0 = h[0][i2c] + h[1][i2c] + h[2][i2c];   // i2r = 0
    const float4 e1 = h[1][i2c] - h[2][i2c] - h[3][i2c];   // i2r = 1
    po[0][2 * i2c + 0] = e0.x;  po[0][2 * i2c + 1] = e0.y;
    po[1][2 * i2c + 0] = e0.z;  po[1][2 * i2c + 1] = e0.w;
    po[2][2 * i2c + 0] = e1.x;  po[2][2 * i2c + 1] = e1.y;
    po[3][2 * i2c + 0] = e1.z;  po[3][2 * i2c + 1] = e1.w;
  }
}

// 2D inner transform (two levels per axis) of a 10 x 10 sub-window S into
// its 256 points as 64 quads.  Point digits (q2r, q2c, q1r, q1c), most
// significant first; put(quad, value) stores quad q2r * 16 + q2c * 4 + q1r
// (q1c over the four lanes of the value).  Q3: level-1 digit 3 is dead, so
// quads q1r = 3 are not formed (put is not called for them), the q1c = 3
// lanes are 0, and S's row and column 9 are not read (rows and columns 1..3
// of B^T of F(2,3) at level 1 take taps 0..2 only).
template <bool SPLIT, bool Q3 = false, class Put>
__device__ __forceinline__ void inner2_xform(const float (&S)[10][10], Put&& put) {
  constexpr int NR = Q3 ? 3 : 4, NJ = Q3 ? 9 : 10;
#pragma unroll
  for (int q2r = 0; q2r < 4; ++q2r) {
    // level 2 along rows (stride 2): Z[u][j], u = 0..3
    float Z[4][10];
    const int a0 = 2 * bt_tap0(q2r), a1 = 2 * bt_tap1(q2r);
    const float s0 = bt_sign0(q2r), s1 = bt_sign1(q2r);
#pragma unroll
    for (int u = 0; u < NR; ++u)
#pragma unroll
      for (int j = 0; j < NJ; ++j) Z[u][j] = s0 * S[u + a0][j] + s1 * S[u + a1][j];
#pragma unroll
    for (int q1r = 0; q1r < NR; ++q1r) {
      // level 1 along rows (stride 1)
      float R[10];
      const int b0 = bt_tap0(q1r), b1 = bt_tap1(q1r);
      const float t0 = bt_sign0(q1r), t1 = bt_sign1(q1r);
#pragma unroll
      for (int j = 0; j < NJ; ++j) R[j] = t0 * Z[b0][j] + t1 * Z[b1][j];
      float o[16];
      bt_inner2<Q3>(R, o);  // columns: index q2c*4 + q1c
#pragma unroll
      for (int q2c = 0; q2c < 4; ++q2c)
        put(q2r * 16 + q2c * 4 + q1r,
            store_quad<SPLIT>(o[q2c * 4 + 0], o[q2c * 4 + 1], o[q2c * 4 + 2], o[q2c * 4 + 3]));
    }
  }
}

// inner2_xform stored to vb, the branch's first quad for this (m, t);
// qstride is the distance between quads (M*T float4).
template <bool SPLIT>
__device__ __forceinline__ void inner2_store(const float (&S)[10][10], float4* __restrict__ vb,
                                             size_t qstride) {
  inner2_xform<SPLIT>(S, [&](int quad, float4 v) { vb[(size_t)quad * qstride] = v; });
}

// ---- F(3,3): B^T, G, A^T (Toom-Cook points 0, 1, -1, 2, infinity) ----------

// B^T[q][a], G[q][k], A^T[i][q] of F(3,3)
__device__ __forceinline__ float bt5(int q, int a) {
  constexpr float T[5][5] = {{1.0f, -0.5f, -1.0f, 0.5f, 0.0f},
                             {0.0f, 1.0f, 0.5f, -0.5f, 0.0f},
                             {0.0f, -1.0f / 3.0f, 0.5f, -1.0f / 6.0f, 0.0f},
                             {0.0f, -1.0f / 6.0f, 0.0f, 1.0f / 6.0f, 0.0f},
                             {0.0f, 2.0f, -1.0f, -2.0f, 1.0f}};
  return T[q][a];
}
__device__ __forceinline__ float g5(int q, int k) {
  constexpr float G[5][3] = {{1.0f, 0.0f, 0.0f}, {1.0f, 1.0f, 1.0f}, {1.0f, -1.0f, 1.0f},
                             {1.0f, 2.0f, 4.0f}, {0.0f, 0.0f, 1.0f}};
  return G[q][k];
}
__host__ __device__ constexpr float at5(int i, int q) {
  return i == 0 ? (q == 4 ? 0.0f : 1.0f)
       : i == 1 ? (q == 0 ? 0.0f : q == 1 ? 1.0f : q == 2 ? -1.0f : q == 3 ? 2.0f : 0.0f)
                : (q == 0 ? 0.0f : q == 3 ? 4.0f : 1.0f);
}

// B^T along a length-5 vector
__device__ __forceinline__ void bt5_vec(const float (&v)[5], float (&o)[5]) {
#pragma unroll
  for (int q = 0; q < 5; ++q) {
    float s = 0.0f;
#pragma unroll
    for (int a = 0; a < 5; ++a)
      if (bt5(q, a) != 0.0f) s = fmaf(bt5(q, a), v[a], s);
    o[q] = s;
  }
}

// ---------------------------------------------------------------------------
// Plan
// ---------------------------------------------------------------------------

struct ContractArgs {
  const float* A;   // [batch][K][Nrows]   (U; N fastest)
  const float* Bm;  // [batch][K][Ncols]   (V or x; columns fastest)
  float* C;         // [batch][Nrows][Ncols]
  long long sA, sB, sC;   // batch strides in elements (sA = 0: shared A)
  int ldA, ldB, ldC;      // row strides in elements
  int Nrows, Ncols, K;
  long long batch;
};

hipError_t launch_kernel_xform_mix(const nwg_plan_info& g, const float* w, float* U,
                                   hipStream_t s);
// X4, Z3: mix_scratch_bytes(g) of scratch at depth 4 (may be NULL at depth 3)
hipError_t launch_input_xform_mix(const nwg_plan_info& g, const float* x, float* V, float* X4,
                                  hipStream_t s);
hipError_t launch_output_xform_mix(const nwg_plan_info& g, const float* Z, float* y, float* Z3,
                                   hipStream_t s);
hipError_t launch_kernel_xform(const nwg_plan_info& g, const float* w, float* U, hipStream_t s);
// part/nparts: at depth 4, the level-4 branches [16 part/nparts, 16 (part+1)/nparts)
// (V quads [4096 part/nparts, ...)); other depths take nparts = 1
hipError_t launch_input_xform(const nwg_plan_info& g, const float* x, float* V, hipStream_t s,
                              int part = 0, int nparts = 1);
// depth 0: y[b] = U^T x[b]
hipError_t launch_gemm_depth0(const ContractArgs& a, hipStream_t s);
// depth >= 1: Z = level-1 A^T of (U^T V per point); G = P / 16 groups
// linear decomposition: U [4][M c^2][N][4] from the c x c sub-kernels of w
hipError_t launch_kernel_xform_ld(const nwg_plan_info& g, const float* w, float* U, hipStream_t s);
// split = true: U, V hold bf16 (hi, lo) pairs (precision NWG_PRECISION_BF16_SPLIT).
// ks > 1: K slices of M / ks channels (deep path: M % (32 ks) == 0, N % 64 == 0,
// T >= 64), slice k writing its partial Z to Z + k G N T 4 floats.
// gm: the plan's group list (G = gm.np^2 entries when gm.np > 0, then ks = 1).
hipError_t launch_contract_fused(const float* U, const float* V, float* Z, int M, int N, int T,
                                 long long G, hipStream_t s, bool split = false, int ks = 1,
                                 const GroupMap& gm = GroupMap{});
// Planar contraction of the mixed nest (mix_planar plans): U [G][9][M][N],
// V [G][9][M][T] over the G = gm.np^2 live groups, Z [P/16][N][T][4] at the
// groups' places; M % 128 == 0, N % 128 == 0, T % 64 == 0.
hipError_t launch_contract_planar(const float* U, const float* V, float* Z, int M, int N, int T,
                                  long long G, const GroupMap& gm, hipStream_t s);
// in place: every fp32 value of buf (n values) -> its packed bf16 (hi, lo) pair
hipError_t launch_split_pairs(float* buf, size_t n, hipStream_t s);
hipError_t launch_input_contract(const nwg_plan_info& g, const float* x, const float* U, float* Z,
                                 hipStream_t s);
// the F(3,3) tile (depth 1-2): U [P][M][N], V [P][M][T], Z [P/25][9][N][T]
hipError_t launch_kernel_xform5(const nwg_plan_info& g, const float* w, float* U, hipStream_t s);
hipError_t launch_input_xform5(const nwg_plan_info& g, const float* x, float* V, hipStream_t s);
hipError_t launch_contract5(const nwg_plan_info& g, const float* U, const float* V, float* Z,
                            hipStream_t s);
// parts > 1 / fold9: the fused kernel's partial Z9 buffers (see f33.hip)
hipError_t launch_output_xform5(const nwg_plan_info& g, const float* Z, float* y, hipStream_t s,
                                int parts = 1, bool fold9 = false);
hipError_t launch_input_contract5(const nwg_plan_info& g, const float* x, const float* U,
                                  float* Zp, hipStream_t s);
hipError_t launch_contract_output5(const nwg_plan_info& g, const float* V, const float* U,
                                   float* y, hipStream_t s);
// Z[i] += Z[k n + i] for k = 1 .. parts-1 (n floats per part)
hipError_t launch_sum_parts(float* Z, size_t n, int parts, hipStream_t s);
hipError_t launch_small_conv(const nwg_plan_info& g, const float* x, const float* U, float* y,
                             hipStream_t s);
// depthwise: y = U[c] x (depth 0); x -> y in one kernel (depth 1-2);
// U, V -> Z element-wise with the level-1 output transform (depth >= 1)
hipError_t launch_dw_scale(const nwg_plan_info& g, const float* x, const float* U, float* y,
                           hipStream_t s);
hipError_t launch_dw_small(const nwg_plan_info& g, const float* x, const float* U, float* y,
                           hipStream_t s);
hipError_t launch_dw_contract(const nwg_plan_info& g, const float* U, const float* V, float* Z,
                              hipStream_t s);
hipError_t launch_output_xform(const nwg_plan_info& g, const float* Yh, float* y, hipStream_t s);

// What nwg_conv2d queues, on workspace the caller provides (the plan's layout:
// U; V when plan_holds_v; Z with its partial sums or scratch when
// plan_holds_z): the kernel transform w -> U, and the steps after it.
// NWG_OK or a status with its message (untimed; pipeline_parts must be 1).
int kernel_transform_into(const nwg_plan_info& g, const float* w, float* U, hipStream_t s);
int conv_steps(const nwg_plan_info& g, const float* U, float* V, float* Yh, const float* x,
               float* y, hipStream_t s);

}  // namespace nwg
