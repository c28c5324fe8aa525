// Nested Winograd with a different base per level (Sec. III.B's level
// recurrence does not need the levels to share a base; Sec. V.A names F(2,3)
// and F(3,3) among its bases): F(2,3) at levels 1 and 2, F(3,3) at the NO =
// 1 or 2 levels above them.  The recurrence s_j = min(M_j, K_j) gives
// strides 1, 2, 4, 12 and
//   NO = 1: M_n = 12, K_n = 15, L_n = 26, 20 points per axis (r = 8..15),
//   NO = 2: M_n = 36, K_n = 39, L_n = 74, 100 points per axis (r = 16..39).
// A 31 x 31 kernel then costs (400 / 36)^2 = 123 general multiplications per
// output instead of (256 / 16)^2 = 256 for four F(2,3) levels.
//
// Point digits (q_n^row, q_n^col, ..., q_1^row, q_1^col), most significant
// first, radix 5 at the F(3,3) levels and 4 at the F(2,3) ones.  With the
// outer branch ob = (q4r, q4c, q3r, q3c) (or (q3r, q3c)) the layouts are the
// F(2x2,3x3) quad layouts: U[P/4][M][N][4], V[P/4][M][T][4] with quad
// 64 ob + 16 q2r + 4 q2c + q1r, and Z[P/16][N][T][4] from the unchanged
// contraction (group g = 16 ob + 4 q2r + q2c after the level-1 A^T).
//
//   kernel transform : one thread per (output channel, outer branch), the
//                      16 output channels of a 512-thread work-group in LDS,
//                      padded to K_n x K_n; the outer G rows fold the kernel
//                      into the 9 x 9 sub-kernel of the two F(2,3) levels.
//   input transform  : 16 (NO = 1) or 32 (NO = 2) tiles x 25 level-3
//                      branches per work-group; at NO = 2 the work-group
//                      owns one level-4 branch, whose
//                      B^T rows the LDS fill applies (74 x 74 -> 26 x 26).
//                      Level 3 runs per output row (rows, then columns), the
//                      two F(2,3) levels in registers (10 x 10 -> 16 x 16).
//   output transform : NO = 1: levels 2 and 3 per (tile, 4 x 4 output
//                      block, channel), straight to y.  NO = 2: levels 2
//                      and 3 per (tile, level-4 branch, channel) into a
//                      12 x 12 block held in a scratch buffer Z3, then a
//                      second kernel applies level 4 to the 25 blocks.
#include "nwg_internal.h"

namespace nwg {
namespace {

constexpr int kStride3 = 4, kStride4 = 12;

// Rank of axis prefix i among the live prefixes (the live ones below it),
// branch-free over the four 32-bit words (a 64-bit shift by a lane-varying
// amount became control flow that stopped the transforms' unrolling).
__device__ __forceinline__ int prefix_rank(unsigned long long m0, unsigned long long m1, int i) {
  const unsigned wd[4] = {(unsigned)m0, (unsigned)(m0 >> 32), (unsigned)m1, (unsigned)(m1 >> 32)};
  int r = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int k = i - 32 * q;
    const unsigned below = k <= 0 ? 0u : (k >= 32 ? 0xffffffffu : (1u << k) - 1u);
    r += __popc(wd[q] & below);
  }
  return r;
}

// The live groups (q2r, q2c) of outer branch (q4r, q4c, q3r, q3c) as a
// 16-bit mask, bit 4 q2r + q2c (NO = 1: no level-4 digits).  A group is live
// when its row prefix (q4r, q3r, q2r) and its column prefix (q4c, q3c, q2c)
// are (masks m0, m1 of nwg_plan_info::live_prefix; all live when both are 0).
template <int NO>
__device__ __forceinline__ unsigned branch_live(unsigned long long m0, unsigned long long m1,
                                                int q4r, int q4c, int q3r, int q3c) {
  if ((m0 | m1) == 0) return 0xffffu;
  return nibble_live(prefix_nibble(m0, m1, NO == 2 ? q4r * 5 + q3r : q3r),
                     prefix_nibble(m0, m1, NO == 2 ? q4c * 5 + q3c : q3c));
}

// How a transform stores its points: every quad of a live branch, the live
// quads only (quad layout), or the live points of the live groups in the
// planar layout (nwg_plan_info::mix_planar).
enum { kStoreAll = 0, kStoreMasked = 1, kStorePlanar = 2 };

// Whether quad q2r * 16 + q2c * 4 + q1r of a branch with live-group mask
// live is stored.
__device__ __forceinline__ bool quad_live(unsigned live, int q3, int quad) {
  return ((live >> (quad >> 2)) & 1u) && !(q3 && (quad & 3) == 3);
}

// Tap of the axis multi-index (k4, k3, k2, k1) (digits < 3, strides 12, 4, 2,
// 1), or -1 when the multi-index is not the greedy split of its tap
// (outermost digit first, each as large as allowed).
template <int NO>
__host__ __device__ constexpr int mix_tap(int k4, int k3, int k2, int k1) {
  const int tap = kStride4 * k4 + kStride3 * k3 + 2 * k2 + k1;
  int rem = tap;
  int d4 = 0;
  if (NO == 2) {
    d4 = rem / kStride4 < 2 ? rem / kStride4 : 2;
    rem -= kStride4 * d4;
  }
  const int d3 = rem / kStride3 < 2 ? rem / kStride3 : 2;
  rem -= kStride3 * d3;
  const int d2 = rem / 2 < 2 ? rem / 2 : 2;
  rem -= 2 * d2;
  const bool ok = rem == k1 && d2 == k2 && d3 == k3 && (NO == 1 ? k4 == 0 : d4 == k4);
  return ok ? tap : -1;
}

// F(3,3) rows with a runtime row index, as selects over compile-time rows
__device__ __forceinline__ void g5_row(int q, float (&c)[3]) {
#pragma unroll
  for (int k = 0; k < 3; ++k) c[k] = 0.0f;
#pragma unroll
  for (int qq = 0; qq < 5; ++qq)
#pragma unroll
    for (int k = 0; k < 3; ++k) c[k] = q == qq ? g5(qq, k) : c[k];
}
__device__ __forceinline__ void bt5_row(int q, float (&c)[5]) {
#pragma unroll
  for (int a = 0; a < 5; ++a) c[a] = 0.0f;
#pragma unroll
  for (int qq = 0; qq < 5; ++qq)
#pragma unroll
    for (int a = 0; a < 5; ++a) c[a] = q == qq ? bt5(qq, a) : c[a];
}

// ---- kernel transform -------------------------------------------------------
// STORE = kStorePlanar: depth 4 only, U [live group][3 q1r + q1c][M][N].
template <int NO, int STORE>
__global__ __launch_bounds__(512) void kernel_xform_mix(const float* __restrict__ w,
                                                        float* __restrict__ U, int M, int N,
                                                        int r, unsigned long long m0,
                                                        unsigned long long m1, int q3) {
  constexpr int K = NO == 2 ? 39 : 15;      // padded taps per axis (odd)
  constexpr int KS = K * K;
  constexpr int NA = NO == 2 ? 3 : 1;       // level-4 digits per axis
  constexpr int NB = NO == 2 ? 625 : 25;    // outer branches
  extern __shared__ float wl[];             // [16][K][K]
  const int m = blockIdx.y;
  const int n0 = blockIdx.x * 16;
  for (int e = threadIdx.x; e < 16 * KS; e += 512) {
    const int c = e / KS, k = e - c * KS;
    const int u = k / K, v = k - u * K;
    const int nn = n0 + c;
    wl[e] = (nn < N && u < r && v < r) ? w[((size_t)nn * M + m) * r * r + u * r + v] : 0.0f;
  }
  __syncthreads();
  const int cl = threadIdx.x & 15, slot = threadIdx.x >> 4;   // 32 slots
  const int nn = n0 + cl;
  if (nn >= N) return;                      // no barrier below
  const float* wk = wl + cl * KS;
  const size_t MN = (size_t)M * N;
  for (int b = slot; b < NB; b += 32) {
    const int q3c = b % 5, q3r = (b / 5) % 5;
    const int q4c = NO == 2 ? (b / 25) % 5 : 0, q4r = NO == 2 ? b / 125 : 0;
    // the groups no real tap reaches are neither computed nor stored
    const unsigned live = branch_live<NO>(m0, m1, q4r, q4c, q3r, q3c);
    if (live == 0) continue;
    float c3r[3], c3c[3], c4r[3], c4c[3];
    g5_row(q3r, c3r);
    g5_row(q3c, c3c);
    g5_row(q4r, c4r);
    g5_row(q4c, c4c);
    float cr[NA][3], cc[NA][3];
#pragma unroll
    for (int a4 = 0; a4 < NA; ++a4)
#pragma unroll
      for (int a3 = 0; a3 < 3; ++a3) {
        cr[a4][a3] = (NO == 2 ? c4r[a4] : 1.0f) * c3r[a3];
        cc[a4][a3] = (NO == 2 ? c4c[a4] : 1.0f) * c3c[a3];
      }
    // S[ir][ic] over the inner digits (k2, k1) of each axis
    float S[9][9];
#pragma unroll
    for (int i = 0; i < 9; ++i)
#pragma unroll
      for (int j = 0; j < 9; ++j) S[i][j] = 0.0f;
#pragma unroll
    for (int a4 = 0; a4 < NA; ++a4)
#pragma unroll
      for (int a3 = 0; a3 < 3; ++a3)
#pragma unroll
        for (int ir = 0; ir < 9; ++ir) {
          const int tr = mix_tap<NO>(a4, a3, ir / 3, ir % 3);
          if (tr < 0) continue;
          // the row's taps folded over the outer column digits
          float rowv[9];
#pragma unroll
          for (int ic = 0; ic < 9; ++ic) rowv[ic] = 0.0f;
#pragma unroll
          for (int b4 = 0; b4 < NA; ++b4)
#pragma unroll
            for (int b3 = 0; b3 < 3; ++b3)
#pragma unroll
              for (int ic = 0; ic < 9; ++ic) {
                const int tc = mix_tap<NO>(b4, b3, ic / 3, ic % 3);
                if (tc < 0) continue;
                rowv[ic] = fmaf(cc[b4][b3], wk[tr * K + tc], rowv[ic]);
              }
#pragma unroll
          for (int ic = 0; ic < 9; ++ic) S[ir][ic] = fmaf(cr[a4][a3], rowv[ic], S[ir][ic]);
        }
    // the two F(2,3) levels: 64 quads of this outer branch
    float4* ub = reinterpret_cast<float4*>(U) + (size_t)b * 64 * MN + (size_t)m * N + nn;
    // kStoreMasked: the wave's four branches b0 .. b0 + 3 share a resource
    const int b0 = __builtin_amdgcn_readfirstlane(b & ~3);
    const auto rs = span_rsrc(reinterpret_cast<float4*>(U) + (size_t)b0 * 64 * MN +
                                  (size_t)m * N + n0,
                              (unsigned)(4 * 64 * MN * 16));
    const unsigned lane0 = (unsigned)(((size_t)(b - b0) * 64 * MN + cl) * 16);
    // kStorePlanar: groups at their live-list places; the wave's resource
    // starts at the lowest row-prefix block (q4r, q3r) of its four branches,
    // and a group's place is at most 20 live row prefixes above it
    unsigned nr = 0, nc = 0;                  // live nibbles of the row / column prefixes
    int lbase = 0, np = 0, r0 = 0, c0 = 0;     // ranks of the first row / column prefix
    __amdgpu_buffer_rsrc_t pr = rs;
    if constexpr (STORE == kStorePlanar) {
      np = __popcll(m0) + __popcll(m1);
      int smin = 1 << 20;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int bi = b0 + i;
        const int si = ((bi / 125) * 5 + (bi / 5) % 5) * 4;
        if (bi < NB && si < smin) smin = si;
      }
      lbase = prefix_rank(m0, m1, smin) * np;
      nr = prefix_nibble(m0, m1, q4r * 5 + q3r);
      nc = prefix_nibble(m0, m1, q4c * 5 + q3c);
      r0 = prefix_rank(m0, m1, (q4r * 5 + q3r) * 4);
      c0 = prefix_rank(m0, m1, (q4c * 5 + q3c) * 4);
      pr = span_rsrc(reinterpret_cast<float4*>(U + (size_t)lbase * 9 * MN + (size_t)m * N + n0),
                     (unsigned)(20 * np * 9 * MN * 4));
    }
#pragma unroll
    for (int rho = 0; rho < 16; ++rho) {
      const int q2r = rho >> 2, q1r = rho & 3;
      if (STORE == kStorePlanar && q1r == 3) continue;   // dead level-1 digit
      float rowv[9];
#pragma unroll
      for (int ic = 0; ic < 9; ++ic) {
        float sacc = 0.0f;
#pragma unroll
        for (int ir = 0; ir < 9; ++ir) {
          const float c = g_coef(q2r, ir / 3) * g_coef(q1r, ir % 3);
          if (c != 0.0f) sacc += c * S[ir][ic];
        }
        rowv[ic] = sacc;
      }
      float o[16];
      g_inner2(rowv, o);
#pragma unroll
      for (int q2c = 0; q2c < 4; ++q2c) {
        const int quad = q2r * 16 + q2c * 4 + q1r;
        const float4 v = make_float4(o[q2c * 4 + 0], o[q2c * 4 + 1], o[q2c * 4 + 2], o[q2c * 4 + 3]);
        if constexpr (STORE == kStorePlanar) {
          const bool on = (live >> (quad >> 2)) & 1u;
          const int ir = r0 + __popc(nr & ((1u << q2r) - 1u));
          const int ic = c0 + __popc(nc & ((1u << q2c) - 1u));
          const unsigned rel = (unsigned)((ir * np + ic - lbase) * 9 + 3 * q1r);
          const unsigned ps = (unsigned)MN * 4u;
          const unsigned o0 = (unsigned)(rel * MN + cl) * 4u;
          drop_store1(pr, on ? o0 : kDrop, v.x);
          drop_store1(pr, on ? o0 + ps : kDrop, v.y);
          drop_store1(pr, on ? o0 + 2 * ps : kDrop, v.z);
        } else if constexpr (STORE == kStoreMasked) {
          drop_store(rs, quad_live(live, q3, quad) ? lane0 + (unsigned)(quad * MN * 16) : kDrop, v);
        } else {
          ub[(size_t)quad * MN] = v;
        }
      }
    }
  }
}

// Planar plans (depth 4, level-1 digit 3 dead): the same transform with the
// outer column fold shared.  The fold of a kernel row over the column digits
// (k4c, k3c) depends on the column branch (q4c, q3c) only, so per column
// branch the work-group first folds every row of its NW kernels into
// C[row tap][column inner digits] in LDS (one thread per (channel, row)),
// and then one thread per (channel, row branch (q4r, q3r)) folds C's rows
// into the 9 x 9 sub-kernel and runs the two F(2,3) levels as above: the
// column fold is computed once per column branch instead of once per outer
// branch.  NW output channels per work-group (32 when their r x r kernels
// fit in LDS, r <= 31): a wavefront's lanes store U in NW-float runs.
// U [live group][3 q1r + q1c][M][N].
template <int NW>
__global__ __launch_bounds__(NW * 32) void kernel_xform_mix_sep(const float* __restrict__ w,
                                                                float* __restrict__ U, int M,
                                                                int N, int r,
                                                                unsigned long long m0,
                                                                unsigned long long m1) {
  constexpr int NT = NW * 32;                // threads
  constexpr int RB = 64 / NW;                // row branches per wavefront
  extern __shared__ float sm[];
  float* wl = sm;                            // [NW][r][r]
  float* cl = sm + NW * r * r;               // [NW][r][9]
  const int m = blockIdx.y;
  const int n0 = blockIdx.x * NW;
  const int rr = r * r;
  for (int e = threadIdx.x; e < NW * rr; e += NT) {
    const int c = e / rr;
    const int nn = n0 + c;
    wl[e] = nn < N ? w[((size_t)nn * M + m) * rr + (e - c * rr)] : 0.0f;
  }
  __syncthreads();
  const int np = __popcll(m0) + __popcll(m1);
  const size_t MN = (size_t)M * N;
  const unsigned ps = (unsigned)MN * 4u;
#pragma unroll 1
  for (int bc = 0; bc < 25; ++bc) {          // column branch: 5 q4c + q3c
    const int q4c = bc / 5, q3c = bc - 5 * q4c;
    const unsigned nc = prefix_nibble(m0, m1, q4c * 5 + q3c);
    if ((m0 | m1) != 0 && nc == 0) continue;   // no live group in this column branch
    // C[c][tr][ic] = sum over (k4c, k3c) of G rows (q4c, q3c) times w[tr][tap]
    // (taps >= r are the kernel's zero padding)
    float c4c[3], c3c[3];
    g5_row(q4c, c4c);
    g5_row(q3c, c3c);
    for (int task = threadIdx.x; task < NW * r; task += NT) {
      const int c = task / r, tr = task - c * r;
      const float* wr = wl + (c * r + tr) * r;
      float cv[9];
#pragma unroll
      for (int ic = 0; ic < 9; ++ic) cv[ic] = 0.0f;
#pragma unroll
      for (int b4 = 0; b4 < 3; ++b4)
#pragma unroll
        for (int b3 = 0; b3 < 3; ++b3) {
          const float cc = c4c[b4] * c3c[b3];
#pragma unroll
          for (int ic = 0; ic < 9; ++ic) {
            const int tc = mix_tap<2>(b4, b3, ic / 3, ic % 3);
            if (tc < 0) continue;
            if (tc < r) cv[ic] = fmaf(cc, wr[tc], cv[ic]);
          }
        }
      float* cr = cl + (c * r + tr) * 9;
#pragma unroll
      for (int ic = 0; ic < 9; ++ic) cr[ic] = cv[ic];
    }
    __syncthreads();
    // one thread per (channel, row branch): lanes on channels, so that the
    // NW lanes of a row branch store NW contiguous floats
    for (int task = threadIdx.x; task < NW * 25; task += NT) {
      const int cln = task % NW, br = task / NW;    // br = 5 q4r + q3r
      const int q4r = br / 5, q3r = br - 5 * q4r;
      const int nn = n0 + cln;
      const unsigned live = branch_live<2>(m0, m1, q4r, q4c, q3r, q3c);
      if (nn >= N || live == 0) continue;
      float c4r[3], c3r[3];
      g5_row(q4r, c4r);
      g5_row(q3r, c3r);
      float S[9][9];
#pragma unroll
      for (int i = 0; i < 9; ++i)
#pragma unroll
        for (int j = 0; j < 9; ++j) S[i][j] = 0.0f;
      const float* cb = cl + cln * r * 9;
#pragma unroll
      for (int a4 = 0; a4 < 3; ++a4)
#pragma unroll
        for (int a3 = 0; a3 < 3; ++a3) {
          const float crr = c4r[a4] * c3r[a3];
#pragma unroll
          for (int ir = 0; ir < 9; ++ir) {
            const int tr = mix_tap<2>(a4, a3, ir / 3, ir % 3);
            if (tr < 0 || tr >= r) continue;   // rows >= r: zero padding
            const float* cv = cb + tr * 9;
#pragma unroll
            for (int ic = 0; ic < 9; ++ic) S[ir][ic] = fmaf(crr, cv[ic], S[ir][ic]);
          }
        }
      // planar places: the wave's RB row branches (readfirstlane of the
      // lowest) share a resource from the lowest row-prefix block; a
      // group's place is at most 20 live row prefixes above it
      const int br0 = __builtin_amdgcn_readfirstlane(br & ~(RB - 1));
      const int lbase = prefix_rank(m0, m1, br0 * 4) * np;
      const unsigned nr = prefix_nibble(m0, m1, q4r * 5 + q3r);
      const int r0 = prefix_rank(m0, m1, (q4r * 5 + q3r) * 4);
      const int c0 = prefix_rank(m0, m1, (q4c * 5 + q3c) * 4);
      const auto pr = span_rsrc(
          reinterpret_cast<float4*>(U + (size_t)lbase * 9 * MN + (size_t)m * N + n0),
          (unsigned)(20 * np * 9 * MN * 4));
#pragma unroll
      for (int rho = 0; rho < 16; ++rho) {
        const int q2r = rho >> 2, q1r = rho & 3;
        if (q1r == 3) continue;              // dead level-1 digit
        float rowv[9];
#pragma unroll
        for (int ic = 0; ic < 9; ++ic) {
          float sacc = 0.0f;
#pragma unroll
          for (int ir = 0; ir < 9; ++ir) {
            const float c = g_coef(q2r, ir / 3) * g_coef(q1r, ir % 3);
            if (c != 0.0f) sacc += c * S[ir][ic];
          }
          rowv[ic] = sacc;
        }
        float o[16];
        g_inner2(rowv, o);
#pragma unroll
        for (int q2c = 0; q2c < 4; ++q2c) {
          const bool on = (live >> (q2r * 4 + q2c)) & 1u;
          const int ir = r0 + __popc(nr & ((1u << q2r) - 1u));
          const int ic = c0 + __popc(nc & ((1u << q2c) - 1u));
          const unsigned rel = (unsigned)((ir * np + ic - lbase) * 9 + 3 * q1r);
          const unsigned o0 = (unsigned)(rel * MN + cln) * 4u;
          drop_store1(pr, on ? o0 : kDrop, o[q2c * 4 + 0]);
          drop_store1(pr, on ? o0 + ps : kDrop, o[q2c * 4 + 1]);
          drop_store1(pr, on ? o0 + 2 * ps : kDrop, o[q2c * 4 + 2]);
        }
      }
    }
    __syncthreads();                         // C is rewritten by the next column branch
  }
}

// ---- input transform --------------------------------------------------------
// Depth 4 runs in two kernels.  input_mix_l4 applies the level-4 B^T rows
// (q4r along the rows, q4c along the columns, stride 12) to every tile's
// 74 x 74 window: X4[q4][m][t][26 x 26].
// input_xform_mix then takes TPW tiles (32 at depth 4, 16 at depth 3) x 25
// level-3 branches per work-group: their 26 x 26 blocks (X4 at depth 4, the
// raw windows at depth 3)
// go to LDS, level 3 runs per output row (rows, then columns) and the two
// F(2,3) levels in registers (10 x 10 -> 16 x 16).
constexpr int kL3 = kMixL3;                 // window side left for levels 1..3
// per-tile stride in LDS: even, so that column pairs are 8-byte aligned
// (float2 reads), and 678 = 38 (mod 64), so that 32 consecutive tiles
// start on 32 different even banks
constexpr int kWS = kL3 * kL3 + 2;

// BS = 26 keeps every level-3 input row and column; BS = 25 (planar plans,
// level-1 digit 3 dead) drops row and column 25, which no live point reads.
template <int BS>
__global__ __launch_bounds__(256) void input_mix_l4(const float* __restrict__ x,
                                                    float* __restrict__ X4, int M, int H, int W,
                                                    int pad, int th, int tw, int T) {
  // work-group (tile t, channel m): the 74 x 74 window, then per level-4
  // row branch the B^T along the rows (BS x 74), then along the columns (5
  // branches of BS x BS), separably through LDS
  constexpr int LW = 74, LS = 75;           // window side, odd LDS stride
  __shared__ float win[LW * LS];
  __shared__ float rw[kL3 * LS];
  const int t = blockIdx.x, m = blockIdx.y;
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  const float* __restrict__ xp = x + ((size_t)b * M + m) * H * W;
  const int gr0 = ty * 36 - pad, gc0 = tx * 36 - pad;
  {
    // all of a thread's loads first (22 in flight), then the LDS writes
    constexpr int PER = (LW * LW + 255) / 256;
    float v[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int i = e / LW, j = e - i * LW;
      const int gr = gr0 + i, gc = gc0 + j;
      v[u] = (e < LW * LW && gr >= 0 && gr < H && gc >= 0 && gc < W) ? xp[(size_t)gr * W + gc]
                                                                    : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int i = e / LW, j = e - i * LW;
      if (e < LW * LW) win[i * LS + j] = v[u];
    }
  }
  __syncthreads();
  // one level-4 row branch at a time, so that rw holds 26 rows: 30 KB of LDS
  // in all, five work-groups per CU to hide the window loads (0.17 -> 0.14
  // ms on the 31 x 31 layer against all five row branches at once)
  const size_t bstride = (size_t)M * T * BS * BS;     // between level-4 branches
  float* __restrict__ dst = X4 + ((size_t)m * T + t) * BS * BS;
#pragma unroll
  for (int q4r = 0; q4r < 5; ++q4r) {
    // rows: rw[i][c] = sum_a B^T[q4r][a] win[i + 12 a][c]
    for (int e = threadIdx.x; e < BS * LW; e += 256) {
      const int i = e / LW, c = e - i * LW;
      float sacc = 0.0f;
#pragma unroll
      for (int a = 0; a < 5; ++a)
        if (bt5(q4r, a) != 0.0f) sacc = fmaf(bt5(q4r, a), win[(i + kStride4 * a) * LS + c], sacc);
      rw[i * LS + c] = sacc;
    }
    __syncthreads();
    // columns: X4[5 q4r + q4c][m][t][i][j] = sum_b B^T[q4c][b] rw[i][j + 12 b]
    for (int k = threadIdx.x; k < BS * BS; k += 256) {
      const int i = k / BS, j = k - i * BS;
      float v[5];
#pragma unroll
      for (int bb = 0; bb < 5; ++bb) v[bb] = rw[i * LS + j + kStride4 * bb];
#pragma unroll
      for (int q = 0; q < 5; ++q) {
        float sacc = 0.0f;
#pragma unroll
        for (int bb = 0; bb < 5; ++bb)
          if (bt5(q, bb) != 0.0f) sacc = fmaf(bt5(q, bb), v[bb], sacc);
        dst[(size_t)(q4r * 5 + q) * bstride + k] = sacc;
      }
    }
    if (q4r < 4) __syncthreads();             // rw is rewritten next
  }
}

// One level-3 branch (slot = 5 q3r + q3c under level-4 branch q4) of one
// tile (lane tl of a TPW-tile chunk starting at t0, channel m): its level-3
// block win in LDS (rows ROW floats apart) -> the branch's points of V.
template <int NO, int STORE, bool Q3, int TPW, int ROW>
__device__ __forceinline__ void mix_branch(const float* win, int slot, int q4, int m, int t0,
                                           int tl, float4* __restrict__ V, int M, int T,
                                           long long qstride, unsigned long long m0,
                                           unsigned long long m1, int q3) {
  const int t = t0 + tl;
  // a row of B^T of F(3,3) has its nonzero taps among 4 consecutive ones,
  // from tap 0 for row 0 and from tap 1 otherwise
  const int q3r = slot / 5, q3c = slot - 5 * q3r;
  // V of the groups no real tap reaches is neither computed nor stored
  const unsigned live = branch_live<NO>(m0, m1, q4 / 5, q4 % 5, q3r, q3c);
  if (live == 0) return;
  const int lr = q3r == 0 ? 0 : 1, lc = q3c == 0 ? 0 : 1;
  float ca5[5], cb5[5], ca[4], cb[4];
  bt5_row(q3r, ca5);
  bt5_row(q3c, cb5);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    ca[u] = lr ? ca5[u + 1] : ca5[u];
    cb[u] = lc ? cb5[u + 1] : cb5[u];
    if constexpr (TPW == 64) {
      // one branch per wavefront: the coefficients are uniform, keep them
      // in scalar registers
      ca[u] = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(ca[u])));
      cb[u] = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(cb[u])));
    }
  }
  // level 3 (stride 4): per output row, the rows' taps over the 22 columns
  // the column taps need (from column 4 lc), read as float2, then the
  // columns' taps
  const float* wb = win + kStride3 * lr * ROW + kStride3 * lc;
  // Q3 (level-1 digit 3 dead): the inner transform reads S[0..8][0..8], so
  // the column taps reach columns 4 lc .. 4 lc + 20 (NC = 21) of the block
  constexpr int NS = Q3 ? 9 : 10, NC = NS + 3 * kStride3;
  float S[10][10];
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    float tr[22];
#pragma unroll
    for (int c = 0; c < 22; c += 2) {
      float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float* p = wb + (i + kStride3 * u) * ROW + c;
        float2 v;
        if constexpr (ROW % 2 == 0) {
          v = *reinterpret_cast<const float2*>(p);
        } else {
          v.x = p[0];                       // odd rows: pairs not 8-byte aligned
          v.y = c + 1 < NC ? p[1] : 0.0f;   // (a 25-wide block has no column 25)
        }
        s0 = fmaf(ca[u], v.x, s0);
        s1 = fmaf(ca[u], v.y, s1);
      }
      tr[c] = s0;
      tr[c + 1] = s1;
    }
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      float sacc = 0.0f;
#pragma unroll
      for (int u = 0; u < 4; ++u) sacc = fmaf(cb[u], tr[j + kStride3 * u], sacc);
      S[i][j] = sacc;
    }
    // one output row at a time: keeps the row's LDS reads from being
    // hoisted across rows (register pressure); with level-1 digit 3 dead the
    // kernel has the registers to let them overlap (0.714 -> 0.672 ms for
    // the stage on the 31 x 31 layer)
    if constexpr (!Q3) __builtin_amdgcn_sched_barrier(0);
  }
  const int ob = q4 * 25 + slot;
  if constexpr (STORE == kStorePlanar) {
    static_assert(NO == 2 && Q3, "planar V: depth 4, level-1 digit 3 dead");
    // groups at their live-list places; the work-group's resource starts at
    // its level-4 row block (q4r), 20 row prefixes
    const int np = __popcll(m0) + __popcll(m1);
    const int q4r = q4 / 5, q4c = q4 - 5 * q4r;
    const int lbase = prefix_rank(m0, m1, q4r * 20) * np;
    const size_t plane = (size_t)M * T;
    const auto pr = span_rsrc(reinterpret_cast<float4*>(reinterpret_cast<float*>(V) +
                                                        (size_t)lbase * 9 * plane +
                                                        (size_t)m * T + t0),
                              (unsigned)(20 * np * 9 * plane * 4));
    // ranks of the branch's first row and column prefixes; the other three
    // follow from the live nibbles
    const int br = q4r * 5 + q3r, bc = q4c * 5 + q3c;
    const unsigned nr = prefix_nibble(m0, m1, br), nc = prefix_nibble(m0, m1, bc);
    const int r0 = prefix_rank(m0, m1, 4 * br), c0 = prefix_rank(m0, m1, 4 * bc);
    const unsigned ps = (unsigned)plane * 4u;
    // byte offset of group (q2r, q2c)'s first point plane, for this lane
    const unsigned gbase = (unsigned)(((r0 * np + c0 - lbase) * 9) * plane) * 4u + (unsigned)tl * 4u;
    inner2_xform<false, true>(S, [=](int quad, float4 v) {
      const int q2r = quad >> 4, q2c = (quad >> 2) & 3, q1r = quad & 3;
      const bool on = (live >> (quad >> 2)) & 1u;
      const int ir = __popc(nr & ((1u << q2r) - 1u)), ic = __popc(nc & ((1u << q2c) - 1u));
      const unsigned o0 = gbase + (unsigned)((ir * np + ic) * 9 + 3 * q1r) * ps;
      const unsigned off = on ? o0 : kDrop;
      drop_store1(pr, off, v.x);
      drop_store1(pr, off, v.y, ps);
      drop_store1(pr, off, v.z, 2 * ps);
    });
  } else if constexpr (STORE == kStoreMasked) {
    // the wave's 64 / TPW consecutive slots share a resource
    constexpr int SPW = 64 / TPW;
    const int slot0 = __builtin_amdgcn_readfirstlane(slot & ~(SPW - 1));
    const auto rs = span_rsrc(V + (size_t)(q4 * 25 + slot0) * 64 * qstride + (size_t)m * T + t0,
                              (unsigned)(SPW * 64 * qstride * 16));
    const unsigned lane0 = (unsigned)(((size_t)(slot - slot0) * 64 * qstride + tl) * 16);
    inner2_xform<false, Q3>(S, [&](int quad, float4 v) {
      drop_store(rs, quad_live(live, q3, quad) ? lane0 + (unsigned)(quad * qstride * 16) : kDrop,
                 v);
    });
  } else {
    float4* vb = V + (size_t)ob * 64 * qstride + (size_t)m * T + t;
    inner2_xform<false, Q3>(S, [&](int quad, float4 v) { vb[(size_t)quad * qstride] = v; });
  }
}

// 16 TPW threads: TPW tiles x 16 slots, slot s taking the level-3 branches s
// and s + 16 (< 25); two wavefronts per SIMD (at depth 3 one work-group's
// stores overlap another's fill and arithmetic).  At depth 4, 32 tiles (512
// threads, one work-group per CU) write each point's V row in 512-byte runs:
// 1.394 -> 1.372 ms on the 31 x 31 layer against 16 tiles.  Work-group ->
// (level-4 branch q4 (NO = 2), TPW-tile chunk, channel m).
// STORE = kStorePlanar: depth 4 and Q3 only, V [live group][3 q1r + q1c][M][T].
template <int NO, int STORE, bool Q3>
__global__ __launch_bounds__(NO == 2 ? 512 : 256) __attribute__((amdgpu_waves_per_eu(2))) void input_xform_mix(
    const float* __restrict__ x, const float* __restrict__ X4, float4* __restrict__ V, int M,
    int H, int W, int pad, int th, int tw, int T, long long qstride, unsigned long long m0,
    unsigned long long m1, int q3) {
  constexpr int Mn = NO == 2 ? 36 : 12;
  constexpr int KK = kL3 * kL3;
  constexpr int TPW = NO == 2 ? 32 : 16, NT = 16 * TPW;   // tiles, threads per work-group
  constexpr int PER = (TPW * KK + NT - 1) / NT;  // fill values per thread
  extern __shared__ float lds[];            // [TPW][kWS]
  const int nchunk = (T + TPW - 1) / TPW;
  int q4, t0, m;
  if (NO == 2) {
    // dispatch order, chunk fastest, then m, then q4: the work-groups that
    // run at once write the quads of one level-4 branch, 512-byte runs side
    // by side (1.37 -> 1.33 ms on the 31 x 31 layer against q4 fastest with
    // a contiguous range per XCD)
    long long lid = blockIdx.x;
    t0 = (int)(lid % nchunk) * TPW;
    lid /= nchunk;
    m = (int)(lid % M);
    q4 = (int)(lid / M);
  } else {
    // depth 3 reads the raw windows: the chunks of one channel, whose
    // windows overlap, run on one XCD
    const long long G = (long long)gridDim.x, i = blockIdx.x;
    const long long q = G / 8, rem = G % 8, xcd = i % 8, sl = i / 8;
    const long long lid = xcd < rem ? xcd * (q + 1) + sl : rem * (q + 1) + (xcd - rem) * q + sl;
    q4 = 0;
    t0 = (int)(lid % nchunk) * TPW;
    m = (int)(lid / nchunk);
  }
  const int nt = T - t0 < TPW ? T - t0 : TPW;   // tiles of this chunk
  // fill: all loads first (PER in flight per thread), then the LDS writes
  {
    float v[PER];
    if (NO == 2) {
      // X4[q4][m][t0 .. t0 + nt) is contiguous
      const float* src = X4 + (((size_t)q4 * M + m) * T + t0) * KK;
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int e = threadIdx.x + NT * u;
        v[u] = e < nt * KK ? src[e] : 0.0f;
      }
    } else {
      const int tpi = th * tw;
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int e = threadIdx.x + NT * u;
        const int tl = e / KK, k = e - tl * KK;
        const int i = k / kL3, j = k - i * kL3;
        float val = 0.0f;
        if (tl < nt) {
          const int t = t0 + tl;
          const int b = t / tpi;
          const int r2 = t - b * tpi;
          const int ty = r2 / tw, tx = r2 - ty * tw;
          const int gr = ty * Mn - pad + i, gc = tx * Mn - pad + j;
          if (gr >= 0 && gr < H && gc >= 0 && gc < W)
            val = x[(((size_t)b * M + m) * H + gr) * W + gc];
        }
        v[u] = val;
      }
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = threadIdx.x + NT * u;
      if (e < TPW * KK) {
        const int tl = e / KK, k = e - tl * KK;
        lds[tl * kWS + k] = v[u];
      }
    }
  }
  __syncthreads();
  const int tl = threadIdx.x & (TPW - 1);
  const int t = t0 + tl;
  if (t >= T) return;                       // no barrier below
  const float* win = lds + tl * kWS;
  for (int slot = threadIdx.x / TPW; slot < 25; slot += 16) {   // slot = 5 q3r + q3c
    mix_branch<NO, STORE, Q3, TPW, kL3>(win, slot, q4, m, t0, tl, V, M, T, qstride, m0, m1, q3);
  }
}

// Planar plans (depth 4, level-1 digit 3 dead, T a multiple of 64): 64 tiles
// per work-group, one wavefront per level-3 branch at a time (its lanes on
// the 64 tiles), so every V store of a wavefront writes 256 contiguous
// bytes and the branch's B^T coefficients are uniform.  The 64 tiles' X4
// blocks are kept 25 x 25 (input_mix_l4<kPB>), one contiguous 160 KB run
// that direct global->LDS loads copy as is.  Work-group -> (64-tile chunk,
// channel m, level-4 branch q4), the chunk fastest.
constexpr int kPB = kL3 - 1, kPKB = kPB * kPB;   // planar X4 block side, floats
constexpr int kPT = 64;                          // tiles per work-group
constexpr int kPRun4 = kPT * kPKB / 4;           // float4 of a work-group's X4 run
constexpr int kPBlk = (kPRun4 + 63) / 64;        // 64-lane load blocks (the last partial)
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2))) void input_xform_mix_p64(
    const float* __restrict__ X4, float4* __restrict__ V, int M, int T, unsigned long long m0,
    unsigned long long m1) {
  extern __shared__ float4 lds4[];           // [kPBlk * 64]: [64][625] floats and a pad
  const int nchunk = T / kPT;
  long long lid = blockIdx.x;
  const int t0 = (int)(lid % nchunk) * kPT;
  lid /= nchunk;
  const int m = (int)(lid % M), q4 = (int)(lid / M);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  {
    // wave w copies 64-float4 blocks w, w + 8, ...; the last block's lanes
    // past the run re-read its last float4 into the pad
    const float4* src =
        reinterpret_cast<const float4*>(X4 + (((size_t)q4 * M + m) * T + t0) * kPKB);
    for (int blk = wave; blk < kPBlk; blk += 8) {
      const int e = blk * 64 + lane;
      __builtin_amdgcn_global_load_lds((const void*)(src + (e < kPRun4 ? e : kPRun4 - 1)),
                                       (__attribute__((address_space(3))) void*)(lds4 + blk * 64),
                                       16, 0, 0);
    }
    wait_vmcnt<0>();
  }
  __syncthreads();
  const float* win = reinterpret_cast<const float*>(lds4) + lane * kPKB;
  for (int slot = wave; slot < 25; slot += 8)
    mix_branch<2, kStorePlanar, true, kPT, kPB>(win, slot, q4, m, t0, lane, V, M, T, 0, m0, m1,
                                                1);
}

// ---- output transform -------------------------------------------------------
// Levels 2 and 3: thread (tile t, level-4 branch q4, channel n), lanes on
// consecutive tiles.  Over the 25 level-3 branches, level2_reduce gives each
// branch's 4 x 4 block and the level-3 A^T accumulates the 12 x 12 block
// acc[i3r][i3c][rr][cc] (row 4 i3r + rr, column 4 i3c + cc), which goes to
// Z3[q4][n][t][e], e = 12 row + column (depth 4).
__global__ __launch_bounds__(64) void output_xform_mix23(const float4* __restrict__ Z,
                                                         float* __restrict__ out, int N, int T,
                                                         long long gstride, unsigned long long m0,
                                                         unsigned long long m1) {
  // grid (tile block, n, q4): consecutive work-groups read adjacent channels
  // of the same Z rows (0.317 -> 0.305 ms per step for the pair on the
  // 31 x 31 layer against q4 before n)
  const int t = blockIdx.x * 64 + threadIdx.x;
  const int n = blockIdx.y;
  const int q4 = blockIdx.z;
  if (t >= T) return;
  float acc[3][3][16];
#pragma unroll
  for (int a = 0; a < 3; ++a)
#pragma unroll
    for (int b = 0; b < 3; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.0f;
  const float4* zt = Z + (size_t)n * T + t;
  // a runtime loop over the 25 branches (one branch's 16 quads in flight at
  // a time: the 144 accumulators leave no room for more)
#pragma unroll 1
  for (int q3 = 0; q3 < 25; ++q3) {
    const int q3r = q3 / 5, q3c = q3 - 5 * q3r;
    const int ob = q4 * 25 + q3;
    // the dead groups' Z is zero and is not read (uniform over the work-group)
    const unsigned live = branch_live<2>(m0, m1, q4 / 5, q4 % 5, q3r, q3c);
    if (live == 0) continue;
    float po[4][4];
    level2_reduce(zt + (size_t)ob * 16 * gstride, (size_t)gstride, po, live);
    float cr[3], cc[3];
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      cr[i] = at5(i, q3r);
      cc[i] = at5(i, q3c);
    }
#pragma unroll
    for (int i3r = 0; i3r < 3; ++i3r)
#pragma unroll
      for (int i3c = 0; i3c < 3; ++i3c) {
        const float c = cr[i3r] * cc[i3c];
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i3r][i3c][e] = fmaf(c, po[e >> 2][e & 3], acc[i3r][i3c][e]);
      }
  }
  // Z3[q4][n][t][e], e = 12 row + column: a thread's 144 values are one
  // contiguous block (36 float4)
  float4* z3 = reinterpret_cast<float4*>(out + (((size_t)q4 * N + n) * T + t) * 144);
#pragma unroll
  for (int i3r = 0; i3r < 3; ++i3r)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr)
#pragma unroll
      for (int i3c = 0; i3c < 3; ++i3c) {
        const float* a = &acc[i3r][i3c][rr * 4];
        z3[(4 * i3r + rr) * 3 + i3c] = make_float4(a[0], a[1], a[2], a[3]);
      }
}

// Depth 3 (NO = 1): levels 2 and 3 straight to y, one thread per (tile t,
// output block (i3r, i3c), channel n), lanes on consecutive tiles: over the
// level-3 branches whose A^T coefficient for its block is nonzero (a
// work-group-uniform test), level2_reduce gives the branch's 4 x 4 block and
// the thread accumulates its own 4 x 4 output block.  Nine times the threads
// of a (tile, channel) split (the 144 accumulators of output_xform_mix23 leave
// one wavefront per CU on layers of a few hundred tiles).  A block's
// branches overlap its neighbours' (each Z value is read by up to nine
// blocks), so the work-groups are numbered per XCD (xcd_remap), tile block
// fastest, then output block, then channel: the 9 ntb work-groups of a
// channel run together on one XCD and share its Z through that XCD's L2.
__global__ __launch_bounds__(64) void output_xform_mix3(const float4* __restrict__ Z,
                                                        float* __restrict__ y, int N, int Ho,
                                                        int Wo, int th, int tw, int T,
                                                        long long gstride, unsigned long long m0,
                                                        unsigned long long m1) {
  const int ntb = (T + 63) / 64;
  const long long lid = xcd_remap(blockIdx.x, gridDim.x);
  const int tb = (int)(lid % ntb);
  const int blk = (int)((lid / ntb) % 9);   // 3 i3r + i3c
  const int n = (int)(lid / (9LL * ntb));
  const int t = tb * 64 + threadIdx.x;
  if (t >= T || n >= N) return;
  const int i3r = blk / 3, i3c = blk - 3 * i3r;
  float acc[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
  const float4* zt = Z + (size_t)n * T + t;
#pragma unroll 1
  for (int q3 = 0; q3 < 25; ++q3) {
    const int q3r = q3 / 5, q3c = q3 - 5 * q3r;
    const float c = at5(i3r, q3r) * at5(i3c, q3c);
    if (c == 0.0f) continue;                // uniform over the work-group
    const unsigned live = branch_live<1>(m0, m1, 0, 0, q3r, q3c);
    if (live == 0) continue;
    float po[4][4];
    level2_reduce(zt + (size_t)q3 * 16 * gstride, (size_t)gstride, po, live);
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = fmaf(c, po[e >> 2][e & 3], acc[e]);
  }
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  float* yo = y + ((size_t)b * N + n) * Ho * Wo;
#pragma unroll
  for (int rr = 0; rr < 4; ++rr) {
    const int row = ty * 12 + 4 * i3r + rr;
    if (row >= Ho) continue;
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) {
      const int col = tx * 12 + 4 * i3c + cc;
      if (col < Wo) yo[(size_t)row * Wo + col] = acc[rr * 4 + cc];
    }
  }
}

// Level 4 (NO = 2): thread (block element e, tile t, channel n), lanes on
// consecutive e (contiguous Z3 reads, 12-column runs of y), combines the 25
// level-4 branches of Z3 into the 3 x 3 blocks of the 36 x 36 tile.
__global__ __launch_bounds__(256) void output_xform_mix4(const float* __restrict__ Z3,
                                                         float* __restrict__ y, int N, int Ho,
                                                         int Wo, int th, int tw, int T,
                                                         long long total) {
  const long long id = (long long)blockIdx.x * 256 + threadIdx.x;
  if (id >= total) return;
  const int e = (int)(id % 144);
  const long long nt = id / 144;            // n T + t
  const int t = (int)(nt % T);
  const int n = (int)(nt / T);
  const size_t bs = (size_t)N * T * 144;    // between level-4 branches
  const float* zp = Z3 + (size_t)nt * 144 + e;
  float h[5][3];                            // [q4r][i4c]
#pragma unroll
  for (int q4r = 0; q4r < 5; ++q4r) {
    float v[5];
#pragma unroll
    for (int q4c = 0; q4c < 5; ++q4c) v[q4c] = zp[(size_t)(q4r * 5 + q4c) * bs];
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      float sacc = 0.0f;
#pragma unroll
      for (int q = 0; q < 5; ++q)
        if (at5(i, q) != 0.0f) sacc = fmaf(at5(i, q), v[q], sacc);
      h[q4r][i] = sacc;
    }
  }
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  const int er = e / 12, ec = e - er * 12;
  float* yo = y + ((size_t)b * N + n) * Ho * Wo;
#pragma unroll
  for (int i4r = 0; i4r < 3; ++i4r) {
    const int row = ty * 36 + 12 * i4r + er;
    if (row >= Ho) continue;
#pragma unroll
    for (int i4c = 0; i4c < 3; ++i4c) {
      const int col = tx * 36 + 12 * i4c + ec;
      if (col >= Wo) continue;
      float sacc = 0.0f;
#pragma unroll
      for (int q = 0; q < 5; ++q)
        if (at5(i4r, q) != 0.0f) sacc = fmaf(at5(i4r, q), h[q][i4c], sacc);
      yo[(size_t)row * Wo + col] = sacc;
    }
  }
}

}  // namespace

hipError_t launch_kernel_xform_mix(const nwg_plan_info& g, const float* w, float* U,
                                   hipStream_t s) {
  const int no = mix_outer_levels(g);
  if ((no != 1 && no != 2) || g.M > 65535 || ((uintptr_t)U & 15)) return hipErrorInvalidValue;
  const int K = no == 2 ? 39 : 15;
  const size_t lds = (size_t)16 * K * K * sizeof(float);
  dim3 grid((unsigned)((g.N + 15) / 16), (unsigned)g.M);
  // the dead quads' stores are dropped when a wave's four branches fit one
  // buffer resource; otherwise every quad of a live branch is stored
  const int q3 = g.level1_live == 0x7 ? 1 : 0;
  const bool mask = ((g.live_prefix[0] | g.live_prefix[1]) != 0 || q3) &&
                    4LL * 64 * g.M * g.N * 16 < (long long)kDrop;
  if (g.mix_planar) {
    // 32 output channels per work-group when their kernels and C fit in LDS
    if (no != 2 || g.r > 39) return hipErrorInvalidValue;
    const auto lds_of = [&](int nw) { return (size_t)nw * (g.r * g.r + 9 * g.r) * sizeof(float); };
    const bool wide = g.N % 32 == 0 && lds_of(32) <= 160 * 1024;
    const int nw = wide ? 32 : 16;
    const size_t ldsp = lds_of(nw);
    const auto fk = wide ? &kernel_xform_mix_sep<32> : &kernel_xform_mix_sep<16>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fk),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)ldsp);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fk, dim3((unsigned)((g.N + nw - 1) / nw), (unsigned)g.M), dim3(nw * 32),
                       ldsp, s, w, U, g.M, g.N, g.r, g.live_prefix[0], g.live_prefix[1]);
    return hipGetLastError();
  }
  const auto fn = no == 2 ? (mask ? &kernel_xform_mix<2, kStoreMasked>
                                       : &kernel_xform_mix<2, kStoreAll>)
                               : (mask ? &kernel_xform_mix<1, kStoreMasked>
                                       : &kernel_xform_mix<1, kStoreAll>);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(fn, grid, dim3(512), lds, s, w, U, g.M, g.N, g.r, g.live_prefix[0],
                     g.live_prefix[1], q3);
  return hipGetLastError();
}

hipError_t launch_input_xform_mix(const nwg_plan_info& g, const float* x, float* Vf,
                                  float* X4, hipStream_t s) {
  const int no = mix_outer_levels(g);
  if ((no != 1 && no != 2) || ((uintptr_t)Vf & 15) || (no == 2 && !X4))
    return hipErrorInvalidValue;
  float4* V = reinterpret_cast<float4*>(Vf);
  const long long qstride = (long long)g.M * g.T;
  const int tpw = no == 2 ? 32 : 16;       // tiles per work-group (TPW)
  const long long nwg = (g.T + tpw - 1) / tpw * g.M * (no == 2 ? 25 : 1);
  if (nwg > 0x7fffffffLL) return hipErrorInvalidValue;
  const size_t lds = (size_t)tpw * kWS * sizeof(float);
  // dead quads' stores dropped when a wave's 64 / TPW branches fit one
  // buffer resource
  const int q3 = g.level1_live == 0x7 ? 1 : 0;
  const bool mask = ((g.live_prefix[0] | g.live_prefix[1]) != 0 || q3) &&
                    (64LL / tpw) * 64 * qstride * 16 < (long long)kDrop;
  constexpr int A = kStoreAll, K = kStoreMasked;
  const auto fn =
      no == 2 ? (q3 ? (mask ? &input_xform_mix<2, K, true> : &input_xform_mix<2, A, true>)
                    : (mask ? &input_xform_mix<2, K, false> : &input_xform_mix<2, A, false>))
              : (q3 ? (mask ? &input_xform_mix<1, K, true> : &input_xform_mix<1, A, true>)
                    : (mask ? &input_xform_mix<1, K, false> : &input_xform_mix<1, A, false>));
  if (g.mix_planar) {
    // 25 x 25 level-4 blocks, then 64 tiles per work-group
    if (no != 2 || !q3 || g.M > 65535 || g.T % kPT) return hipErrorInvalidValue;
    hipLaunchKernelGGL(input_mix_l4<kPB>, dim3((unsigned)g.T, (unsigned)g.M), dim3(256), 0, s, x,
                       X4, g.M, g.H, g.W, g.pad, g.th, g.tw, (int)g.T);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t ldsp = (size_t)kPBlk * 64 * sizeof(float4);
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&input_xform_mix_p64),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)ldsp);
    if (e != hipSuccess) return e;
    const long long nwgp = (long long)(g.T / kPT) * g.M * 25;
    if (nwgp > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(input_xform_mix_p64, dim3((unsigned)nwgp), dim3(512), ldsp, s, X4, V, g.M,
                       (int)g.T, g.live_prefix[0], g.live_prefix[1]);
    return hipGetLastError();
  }
  if (no == 2) {
    if (g.M > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL(input_mix_l4<kL3>, dim3((unsigned)g.T, (unsigned)g.M), dim3(256), 0, s, x,
                       X4, g.M, g.H, g.W, g.pad, g.th, g.tw, (int)g.T);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const hipError_t ea = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (ea != hipSuccess) return ea;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)nwg), dim3(no == 2 ? 512 : 256), lds, s, x, X4, V, g.M,
                     g.H, g.W, g.pad, g.th, g.tw, (int)g.T, qstride, g.live_prefix[0],
                     g.live_prefix[1], q3);
  return hipGetLastError();
}

hipError_t launch_output_xform_mix(const nwg_plan_info& g, const float* Zf, float* y,
                                   float* Z3, hipStream_t s) {
  const int no = mix_outer_levels(g);
  if ((no != 1 && no != 2) || ((uintptr_t)Zf & 15) || g.N > 65535) return hipErrorInvalidValue;
  const float4* Z = reinterpret_cast<const float4*>(Zf);
  const long long gstride = (long long)g.N * g.T;
  const unsigned tb = (unsigned)((g.T + 63) / 64);
  if (no == 1) {
    const long long nwg = 9LL * tb * g.N;
    if (nwg > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(output_xform_mix3, dim3((unsigned)nwg), dim3(64), 0, s, Z, y, g.N,
                       g.Ho, g.Wo, g.th, g.tw, (int)g.T, gstride, g.live_prefix[0],
                       g.live_prefix[1]);
    return hipGetLastError();
  }
  if (!Z3) return hipErrorInvalidValue;
  hipLaunchKernelGGL(output_xform_mix23, dim3(tb, (unsigned)g.N, 25), dim3(64), 0, s, Z, Z3, g.N,
                     (int)g.T, gstride, g.live_prefix[0], g.live_prefix[1]);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long long total = 144LL * g.N * g.T;
  const long long blocks = (total + 255) / 256;
  if (blocks > 0x7fffffffLL || ((uintptr_t)Z3 & 15)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(output_xform_mix4, dim3((unsigned)blocks), dim3(256), 0, s, Z3, y, g.N, g.Ho,
                     g.Wo, g.th, g.tw, (int)g.T, total);
  return hipGetLastError();
}

}  // namespace nwg
