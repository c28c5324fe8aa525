// Nested output transformation (Sec. III.B, final step; 2D per Fig. 4 text),
// levels 2..n.  Level 1 is already applied by the contraction, which writes
//
//     Z[g][n][t][2*i1r + i1c],   g = p / 16 (the point's digits above level 1).
//
// For every tile t and output channel n this applies A^T of F(2,3) along
// both axes for levels 2..n, giving the output reordered tensor Y[i;k]
// (i_j, k_j in {0,1}), flattened to the M_n x M_n output tile: row
// sum_j 2^(j-1) i_j, column sum_j 2^(j-1) k_j.  Outputs beyond Ho x Wo are
// cropped.
//
// Reads are float4 quads Z[g][n][t] with consecutive lanes on consecutive
// tiles: 256 contiguous bytes per quarter-wave.  Each thread reduces the
// 16 level-2 groups of one branch in registers (4x4 partial tile).  At depth
// >= 3 a lane sums the 4 branches of one level-3 row digit, and the 4 rows
// of a tile, held by the 4 quarter-waves of one wavefront, are combined by
// lane shuffles (no LDS); at depth 4 the level-4 A^T accumulates the 16
// level-4 branches in registers.
#include "nwg_internal.h"

namespace nwg {
namespace {

// ---- depth 1 and 2: one thread per tile -----------------------------------
template <int NLEV>
__global__ __launch_bounds__(256) void output_xform_tile(
    const float4* __restrict__ Z, float* __restrict__ y, int N, int Ho, int Wo, int th, int tw,
    int T, long long gstride) {
  constexpr int Mn = 1 << NLEV;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int n = blockIdx.y;
  if (t >= T) return;
  const float4* zb = Z + (size_t)n * T + t;
  float po[4][4];
  if constexpr (NLEV == 2) {
    level2_reduce(zb, (size_t)gstride, po);
  } else {
    const float4 v = zb[0];
    po[0][0] = v.x;  po[0][1] = v.y;
    po[1][0] = v.z;  po[1][1] = v.w;
  }
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  float* yo = y + ((size_t)b * N + n) * Ho * Wo;
#pragma unroll
  for (int i = 0; i < Mn; ++i) {
    const int row = ty * Mn + i;
    if (row >= Ho) continue;
#pragma unroll
    for (int k = 0; k < Mn; ++k) {
      const int col = tx * Mn + k;
      if (col < Wo) yo[(size_t)row * Wo + col] = po[i][k];
    }
  }
}

// ---- depth 3 and 4: one wavefront per 16 tiles, level 3 by shuffles -------
// Lane (tl, q3r): tile tl of the wavefront's 16, level-3 row digit q3r.
// Per level-4 branch the lane reduces the 4 branches q3c of its row (levels
// 2 and the column half of level 3) in registers, giving C[i3c][rr][cc].
// The row half of level 3, y3[i3r] = sum_q3r A^T[i3r][q3r] C_q3r, combines
// the 4 quarter-waves holding q3r = 0..3 in two shuffle steps (lane xor 16,
// then xor 32), each moving 16 values, after which the lane owns the 4x4
// block (i3r, i3c) = (q3r >> 1, q3r & 1) of the tile.  Level 4 accumulates
// over the 16 level-4 branches in registers.  Z reads are float4 with 16
// consecutive tiles per quarter-wave; y is written as float4 row segments.
//
// Shuffle step 1 (partner q3r ^ 1) keeps half k = q3r & 1 (i3c = k):
//   q3r = 0: u = a0 + a1, w = a1      q3r = 1: u = a0 + a1, w = a1
//   q3r = 2: u = a2,      w = a2 + a3 q3r = 3: u = a2,      w = a2 + a3
// (a_q = C of row q, for column half k).  Step 2 (partner q3r ^ 2):
//   q3r < 2: y3[0] = u + u(partner)   q3r >= 2: y3[1] = w(partner) - w
// which are the two A^T rows (1, 1, 1, 0) and (0, 1, -1, -1).
// m0, m1: the plan's live digit prefixes (nwg_plan_info::live_prefix; both 0
// when every group is live): the groups no tap reaches are not read (the
// contraction does not write them; their Z is zero).
template <int NLEV>
__global__ __launch_bounds__(64) void output_xform_shfl(
    const float4* __restrict__ Z, float* __restrict__ y, int N, int Ho, int Wo, int th, int tw,
    int T, long long gstride, int vec, unsigned long long m0, unsigned long long m1) {
  constexpr int Mn = 1 << NLEV;
  constexpr int PASSES = NLEV == 4 ? 16 : 1;
  constexpr int NI4 = NLEV == 4 ? 2 : 1;
  const int n = blockIdx.y;
  const int lane = threadIdx.x;
  const int tl = lane & 15, q3r = lane >> 4;
  const int t = blockIdx.x * 16 + tl;
  const bool valid = t < T;
  const int k = q3r & 1;
  // step-1 and step-2 coefficients of this lane (see above)
  const float cu0 = q3r == 3 ? 0.0f : 1.0f, cu1 = q3r == 2 ? 0.0f : 1.0f;
  const float cw0 = q3r == 0 ? 0.0f : 1.0f, cw1 = q3r == 1 ? 0.0f : 1.0f;
  const bool low = q3r < 2;
  float acc[NI4][NI4][16];
#pragma unroll
  for (int a = 0; a < NI4; ++a)
#pragma unroll
    for (int b = 0; b < NI4; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.0f;

  const float4* zt = Z + (size_t)n * T + (valid ? t : 0);
  for (int pass = 0; pass < PASSES; ++pass) {
    // levels 2 and the column half of level 3 over this row's 4 branches
    float C[2][16];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 16; ++e) C[h][e] = 0.0f;
    if (valid) {
      // depth 4: two branches' 32 quad loads in flight at a time (240
      // registers, two wavefronts per SIMD); depth 3 has one pass and keeps
      // all four branches in flight
      const int p4r = pass >> 2, p4c = pass & 3;
      const unsigned nr = prefix_nibble(m0, m1, NLEV == 4 ? p4r * 4 + q3r : q3r);
#pragma unroll (NLEV == 3 ? 4 : 2)
      for (int q3c = 0; q3c < 4; ++q3c) {
        const int branch = pass * 16 + q3r * 4 + q3c;
        const unsigned live = (m0 | m1) == 0
            ? 0xffffu
            : nibble_live(nr, prefix_nibble(m0, m1, NLEV == 4 ? p4c * 4 + q3c : q3c));
        float po[4][4];
        level2_reduce(zt + (size_t)branch * 16 * gstride, (size_t)gstride, po, live);
        const float c0 = at_coef(0, q3c), c1 = at_coef(1, q3c);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          C[0][e] += c0 * po[e >> 2][e & 3];
          C[1][e] += c1 * po[e >> 2][e & 3];
        }
      }
    }
    // row half of level 3 across the four quarter-waves
    float out[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float keep = k ? C[1][e] : C[0][e];
      const float give = k ? C[0][e] : C[1][e];
      const float r = __shfl_xor(give, 16);
      const float u = cu0 * keep + cu1 * r;
      const float w = cw0 * keep + cw1 * r;
      const float r2 = __shfl_xor(low ? w : u, 32);
      out[e] = low ? u + r2 : r2 - w;
    }
    const int q4r = pass >> 2, q4c = pass & 3;
#pragma unroll
    for (int a = 0; a < NI4; ++a)
#pragma unroll
      for (int b = 0; b < NI4; ++b) {
        const float c4 = NLEV == 4 ? at_coef(a, q4r) * at_coef(b, q4c) : 1.0f;
        if (NLEV == 4) {
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[a][b][e] += c4 * out[e];
        } else {
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[a][b][e] = out[e];
        }
      }
  }
  if (!valid) return;
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  float* yo = y + ((size_t)b * N + n) * Ho * Wo;
  const int i3r = q3r >> 1, i3c = q3r & 1;
#pragma unroll
  for (int a = 0; a < NI4; ++a)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int row = ty * Mn + 8 * a + 4 * i3r + rr;
      if (row >= Ho) continue;
      float* yr = yo + (size_t)row * Wo;
#pragma unroll
      for (int c = 0; c < NI4; ++c) {
        const int col = tx * Mn + 8 * c + 4 * i3c;
        const float* v = &acc[a][c][rr * 4];
        if (vec && col + 3 < Wo) {
          *reinterpret_cast<float4*>(yr + col) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
#pragma unroll
          for (int cc = 0; cc < 4; ++cc)
            if (col + cc < Wo) yr[col + cc] = v[cc];
        }
      }
    }
}

}  // namespace

hipError_t launch_output_xform(const nwg_plan_info& g, const float* Zf, float* y, hipStream_t s) {
  if ((uintptr_t)Zf & 15) return hipErrorInvalidValue;
  const float4* Z = reinterpret_cast<const float4*>(Zf);
  const long long gstride = (long long)g.N * g.T;    // float4 quads between groups
  const int T = (int)g.T;
  if (g.n >= 3) {
    // float4 stores of y rows need 16-byte aligned rows
    const int vec = (g.Wo % 4 == 0 && ((uintptr_t)y & 15) == 0) ? 1 : 0;
    // the dead groups of a dense F(2,3) chain (none elsewhere)
    const bool dead = g.tile == NWG_TILE_F2X2_3X3 && !g.depthwise && g.live_np > 0;
    const unsigned long long m0 = dead ? g.live_prefix[0] : 0, m1 = dead ? g.live_prefix[1] : 0;
    dim3 grid((unsigned)((g.T + 15) / 16), (unsigned)g.N);
    if (g.n == 3)
      hipLaunchKernelGGL(output_xform_shfl<3>, grid, dim3(64), 0, s, Z, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, gstride, vec, m0, m1);
    else
      hipLaunchKernelGGL(output_xform_shfl<4>, grid, dim3(64), 0, s, Z, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, gstride, vec, m0, m1);
  } else {
    dim3 grid((unsigned)((g.T + 255) / 256), (unsigned)g.N);
    if (g.n == 2)
      hipLaunchKernelGGL(output_xform_tile<2>, grid, dim3(256), 0, s, Z, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, gstride);
    else
      hipLaunchKernelGGL(output_xform_tile<1>, grid, dim3(256), 0, s, Z, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, gstride);
  }
  return hipGetLastError();
}

}  // namespace nwg
