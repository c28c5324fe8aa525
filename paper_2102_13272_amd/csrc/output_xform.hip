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
// >= 3 the 16 level-3 branches of a tile sit in 16 different threads; their
// partial tiles go through LDS, where the level-3 A^T combines them, and at
// depth 4 the level-4 A^T accumulates the 16 level-4 branches in registers
// over 16 passes.
#include "nwg_internal.h"

namespace nwg {
namespace {

// Level 2 for one branch: 16 quads (q2r, q2c) -> 4x4 partial tile
// po[rr][cc], rr = i1r + 2*i2r, cc = i1c + 2*i2c.  zb points at the branch's
// first quad for this (n, t); gstride is the distance between groups.
__device__ __forceinline__ void level2_reduce(const float4* __restrict__ zb, size_t gstride,
                                              float (&po)[4][4]) {
  float4 v[4][4];
#pragma unroll
  for (int q2r = 0; q2r < 4; ++q2r)
#pragma unroll
    for (int q2c = 0; q2c < 4; ++q2c) v[q2r][q2c] = zb[(size_t)(q2r * 4 + q2c) * gstride];
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

// ---- depth 3 and 4: 16 tiles x 16 level-3 branches per work-group ---------
template <int NLEV>
__global__ __launch_bounds__(256) void output_xform_branches(
    const float4* __restrict__ Z, float* __restrict__ y, int N, int Ho, int Wo, int th, int tw,
    int T, long long gstride) {
  constexpr int Mn = 1 << NLEV;
  constexpr int PASSES = NLEV == 4 ? 16 : 1;
  // [tile][level-3 branch][partial output]; odd tile stride (16*17+1): the
  // 16 tiles of a quarter-wave hit 16 different banks
  constexpr int TS = 16 * 17 + 1;
  __shared__ float part[16 * TS];
  const int n = blockIdx.y;
  const int tl = threadIdx.x & 15;
  const int slot = threadIdx.x >> 4;
  const int t = blockIdx.x * 16 + tl;
  const bool valid = t < T;
  // phase-2 role: this thread finalises partial output e = slot of tile tl
  const int e = slot;
  float acc[2][2][2][2];                    // [i4r][i4c][i3r][i3c]
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int d = 0; d < 2; ++d) acc[a][b][c][d] = 0.0f;

  const float4* zslot = Z + (size_t)slot * 16 * gstride + (size_t)n * T + t;
  for (int pass = 0; pass < PASSES; ++pass) {
    float po[4][4];
    if (valid) {
      level2_reduce(zslot + (size_t)pass * 256 * gstride, (size_t)gstride, po);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int k = 0; k < 4; ++k) po[i][k] = 0.0f;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) part[tl * TS + slot * 17 + i * 4 + k] = po[i][k];
    __syncthreads();
    // level 3 across the 16 branches of tile tl, for partial output e
    float pv[4][4];
#pragma unroll
    for (int q3r = 0; q3r < 4; ++q3r)
#pragma unroll
      for (int q3c = 0; q3c < 4; ++q3c) pv[q3r][q3c] = part[tl * TS + (q3r * 4 + q3c) * 17 + e];
    const int q4r = pass >> 2, q4c = pass & 3;
#pragma unroll
    for (int i3r = 0; i3r < 2; ++i3r)
#pragma unroll
      for (int i3c = 0; i3c < 2; ++i3c) {
        float s = 0.0f;
#pragma unroll
        for (int q3r = 0; q3r < 4; ++q3r)
#pragma unroll
          for (int q3c = 0; q3c < 4; ++q3c) {
            const float c = at_coef(i3r, q3r) * at_coef(i3c, q3c);
            if (c != 0.0f) s += c * pv[q3r][q3c];
          }
#pragma unroll
        for (int i4r = 0; i4r < 2; ++i4r)
#pragma unroll
          for (int i4c = 0; i4c < 2; ++i4c) {
            const float c4 = NLEV == 4 ? at_coef(i4r, q4r) * at_coef(i4c, q4c)
                                       : (i4r == 0 && i4c == 0 ? 1.0f : 0.0f);
            acc[i4r][i4c][i3r][i3c] += c4 * s;
          }
      }
    __syncthreads();
  }
  if (!valid) return;
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  float* yo = y + ((size_t)b * N + n) * Ho * Wo;
  const int rr = e >> 2, cc = e & 3;
  constexpr int NI4 = NLEV == 4 ? 2 : 1;
#pragma unroll
  for (int i4r = 0; i4r < NI4; ++i4r)
#pragma unroll
    for (int i3r = 0; i3r < 2; ++i3r) {
      const int row = ty * Mn + 8 * i4r + 4 * i3r + rr;
      if (row >= Ho) continue;
#pragma unroll
      for (int i4c = 0; i4c < NI4; ++i4c)
#pragma unroll
        for (int i3c = 0; i3c < 2; ++i3c) {
          const int col = tx * Mn + 8 * i4c + 4 * i3c + cc;
          if (col < Wo) yo[(size_t)row * Wo + col] = acc[i4r][i4c][i3r][i3c];
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
    dim3 grid((unsigned)((g.T + 15) / 16), (unsigned)g.N);
    if (g.n == 3)
      hipLaunchKernelGGL(output_xform_branches<3>, grid, dim3(256), 0, s, Z, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, gstride);
    else
      hipLaunchKernelGGL(output_xform_branches<4>, grid, dim3(256), 0, s, Z, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, gstride);
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
