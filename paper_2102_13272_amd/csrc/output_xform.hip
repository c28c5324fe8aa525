// Nested output transformation (Sec. III.B, final step; 2D per Fig. 4 text).
//
// For every tile t and output channel n, the P = 4^(2n) values Yhat[p][n][t]
// are transformed by A^T of F(2,3) along every axis, giving the output
// reordered tensor Y[i;k] (i_j, k_j in {0,1}), which is flattened to the
// M_n x M_n output tile: row sum_j s_{j-1} i_j, column sum_j s_{j-1} k_j,
// with s_{j-1} = 2^(j-1).  Outputs beyond Ho x Wo are cropped.
//
// Reads are Yhat[p][n][t] with consecutive lanes on consecutive tiles
// (contiguous runs of the T axis).  Each thread reduces the 256 points of
// one branch through the two innermost levels in registers (16 -> 4 per
// axis).  At depth >= 3 the 16 level-3 branches of a tile sit in 16
// different threads; their 4x4 partial outputs go through LDS, where the
// level-3 A^T combines them, and at depth 4 the level-4 A^T accumulates the
// 16 level-4 branches in registers over 16 passes.
#include "nwg_internal.h"

namespace nwg {
namespace {

// Two inner levels for one branch: 256 points -> 4x4 partial tile.
// po[rr][cc], rr = i1r + 2*i2r, cc = i1c + 2*i2c.  yb points at the branch's
// first point; points are (q2r, q2c, q1r, q1c), most significant first.
__device__ __forceinline__ void inner2_reduce(const float* __restrict__ yb, size_t pstride,
                                              float (&po)[4][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) po[i][k] = 0.0f;
#pragma unroll
  for (int q2r = 0; q2r < 4; ++q2r) {
#pragma unroll
    for (int q2c = 0; q2c < 4; ++q2c) {
      float v[4][4];
#pragma unroll
      for (int q1r = 0; q1r < 4; ++q1r)
#pragma unroll
        for (int q1c = 0; q1c < 4; ++q1c)
          v[q1r][q1c] = yb[(size_t)(q2r * 64 + q2c * 16 + q1r * 4 + q1c) * pstride];
      // level 1 along columns then rows: 4x4 -> 2x2
      float h[4][2];
#pragma unroll
      for (int q1r = 0; q1r < 4; ++q1r) {
        h[q1r][0] = v[q1r][0] + v[q1r][1] + v[q1r][2];
        h[q1r][1] = v[q1r][1] - v[q1r][2] - v[q1r][3];
      }
      float e[2][2];
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        e[0][c] = h[0][c] + h[1][c] + h[2][c];
        e[1][c] = h[1][c] - h[2][c] - h[3][c];
      }
      // level 2: add with A^T[i2r][q2r] * A^T[i2c][q2c]
#pragma unroll
      for (int i2r = 0; i2r < 2; ++i2r)
#pragma unroll
        for (int i2c = 0; i2c < 2; ++i2c) {
          const float c = at_coef(i2r, q2r) * at_coef(i2c, q2c);
          if (c != 0.0f) {
#pragma unroll
            for (int i1r = 0; i1r < 2; ++i1r)
#pragma unroll
              for (int i1c = 0; i1c < 2; ++i1c)
                po[i1r + 2 * i2r][i1c + 2 * i2c] += c * e[i1r][i1c];
          }
        }
    }
  }
}

// ---- depth 1 and 2: one thread per tile -----------------------------------
template <int NLEV>
__global__ __launch_bounds__(256) void output_xform_tile(
    const float* __restrict__ Yh, float* __restrict__ y, int N, int Ho, int Wo, int th, int tw,
    int T, long long NT) {
  constexpr int Mn = 1 << NLEV;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int n = blockIdx.y;
  if (t >= T) return;
  const float* yb = Yh + (size_t)n * T + t;
  float po[4][4];
  if constexpr (NLEV == 2) {
    inner2_reduce(yb, (size_t)NT, po);
  } else {
    float v[4][4];
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r)
#pragma unroll
      for (int q1c = 0; q1c < 4; ++q1c) v[q1r][q1c] = yb[(size_t)(q1r * 4 + q1c) * NT];
    float h[4][2];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      h[q][0] = v[q][0] + v[q][1] + v[q][2];
      h[q][1] = v[q][1] - v[q][2] - v[q][3];
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      po[0][c] = h[0][c] + h[1][c] + h[2][c];
      po[1][c] = h[1][c] - h[2][c] - h[3][c];
    }
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
    const float* __restrict__ Yh, float* __restrict__ y, int N, int Ho, int Wo, int th, int tw,
    int T, long long NT) {
  constexpr int Mn = 1 << NLEV;
  constexpr int PASSES = NLEV == 4 ? 16 : 1;
  __shared__ float part[16][16][17];        // [tile][level-3 branch][partial output]
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

  const float* yslot = Yh + (size_t)slot * 256 * NT + (size_t)n * T + t;
  for (int pass = 0; pass < PASSES; ++pass) {
    float po[4][4];
    if (valid) {
      inner2_reduce(yslot + (size_t)pass * 4096 * NT, (size_t)NT, po);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int k = 0; k < 4; ++k) po[i][k] = 0.0f;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) part[tl][slot][i * 4 + k] = po[i][k];
    __syncthreads();
    // level 3 across the 16 branches of tile tl, for partial output e
    float pv[4][4];
#pragma unroll
    for (int q3r = 0; q3r < 4; ++q3r)
#pragma unroll
      for (int q3c = 0; q3c < 4; ++q3c) pv[q3r][q3c] = part[tl][q3r * 4 + q3c][e];
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

hipError_t launch_output_xform(const nwg_plan_info& g, const float* Yh, float* y, hipStream_t s) {
  const long long NT = (long long)g.N * g.T;
  const int T = (int)g.T;
  if (g.n >= 3) {
    dim3 grid((unsigned)((g.T + 15) / 16), (unsigned)g.N);
    if (g.n == 3)
      hipLaunchKernelGGL(output_xform_branches<3>, grid, dim3(256), 0, s, Yh, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, NT);
    else
      hipLaunchKernelGGL(output_xform_branches<4>, grid, dim3(256), 0, s, Yh, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, NT);
  } else {
    dim3 grid((unsigned)((g.T + 255) / 256), (unsigned)g.N);
    if (g.n == 2)
      hipLaunchKernelGGL(output_xform_tile<2>, grid, dim3(256), 0, s, Yh, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, NT);
    else
      hipLaunchKernelGGL(output_xform_tile<1>, grid, dim3(256), 0, s, Yh, y, g.N, g.Ho, g.Wo,
                         g.th, g.tw, T, NT);
  }
  return hipGetLastError();
}

}  // namespace nwg
