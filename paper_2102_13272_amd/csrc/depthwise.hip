// Depthwise nested-Winograd convolution (Table I's depth-wise row): each of
// the C channels is correlated with its own r x r kernel and there is no sum
// over channels, so the Winograd-domain step is an element-wise product
// Yhat[p][c][t] = U[p][c] V[p][c][t] instead of a contraction (Sec. III.B
// with M = 1 per channel).  The transforms are those of the dense path.
//
//   depth 0 (r = 1):  y = w[c] x                         (dw_scale)
//   depth 1, 2:       one lane per (tile, channel) runs the input
//                     transform, the product and the whole output
//                     transform in registers: x -> y     (dw_small)
//   depth 3, 4:       the fused input-transform kernel writes Z (see
//                     fused_small.hip), then the output transform
//   stage call:       U, V -> Z, the product and the level-1 output
//                     transform                          (dw_contract)
//
// U is the kernel transform of w [C][1][r][r] seen as N = C kernels of one
// input channel: U[P/4][1][C][4] (float4 quads over the level-1 column
// digit), so a wavefront of one channel reads the same U quads (scalar
// loads).
#include "nwg_internal.h"

namespace nwg {
namespace {

// ---- depth 0: y[b][c] = U[c] x[b][c] ----------------------------------------
__global__ __launch_bounds__(256) void dw_scale(const float* __restrict__ x,
                                                const float* __restrict__ U, float* __restrict__ y,
                                                int C, long long HW, long long total) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int c = (int)((i / HW) % C);
  y[i] = U[c] * x[i];
}

// ---- depth 1 and 2: lane per (tile, channel), x -> y ------------------------
template <int NLEV>
__global__ __launch_bounds__(256) void dw_small(const float* __restrict__ x,
                                                const float4* __restrict__ U,
                                                float* __restrict__ y, int C, int H, int W,
                                                int pad, int Ho, int Wo, int th, int tw, int T) {
  constexpr int Mn = 1 << NLEV;
  constexpr int Ln = 3 * Mn - 2;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int c = blockIdx.y;
  if (t >= T) return;
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  const int gr0 = ty * Mn - pad, gc0 = tx * Mn - pad;
  const float* __restrict__ xp = x + ((size_t)b * C + c) * H * W;
  // the L_n x L_n window, zero outside the image (clamped loads, then masked)
  float win[Ln][Ln];
  {
    int col[Ln];
    float cm[Ln];
#pragma unroll
    for (int j = 0; j < Ln; ++j) {
      const int gc = gc0 + j;
      cm[j] = (gc >= 0 && gc < W) ? 1.0f : 0.0f;
      col[j] = gc < 0 ? 0 : (gc > W - 1 ? W - 1 : gc);
    }
#pragma unroll
    for (int i = 0; i < Ln; ++i) {
      const int gr = gr0 + i;
      const float rm = (gr >= 0 && gr < H) ? 1.0f : 0.0f;
      const float* row = xp + (size_t)(gr < 0 ? 0 : (gr > H - 1 ? H - 1 : gr)) * W;
#pragma unroll
      for (int j = 0; j < Ln; ++j) win[i][j] = rm * cm[j] * row[col[j]];
    }
  }
  const float4* __restrict__ Uc = U + c;     // quad q of this channel at Uc[q * C]
  // output accumulators, rows and columns ordered (i_n, ..., i_1)
  float acc[Mn][Mn];
#pragma unroll
  for (int i = 0; i < Mn; ++i)
#pragma unroll
    for (int k = 0; k < Mn; ++k) acc[i][k] = 0.0f;

  if constexpr (NLEV == 1) {
    // B^T along the rows, then along the columns: o[q1r][q1c]
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r) {
      float R[4], o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        R[j] = bt_sign0(q1r) * win[bt_tap0(q1r)][j] + bt_sign1(q1r) * win[bt_tap1(q1r)][j];
      bt_one(R, o);
      const float4 u = Uc[(size_t)q1r * C];
      const float p0 = o[0] * u.x, p1 = o[1] * u.y, p2 = o[2] * u.z, p3 = o[3] * u.w;
      const float z0 = p0 + p1 + p2, z1 = p1 - p2 - p3;
#pragma unroll
      for (int i1r = 0; i1r < 2; ++i1r) {
        const float e = at_coef(i1r, q1r);
        acc[i1r][0] += e * z0;
        acc[i1r][1] += e * z1;
      }
    }
  } else {
#pragma unroll
    for (int q2r = 0; q2r < 4; ++q2r) {
      float Zr[4][Ln];
      const int a0 = 2 * bt_tap0(q2r), a1 = 2 * bt_tap1(q2r);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int j = 0; j < Ln; ++j)
          Zr[u][j] = bt_sign0(q2r) * win[u + a0][j] + bt_sign1(q2r) * win[u + a1][j];
#pragma unroll
      for (int q1r = 0; q1r < 4; ++q1r) {
        float R[10], o[16];
#pragma unroll
        for (int j = 0; j < 10; ++j)
          R[j] = bt_sign0(q1r) * Zr[bt_tap0(q1r)][j] + bt_sign1(q1r) * Zr[bt_tap1(q1r)][j];
        bt_inner2(R, o);   // index q2c * 4 + q1c
        // product, then the output transform along the columns (levels 1, 2)
        float col1[4][2];
#pragma unroll
        for (int q2c = 0; q2c < 4; ++q2c) {
          const float4 u = Uc[(size_t)(q2r * 16 + q2c * 4 + q1r) * C];
          const float p0 = o[q2c * 4 + 0] * u.x, p1 = o[q2c * 4 + 1] * u.y;
          const float p2 = o[q2c * 4 + 2] * u.z, p3 = o[q2c * 4 + 3] * u.w;
          col1[q2c][0] = p0 + p1 + p2;
          col1[q2c][1] = p1 - p2 - p3;
        }
        float colf[2][2];   // [i2c][i1c]
#pragma unroll
        for (int i1c = 0; i1c < 2; ++i1c) {
          colf[0][i1c] = col1[0][i1c] + col1[1][i1c] + col1[2][i1c];
          colf[1][i1c] = col1[1][i1c] - col1[2][i1c] - col1[3][i1c];
        }
        // then along the rows
#pragma unroll
        for (int i2r = 0; i2r < 2; ++i2r)
#pragma unroll
          for (int i1r = 0; i1r < 2; ++i1r) {
            const float e = at_coef(i2r, q2r) * at_coef(i1r, q1r);
            if (e == 0.0f) continue;
#pragma unroll
            for (int i2c = 0; i2c < 2; ++i2c)
#pragma unroll
              for (int i1c = 0; i1c < 2; ++i1c)
                acc[2 * i2r + i1r][2 * i2c + i1c] += e * colf[i2c][i1c];
          }
      }
    }
  }
  float* __restrict__ yo = y + ((size_t)b * C + c) * Ho * Wo;
#pragma unroll
  for (int i = 0; i < Mn; ++i) {
    const int row = ty * Mn + i;
    if (row >= Ho) continue;
#pragma unroll
    for (int k = 0; k < Mn; ++k) {
      const int colo = tx * Mn + k;
      if (colo < Wo) yo[(size_t)row * Wo + colo] = acc[i][k];
    }
  }
}

// ---- stage call: U, V -> Z (product and level-1 output transform) ----------
__global__ __launch_bounds__(256) void dw_contract(const float4* __restrict__ U,
                                                   const float4* __restrict__ V,
                                                   float4* __restrict__ Z, int C, int T) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int c = blockIdx.y;
  const long long g = blockIdx.z;
  if (t >= T) return;
  float z[2][2] = {{0.0f, 0.0f}, {0.0f, 0.0f}};
#pragma unroll
  for (int q1r = 0; q1r < 4; ++q1r) {
    const size_t quad = (size_t)(4 * g + q1r);
    const float4 u = U[quad * C + c];
    const float4 v = V[(quad * C + c) * T + t];
    const float p0 = u.x * v.x, p1 = u.y * v.y, p2 = u.z * v.z, p3 = u.w * v.w;
    const float z0 = p0 + p1 + p2, z1 = p1 - p2 - p3;
#pragma unroll
    for (int i1r = 0; i1r < 2; ++i1r) {
      const float e = at_coef(i1r, q1r);
      z[i1r][0] += e * z0;
      z[i1r][1] += e * z1;
    }
  }
  Z[((size_t)g * C + c) * T + t] = make_float4(z[0][0], z[0][1], z[1][0], z[1][1]);
}

}  // namespace

hipError_t launch_dw_scale(const nwg_plan_info& g, const float* x, const float* U, float* y,
                           hipStream_t s) {
  const long long HW = (long long)g.H * g.W;
  const long long total = (long long)g.B * g.N * HW;
  const long long blocks = (total + 255) / 256;
  if (g.n != 0 || blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dw_scale, dim3((unsigned)blocks), dim3(256), 0, s, x, U, y, g.N, HW, total);
  return hipGetLastError();
}

hipError_t launch_dw_small(const nwg_plan_info& g, const float* x, const float* Uf, float* y,
                           hipStream_t s) {
  if ((g.n != 1 && g.n != 2) || ((uintptr_t)Uf & 15)) return hipErrorInvalidValue;
  if (g.N > 65535 || g.T > 0x7fffffffLL - 255) return hipErrorInvalidValue;
  const int T = (int)g.T;
  const float4* U = reinterpret_cast<const float4*>(Uf);
  dim3 grid((unsigned)((T + 255) / 256), (unsigned)g.N);
  if (g.n == 1)
    hipLaunchKernelGGL(dw_small<1>, grid, dim3(256), 0, s, x, U, y, g.N, g.H, g.W, g.pad, g.Ho,
                       g.Wo, g.th, g.tw, T);
  else
    hipLaunchKernelGGL(dw_small<2>, grid, dim3(256), 0, s, x, U, y, g.N, g.H, g.W, g.pad, g.Ho,
                       g.Wo, g.th, g.tw, T);
  return hipGetLastError();
}

hipError_t launch_dw_contract(const nwg_plan_info& g, const float* Uf, const float* Vf,
                              float* Zf, hipStream_t s) {
  if (g.n < 1 || (((uintptr_t)Uf | (uintptr_t)Vf | (uintptr_t)Zf) & 15))
    return hipErrorInvalidValue;
  const long long G = g.P / 16;
  if (g.N > 65535 || G > 65535 || g.T > 0x7fffffffLL - 255) return hipErrorInvalidValue;
  const int T = (int)g.T;
  dim3 grid((unsigned)((T + 255) / 256), (unsigned)g.N, (unsigned)G);
  hipLaunchKernelGGL(dw_contract, grid, dim3(256), 0, s, reinterpret_cast<const float4*>(Uf),
                     reinterpret_cast<const float4*>(Vf), reinterpret_cast<float4*>(Zf), g.N, T);
  return hipGetLastError();
}

}  // namespace nwg
