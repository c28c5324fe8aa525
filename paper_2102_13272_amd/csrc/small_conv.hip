// Layers with few channels at depth 1 or 2: the whole nested convolution
// (input transform, per-point channel sum, output transform; Sec. III.B) in
// one kernel, x -> y.  With M and N in the single digits the transformed
// tensors V and Z are 4x (depth 1) to 16x (depth 2) larger than x and y,
// and the three-kernel path spends its time moving them through HBM; here
// they stay in registers.
//
//   depth 1, M <= 8, N <= 16 (small_d1<M>): one lane per tile.  The lane
//     reads its 4 x 4 window of every input channel from an LDS-staged box,
//     forms V_m (16 points each) in registers, and for each output channel
//     n accumulates sum_m U[p][m][n] V_m[p], applies A^T along both axes and
//     writes the 2 x 2 outputs.
//   depth 2, M <= 2, M N <= 64 (small_d2<M>): four lanes per tile, lane q2r
//     holds the 64 points of its level-2 row digit for each input channel;
//     for each n it multiplies by U, applies the column output transform and
//     its row coefficients, and the tile's four lanes add their 4 x 4 partial
//     tiles with two xor shuffles, each writing one output row as a float4.
//
// U (the kernel transform, [P/4][M][N][4] quads) is staged in LDS per work-
// group.  Windows of a box of tiles of one image are staged in LDS with
// coalesced, clamped, masked loads (zero outside the image).
#include "nwg_internal.h"

namespace nwg {
namespace {

// The boxes of RX x RY tiles of image b for all MC input channels: rows
// r0 .., columns c0 .., MC x BH x BW floats at dst (channel-major); 256
// threads walk the flat box with batches of FB independent clamped loads,
// so the whole fill costs one or two memory round trips.
template <int MC>
__device__ __forceinline__ void stage_boxes(const float* __restrict__ xb, float* dst, int H,
                                            int W, int r0, int c0, int BH, int BW) {
  constexpr int FB = 16;
  const int plane = BH * BW;
  const int nel = MC * plane;
  const int tid = threadIdx.x;
  // position of element tid, and the step of 256 elements, as (channel, row, col)
  int m = tid / plane;
  int row = (tid - m * plane) / BW;
  int col = tid - m * plane - row * BW;
  const int dm = 256 / plane, drow = (256 - dm * plane) / BW, dcol = 256 - dm * plane - drow * BW;
  for (int e0 = 0; e0 < nel; e0 += 256 * FB) {
    float v[FB];
    bool ok[FB];
#pragma unroll
    for (int k = 0; k < FB; ++k) {
      const int gr = r0 + row, gc = c0 + col;
      const int mc = m < MC ? m : MC - 1;
      ok[k] = m < MC && gr >= 0 && gr < H && gc >= 0 && gc < W;
      const int grc = gr < 0 ? 0 : (gr > H - 1 ? H - 1 : gr);
      const int gcc = gc < 0 ? 0 : (gc > W - 1 ? W - 1 : gc);
      v[k] = xb[(size_t)mc * H * W + (size_t)grc * W + gcc];
      m += dm;
      row += drow;
      col += dcol;
      if (col >= BW) {
        col -= BW;
        ++row;
      }
      if (row >= BH) {
        row -= BH;
        ++m;
      }
    }
#pragma unroll
    for (int k = 0; k < FB; ++k) {
      const int e = e0 + k * 256 + tid;
      if (e < nel) dst[e] = ok[k] ? v[k] : 0.0f;
    }
  }
}

// ---- depth 1 ----------------------------------------------------------------
// Work-group (box of tiles, output-channel group blockIdx.y): the group's
// channels [n0, n0 + NG) of the N; more groups give more wavefronts for
// the same tiles (each group recomputes the tiles' V).
template <int MC>
__global__ __launch_bounds__(256) void small_d1(const float* __restrict__ x,
                                                const float4* __restrict__ U,
                                                float* __restrict__ y, int N, int NG, int H, int W,
                                                int pad, int Ho, int Wo, int th, int tw, int RX,
                                                int RY, int nbx, int nby, int BW, int vec) {
  constexpr int Mn = 2, Ln = 4;
  extern __shared__ float4 smem4[];
  const int n0 = blockIdx.y * NG;
  const int nc = N - n0 < NG ? N - n0 : NG;            // channels of this group
  float4* Us = smem4;                                  // [n - n0][m][q1r], 4 * MC * NG quads
  float* box = reinterpret_cast<float*>(smem4 + 4 * MC * NG);
  int bid = blockIdx.x;
  const int bx = bid % nbx;
  bid /= nbx;
  const int by = bid % nby;
  const int b = bid / nby;
  const int ty0 = by * RY, tx0 = bx * RX;
  const int BH = (RY - 1) * Mn + Ln;
  const int r0 = ty0 * Mn - pad, c0 = tx0 * Mn - pad;
  for (int i = threadIdx.x; i < 4 * MC * nc; i += 256) {
    // U quad (q1r, m, n) is at q1r * M * N + m * N + n
    const int q1r = i & 3, mn = i >> 2;
    const int n = mn / MC, m = mn - n * MC;
    Us[i] = U[(size_t)q1r * MC * N + (size_t)m * N + n0 + n];
  }
  stage_boxes<MC>(x + (size_t)b * MC * H * W, box, H, W, r0, c0, BH, BW);
  __syncthreads();
  const int s = threadIdx.x;
  if (s >= RX * RY) return;
  const int ly = s / RX, lx = s - ly * RX;
  const int ty = ty0 + ly, tx = tx0 + lx;
  if (ty >= th || tx >= tw) return;
  // V_m[q1r][q1c] for every input channel
  float V[MC][4][4];
#pragma unroll
  for (int m = 0; m < MC; ++m) {
    const float* wb = box + m * BH * BW + ly * Mn * BW + lx * Mn;
    float win[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float2 a = *reinterpret_cast<const float2*>(wb + i * BW);
      const float2 c = *reinterpret_cast<const float2*>(wb + i * BW + 2);
      win[i][0] = a.x;  win[i][1] = a.y;  win[i][2] = c.x;  win[i][3] = c.y;
    }
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r) {
      float R[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        R[j] = bt_sign0(q1r) * win[bt_tap0(q1r)][j] + bt_sign1(q1r) * win[bt_tap1(q1r)][j];
      bt_one(R, V[m][q1r]);
    }
  }
  const size_t plane = (size_t)Ho * Wo;
  float* __restrict__ yb = y + (size_t)b * N * plane;
  const int row0 = ty * Mn, col = tx * Mn;
  for (int n = 0; n < nc; ++n) {
    float acc[2][2] = {{0.0f, 0.0f}, {0.0f, 0.0f}};
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r) {
      float p[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int m = 0; m < MC; ++m) {
        const float4 u = Us[(n * MC + m) * 4 + q1r];
        p[0] = fmaf(u.x, V[m][q1r][0], p[0]);
        p[1] = fmaf(u.y, V[m][q1r][1], p[1]);
        p[2] = fmaf(u.z, V[m][q1r][2], p[2]);
        p[3] = fmaf(u.w, V[m][q1r][3], p[3]);
      }
      const float z0 = p[0] + p[1] + p[2], z1 = p[1] - p[2] - p[3];
#pragma unroll
      for (int i1r = 0; i1r < 2; ++i1r) {
        const float e = at_coef(i1r, q1r);
        acc[i1r][0] += e * z0;
        acc[i1r][1] += e * z1;
      }
    }
    float* yo = yb + (size_t)(n0 + n) * plane;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int row = row0 + i;
      if (row >= Ho) continue;
      float* yr = yo + (size_t)row * Wo;
      if (vec && col + 1 < Wo) {
        *reinterpret_cast<float2*>(yr + col) = make_float2(acc[i][0], acc[i][1]);
      } else {
        if (col < Wo) yr[col] = acc[i][0];
        if (col + 1 < Wo) yr[col + 1] = acc[i][1];
      }
    }
  }
}

// ---- depth 2 ----------------------------------------------------------------
template <int MC>
__global__ __launch_bounds__(256) void small_d2(const float* __restrict__ x,
                                                const float4* __restrict__ U,
                                                float* __restrict__ y, int N, int NG, int H, int W,
                                                int pad, int Ho, int Wo, int th, int tw, int RX,
                                                int RY, int nbx, int nby, int BW, int vec) {
  constexpr int Mn = 4, Ln = 10;
  constexpr int QS = 68;                               // quads per (n, m): 17 per row digit
  extern __shared__ float4 smem4[];
  const int n0 = blockIdx.y * NG;
  const int nc = N - n0 < NG ? N - n0 : NG;            // channels of this group
  // U quads [n - n0][m][q2r * 17 + q2c * 4 + q1r]: the four row digits' lanes
  // of a tile read 272 bytes apart, in different banks
  float4* Us = smem4;
  float* box = reinterpret_cast<float*>(smem4 + QS * MC * NG);
  int bid = blockIdx.x;
  const int bx = bid % nbx;
  bid /= nbx;
  const int by = bid % nby;
  const int b = bid / nby;
  const int ty0 = by * RY, tx0 = bx * RX;
  const int BH = (RY - 1) * Mn + Ln;
  const int r0 = ty0 * Mn - pad, c0 = tx0 * Mn - pad;
  for (int i = threadIdx.x; i < 64 * MC * nc; i += 256) {
    // source U quad (q, m, n) at q * M * N + m * N + n, q = q2r*16 + q2c*4 + q1r
    const int q = i & 63, mn = i >> 6;
    const int n = mn / MC, m = mn - n * MC;
    Us[(size_t)mn * QS + (q >> 4) * 17 + (q & 15)] =
        U[(size_t)q * MC * N + (size_t)m * N + n0 + n];
  }
  stage_boxes<MC>(x + (size_t)b * MC * H * W, box, H, W, r0, c0, BH, BW);
  __syncthreads();
  const int q2r = threadIdx.x & 3;
  const int s = threadIdx.x >> 2;                      // tile within the box
  const int ly = s / RX, lx = s - ly * RX;
  const int ty = ty0 + ly, tx = tx0 + lx;
  // lanes past the box or the image still take part in the shuffles
  const bool valid = s < RX * RY && ty < th && tx < tw;
  // this lane's 64 points (q1r, q2c, q1c) of row digit q2r, per input channel
  // (the factor sg0 = +-1 of the level-2 row goes into the output coefficients)
  float V[MC][4][16];
  const float sg0 = bt_sign0(q2r), s01 = bt_sign0(q2r) * bt_sign1(q2r);
  const int a0 = 2 * bt_tap0(q2r), a1 = 2 * bt_tap1(q2r);
#pragma unroll
  for (int m = 0; m < MC; ++m) {
    if (!valid) {
#pragma unroll
      for (int q1r = 0; q1r < 4; ++q1r)
#pragma unroll
        for (int j = 0; j < 16; ++j) V[m][q1r][j] = 0.0f;
      continue;
    }
    const float* wb = box + m * BH * BW + ly * Mn * BW + lx * Mn;
    float Zr[4][Ln];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float* ra = wb + (u + a0) * BW;
      const float* rb = wb + (u + a1) * BW;
      const float4 a_0 = *reinterpret_cast<const float4*>(ra);
      const float4 a_1 = *reinterpret_cast<const float4*>(ra + 4);
      const float2 a_2 = *reinterpret_cast<const float2*>(ra + 8);
      const float4 b_0 = *reinterpret_cast<const float4*>(rb);
      const float4 b_1 = *reinterpret_cast<const float4*>(rb + 4);
      const float2 b_2 = *reinterpret_cast<const float2*>(rb + 8);
      const float av[Ln] = {a_0.x, a_0.y, a_0.z, a_0.w, a_1.x, a_1.y, a_1.z, a_1.w, a_2.x, a_2.y};
      const float bv[Ln] = {b_0.x, b_0.y, b_0.z, b_0.w, b_1.x, b_1.y, b_1.z, b_1.w, b_2.x, b_2.y};
#pragma unroll
      for (int j = 0; j < Ln; ++j) Zr[u][j] = fmaf(s01, bv[j], av[j]);
    }
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r) {
      float R[10];
#pragma unroll
      for (int j = 0; j < 10; ++j)
        R[j] = bt_sign0(q1r) * Zr[bt_tap0(q1r)][j] + bt_sign1(q1r) * Zr[bt_tap1(q1r)][j];
      bt_inner2(R, V[m][q1r]);                         // index q2c * 4 + q1c
    }
  }
  const float e2[2] = {sg0 * at_coef(0, q2r), sg0 * at_coef(1, q2r)};
  const int b0 = q2r & 1, b1 = q2r >> 1;
  const size_t plane = (size_t)Ho * Wo;
  const int row = ty * Mn + q2r, col = tx * Mn;
  for (int n = 0; n < nc; ++n) {
    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[i][k] = 0.0f;
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r) {
      float col1[4][2];
#pragma unroll
      for (int q2c = 0; q2c < 4; ++q2c) {
        float p[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int m = 0; m < MC; ++m) {
          const float4 u = Us[(size_t)(n * MC + m) * QS + q2r * 17 + q2c * 4 + q1r];
          p[0] = fmaf(u.x, V[m][q1r][q2c * 4 + 0], p[0]);
          p[1] = fmaf(u.y, V[m][q1r][q2c * 4 + 1], p[1]);
          p[2] = fmaf(u.z, V[m][q1r][q2c * 4 + 2], p[2]);
          p[3] = fmaf(u.w, V[m][q1r][q2c * 4 + 3], p[3]);
        }
        col1[q2c][0] = p[0] + p[1] + p[2];
        col1[q2c][1] = p[1] - p[2] - p[3];
      }
      float colf[2][2];   // [i2c][i1c]
#pragma unroll
      for (int i1c = 0; i1c < 2; ++i1c) {
        colf[0][i1c] = col1[0][i1c] + col1[1][i1c] + col1[2][i1c];
        colf[1][i1c] = col1[1][i1c] - col1[2][i1c] - col1[3][i1c];
      }
#pragma unroll
      for (int i2r = 0; i2r < 2; ++i2r)
#pragma unroll
        for (int i1r = 0; i1r < 2; ++i1r) {
          if (at_coef(i1r, q1r) == 0.0f) continue;
          const float e = e2[i2r] * at_coef(i1r, q1r);
#pragma unroll
          for (int i2c = 0; i2c < 2; ++i2c)
#pragma unroll
            for (int i1c = 0; i1c < 2; ++i1c)
              acc[2 * i2r + i1r][2 * i2c + i1c] += e * colf[i2c][i1c];
        }
    }
    // sum over the tile's 4 lanes; lane q2r ends with output row q2r
    float h[2][4];                                     // rows b0 and b0 + 2
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float give0 = b0 ? acc[0][k] : acc[1][k];
      const float give1 = b0 ? acc[2][k] : acc[3][k];
      h[0][k] = (b0 ? acc[1][k] : acc[0][k]) + __shfl_xor(give0, 1);
      h[1][k] = (b0 ? acc[3][k] : acc[2][k]) + __shfl_xor(give1, 1);
    }
    float out[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float give = b1 ? h[0][k] : h[1][k];
      out[k] = (b1 ? h[1][k] : h[0][k]) + __shfl_xor(give, 2);
    }
    if (valid && row < Ho) {
      float* yr = y + ((size_t)b * N + n0 + n) * plane + (size_t)row * Wo;
      if (vec && col + 3 < Wo) {
        *reinterpret_cast<float4*>(yr + col) = make_float4(out[0], out[1], out[2], out[3]);
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (col + k < Wo) yr[col + k] = out[k];
      }
    }
  }
}

// output-channel groups per box: enough work-groups for four per CU (256
// CUs), at most one group per channel
int n_groups(long long boxes, int N) {
  long long ng = (1024 + boxes - 1) / boxes;
  if (ng > N) ng = N;
  return ng < 1 ? 1 : (int)ng;
}

template <int MC>
hipError_t launch_small_d1(const nwg_plan_info& g, const float* x, const float4* U, float* y,
                           hipStream_t s) {
  const int RX = g.tw < 256 ? g.tw : 256;
  int RY = 256 / RX;
  if (RY > g.th) RY = g.th;
  const int nbx = (g.tw + RX - 1) / RX, nby = (g.th + RY - 1) / RY;
  const long long blocks = (long long)nbx * nby * g.B;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  const int BW = ((RX - 1) * 2 + 4 + 1) & ~1;          // even: 8-byte aligned window rows
  const int BH = (RY - 1) * 2 + 4;
  const int ngroups = n_groups(blocks, g.N), NG = (g.N + ngroups - 1) / ngroups;
  const size_t lds = (size_t)4 * MC * NG * 16 + (size_t)MC * BH * BW * sizeof(float);
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  const int vec = (g.Wo % 2 == 0 && ((uintptr_t)y & 7) == 0) ? 1 : 0;
  hipLaunchKernelGGL(small_d1<MC>, dim3((unsigned)blocks, (unsigned)((g.N + NG - 1) / NG)),
                     dim3(256), lds, s, x, U, y, g.N, NG, g.H, g.W, g.pad, g.Ho, g.Wo, g.th, g.tw,
                     RX, RY, nbx, nby, BW, vec);
  return hipGetLastError();
}

template <int MC>
hipError_t launch_small_d2(const nwg_plan_info& g, const float* x, const float4* U, float* y,
                           hipStream_t s) {
  const int RX = g.tw < 64 ? g.tw : 64;                // 64 tiles x 4 lanes
  int RY = 64 / RX;
  if (RY > g.th) RY = g.th;
  const int nbx = (g.tw + RX - 1) / RX, nby = (g.th + RY - 1) / RY;
  const long long blocks = (long long)nbx * nby * g.B;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  const int BW = ((RX - 1) * 4 + 10 + 3) & ~3;         // 16-byte aligned window rows
  const int BH = (RY - 1) * 4 + 10;
  const int ngroups = n_groups(blocks, g.N), NG = (g.N + ngroups - 1) / ngroups;
  const size_t lds = (size_t)68 * MC * NG * 16 + (size_t)MC * BH * BW * sizeof(float);
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  const int vec = (g.Wo % 4 == 0 && ((uintptr_t)y & 15) == 0) ? 1 : 0;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&small_d2<MC>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(small_d2<MC>, dim3((unsigned)blocks, (unsigned)((g.N + NG - 1) / NG)),
                     dim3(256), lds, s, x, U, y, g.N, NG, g.H, g.W, g.pad, g.Ho, g.Wo, g.th, g.tw,
                     RX, RY, nbx, nby, BW, vec);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_small_conv(const nwg_plan_info& g, const float* x, const float* Uf, float* y,
                             hipStream_t s) {
  if (!small_conv_applies(g) || ((uintptr_t)Uf & 15)) return hipErrorInvalidValue;
  const float4* U = reinterpret_cast<const float4*>(Uf);
  if (g.n == 1) {
    switch (g.M) {
      case 1: return launch_small_d1<1>(g, x, U, y, s);
      case 2: return launch_small_d1<2>(g, x, U, y, s);
      case 3: return launch_small_d1<3>(g, x, U, y, s);
      case 4: return launch_small_d1<4>(g, x, U, y, s);
      case 5: return launch_small_d1<5>(g, x, U, y, s);
      case 6: return launch_small_d1<6>(g, x, U, y, s);
      case 7: return launch_small_d1<7>(g, x, U, y, s);
      default: return launch_small_d1<8>(g, x, U, y, s);
    }
  }
  return g.M == 1 ? launch_small_d2<1>(g, x, U, y, s) : launch_small_d2<2>(g, x, U, y, s);
}

}  // namespace nwg
