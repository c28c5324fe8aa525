// Depthwise nested-Winograd convolution (Table I's depth-wise row): each of
// the C channels is correlated with its own r x r kernel and there is no sum
// over channels, so the Winograd-domain step is an element-wise product
// Yhat[p][c][t] = U[p][c] V[p][c][t] instead of a contraction (Sec. III.B
// with M = 1 per channel).  The transforms are those of the dense path.
//
//   depth 0 (r = 1):  y = w[c] x                         (dw_scale)
//   depth 1, 2:       the input transform, the product and the whole
//                     output transform in one kernel, windows staged in
//                     LDS: x -> y; one lane per (tile, channel) at depth 1
//                     (dw_small_d1), four at depth 2 (dw_small_d2)
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

// ---- depth 1: lane per (tile, channel), x -> y ------------------------------
// A work-group takes one channel and a box of up to 256 tiles: the union of
// their 4 x 4 windows is staged in LDS with coalesced row reads (zero
// outside the image), together with the channel's 4 U quads; each lane then
// reads its window as aligned 8-byte LDS rows.
__global__ __launch_bounds__(256) void dw_small_d1(const float* __restrict__ x,
                                                   const float4* __restrict__ U,
                                                   float* __restrict__ y, int C, int H, int W,
                                                   int pad, int Ho, int Wo, int th, int tw, int RX,
                                                   int RY, int nbx, int nby, int BW) {
  constexpr int Mn = 2, Ln = 4;
  extern __shared__ float4 smem4[];
  float4* Us = smem4;
  float* box = reinterpret_cast<float*>(smem4 + 4);
  const int c = blockIdx.y;
  int bid = blockIdx.x;
  const int bx = bid % nbx;
  bid /= nbx;
  const int by = bid % nby;
  const int b = bid / nby;
  const int ty0 = by * RY, tx0 = bx * RX;
  const int BH = (RY - 1) * Mn + Ln;
  const int r0 = ty0 * Mn - pad, c0 = tx0 * Mn - pad;
  const float* __restrict__ xp = x + ((size_t)b * C + c) * H * W;
  if (threadIdx.x < 4) Us[threadIdx.x] = U[(size_t)threadIdx.x * C + c];
  for (int e = threadIdx.x; e < BH * BW; e += 256) {
    const int row = e / BW, col = e - row * BW;
    const int gr = r0 + row, gc = c0 + col;
    float v = 0.0f;
    if (gr >= 0 && gr < H && gc >= 0 && gc < W) v = xp[(size_t)gr * W + gc];
    box[e] = v;
  }
  __syncthreads();
  const int s = threadIdx.x;
  if (s >= RX * RY) return;
  const int ly = s / RX, lx = s - ly * RX;
  const int ty = ty0 + ly, tx = tx0 + lx;
  if (ty >= th || tx >= tw) return;
  const float* wb = box + ly * Mn * BW + lx * Mn;
  float win[Ln][Ln];
#pragma unroll
  for (int i = 0; i < Ln; ++i) {
    const float2 a = *reinterpret_cast<const float2*>(wb + i * BW);
    const float2 bq = *reinterpret_cast<const float2*>(wb + i * BW + 2);
    win[i][0] = a.x;  win[i][1] = a.y;  win[i][2] = bq.x; win[i][3] = bq.y;
  }
  float acc[2][2] = {{0.0f, 0.0f}, {0.0f, 0.0f}};
  // B^T along the rows, then along the columns: o[q1c] for row digit q1r
#pragma unroll
  for (int q1r = 0; q1r < 4; ++q1r) {
    float R[4], o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      R[j] = bt_sign0(q1r) * win[bt_tap0(q1r)][j] + bt_sign1(q1r) * win[bt_tap1(q1r)][j];
    bt_one(R, o);
    const float4 u = Us[q1r];
    const float p0 = o[0] * u.x, p1 = o[1] * u.y, p2 = o[2] * u.z, p3 = o[3] * u.w;
    const float z0 = p0 + p1 + p2, z1 = p1 - p2 - p3;
#pragma unroll
    for (int i1r = 0; i1r < 2; ++i1r) {
      const float e = at_coef(i1r, q1r);
      acc[i1r][0] += e * z0;
      acc[i1r][1] += e * z1;
    }
  }
  float* __restrict__ yo = y + ((size_t)b * C + c) * Ho * Wo;
#pragma unroll
  for (int i = 0; i < Mn; ++i) {
    const int row = ty * Mn + i;
    if (row >= Ho) continue;
#pragma unroll
    for (int k = 0; k < Mn; ++k) {
      const int col = tx * Mn + k;
      if (col < Wo) yo[(size_t)row * Wo + col] = acc[i][k];
    }
  }
}

// ---- depth 2: four lanes per (tile, channel) ---------------------------------
// Lane (tile, q2r): the lane runs the level-2 row digit q2r of its tile (the
// window's 8 rows that digit reads, levels 1-2 of the columns, the product
// and the column output transform) and keeps 16 partial outputs.  The 4
// lanes of a tile then add their partials in two shuffle steps (xor 1, xor
// 2; 8 then 4 values), after which lane q2r owns output row q2r of the tile
// and stores it as one float4.  64 tiles per work-group.
__global__ __launch_bounds__(256) void dw_small_d2(const float* __restrict__ x,
                                                   const float4* __restrict__ U,
                                                   float* __restrict__ y, int C, int H, int W,
                                                   int pad, int Ho, int Wo, int th, int tw, int RX,
                                                   int RY, int nbx, int nby, int BW, int vec) {
  constexpr int Mn = 4, Ln = 10;
  extern __shared__ float4 smem4[];
  // the channel's 64 U quads, 17 quads per level-2 row digit: the four
  // digits' lanes of a tile read 272 bytes apart, in different banks
  float4* Us = smem4;
  float* box = reinterpret_cast<float*>(smem4 + 68);
  const int c = blockIdx.y;
  int bid = blockIdx.x;
  const int bx = bid % nbx;
  bid /= nbx;
  const int by = bid % nby;
  const int b = bid / nby;
  const int ty0 = by * RY, tx0 = bx * RX;
  const int BH = (RY - 1) * Mn + Ln;
  const int r0 = ty0 * Mn - pad, c0 = tx0 * Mn - pad;
  const float* __restrict__ xp = x + ((size_t)b * C + c) * H * W;
  if (threadIdx.x < 64)
    Us[(threadIdx.x >> 4) * 17 + (threadIdx.x & 15)] = U[(size_t)threadIdx.x * C + c];
  {
    // element e = tid + 256 k of the box, walked incrementally; batches of FB
    // clamped (always in-bounds) loads are issued together, then masked
    constexpr int FB = 4;
    const int nel = BH * BW;
    const int tid = threadIdx.x;
    const int drow = 256 / BW, dcol = 256 - drow * BW;
    int row = tid / BW, col = tid - row * BW;
    for (int e0 = 0; e0 < nel; e0 += 256 * FB) {
      float v[FB];
      bool ok[FB];
#pragma unroll
      for (int k = 0; k < FB; ++k) {
        const int gr = r0 + row, gc = c0 + col;
        ok[k] = gr >= 0 && gr < H && gc >= 0 && gc < W;
        const int grc = gr < 0 ? 0 : (gr > H - 1 ? H - 1 : gr);
        const int gcc = gc < 0 ? 0 : (gc > W - 1 ? W - 1 : gc);
        v[k] = xp[(size_t)grc * W + gcc];
        row += drow;
        col += dcol;
        if (col >= BW) {
          col -= BW;
          ++row;
        }
      }
#pragma unroll
      for (int k = 0; k < FB; ++k) {
        const int e = e0 + k * 256 + tid;
        if (e < nel) box[e] = ok[k] ? v[k] : 0.0f;
      }
    }
  }
  __syncthreads();
  const int q2r = threadIdx.x & 3;
  const int s = threadIdx.x >> 2;               // tile within the box
  const int ly = s / RX, lx = s - ly * RX;
  const int ty = ty0 + ly, tx = tx0 + lx;
  // lanes past the box or the image still take part in the shuffles
  const bool valid = s < RX * RY && ty < th && tx < tw;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[i][k] = 0.0f;
  if (valid) {
    const float* wb = box + ly * Mn * BW + lx * Mn;
    auto read_row = [&](int i, float (&v)[Ln]) {
      const float4 a = *reinterpret_cast<const float4*>(wb + i * BW);
      const float4 bq = *reinterpret_cast<const float4*>(wb + i * BW + 4);
      const float2 cq = *reinterpret_cast<const float2*>(wb + i * BW + 8);
      v[0] = a.x;  v[1] = a.y;  v[2] = a.z;  v[3] = a.w;
      v[4] = bq.x; v[5] = bq.y; v[6] = bq.z; v[7] = bq.w;
      v[8] = cq.x; v[9] = cq.y;
    };
    // level 2 along the rows: sg0 (ra + sg0 sg1 rb), the factor sg0 = +-1
    // moved into the digit's output coefficients e2
    float Zr[4][Ln];
    const int a0 = 2 * bt_tap0(q2r), a1 = 2 * bt_tap1(q2r);
    const float sg0 = bt_sign0(q2r), s01 = bt_sign0(q2r) * bt_sign1(q2r);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      float ra[Ln], rb[Ln];
      read_row(u + a0, ra);
      read_row(u + a1, rb);
#pragma unroll
      for (int j = 0; j < Ln; ++j) Zr[u][j] = fmaf(s01, rb[j], ra[j]);
    }
    const float e2[2] = {sg0 * at_coef(0, q2r), sg0 * at_coef(1, q2r)};
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r) {
      float R[10], o[16];
#pragma unroll
      for (int j = 0; j < 10; ++j)
        R[j] = bt_sign0(q1r) * Zr[bt_tap0(q1r)][j] + bt_sign1(q1r) * Zr[bt_tap1(q1r)][j];
      bt_inner2(R, o);   // index q2c * 4 + q1c
      float col1[4][2];
#pragma unroll
      for (int q2c = 0; q2c < 4; ++q2c) {
        const float4 u = Us[q2r * 17 + q2c * 4 + q1r];
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
  }
  // sum over the tile's 4 lanes; lane q2r ends with output row q2r
  const int b0 = q2r & 1, b1 = q2r >> 1;
  float h[2][4];                                // rows b0 and b0 + 2
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
  if (!valid) return;
  const int row = ty * Mn + q2r;
  if (row >= Ho) return;
  float* __restrict__ yr = y + ((size_t)b * C + c) * Ho * Wo + (size_t)row * Wo;
  const int col = tx * Mn;
  if (vec && col + 3 < Wo) {
    *reinterpret_cast<float4*>(yr + col) = make_float4(out[0], out[1], out[2], out[3]);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (col + k < Wo) yr[col + k] = out[k];
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
  if (g.N > 65535) return hipErrorInvalidValue;
  const int Mn = 1 << g.n, Ln = 3 * Mn - 2;
  // depth 2: 64 tiles x 4 lanes per work-group; depth 1: 256 tiles
  const int tiles = g.n == 2 ? 64 : 256;
  const int RX = g.tw < tiles ? g.tw : tiles;
  int RY = tiles / RX;
  if (RY > g.th) RY = g.th;
  const int nbx = (g.tw + RX - 1) / RX, nby = (g.th + RY - 1) / RY;
  const long long blocks = (long long)nbx * nby * g.B;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  // box rows padded to 16 bytes, so every window row starts aligned
  const int BW = ((RX - 1) * Mn + Ln + 3) & ~3;
  const int BH = (RY - 1) * Mn + Ln;
  const int P4 = g.n == 1 ? 4 : 68;            // U quads in LDS (depth 2: padded)
  const size_t lds = (size_t)P4 * 16 + (size_t)BH * BW * sizeof(float);
  const int vec = (g.Wo % 4 == 0 && ((uintptr_t)y & 15) == 0) ? 1 : 0;
  const float4* U = reinterpret_cast<const float4*>(Uf);
  dim3 grid((unsigned)blocks, (unsigned)g.N);
  if (g.n == 1)
    hipLaunchKernelGGL(dw_small_d1, grid, dim3(256), lds, s, x, U, y, g.N, g.H, g.W, g.pad, g.Ho,
                       g.Wo, g.th, g.tw, RX, RY, nbx, nby, BW);
  else
    hipLaunchKernelGGL(dw_small_d2, grid, dim3(256), lds, s, x, U, y, g.N, g.H, g.W, g.pad, g.Ho,
                       g.Wo, g.th, g.tw, RX, RY, nbx, nby, BW, vec);
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
