// Fused nested input transformation + channel contraction + level-1 output
// transformation for layers with one or two output channels at depth 3 or 4,
// and for depthwise layers at depth 3 or 4
// (Sec. III.B: the input-transform and element-wise steps, and the first
// level of the output transform).
//
// With N <= 2 output channels the contraction does 2 N flops per transformed
// input value, while the transformed input V is (L_n / M_n)^2 = 64x (depth 3)
// or ~100x (depth 4) larger than the input: the unfused path spends nearly
// all its time writing V to HBM and reading it back.  This kernel never
// forms V in memory.  For every input channel it stages the tiles' windows
// in LDS, computes each level-3 branch's 256 points in registers (the same
// level order as the input-transform kernel), multiplies them by
// U[p][m][n] and folds the level-1 A^T into 64 accumulators per output
// channel.  After the last channel it writes Z[g][n][t][4] (float4, the
// layout the output transform reads).
//
// Work decomposition: a wavefront owns 4 consecutive tiles x 16 level-3
// branches (lane = 4 * branch + tile) and a subset of the input channels;
// the CS wavefronts of a work-group split the channels (m = wave, wave + CS,
// ...) with private LDS windows and add their partial sums at the end.  At
// depth 4 a work-group owns one level-4 branch (q4r, q4c), whose B^T rows
// are applied while filling the 22 x 22 windows.
//
// Per lane the branch's sub-window is S = k (a + rr c), a = w00 + cc w01,
// c = w10 + cc w11, with the sign products rr, cc and k = +-1 of the
// level-3 rows: three FMAs per value, and k is applied to the accumulators
// once at the end (every product with S is linear in S).
#include "nwg_internal.h"

namespace nwg {
namespace {

// Orders the LDS accesses of one wavefront: stores issued before it are seen
// by loads issued after it, from any lane of the same wavefront.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

constexpr int kTilesPerWave = 4;
constexpr int kWin = 22;                    // window side left for levels 1..3
constexpr int kWinStride = kWin * kWin + 1; // odd: the 4 tiles' windows start in different banks

// DW: depthwise, one channel per launch row (blockIdx.y): x channel ch is
// multiplied by U quad (p/4, 0, ch) of U[P/4][1][C][4] and written to Z
// channel ch; no sum over channels (M = N = C, NC = 1, CS = 1).
template <int NLEV, int NC, int CS, bool DW>
__global__ __launch_bounds__(64 * CS) void input_contract_small(
    const float* __restrict__ x, const float4* __restrict__ U, float4* __restrict__ Z, int M,
    int N, int H, int W, int pad, int th, int tw, int T) {
  static_assert(!DW || (NC == 1 && CS == 1), "depthwise: one channel, one wavefront");
  constexpr int Mn = 1 << NLEV;
  constexpr int L3 = kWin, WS = kWinStride, TW = kTilesPerWave;
  constexpr int NTASK = (TW * L3 + 63) / 64;   // window columns filled per lane
  __shared__ float lds[CS * TW * WS];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // Work-group -> (level-4 branch, tile chunk), the branch fastest.  The
  // dispatcher deals work-groups round-robin over the 8 XCDs; this numbering
  // gives each XCD a contiguous range, so the 16 branches that read the same
  // windows run on one XCD and share its L2.
  long long lid;
  {
    const long long G = (long long)gridDim.x, i = blockIdx.x;
    const long long q = G / 8, rem = G % 8, xcd = i % 8, sl = i / 8;
    lid = xcd < rem ? xcd * (q + 1) + sl : rem * (q + 1) + (xcd - rem) * q + sl;
  }
  const int q4 = NLEV == 4 ? (int)(lid % 16) : 0;
  const int t0 = (int)(NLEV == 4 ? lid / 16 : lid) * TW;
  const int q4r = q4 >> 2, q4c = q4 & 3;
  const int tpi = th * tw;
  float* wbuf = lds + wave * TW * WS;

  // ---- fill tasks: window column c of tile ftl, for idx = lane + 64 k
  const int a4r0 = 8 * bt_tap0(q4r), a4r1 = 8 * bt_tap1(q4r);
  const float s4r0 = bt_sign0(q4r), s4r1 = bt_sign1(q4r);
  bool f_ok[NTASK];
  int f_img[NTASK];                                // b M H W (< 2^31, checked at launch)
  int f_dst[NTASK], f_gr0[NTASK], f_ca[NTASK], f_cb[NTASK];
  float f_ma[NTASK], f_mb[NTASK];
#pragma unroll
  for (int k = 0; k < NTASK; ++k) {
    const int idx = lane + 64 * k;
    const int ftl = idx / L3, c = idx - ftl * L3;
    const int ft = t0 + ftl;
    f_ok[k] = idx < TW * L3 && ft < T;
    f_img[k] = 0;
    f_dst[k] = 0;
    f_gr0[k] = 0;
    f_ca[k] = f_cb[k] = 0;
    f_ma[k] = f_mb[k] = 0.0f;
    if (f_ok[k]) {
      const int b = ft / tpi;
      const int r2 = ft - b * tpi;
      const int ty = r2 / tw, tx = r2 - ty * tw;
      f_img[k] = b * M * H * W;
      f_dst[k] = ftl * WS + c;
      f_gr0[k] = ty * Mn - pad;
      const int gc = tx * Mn - pad + c;
      if (NLEV == 4) {
        const int ca = gc + 8 * bt_tap0(q4c), cb = gc + 8 * bt_tap1(q4c);
        f_ma[k] = (ca >= 0 && ca < W) ? bt_sign0(q4c) : 0.0f;
        f_mb[k] = (cb >= 0 && cb < W) ? bt_sign1(q4c) : 0.0f;
        f_ca[k] = ca < 0 ? 0 : (ca > W - 1 ? W - 1 : ca);
        f_cb[k] = cb < 0 ? 0 : (cb > W - 1 ? W - 1 : cb);
      } else {
        f_ma[k] = (gc >= 0 && gc < W) ? 1.0f : 0.0f;
        f_ca[k] = gc < 0 ? 0 : (gc > W - 1 ? W - 1 : gc);
      }
    }
  }

  // ---- compute role: tile tl, level-3 branch slot = (q3r, q3c)
  const int tl = lane & 3, slot = lane >> 2;
  const int t = t0 + tl;
  const bool valid = t < T;
  const int q3r = slot >> 2, q3c = slot & 3;
  const float* win = wbuf + tl * WS;
  const float* w00 = win + 4 * bt_tap0(q3r) * L3 + 4 * bt_tap0(q3c);
  const float* w01 = win + 4 * bt_tap0(q3r) * L3 + 4 * bt_tap1(q3c);
  const float* w10 = win + 4 * bt_tap1(q3r) * L3 + 4 * bt_tap0(q3c);
  const float* w11 = win + 4 * bt_tap1(q3r) * L3 + 4 * bt_tap1(q3c);
  const float cc = bt_sign0(q3c) * bt_sign1(q3c);
  const float rr = bt_sign0(q3r) * bt_sign1(q3r);
  const float ksign = bt_sign0(q3c) * bt_sign0(q3r);
  const int branch = q4 * 16 + slot;              // 256-point block
  // U quad (p/4, m, n) sits at float4 index (p/4) M N + m N + n; the
  // branch's 64 quads start at branch * 64 M N (a per-lane offset, < 2^31
  // by the launch check), the rest is uniform
  const unsigned qsU = (unsigned)(DW ? N : M * N); // float4 quads between U quads
  const unsigned ulane = (unsigned)branch * 64u * qsU;
  const int ch = DW ? (int)blockIdx.y : 0;

  float acc[NC][4][4][4];                         // [n][q2r][q2c][2 i1r + i1c]
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int d = 0; d < 4; ++d) acc[c][a][b][d] = 0.0f;

  const int m_begin = DW ? ch : wave, m_end = DW ? ch + 1 : M;
  for (int m = m_begin; m < m_end; m += CS) {
    // fill: this wavefront's 4 windows of channel m (after the level-4 rows)
    const float* __restrict__ xm = x + (size_t)m * H * W;
#pragma unroll
    for (int k = 0; k < NTASK; ++k) {
      if (!f_ok[k]) continue;
      const int img = f_img[k];
      float* dst = wbuf + f_dst[k];
      // opaque per channel: keeps the 22 clamped row offsets and masks from
      // being hoisted out of the channel loop (they would hold ~90 registers)
      int gr0 = f_gr0[k];
      asm volatile("" : "+v"(gr0));
      if (NLEV == 4) {
        constexpr int RB = 11;   // rows per batch: 4 RB loads in flight
#pragma unroll
        for (int r0 = 0; r0 < L3; r0 += RB) {
          float va[RB], vb[RB], vc[RB], vd[RB];
#pragma unroll
          for (int i = 0; i < RB; ++i) {
            const int ra = gr0 + r0 + i + a4r0, rb = gr0 + r0 + i + a4r1;
            const int rac = ra < 0 ? 0 : (ra > H - 1 ? H - 1 : ra);
            const int rbc = rb < 0 ? 0 : (rb > H - 1 ? H - 1 : rb);
            // uniform channel base plus a 32-bit per-lane offset
            va[i] = xm[img + rac * W + f_ca[k]];
            vb[i] = xm[img + rac * W + f_cb[k]];
            vc[i] = xm[img + rbc * W + f_ca[k]];
            vd[i] = xm[img + rbc * W + f_cb[k]];
          }
#pragma unroll
          for (int i = 0; i < RB; ++i) {
            const int ra = gr0 + r0 + i + a4r0, rb = gr0 + r0 + i + a4r1;
            const float mra = (ra >= 0 && ra < H) ? s4r0 : 0.0f;
            const float mrb = (rb >= 0 && rb < H) ? s4r1 : 0.0f;
            dst[(r0 + i) * L3] = mra * (f_ma[k] * va[i] + f_mb[k] * vb[i]) +
                                 mrb * (f_ma[k] * vc[i] + f_mb[k] * vd[i]);
          }
        }
      } else {
        float va[L3];
#pragma unroll
        for (int i = 0; i < L3; ++i) {
          const int gr = gr0 + i;
          va[i] = xm[img + (gr < 0 ? 0 : (gr > H - 1 ? H - 1 : gr)) * W + f_ca[k]];
        }
#pragma unroll
        for (int i = 0; i < L3; ++i) {
          const int gr = gr0 + i;
          dst[i * L3] = (gr >= 0 && gr < H) ? f_ma[k] * va[i] : 0.0f;
        }
      }
    }
    wave_sync();
    if (valid) {
      // opaque per channel, so the 64 uniform quad offsets are recomputed
      // (scalar ALU) instead of being held across the loop
      unsigned qs = qsU;
      asm volatile("" : "+s"(qs));
      const float4* __restrict__ Um = U + (DW ? (size_t)ch : (size_t)m * N);
      // Two passes over column halves: pass hc produces the level-2 column
      // digits q2c = 2 hc, 2 hc + 1, which read sub-window columns
      // [2 hc, 2 hc + 8) only; the halves share rows 2..9, recomputed.
#pragma unroll
      for (int hc = 0; hc < 2; ++hc) {
        const int c0 = 2 * hc;
        // keeps the second pass from reusing the first pass's window reads
        // (which would keep all 10 x 10 values live)
        asm volatile("" ::: "memory");
        // level 3 (stride 4) in both directions, up to the sign ksign
        float S[10][8];
#pragma unroll
        for (int i = 0; i < 10; ++i)
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
            const int o = i * L3 + c0 + jj;
            S[i][jj] = fmaf(rr, fmaf(cc, w11[o], w10[o]), fmaf(cc, w01[o], w00[o]));
          }
#pragma unroll
        for (int q2r = 0; q2r < 4; ++q2r) {
          // this block's 8 U quads per output channel, issued together
          float4 uq[4][2][NC];
#pragma unroll
          for (int q1r = 0; q1r < 4; ++q1r)
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
              for (int c = 0; c < NC; ++c)
                uq[q1r][h][c] =
                    (Um + (size_t)((q2r * 16 + (c0 + h) * 4 + q1r) * qs + c))[ulane];
          asm volatile("" ::: "memory");
          // level 2 along the rows (stride 2)
          float Zr[4][8];
          const int a0 = 2 * bt_tap0(q2r), a1 = 2 * bt_tap1(q2r);
          const float s0 = bt_sign0(q2r), s1 = bt_sign1(q2r);
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) Zr[u][jj] = s0 * S[u + a0][jj] + s1 * S[u + a1][jj];
#pragma unroll
          for (int q1r = 0; q1r < 4; ++q1r) {
            // level 1 along the rows
            float R[8];
            const int b0 = bt_tap0(q1r), b1 = bt_tap1(q1r);
            const float t0s = bt_sign0(q1r), t1s = bt_sign1(q1r);
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) R[jj] = t0s * Zr[b0][jj] + t1s * Zr[b1][jj];
            const float e0 = at_coef(0, q1r), e1 = at_coef(1, q1r);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              // levels 2 and 1 along the columns
              const int q2c = c0 + h;
              const int d0 = 2 * bt_tap0(q2c) - c0, d1 = 2 * bt_tap1(q2c) - c0;
              const float g0 = bt_sign0(q2c), g1 = bt_sign1(q2c);
              float zc[4], o[4];
#pragma unroll
              for (int u = 0; u < 4; ++u) zc[u] = g0 * R[u + d0] + g1 * R[u + d1];
              bt_one(zc, o);  // index q1c
#pragma unroll
              for (int c = 0; c < NC; ++c) {
                const float4 u = uq[q1r][h][c];
                const float p0 = o[0] * u.x, p1 = o[1] * u.y, p2 = o[2] * u.z, p3 = o[3] * u.w;
                // level-1 A^T along the columns, then along the rows
                const float z0 = p0 + p1 + p2, z1 = p1 - p2 - p3;
                acc[c][q2r][q2c][0] += e0 * z0;
                acc[c][q2r][q2c][1] += e0 * z1;
                acc[c][q2r][q2c][2] += e1 * z0;
                acc[c][q2r][q2c][3] += e1 * z1;
              }
            }
          }
        }
      }
    }
    wave_sync();   // the next channel's fill overwrites the windows
  }

  if (CS > 1) {
    // add the other wavefronts' partial sums into wavefront 0, 16 values per pass
    float* red = lds;
    __syncthreads();
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        if (wave > 0) {
#pragma unroll
          for (int v = 0; v < 16; ++v) red[((wave - 1) * 16 + v) * 64 + lane] = acc[c][a][v >> 2][v & 3];
        }
        __syncthreads();
        if (wave == 0) {
#pragma unroll
          for (int w = 1; w < CS; ++w)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[c][a][v >> 2][v & 3] += red[((w - 1) * 16 + v) * 64 + lane];
        }
        __syncthreads();
      }
  }
  if (wave != 0 || !valid) return;
  // Z[g][n][t], g = branch * 16 + q2r * 4 + q2c
  const size_t gstride = (size_t)N * T;
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int q2r = 0; q2r < 4; ++q2r)
#pragma unroll
      for (int q2c = 0; q2c < 4; ++q2c) {
        const size_t g = (size_t)branch * 16 + q2r * 4 + q2c;
        const float* a = acc[c][q2r][q2c];
        Z[g * gstride + (size_t)(DW ? ch : c) * T + t] =
            make_float4(ksign * a[0], ksign * a[1], ksign * a[2], ksign * a[3]);
      }
}

template <int NLEV, int NC>
hipError_t launch_ics(const nwg_plan_info& g, const float* x, const float4* U, float4* Z,
                      unsigned nwg, int cs, hipStream_t s) {
  const int T = (int)g.T;
  if (cs == 4)
    hipLaunchKernelGGL((input_contract_small<NLEV, NC, 4, false>), dim3(nwg), dim3(256), 0, s, x,
                       U, Z, g.M, g.N, g.H, g.W, g.pad, g.th, g.tw, T);
  else if (cs == 2)
    hipLaunchKernelGGL((input_contract_small<NLEV, NC, 2, false>), dim3(nwg), dim3(128), 0, s, x,
                       U, Z, g.M, g.N, g.H, g.W, g.pad, g.th, g.tw, T);
  else
    hipLaunchKernelGGL((input_contract_small<NLEV, NC, 1, false>), dim3(nwg), dim3(64), 0, s, x,
                       U, Z, g.M, g.N, g.H, g.W, g.pad, g.th, g.tw, T);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_input_contract(const nwg_plan_info& g, const float* x, const float* Uf,
                                 float* Zf, hipStream_t s) {
  if (!input_contract_applies(g)) return hipErrorInvalidValue;
  if (((uintptr_t)Uf | (uintptr_t)Zf) & 15) return hipErrorInvalidValue;
  const long long chunks = (g.T + kTilesPerWave - 1) / kTilesPerWave;
  const long long nwg = chunks * (g.n == 4 ? 16 : 1);
  if (nwg > 0x7fffffffLL) return hipErrorInvalidValue;
  const long long uquads = (long long)g.P / 4 * (g.depthwise ? 1 : g.M) * g.N;
  if (uquads > 0x7fffffffLL) return hipErrorInvalidValue;
  if ((long long)g.B * g.M * g.H * g.W > 0x7fffffffLL) return hipErrorInvalidValue;
  const float4* U = reinterpret_cast<const float4*>(Uf);
  float4* Z = reinterpret_cast<float4*>(Zf);
  const int T = (int)g.T;
  if (g.depthwise) {
    if (g.N > 65535) return hipErrorInvalidValue;
    dim3 grid((unsigned)nwg, (unsigned)g.N);
    if (g.n == 3)
      hipLaunchKernelGGL((input_contract_small<3, 1, 1, true>), grid, dim3(64), 0, s, x, U, Z,
                         g.M, g.N, g.H, g.W, g.pad, g.th, g.tw, T);
    else
      hipLaunchKernelGGL((input_contract_small<4, 1, 1, true>), grid, dim3(64), 0, s, x, U, Z,
                         g.M, g.N, g.H, g.W, g.pad, g.th, g.tw, T);
    return hipGetLastError();
  }
  // channel split: enough wavefronts for two per SIMD (1024 SIMDs), at
  // least one channel per wavefront
  int cs = 1;
  while (cs < 4 && nwg * cs < 2048 && 2 * cs <= g.M) cs *= 2;
  if (g.n == 3)
    return g.N == 1 ? launch_ics<3, 1>(g, x, U, Z, (unsigned)nwg, cs, s)
                    : launch_ics<3, 2>(g, x, U, Z, (unsigned)nwg, cs, s);
  return g.N == 1 ? launch_ics<4, 1>(g, x, U, Z, (unsigned)nwg, cs, s)
                  : launch_ics<4, 2>(g, x, U, Z, (unsigned)nwg, cs, s);
}

}  // namespace nwg
