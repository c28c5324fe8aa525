// Nested input transformation (Sec. III.B, first step; 2D per Fig. 4 text).
//
// For every tile t and input channel m, the L_n x L_n input window starting
// at (ty*M_n - pad, tx*M_n - pad) (zero outside the image) is reordered into
// the 2n-dim tensor D[a;b] = x[sum_j s_{j-1} a_j][sum_j s_{j-1} b_j] and
// transformed by B^T of F(2,3) along every axis, giving the P = 4^(2n)
// values V[p][m][t].
//
// Level by level, outermost first: a B^T row at stride s combines two
// windows shifted by s * tap, so the outer levels turn the window into
// independent sub-windows ("branches"), and the two innermost levels
// (10 -> 16 per axis) run in registers.
//
//   depth 1      : one thread per tile; the work-group stages the union of
//                  its tiles' windows (a box of whole-row tile runs) in LDS.
//   depth 2      : the same box staging for 16 tiles, with 16 threads per
//                  tile (one per row of the two-level transform).
//   depth n >= 3 : one thread per (tile, level-3 branch); the work-group
//                  stages each of its 16 tiles' windows separately in LDS
//                  (odd window stride, so that the 16 tiles of a
//                  quarter-wave read 16 different banks).  At depth 4 the
//                  work-group also owns one level-4 branch (q4r, q4c): the
//                  fill already applies those B^T rows along both axes of
//                  the 46 x 46 window (-> 22 x 22).  A branch's 10 x 10
//                  sub-window is then a signed sum of 2 x 2 level-3 shifted
//                  window reads at compile-time offsets.
//
// V is quad-interleaved, V[p/4][m][t][p%4] (p%4 is the level-1 column digit
// q1c): every thread stores float4 quads, and the consecutive tiles of a
// quarter-wave write 256 contiguous bytes.
#include "nwg_internal.h"

namespace nwg {
namespace {

// ---- depth 1: union box of tiles in LDS, one thread per tile ----------------
template <int NLEV, bool SPLIT>
__global__ __launch_bounds__(256) void input_xform_box(
    const float* __restrict__ x, float4* __restrict__ V, int M, int H, int W, int pad, int th,
    int tw, int T, long long qstride, int RX, int RY, int nbx, int nby, int ldc) {
  constexpr int Mn = 1 << NLEV;
  constexpr int Ln = 3 * Mn - 2;
  extern __shared__ float lds[];
  // V channel mv; in a linear-decomposition plan (ldc > 0) it is
  // (sub-kernel (cu, cv), input channel m), mv = (cu ldc + cv) M + m, and the
  // window moves by (3 cu, 3 cv)
  const int mv = blockIdx.y;
  int m = mv, sr = 0, sc = 0;
  if (ldc > 0) {
    m = mv % M;
    const int sub = mv / M;
    sr = 3 * (sub / ldc);
    sc = 3 * (sub % ldc);
  }
  int bid = blockIdx.x;
  const int bx = bid % nbx;
  bid /= nbx;
  const int by = bid % nby;
  const int b = bid / nby;
  const int ty0 = by * RY, tx0 = bx * RX;
  const int BH = (RY - 1) * Mn + Ln, BW = (RX - 1) * Mn + Ln;
  const int r0 = ty0 * Mn - pad + sr, c0 = tx0 * Mn - pad + sc;
  const float* __restrict__ xp = x + ((size_t)b * M + m) * H * W;
  const int nth = blockDim.x;
  for (int e = threadIdx.x; e < BH * BW; e += nth) {
    const int row = e / BW, col = e - row * BW;
    const int gr = r0 + row, gc = c0 + col;
    float v = 0.0f;
    if (gr >= 0 && gr < H && gc >= 0 && gc < W) v = xp[(size_t)gr * W + gc];
    lds[e] = v;
  }
  __syncthreads();
  const int s = threadIdx.x;
  if (s >= RX * RY) return;
  const int ly = s / RX, lx = s - ly * RX;
  const int ty = ty0 + ly, tx = tx0 + lx;
  if (ty >= th || tx >= tw) return;
  const int t = (b * th + ty) * tw + tx;
  const float* win = lds + ly * Mn * BW + lx * Mn;
  float4* vb = V + (size_t)mv * T + t;
  static_assert(NLEV == 1, "the box kernel serves depth 1");
  {
    float X[4][4], Rw[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float row[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) row[j] = win[i * BW + j];
      float o[4];
      bt_one(row, o);                    // along the row: index q1c
#pragma unroll
      for (int j = 0; j < 4; ++j) X[i][j] = o[j];
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float col[4] = {X[0][c], X[1][c], X[2][c], X[3][c]};
      float o[4];
      bt_one(col, o);                    // along the column: index q1r
#pragma unroll
      for (int q = 0; q < 4; ++q) Rw[q][c] = o[q];
    }
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r)
      vb[(size_t)q1r * qstride] = store_quad<SPLIT>(Rw[q1r][0], Rw[q1r][1], Rw[q1r][2], Rw[q1r][3]);
  }
}

// ---- depth 2: 16 tiles per work-group, 16 threads per tile -----------------
// Thread (tile, rho = (q2r, q1r)) applies that row of the two-level B^T to
// the tile's 10 x 10 window (4 window rows per output row) and the two
// levels along the columns to the result, storing 4 quads.  The work-group's
// 16 tiles form a box of RX x RY tiles whose windows are staged in LDS.
template <bool SPLIT>
__global__ __launch_bounds__(256) void input_xform_d2(
    const float* __restrict__ x, float4* __restrict__ V, int M, int H, int W, int pad, int th,
    int tw, int T, long long qstride, int RX, int RY, int nbx, int nby) {
  constexpr int Mn = 4, Ln = 10;
  extern __shared__ float lds[];
  const int m = blockIdx.y;
  int bid = blockIdx.x;
  const int bx = bid % nbx;
  bid /= nbx;
  const int by = bid % nby;
  const int b = bid / nby;
  const int ty0 = by * RY, tx0 = bx * RX;
  const int BH = (RY - 1) * Mn + Ln, BW = (RX - 1) * Mn + Ln;
  const int r0 = ty0 * Mn - pad, c0 = tx0 * Mn - pad;
  const float* __restrict__ xp = x + ((size_t)b * M + m) * H * W;
  for (int e = threadIdx.x; e < BH * BW; e += 256) {
    const int row = e / BW, col = e - row * BW;
    const int gr = r0 + row, gc = c0 + col;
    float v = 0.0f;
    if (gr >= 0 && gr < H && gc >= 0 && gc < W) v = xp[(size_t)gr * W + gc];
    lds[e] = v;
  }
  __syncthreads();
  const int s = threadIdx.x & 15, rho = threadIdx.x >> 4;
  if (s >= RX * RY) return;
  const int ly = s / RX, lx = s - ly * RX;
  const int ty = ty0 + ly, tx = tx0 + lx;
  if (ty >= th || tx >= tw) return;
  const int t = (b * th + ty) * tw + tx;
  const float* win = lds + ly * Mn * BW + lx * Mn;
  const int q2r = rho >> 2, q1r = rho & 3;
  // row rho of the two-level B^T: taps 2 a2 + a1 with sign s2 * s1
  const int a20 = 2 * bt_tap0(q2r), a21 = 2 * bt_tap1(q2r);
  const int a10 = bt_tap0(q1r), a11 = bt_tap1(q1r);
  const float s20 = bt_sign0(q2r), s21 = bt_sign1(q2r), s10 = bt_sign0(q1r), s11 = bt_sign1(q1r);
  float R[10];
#pragma unroll
  for (int j = 0; j < 10; ++j)
    R[j] = s20 * (s10 * win[(a20 + a10) * BW + j] + s11 * win[(a20 + a11) * BW + j]) +
           s21 * (s10 * win[(a21 + a10) * BW + j] + s11 * win[(a21 + a11) * BW + j]);
  float o[16];
  bt_inner2(R, o);  // columns: index q2c*4 + q1c
  float4* vb = V + (size_t)m * T + t;
#pragma unroll
  for (int q2c = 0; q2c < 4; ++q2c) {
    const int quad = q2r * 16 + q2c * 4 + q1r;
    vb[(size_t)quad * qstride] =
        store_quad<SPLIT>(o[q2c * 4 + 0], o[q2c * 4 + 1], o[q2c * 4 + 2], o[q2c * 4 + 3]);
  }
}

// ---- depth 3 and 4: 16 tiles per work-group, per-tile windows in LDS -------
template <int NLEV, bool SPLIT>
__global__ __launch_bounds__(256) void input_xform_tiles(
    const float* __restrict__ x, float4* __restrict__ V, int M, int H, int W, int pad, int th,
    int tw, int T, long long qstride, int q4_0, int nq4, unsigned long long live) {
  constexpr int Mn = 1 << NLEV;
  constexpr int L3 = 22;                     // window side left for levels 1..3
  constexpr int WS = L3 * L3 + 1;            // odd window stride: 16 tiles -> 16 banks
  extern __shared__ float lds[];
  // Work-group -> (level-4 branch q4, 16-tile chunk, channel m), q4 fastest.
  // The dispatcher deals work-groups round-robin over the 8 XCDs; this
  // numbering gives each XCD a contiguous range, so the 16 branches that
  // re-read the same input windows run back to back on one XCD and find
  // them in its L2.
  long long lid;
  {
    const long long G = (long long)gridDim.x, i = blockIdx.x;
    const long long q = G / 8, rem = G % 8, xcd = i % 8, sl = i / 8;
    lid = xcd < rem ? xcd * (q + 1) + sl : rem * (q + 1) + (xcd - rem) * q + sl;
  }
  // level-4 branch (q4r, q4c) in [q4_0, q4_0 + nq4), else 0
  const int q4 = NLEV == 4 ? q4_0 + (int)(lid % nq4) : 0;
  const long long rest = NLEV == 4 ? lid / nq4 : lid;
  const int nchunk = (T + 15) / 16;
  const int t0 = (int)(rest % nchunk) * 16;
  const int m = (int)(rest / nchunk);
  const int q4r = q4 >> 2, q4c = q4 & 3;
  const int tpi = th * tw;
  // fill: per tile, the 22 x 22 window after the level-4 B^T rows q4r (along
  // the rows) and q4c (along the columns) at depth 4, the window itself at 3
  const int a4r0 = 8 * bt_tap0(q4r), a4r1 = 8 * bt_tap1(q4r);
  const int a4c0 = 8 * bt_tap0(q4c), a4c1 = 8 * bt_tap1(q4c);
  const float s4r0 = bt_sign0(q4r), s4r1 = bt_sign1(q4r);
  const float s4c0 = bt_sign0(q4c), s4c1 = bt_sign1(q4c);
  // 16 threads per tile: thread (ftl, fj) fills columns fj and fj + 16 of
  // tile ftl's window, walking its 22 rows with independent loads
  {
    const int ftl = threadIdx.x >> 4, fj = threadIdx.x & 15;
    const int t = t0 + ftl;
    if (t < T) {
      const int b = t / tpi;
      const int r2 = t - b * tpi;
      const int ty = r2 / tw, tx = r2 - ty * tw;
      const float* __restrict__ xp = x + ((size_t)b * M + m) * H * W;
      const int gr0 = ty * Mn - pad, gc0 = tx * Mn - pad;
      float* dst = lds + ftl * WS;
      // Loads are unconditional, from addresses clamped into the image, and
      // masked afterwards: no branches, so a whole column of loads can be in
      // flight at once.
      auto clampi = [](int v, int hi) { return v < 0 ? 0 : (v > hi ? hi : v); };
#pragma unroll
      for (int c = fj; c < L3; c += 16) {
        const int gc = gc0 + c;
        if (NLEV == 4) {
          const int ca = gc + a4c0, cb = gc + a4c1;
          const float mca = (ca >= 0 && ca < W) ? s4c0 : 0.0f;
          const float mcb = (cb >= 0 && cb < W) ? s4c1 : 0.0f;
          const int cac = clampi(ca, W - 1), cbc = clampi(cb, W - 1);
          constexpr int RB = 11;   // rows per batch: 4*RB loads in flight
#pragma unroll
          for (int r0 = 0; r0 < L3; r0 += RB) {
            float va[RB], vb[RB], vc[RB], vd[RB];
#pragma unroll
            for (int k = 0; k < RB; ++k) {
              const int row = r0 + k;
              const int rac = clampi(gr0 + row + a4r0, H - 1), rbc = clampi(gr0 + row + a4r1, H - 1);
              va[k] = xp[(size_t)rac * W + cac];
              vb[k] = xp[(size_t)rac * W + cbc];
              vc[k] = xp[(size_t)rbc * W + cac];
              vd[k] = xp[(size_t)rbc * W + cbc];
            }
#pragma unroll
            for (int k = 0; k < RB; ++k) {
              const int row = r0 + k;
              const int ra = gr0 + row + a4r0, rb = gr0 + row + a4r1;
              const float mra = (ra >= 0 && ra < H) ? s4r0 : 0.0f;
              const float mrb = (rb >= 0 && rb < H) ? s4r1 : 0.0f;
              dst[row * L3 + c] = mra * (mca * va[k] + mcb * vb[k]) +
                                  mrb * (mca * vc[k] + mcb * vd[k]);
            }
          }
        } else {
          const float mc = (gc >= 0 && gc < W) ? 1.0f : 0.0f;
          const int gcc = clampi(gc, W - 1);
          float va[L3];
#pragma unroll
          for (int row = 0; row < L3; ++row) va[row] = xp[(size_t)clampi(gr0 + row, H - 1) * W + gcc];
#pragma unroll
          for (int row = 0; row < L3; ++row) {
            const int gr = gr0 + row;
            dst[row * L3 + c] = (gr >= 0 && gr < H) ? mc * va[row] : 0.0f;
          }
        }
      }
    }
  }
  __syncthreads();
  const int tl = threadIdx.x & 15;
  const int slot = threadIdx.x >> 4;        // level-3 branch (q3r, q3c)
  const int t = t0 + tl;
  if (t >= T) return;                       // no barrier below
  const int q3r = slot >> 2, q3c = slot & 3;
  const float* win = lds + tl * WS;
  // level 3 (stride 4): two row taps and two column taps
  const int ro0 = 4 * bt_tap0(q3r), ro1 = 4 * bt_tap1(q3r);
  const int co0 = 4 * bt_tap0(q3c), co1 = 4 * bt_tap1(q3c);
  const float rs0 = bt_sign0(q3r), rs1 = bt_sign1(q3r);
  const float cs0 = bt_sign0(q3c), cs1 = bt_sign1(q3c);
  const float* w00 = win + ro0 * L3 + co0;
  const float* w01 = win + ro0 * L3 + co1;
  const float* w10 = win + ro1 * L3 + co0;
  const float* w11 = win + ro1 * L3 + co1;
  float S[10][10];
#pragma unroll
  for (int i = 0; i < 10; ++i)
#pragma unroll
    for (int j = 0; j < 10; ++j) {
      const float a = cs0 * w00[i * L3 + j] + cs1 * w01[i * L3 + j];
      const float c = cs0 * w10[i * L3 + j] + cs1 * w11[i * L3 + j];
      S[i][j] = rs0 * a + rs1 * c;
    }
  // 256-point block of this branch: (q4r, q4c, q3r, q3c) at depth 4, (q3r, q3c) at depth 3
  const int branch = q4 * 16 + slot;
  if (live == 0) {
    inner2_store<SPLIT>(S, V + (size_t)branch * 64 * qstride + (size_t)m * T + t, (size_t)qstride);
    return;
  }
  // only the live groups (q2r, q2c) of the branch are written (the groups
  // no tap reaches are never read): one buffer resource over the wave's
  // four branches, (q3r, q3c = 0..3), dead quads' lanes sent past its range
  const int wv = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const unsigned g16 = nibble_live(prefix_nibble(live, 0, NLEV == 4 ? 4 * q4r + q3r : q3r),
                                   prefix_nibble(live, 0, NLEV == 4 ? 4 * q4c + q3c : q3c));
  const __amdgpu_buffer_rsrc_t rs =
      span_rsrc(V + (size_t)(q4 * 16 + 4 * wv) * 64 * qstride, (unsigned)(256 * qstride * 16));
  const unsigned lane0 = (unsigned)((((size_t)(slot & 3) * 64) * qstride + (size_t)m * T + t) * 16);
  const unsigned qs = (unsigned)(qstride * 16);
  inner2_xform<SPLIT>(S, [&](int quad, float4 v) {
    const int grp = (quad >> 4) * 4 + ((quad >> 2) & 3);      // 4 q2r + q2c
    drop_store(rs, ((g16 >> grp) & 1u) ? lane0 + (unsigned)quad * qs : kDrop, v);
  });
}

}  // namespace

hipError_t launch_input_xform(const nwg_plan_info& g, const float* x, float* Vf, hipStream_t s,
                              int part, int nparts) {
  float4* V = reinterpret_cast<float4*>(Vf);
  if ((uintptr_t)Vf & 15) return hipErrorInvalidValue;
  // split precision: every quad holds the four values' bf16 (hi, lo) pairs
  const bool split = g.precision == NWG_PRECISION_BF16_SPLIT;
  // V channels: M, or M c^2 for a linear-decomposition plan (c = ld_c)
  const long long mv = (long long)g.M * (g.ld_c > 0 ? g.ld_c * g.ld_c : 1);
  const long long qstride = mv * g.T;   // float4 quads between consecutive quads
  const int T = (int)g.T;
  if (g.n >= 3) {
    const size_t lds = (size_t)16 * (22 * 22 + 1) * sizeof(float);
    // depth 4: part k of nparts covers level-4 branches [16k/nparts, 16(k+1)/nparts)
    int q4_0 = 0, nq4 = 1;
    if (g.n == 4) {
      if (nparts < 1 || 16 % nparts || part < 0 || part >= nparts) return hipErrorInvalidValue;
      nq4 = 16 / nparts;
      q4_0 = part * nq4;
    } else if (nparts != 1) {
      return hipErrorInvalidValue;
    }
    const long long nwg = (g.T + 15) / 16 * g.M * nq4;
    if (nwg > 0x7fffffffLL) return hipErrorInvalidValue;
    dim3 grid((unsigned)nwg);
    // dense F(2,3) chains write the live groups only, when a wave's four
    // branches (256 quads of M T float4) span at most 2^30 bytes
    const unsigned long long live =
        g.tile == NWG_TILE_F2X2_3X3 && g.live_np > 0 && g.ld_c == 0 &&
                256.0 * (double)qstride * 16.0 <= (double)(1u << 30)
            ? g.live_prefix[0]
            : 0ull;
#define NWG_TILES(L, SP)                                                                       \
  hipLaunchKernelGGL((input_xform_tiles<L, SP>), grid, dim3(256), lds, s, x, V, g.M, g.H, g.W,  \
                     g.pad, g.th, g.tw, T, qstride, q4_0, nq4, live)
    if (g.n == 3) {
      if (split) NWG_TILES(3, true); else NWG_TILES(3, false);
    } else {
      if (split) NWG_TILES(4, true); else NWG_TILES(4, false);
    }
#undef NWG_TILES
  } else if (g.n == 2) {
    if (nparts != 1) return hipErrorInvalidValue;
    const int Mn = 4, Ln = 10;
    const int RX = g.tw < 16 ? g.tw : 16;
    int RY = 16 / RX;
    if (RY > g.th) RY = g.th;
    const int nbx = (g.tw + RX - 1) / RX, nby = (g.th + RY - 1) / RY;
    const size_t lds = (size_t)((RY - 1) * Mn + Ln) * ((RX - 1) * Mn + Ln) * sizeof(float);
    dim3 grid((unsigned)(nbx * nby * g.B), (unsigned)g.M);
    if (split)
      hipLaunchKernelGGL(input_xform_d2<true>, grid, dim3(256), lds, s, x, V, g.M, g.H, g.W,
                         g.pad, g.th, g.tw, T, qstride, RX, RY, nbx, nby);
    else
      hipLaunchKernelGGL(input_xform_d2<false>, grid, dim3(256), lds, s, x, V, g.M, g.H, g.W,
                         g.pad, g.th, g.tw, T, qstride, RX, RY, nbx, nby);
  } else {
    if (nparts != 1 || mv > 65535) return hipErrorInvalidValue;
    const int Mn = 1 << g.n, Ln = 3 * Mn - 2;
    // tiles per work-group: 256, or 64 when that leaves too few work-groups
    int tpb = 256;
    for (int pass = 0; pass < 2; ++pass) {
      const int RX = g.tw < tpb ? g.tw : tpb;
      int RY = tpb / RX;
      if (RY > g.th) RY = g.th;
      const long long nwg = (long long)((g.tw + RX - 1) / RX) * ((g.th + RY - 1) / RY) * g.B * mv;
      if (nwg >= 1024 || tpb == 64) break;
      tpb = 64;
    }
    const int RX = g.tw < tpb ? g.tw : tpb;
    int RY = tpb / RX;
    if (RY > g.th) RY = g.th;
    const int nbx = (g.tw + RX - 1) / RX, nby = (g.th + RY - 1) / RY;
    const size_t lds = (size_t)((RY - 1) * Mn + Ln) * ((RX - 1) * Mn + Ln) * sizeof(float);
    dim3 grid((unsigned)(nbx * nby * g.B), (unsigned)mv);
    if (split)
      hipLaunchKernelGGL((input_xform_box<1, true>), grid, dim3(tpb), lds, s, x, V, g.M, g.H, g.W,
                         g.pad, g.th, g.tw, T, qstride, RX, RY, nbx, nby, g.ld_c);
    else
      hipLaunchKernelGGL((input_xform_box<1, false>), grid, dim3(tpb), lds, s, x, V, g.M, g.H,
                         g.W, g.pad, g.th, g.tw, T, qstride, RX, RY, nbx, nby, g.ld_c);
  }
  return hipGetLastError();
}

}  // namespace nwg
