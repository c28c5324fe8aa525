// Nested Winograd on the base F(3,3) (Sec. III.B with m = r = 3, l = 5),
// depth 1 or 2 (kernels up to 9 x 9): the level recurrence gives strides
// 1, 3, M_n = K_n = 3^n, L_n = 5 at depth 1 and 17 at depth 2, and
// P = 5^(2n) = 25 or 625 points per tile.  Sec. V.A names F(3,3) among the
// bases of its comparison; at depth <= 2 its fp32 error stays near 1e-6.
//
// Base matrices from the Toom-Cook construction with interpolation points
// 0, 1, -1, 2 and infinity (correlation form y = A^T[(G w) (.) (B^T x)]):
//   G (5x3):  [1,0,0] [1,1,1] [1,-1,1] [1,2,4] [0,0,1]
//   A^T (3x5): [1,1,1,1,0] [0,1,-1,2,0] [0,1,1,4,1]
//   B^T (5x5) = (Vandermonde of the points)^-T:
//     [1,-1/2,-1,1/2,0] [0,1,1/2,-1/2,0] [0,-1/3,1/2,-1/6,0] [0,-1/6,0,1/6,0] [0,2,-1,-2,1]
// (the inverse of the Vandermonde map f = V c of a degree-4 polynomial
// sampled at 0, 1, -1, 2 with its leading coefficient, solved by hand).
//
// Layouts (plain fp32; p has base-5 digits (q2r, q2c, q1r, q1c), most
// significant first, the level-2 digits absent at depth 1):
//   U [P][M][N], V [P][M][T],
//   Z [P/25][5][3][N][T]: the contraction applies the level-1 A^T along the
//       columns, Z[g][q1r][i1c][n][t] = sum_q1c A^T[i1c][q1c] Yhat[25 g + 5 q1r + q1c][n][t].
// Consecutive lanes take consecutive tiles (or output channels), so every
// store and load of a wavefront covers 256 contiguous bytes.
#include "nwg_internal.h"

namespace nwg {
namespace {

constexpr int L5 = 5;

// ---- kernel transform: one thread per (n, m) --------------------------------
// w (r x r, zero-padded to K_n x K_n at its end) -> U[p][m][n].  Tap k splits
// as k = k1 + 3 k2 (k1, k2 < 3).  For every pair of row digits (q2r, q1r)
// the weighted rows give a length-K_n row wr, transformed along the columns.
template <int NLEV>
__global__ __launch_bounds__(256) void kernel_xform5(const float* __restrict__ w,
                                                     float* __restrict__ U, int M, int N, int r,
                                                     long long nthreads) {
  constexpr int K = NLEV == 1 ? 3 : 9;
  const long long id = (long long)blockIdx.x * 256 + threadIdx.x;
  if (id >= nthreads) return;
  const int n = (int)(id % N), m = (int)(id / N);
  const float* __restrict__ wp = w + ((size_t)n * M + m) * r * r;
  float wk[K][K];
#pragma unroll
  for (int i = 0; i < K; ++i)
#pragma unroll
    for (int j = 0; j < K; ++j) wk[i][j] = (i < r && j < r) ? wp[i * r + j] : 0.0f;
  const size_t pstride = (size_t)M * N;
  float* __restrict__ up = U + (size_t)m * N + n;
  constexpr int R1 = NLEV == 1 ? 1 : 5;     // level-2 digits per axis
#pragma unroll
  for (int q2r = 0; q2r < R1; ++q2r)
#pragma unroll
    for (int q1r = 0; q1r < 5; ++q1r) {
      // row combination: coefficient of kernel row k1 + 3 k2
      float wr[K];
#pragma unroll
      for (int j = 0; j < K; ++j) {
        float s = 0.0f;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const float c = NLEV == 1 ? g5(q1r, k) : g5(q2r, k / 3) * g5(q1r, k % 3);
          s = fmaf(c, wk[k][j], s);
        }
        wr[j] = s;
      }
#pragma unroll
      for (int q2c = 0; q2c < R1; ++q2c)
#pragma unroll
        for (int q1c = 0; q1c < 5; ++q1c) {
          float s = 0.0f;
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const float c = NLEV == 1 ? g5(q1c, k) : g5(q2c, k / 3) * g5(q1c, k % 3);
            s = fmaf(c, wr[k], s);
          }
          const int p = NLEV == 1 ? q1r * 5 + q1c : ((q2r * 5 + q2c) * 5 + q1r) * 5 + q1c;
          up[(size_t)p * pstride] = s;
        }
    }
}

// ---- input transform --------------------------------------------------------
// Work-group: a box of RX x RY tiles of one (image, channel) staged in LDS;
// depth 1: one thread per tile; depth 2: wavefront q2r (5 wavefronts) of 64
// tiles, each lane computing the 125 points of its level-2 row digit.
template <int NLEV>
__global__ __launch_bounds__(320) void input_xform5(const float* __restrict__ x,
                                                    float* __restrict__ V, int M, int H, int W,
                                                    int pad, int th, int tw, int T, int RX, int RY,
                                                    int nbx, int nby) {
  constexpr int Mn = NLEV == 1 ? 3 : 9;
  constexpr int Ln = NLEV == 1 ? 5 : 17;
  extern __shared__ float box[];
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
  const int nth = blockDim.x;
  const int nbox = BH * BW;
  // batches of FB loads per thread, all issued before the first LDS store,
  // so that the fill waits for memory once per batch, not once per element
  constexpr int FB = 8;
  for (int e0 = threadIdx.x; e0 < nbox; e0 += FB * nth) {
    float v[FB];
#pragma unroll
    for (int u = 0; u < FB; ++u) {
      const int e = e0 + u * nth;
      const int row = e / BW, col = e - row * BW;
      const int gr = r0 + row, gc = c0 + col;
      v[u] = 0.0f;
      if (e < nbox && gr >= 0 && gr < H && gc >= 0 && gc < W) v[u] = xp[(size_t)gr * W + gc];
    }
#pragma unroll
    for (int u = 0; u < FB; ++u)
      if (e0 + u * nth < nbox) box[e0 + u * nth] = v[u];
  }
  __syncthreads();
  const int s = threadIdx.x & 63;                      // tile within the box (<= 64)
  const int q2r = NLEV == 1 ? 0 : (int)(threadIdx.x >> 6);
  if (NLEV == 1 && threadIdx.x >= 64) return;
  if (s >= RX * RY) return;
  const int ly = s / RX, lx = s - ly * RX;
  const int ty = ty0 + ly, tx = tx0 + lx;
  if (ty >= th || tx >= tw) return;
  const int t = (b * th + ty) * tw + tx;
  const float* win = box + ly * Mn * BW + lx * Mn;
  const size_t pstride = (size_t)M * T;
  float* __restrict__ vp = V + (size_t)m * T + t;
  if constexpr (NLEV == 1) {
    float X[5][5];
#pragma unroll
    for (int i = 0; i < 5; ++i)
#pragma unroll
      for (int j = 0; j < 5; ++j) X[i][j] = win[i * BW + j];
    float C[5][5];                                     // rows transformed: C[q1r][col]
#pragma unroll
    for (int j = 0; j < 5; ++j) {
      const float col[5] = {X[0][j], X[1][j], X[2][j], X[3][j], X[4][j]};
      float o[5];
      bt5_vec(col, o);
#pragma unroll
      for (int q = 0; q < 5; ++q) C[q][j] = o[q];
    }
#pragma unroll
    for (int q1r = 0; q1r < 5; ++q1r) {
      float o[5];
      bt5_vec(C[q1r], o);
#pragma unroll
      for (int q1c = 0; q1c < 5; ++q1c) vp[(size_t)(q1r * 5 + q1c) * pstride] = o[q1c];
    }
  } else {
    // level 2 along the rows (stride 3) for this wavefront's digit q2r:
    // Rw[a1][c] = sum_a2 B^T[q2r][a2] win[a1 + 3 a2][c]; the row of B^T is
    // selected, since q2r is not a compile-time index
    float c2v[5] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int q = 0; q < 5; ++q)
#pragma unroll
      for (int a2 = 0; a2 < 5; ++a2) c2v[a2] = q2r == q ? bt5(q, a2) : c2v[a2];
    float Rw[5][17];
#pragma unroll
    for (int a1 = 0; a1 < 5; ++a1) {
#pragma unroll
      for (int c = 0; c < 17; ++c) Rw[a1][c] = 0.0f;
#pragma unroll
      for (int a2 = 0; a2 < 5; ++a2) {
        const float* rowp = win + (a1 + 3 * a2) * BW;
#pragma unroll
        for (int c = 0; c < 17; ++c) Rw[a1][c] = fmaf(c2v[a2], rowp[c], Rw[a1][c]);
      }
    }
#pragma unroll
    for (int q1r = 0; q1r < 5; ++q1r) {
      // level 1 along the rows
      float R[17];
#pragma unroll
      for (int c = 0; c < 17; ++c) {
        float sr = 0.0f;
#pragma unroll
        for (int a1 = 0; a1 < 5; ++a1)
          if (bt5(q1r, a1) != 0.0f) sr = fmaf(bt5(q1r, a1), Rw[a1][c], sr);
        R[c] = sr;
      }
      // columns: level 2 (stride 3), then level 1
#pragma unroll
      for (int q2c = 0; q2c < 5; ++q2c) {
        float v5[5];
#pragma unroll
        for (int b1 = 0; b1 < 5; ++b1) {
          float s2 = 0.0f;
#pragma unroll
          for (int b2 = 0; b2 < 5; ++b2)
            if (bt5(q2c, b2) != 0.0f) s2 = fmaf(bt5(q2c, b2), R[b1 + 3 * b2], s2);
          v5[b1] = s2;
        }
        float o[5];
        bt5_vec(v5, o);
#pragma unroll
        for (int q1c = 0; q1c < 5; ++q1c) {
          const int p = ((q2r * 5 + q2c) * 5 + q1r) * 5 + q1c;
          vp[(size_t)p * pstride] = o[q1c];
        }
      }
    }
  }
}

// ---- contraction: per point U[p]^T V[p] on fp32 MFMA ----------------------
// Work-group (256 threads, 2 x 2 wavefronts of 32 x 32): a 64 x 64 block of
// (n, t) for the 5 points of one level-1 row digit (group g, digit q1r).
// The 5 products are folded along the level-1 columns in registers,
//   Z[g][q1r][i1c] = sum_q1c A^T[i1c][q1c] Yhat[25 g + 5 q1r + q1c],
// and the output transform applies the level-1 rows.  Splitting the 25
// points of a group over 5 work-groups keeps 48 accumulator registers per
// lane instead of 144 and gives 5x the work-groups.
//
// The K loop runs over chunks of BK channels (5 points x M/BK chunks in a
// row) through a ring of 4 LDS stages, each a distinct LDS object, filled by
// direct global->LDS loads; three chunks are in flight while one is
// multiplied.  Columns past N or T re-read the last valid column (those
// results are not stored).  Two loaders:
//   VEC (N, T multiples of 4, 16-byte aligned buffers): global_load_lds_dwordx4,
//     lane l of a load writes LDS floats [4 l, 4 l + 4) of a 4-row slab of
//     64-float rows; the lane fetches column quad (l % 16) ^ 4 (row % 4), so
//     that the 4 rows one MFMA operand read touches fall in distinct
//     16-bank groups (the reader undoes the XOR);
//   otherwise global_load_lds_dword, lane l writing word l of one row,
//     rows padded to 80 floats for the same bank spread.
//   EVEN (M a multiple of 4 BK): every point takes a whole number of ring
//     turns, so the loop body is four unconditional steps and the fold
//     follows each point;
//   otherwise every step is guarded, the fold is tested per step, and in a
//     ragged last chunk the operand values of channels >= M are zeroed in
//     registers before the MFMA.
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int C5_BM = 64, C5_BN = 64;

template <int BK, bool VEC>
using C5Buf = float[BK][VEC ? 64 : 80];

// LDS word of (row, col) in a VEC buffer: column quad XOR 4 (row % 4)
__device__ __forceinline__ int c5_swz(int row, int col) {
  return row * 64 + ((((col >> 2) ^ ((row & 3) << 2))) << 2) + (col & 3);
}

template <int BK, bool EVEN, bool VEC>
__global__ __launch_bounds__(256) void contract5(const float* __restrict__ U,
                                                 const float* __restrict__ V,
                                                 float* __restrict__ Z, int M, int N, int T,
                                                 int ntb, int nnb) {
  // loads per wavefront per chunk: VEC, 2 BK / 4 slabs of 4 rows over 4
  // wavefronts (BK = 8: wavefronts 0-1 load U, 2-3 load V); else BK / 4
  // rows of each operand
  static_assert(!VEC || BK == 8 || BK == 16, "VEC chunks of 8 or 16 channels");
  constexpr int RPW = BK / 4;
  constexpr int LPC = VEC ? BK / 8 : 2 * RPW;
  using Buf = C5Buf<BK, VEC>;
  __shared__ Buf A0, A1, A2, A3, B0, B1, B2, B3;
  long long bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tb = (int)(bid % ntb);
  bid /= ntb;
  const int nb = (int)(bid % nnb);
  const long long gq = bid / nnb;                      // 5 g + q1r
  const int n0 = nb * C5_BM, c0 = tb * C5_BN;
  const int lane = threadIdx.x & 63;
  // the wavefront index is uniform: in a scalar register, the row addresses
  // and LDS bases below are scalar too
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 15, lk = lane >> 4;
  const size_t pU = (size_t)M * N, pV = (size_t)M * T;
  const float* __restrict__ Ub = U + (size_t)(5 * gq) * pU;
  const float* __restrict__ Vb = V + (size_t)(5 * gq) * pV;
  int ulane, vlane;
  if constexpr (VEC) {
    // slab lane l -> row l / 16, column quad (l % 16) ^ 4 (l / 16), clamped
    const int q = (lane & 15) ^ ((lane >> 4) << 2);
    const int qu = (n0 >> 2) + q, qv = (c0 >> 2) + q;
    ulane = 4 * (qu < (N >> 2) ? qu : (N >> 2) - 1);
    vlane = 4 * (qv < (T >> 2) ? qv : (T >> 2) - 1);
  } else {
    ulane = n0 + lane < N ? n0 + lane : N - 1;
    vlane = c0 + lane < T ? c0 + lane : T - 1;
  }
  const int nk = (M + BK - 1) / BK;
  const int total = 5 * nk;

  floatx4 acc[2][2], w[3][2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int o = 0; o < 3; ++o) w[o][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

  // chunk c: point q1c = c / nk, channels [BK (c % nk), +BK)
  auto request = [&](int c, Buf& An, Buf& Bn) {
    const int q1c = c / nk;
    const int kc0 = (c - q1c * nk) * BK;
    if constexpr (VEC) {
      // slabs of 4 rows: BK = 16, wavefront w loads slab w of U and of V;
      // BK = 8, wavefront w loads slab w % 2 of U (w < 2) or of V (w >= 2)
#pragma unroll
      for (int j = 0; j < LPC; ++j) {
        const bool isU = BK == 16 ? j == 0 : wave < 2;
        const int slab = BK == 16 ? wave : (wave & 1);
        int k = kc0 + 4 * slab + lk;
        if (!EVEN) k = k < M ? k : M - 1;
        const float* src = isU ? Ub + (size_t)q1c * pU + (size_t)k * N + ulane
                               : Vb + (size_t)q1c * pV + (size_t)k * T + vlane;
        float* dst = isU ? &An[4 * slab][0] : &Bn[4 * slab][0];
        __builtin_amdgcn_global_load_lds((const void*)src,
                                         (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
      }
    } else {
      const int k0 = kc0 + RPW * wave;
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
        const int k = EVEN || k0 + r < M ? k0 + r : M - 1;
        const float* urow = Ub + (size_t)q1c * pU + (size_t)k * N;
        const float* vrow = Vb + (size_t)q1c * pV + (size_t)k * T;
        __builtin_amdgcn_global_load_lds(
            (const void*)(urow + ulane),
            (__attribute__((address_space(3))) void*)&An[RPW * wave + r][0], 4, 0, 0);
        __builtin_amdgcn_global_load_lds(
            (const void*)(vrow + vlane),
            (__attribute__((address_space(3))) void*)&Bn[RPW * wave + r][0], 4, 0, 0);
      }
    }
  };

  // all operand reads of the chunk first, then its MFMAs
  auto compute = [&](const Buf& Ac, const Buf& Bc, int kvalid) {
    float af[BK / 4][2], bf[BK / 4][2];
#pragma unroll
    for (int kk = 0; kk < BK / 4; ++kk) {
      const int row = kk * 4 + lk;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int col = wm * 32 + i * 16 + lr;
        af[kk][i] = VEC ? (&Ac[0][0])[c5_swz(row, col)] : Ac[row][col];
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = wn * 32 + j * 16 + lr;
        bf[kk][j] = VEC ? (&Bc[0][0])[c5_swz(row, col)] : Bc[row][col];
      }
      if (!EVEN && kk * 4 + lk >= kvalid) af[kk][0] = af[kk][1] = bf[kk][0] = bf[kk][1] = 0.0f;
    }
#pragma unroll
    for (int kk = 0; kk < BK / 4; ++kk)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[kk][i], bf[kk][j], acc[i][j], 0, 0, 0);
  };

  // w[i1c] += A^T[i1c][q1c] acc (F(3,3)'s A^T, selected for the runtime digit)
  auto fold = [&](int q1c) {
    const float a0 = q1c < 4 ? 1.0f : 0.0f;
    const float a1 = q1c == 1 ? 1.0f : q1c == 2 ? -1.0f : q1c == 3 ? 2.0f : 0.0f;
    const float a2 = q1c == 0 ? 0.0f : q1c == 3 ? 4.0f : 1.0f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        w[0][i][j] += a0 * acc[i][j];
        w[1][i][j] += a1 * acc[i][j];
        w[2][i][j] += a2 * acc[i][j];
        acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
  };

  // one pipeline step: wait for chunk it (own loads, then the barrier for
  // everyone's), request chunk it + 3 (clamped to the last chunk, into the
  // buffer read in step it - 1), multiply chunk it
  auto step = [&](int it, const Buf& Ac, const Buf& Bc, Buf& An, Buf& Bn) {
    wait_vmcnt<2 * LPC>();
    __builtin_amdgcn_s_barrier();
    const int c = it + 3;
    request(c < total ? c : total - 1, An, Bn);
    if constexpr (EVEN) {
      compute(Ac, Bc, BK);
    } else {
      const int q1c = it / nk, kc = it - q1c * nk;
      compute(Ac, Bc, kc == nk - 1 ? M - kc * BK : BK);
      if (kc == nk - 1) fold(q1c);
    }
  };

  request(0, A0, B0);
  request(1 < total ? 1 : total - 1, A1, B1);
  request(2 < total ? 2 : total - 1, A2, B2);
  if constexpr (EVEN) {
    for (int q1c = 0; q1c < 5; ++q1c) {
      for (int kb = 0; kb < nk; kb += 4) {
        const int c = q1c * nk + kb;
        step(c, A0, B0, A3, B3);
        step(c + 1, A1, B1, A0, B0);
        step(c + 2, A2, B2, A1, B1);
        step(c + 3, A3, B3, A2, B2);
      }
      fold(q1c);
    }
  } else {
    for (int base = 0; base < total; base += 4) {
      step(base, A0, B0, A3, B3);
      if (base + 1 < total) step(base + 1, A1, B1, A0, B0);
      if (base + 2 < total) step(base + 2, A2, B2, A1, B1);
      if (base + 3 < total) step(base + 3, A3, B3, A2, B2);
    }
  }
  wait_vmcnt<0>();   // the clamped requests of the last steps

  // D layout of v_mfma_f32_16x16x4f32: lane l, register v -> row 4 (l / 16) + v, column l % 16
  const size_t plane = (size_t)N * T;
  float* __restrict__ Zg = Z + (size_t)gq * 3 * plane;
#pragma unroll
  for (int o = 0; o < 3; ++o)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = n0 + wm * 32 + i * 16 + lk * 4 + v;
        if (row >= N) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int col = c0 + wn * 32 + j * 16 + lr;
          if (col < T) Zg[(size_t)o * plane + (size_t)row * T + col] = w[o][i][j][v];
        }
      }
}

// ---- output transform: one thread per (tile, n) ----------------------------
// Z [P/25][5][3][N][T] (level-1 columns applied) -> the level-1 rows, then
// at depth 2 the level-2 A^T on both axes (output row i1r + 3 i2r).
// FOLD9 (the fused kernel's parts, depth 2): Z9 [P/25][3][3][N][T], level 1
// already applied on both axes.  parts > 1: the sum of `parts` buffers
// zpart floats apart.
template <int NLEV, bool FOLD9 = false>
__global__ __launch_bounds__(256) void output_xform5(const float* __restrict__ Z,
                                                     float* __restrict__ y, int N, int Ho,
                                                     int Wo, int th, int tw, int T, int parts,
                                                     size_t zpart) {
  constexpr int Mn = NLEV == 1 ? 3 : 9;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int n = blockIdx.y;
  if (t >= T) return;
  const size_t plane = (size_t)N * T;
  const float* __restrict__ zp = Z + (size_t)n * T + t;
  // level-1 rows: z9[i1r][i1c] = sum_q1r A^T[i1r][q1r] zr[q1r][i1c]
  auto level1_rows = [&](const float (&zr)[5][3], float (&z9)[3][3]) {
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        float sacc = 0.0f;
#pragma unroll
        for (int q = 0; q < 5; ++q)
          if (at5(i, q) != 0.0f) sacc = fmaf(at5(i, q), zr[q][c], sacc);
        z9[i][c] = sacc;
      }
  };
  float out[Mn][Mn];
  if constexpr (NLEV == 1) {
    float zr[5][3];
#pragma unroll
    for (int q = 0; q < 5; ++q)
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        float v = 0.0f;
        for (int k = 0; k < parts; ++k) v += zp[(size_t)k * zpart + (size_t)(q * 3 + c) * plane];
        zr[q][c] = v;
      }
    level1_rows(zr, out);
  } else {
#pragma unroll
    for (int i = 0; i < 9; ++i)
#pragma unroll
      for (int k = 0; k < 9; ++k) out[i][k] = 0.0f;
    // one level-2 row digit q2r per iteration: its 5 groups' 75 values are
    // loaded together (one wait for memory per row digit).  The plane
    // stride is made opaque so the loop-invariant offsets of the 75 loads
    // are not all precomputed and kept in scalar registers.
    const float* zq = zp;
#pragma unroll 1
    for (int q2r = 0; q2r < 5; ++q2r) {
      float zv9[5][3][3];
      size_t pl = plane;
      asm volatile("" : "+s"(pl));
      if constexpr (FOLD9) {
#pragma unroll
        for (int q2c = 0; q2c < 5; ++q2c)
#pragma unroll
          for (int i = 0; i < 3; ++i)
#pragma unroll
            for (int c = 0; c < 3; ++c) {
              zv9[q2c][i][c] = *zq;
              zq += pl;
            }
        for (int k = 1; k < parts; ++k) {
          const float* zk = zq - 45 * pl + (size_t)k * zpart;
#pragma unroll
          for (int q2c = 0; q2c < 5; ++q2c)
#pragma unroll
            for (int i = 0; i < 3; ++i)
#pragma unroll
              for (int c = 0; c < 3; ++c) {
                zv9[q2c][i][c] += *zk;
                zk += pl;
              }
        }
      } else {
        float zr[5][5][3];
#pragma unroll
        for (int q2c = 0; q2c < 5; ++q2c)
#pragma unroll
          for (int q = 0; q < 5; ++q)
#pragma unroll
            for (int c = 0; c < 3; ++c) {
              zr[q2c][q][c] = *zq;
              zq += pl;
            }
        // partial sums of a channel-split contraction (parts > 1)
        for (int k = 1; k < parts; ++k) {
          const float* zk = zq - 75 * pl + (size_t)k * zpart;
#pragma unroll
          for (int q2c = 0; q2c < 5; ++q2c)
#pragma unroll
            for (int q = 0; q < 5; ++q)
#pragma unroll
              for (int c = 0; c < 3; ++c) {
                zr[q2c][q][c] += *zk;
                zk += pl;
              }
        }
#pragma unroll
        for (int q2c = 0; q2c < 5; ++q2c) level1_rows(zr[q2c], zv9[q2c]);
      }
      float cr[3];
#pragma unroll
      for (int i = 0; i < 3; ++i) {
        cr[i] = 0.0f;
#pragma unroll
        for (int q = 0; q < 5; ++q) cr[i] = q2r == q ? at5(i, q) : cr[i];
      }
#pragma unroll
      for (int q2c = 0; q2c < 5; ++q2c) {
        const float (&zv)[3][3] = zv9[q2c];
#pragma unroll
        for (int i2r = 0; i2r < 3; ++i2r)
#pragma unroll
          for (int i2c = 0; i2c < 3; ++i2c) {
            if (at5(i2c, q2c) == 0.0f) continue;
            const float cf = cr[i2r] * at5(i2c, q2c);
#pragma unroll
            for (int i1r = 0; i1r < 3; ++i1r)
#pragma unroll
              for (int i1c = 0; i1c < 3; ++i1c)
                out[3 * i2r + i1r][3 * i2c + i1c] =
                    fmaf(cf, zv[i1r][i1c], out[3 * i2r + i1r][3 * i2c + i1c]);
          }
      }
    }
  }
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  float* __restrict__ yo = y + ((size_t)b * N + n) * Ho * Wo;
#pragma unroll
  for (int i = 0; i < Mn; ++i) {
    const int row = ty * Mn + i;
    if (row >= Ho) continue;
#pragma unroll
    for (int k = 0; k < Mn; ++k) {
      const int col = tx * Mn + k;
      if (col < Wo) yo[(size_t)row * Wo + col] = out[i][k];
    }
  }
}

// ---- contraction fused into the output transform: one or two input channels
// With M <= 2 the contraction is one or two multiply-adds per point, while Z
// would hold 3P/5 values per (output channel, tile): the output transform
// forms each point's sum from V and U itself and no Z reaches memory.
// Thread per (tile, n); U[.][.][n] (P x M values) is staged in LDS and read
// as broadcasts; V reads are coalesced over the tiles of a wavefront.
template <int NLEV, int MM>
__global__ __launch_bounds__(256) void contract_output5(const float* __restrict__ V,
                                                        const float* __restrict__ U,
                                                        float* __restrict__ y, int N, int Ho,
                                                        int Wo, int th, int tw, int T) {
  constexpr int Mn = NLEV == 1 ? 3 : 9;
  constexpr int P = NLEV == 1 ? 25 : 625;
  __shared__ float Us[P * MM];
  const int n = blockIdx.y;
  for (int e = threadIdx.x; e < P * MM; e += 256) {
    const int p = e / MM, m = e - p * MM;
    Us[e] = U[((size_t)p * MM + m) * N + n];
  }
  __syncthreads();
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  const float* __restrict__ vp = V + t;
  // the 25 points of group grp, their V values in vv -> level 1 on both axes
  auto group = [&](int grp, const float (&vv)[25][MM], float (&z9)[3][3]) {
    float zr[5][3];
#pragma unroll
    for (int q1r = 0; q1r < 5; ++q1r) {
      float a[5];
#pragma unroll
      for (int q1c = 0; q1c < 5; ++q1c) {
        const int p = grp * 25 + q1r * 5 + q1c;
        float sacc = 0.0f;
#pragma unroll
        for (int m = 0; m < MM; ++m) sacc = fmaf(Us[p * MM + m], vv[q1r * 5 + q1c][m], sacc);
        a[q1c] = sacc;
      }
#pragma unroll
      for (int i1c = 0; i1c < 3; ++i1c) {
        float sc = 0.0f;
#pragma unroll
        for (int q1c = 0; q1c < 5; ++q1c)
          if (at5(i1c, q1c) != 0.0f) sc = fmaf(at5(i1c, q1c), a[q1c], sc);
        zr[q1r][i1c] = sc;
      }
    }
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        float sacc = 0.0f;
#pragma unroll
        for (int q = 0; q < 5; ++q)
          if (at5(i, q) != 0.0f) sacc = fmaf(at5(i, q), zr[q][c], sacc);
        z9[i][c] = sacc;
      }
  };
  auto load_group = [&](int grp, float (&vv)[25][MM]) {
#pragma unroll
    for (int k = 0; k < 25; ++k)
#pragma unroll
      for (int m = 0; m < MM; ++m) vv[k][m] = vp[((size_t)(grp * 25 + k) * MM + m) * T];
  };
  float out[Mn][Mn];
  if constexpr (NLEV == 1) {
    float vv[25][MM];
    load_group(0, vv);
    group(0, vv, out);
  } else {
#pragma unroll
    for (int i = 0; i < 9; ++i)
#pragma unroll
      for (int k = 0; k < 9; ++k) out[i][k] = 0.0f;
    // one group per iteration (batching three groups' loads measured slower)
    constexpr int GB = 1;
#pragma unroll 1
    for (int g0 = 0; g0 < 25; g0 += GB) {
      float vv[GB][25][MM];
#pragma unroll
      for (int j = 0; j < GB; ++j) load_group(g0 + j < 25 ? g0 + j : 24, vv[j]);
#pragma unroll
      for (int j = 0; j < GB; ++j) {
        // past the last group (25 is not a multiple of GB): q2r = 5 selects
        // zero coefficients, the data are group 24's
        const int grp = g0 + j;
        const int q2r = grp / 5, q2c = grp - 5 * q2r;
        float zv[3][3];
        group(grp < 25 ? grp : 24, vv[j], zv);
        float cr[3], cc[3];
#pragma unroll
        for (int i = 0; i < 3; ++i) {
          cr[i] = 0.0f;
          cc[i] = 0.0f;
#pragma unroll
          for (int q = 0; q < 5; ++q) {
            cr[i] = q2r == q ? at5(i, q) : cr[i];
            cc[i] = q2c == q ? at5(i, q) : cc[i];
          }
        }
#pragma unroll
        for (int i2r = 0; i2r < 3; ++i2r)
#pragma unroll
          for (int i2c = 0; i2c < 3; ++i2c) {
            const float cf = cr[i2r] * cc[i2c];
#pragma unroll
            for (int i1r = 0; i1r < 3; ++i1r)
#pragma unroll
              for (int i1c = 0; i1c < 3; ++i1c)
                out[3 * i2r + i1r][3 * i2c + i1c] =
                    fmaf(cf, zv[i1r][i1c], out[3 * i2r + i1r][3 * i2c + i1c]);
          }
      }
    }
  }
  const int tpi = th * tw;
  const int b = t / tpi;
  const int r2 = t - b * tpi;
  const int ty = r2 / tw, tx = r2 - ty * tw;
  float* __restrict__ yo = y + ((size_t)b * N + n) * Ho * Wo;
#pragma unroll
  for (int i = 0; i < Mn; ++i) {
    const int row = ty * Mn + i;
    if (row >= Ho) continue;
#pragma unroll
    for (int k = 0; k < Mn; ++k) {
      const int col = tx * Mn + k;
      if (col < Wo) yo[(size_t)row * Wo + col] = out[i][k];
    }
  }
}

// ---- fused input transform + contraction: depth 2, one output channel -----
// x -> Z with no V in memory (the F(3,3) counterpart of the F(2,3) fused
// kernel): work-group = a box of up to 64 tiles of one image and a group of
// input channels; wavefront q2r (5 of them) and lane = tile, as in the input
// transform.  Per channel the box and U[.][m][0] are staged in LDS; each
// lane forms its 125 points (q2c, q1r, q1c), multiplies them by U (LDS
// broadcast reads) and folds level 1 on both axes into 45 accumulators
// acc[q2c][i1r][i1c].  Channel group cg writes its partial Z9 (P/25 x 9
// values per tile: level 1 fully applied) to part cg; the output
// transform adds the parts.
__global__ __launch_bounds__(320) void input_contract5(
    const float* __restrict__ x, const float* __restrict__ U, float* __restrict__ Zp, int M,
    int H, int W, int pad, int th, int tw, int T, int RX, int RY, int nbx, int nby, int mper,
    size_t zpart) {
  constexpr int Mn = 9, Ln = 17, P = 625;
  extern __shared__ float lds[];
  const int BH = (RY - 1) * Mn + Ln, BW = (RX - 1) * Mn + Ln;
  const int nbox = BH * BW;
  float* box = lds;
  float* Us = lds + nbox;
  int bid = blockIdx.x;
  const int bx = bid % nbx;
  bid /= nbx;
  const int by = bid % nby;
  const int b = bid / nby;
  const int cg = blockIdx.y;
  const int m0 = cg * mper, m1 = M < m0 + mper ? M : m0 + mper;
  const int ty0 = by * RY, tx0 = bx * RX;
  const int r0 = ty0 * Mn - pad, c0 = tx0 * Mn - pad;
  const int s = threadIdx.x & 63;
  const int q2r = threadIdx.x >> 6;
  const int ly = s / RX, lx = s - ly * RX;
  const int ty = ty0 + ly, tx = tx0 + lx;
  const bool active = s < RX * RY && ty < th && tx < tw;
  float c2v[5] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int q = 0; q < 5; ++q)
#pragma unroll
    for (int a2 = 0; a2 < 5; ++a2) c2v[a2] = q2r == q ? bt5(q, a2) : c2v[a2];
  float acc[5][3][3];   // [q2c][i1r][i1c]
#pragma unroll
  for (int i = 0; i < 5; ++i)
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
      for (int k = 0; k < 3; ++k) acc[i][j][k] = 0.0f;

  for (int m = m0; m < m1; ++m) {
    const float* __restrict__ xp = x + ((size_t)b * M + m) * H * W;
    // batches of FB loads per thread (a 64-tile box of 9 x 9 tiles is
    // about 7000 floats: one batch), all issued before the LDS stores
    constexpr int FB = 24;
    for (int e0 = threadIdx.x; e0 < nbox; e0 += FB * 320) {
      float v[FB];
#pragma unroll
      for (int u = 0; u < FB; ++u) {
        const int e = e0 + u * 320;
        const int row = e / BW, col = e - row * BW;
        const int gr = r0 + row, gc = c0 + col;
        v[u] = 0.0f;
        if (e < nbox && gr >= 0 && gr < H && gc >= 0 && gc < W) v[u] = xp[(size_t)gr * W + gc];
      }
#pragma unroll
      for (int u = 0; u < FB; ++u)
        if (e0 + u * 320 < nbox) box[e0 + u * 320] = v[u];
    }
    for (int e = threadIdx.x; e < P; e += 320) Us[e] = U[(size_t)e * M + m];
    __syncthreads();
    if (active) {
      const float* win = box + ly * Mn * BW + lx * Mn;
      float Rw[5][17];
#pragma unroll
      for (int a1 = 0; a1 < 5; ++a1) {
#pragma unroll
        for (int c = 0; c < 17; ++c) Rw[a1][c] = 0.0f;
#pragma unroll
        for (int a2 = 0; a2 < 5; ++a2) {
          const float* rowp = win + (a1 + 3 * a2) * BW;
#pragma unroll
          for (int c = 0; c < 17; ++c) Rw[a1][c] = fmaf(c2v[a2], rowp[c], Rw[a1][c]);
        }
      }
      const float* ub = Us + q2r * 125;
#pragma unroll
      for (int q1r = 0; q1r < 5; ++q1r) {
        float R[17];
#pragma unroll
        for (int c = 0; c < 17; ++c) {
          float sr = 0.0f;
#pragma unroll
          for (int a1 = 0; a1 < 5; ++a1)
            if (bt5(q1r, a1) != 0.0f) sr = fmaf(bt5(q1r, a1), Rw[a1][c], sr);
          R[c] = sr;
        }
#pragma unroll
        for (int q2c = 0; q2c < 5; ++q2c) {
          float v5[5];
#pragma unroll
          for (int b1 = 0; b1 < 5; ++b1) {
            float s2 = 0.0f;
#pragma unroll
            for (int b2 = 0; b2 < 5; ++b2)
              if (bt5(q2c, b2) != 0.0f) s2 = fmaf(bt5(q2c, b2), R[b1 + 3 * b2], s2);
            v5[b1] = s2;
          }
          float o[5];
          bt5_vec(v5, o);
          const float* up = ub + (q2c * 5 + q1r) * 5;   // the same LDS word for every lane
          float pr[5];
#pragma unroll
          for (int q1c = 0; q1c < 5; ++q1c) pr[q1c] = up[q1c] * o[q1c];
#pragma unroll
          for (int i1c = 0; i1c < 3; ++i1c) {
            float wc = 0.0f;
#pragma unroll
            for (int q1c = 0; q1c < 5; ++q1c)
              if (at5(i1c, q1c) != 0.0f) wc = fmaf(at5(i1c, q1c), pr[q1c], wc);
#pragma unroll
            for (int i1r = 0; i1r < 3; ++i1r)
              if (at5(i1r, q1r) != 0.0f)
                acc[q2c][i1r][i1c] = fmaf(at5(i1r, q1r), wc, acc[q2c][i1r][i1c]);
          }
        }
      }
    }
    __syncthreads();   // the next channel's fill overwrites box and Us
  }
  if (active) {
    const int t = (b * th + ty) * tw + tx;
    float* __restrict__ zp = Zp + (size_t)cg * zpart + t;
#pragma unroll
    for (int q2c = 0; q2c < 5; ++q2c)
#pragma unroll
      for (int i1r = 0; i1r < 3; ++i1r)
#pragma unroll
        for (int i1c = 0; i1c < 3; ++i1c)
          zp[(size_t)((q2r * 5 + q2c) * 9 + i1r * 3 + i1c) * T] = acc[q2c][i1r][i1c];
  }
}

}  // namespace

hipError_t launch_kernel_xform5(const nwg_plan_info& g, const float* w, float* U, hipStream_t s) {
  const long long nthreads = (long long)g.N * g.M;
  dim3 grid((unsigned)((nthreads + 255) / 256));
  if (g.n == 1)
    hipLaunchKernelGGL(kernel_xform5<1>, grid, dim3(256), 0, s, w, U, g.M, g.N, g.r, nthreads);
  else if (g.n == 2)
    hipLaunchKernelGGL(kernel_xform5<2>, grid, dim3(256), 0, s, w, U, g.M, g.N, g.r, nthreads);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_input_xform5(const nwg_plan_info& g, const float* x, float* V, hipStream_t s) {
  if (g.n != 1 && g.n != 2) return hipErrorInvalidValue;
  const int Mn = g.n == 1 ? 3 : 9, Ln = g.n == 1 ? 5 : 17;
  // up to 64 tiles per box
  const int RX = g.tw < 64 ? g.tw : 64;
  int RY = 64 / RX;
  if (RY > g.th) RY = g.th;
  const int nbx = (g.tw + RX - 1) / RX, nby = (g.th + RY - 1) / RY;
  const long long blocks = (long long)nbx * nby * g.B;
  if (blocks > 0x7fffffffLL || g.M > 65535) return hipErrorInvalidValue;
  const size_t lds = (size_t)((RY - 1) * Mn + Ln) * ((RX - 1) * Mn + Ln) * sizeof(float);
  dim3 grid((unsigned)blocks, (unsigned)g.M);
  const int T = (int)g.T;
  if (g.n == 1)
    hipLaunchKernelGGL(input_xform5<1>, grid, dim3(64), lds, s, x, V, g.M, g.H, g.W, g.pad, g.th,
                       g.tw, T, RX, RY, nbx, nby);
  else
    hipLaunchKernelGGL(input_xform5<2>, grid, dim3(320), lds, s, x, V, g.M, g.H, g.W, g.pad,
                       g.th, g.tw, T, RX, RY, nbx, nby);
  return hipGetLastError();
}

hipError_t launch_contract5(const nwg_plan_info& g, const float* U, const float* V, float* Z,
                            hipStream_t s) {
  if (g.n != 1 && g.n != 2) return hipErrorInvalidValue;
  const int T = (int)g.T;
  const int ntb = (T + C5_BN - 1) / C5_BN, nnb = (g.N + C5_BM - 1) / C5_BM;
  const long long blocks = (long long)ntb * nnb * (g.P / 5);
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks), block(256);
  const bool vec = g.N % 4 == 0 && T % 4 == 0 && !(((uintptr_t)U | (uintptr_t)V) & 15);
#define NWG_C5(BK, EVEN, VEC)                                                                 \
  hipLaunchKernelGGL((contract5<BK, EVEN, VEC>), grid, block, 0, s, U, V, Z, g.M, g.N, T, ntb, \
                     nnb)
  if (g.M % 64 == 0) {
    if (vec) NWG_C5(16, true, true); else NWG_C5(16, true, false);
  } else if (g.M % 32 == 0) {
    if (vec) NWG_C5(8, true, true); else NWG_C5(8, true, false);
  } else {
    if (vec) NWG_C5(16, false, true); else NWG_C5(16, false, false);
  }
#undef NWG_C5
  return hipGetLastError();
}

hipError_t launch_output_xform5(const nwg_plan_info& g, const float* Z, float* y, hipStream_t s,
                                int parts, bool fold9) {
  if (g.N > 65535 || parts < 1 || (fold9 && g.n != 2)) return hipErrorInvalidValue;
  const int T = (int)g.T;
  // parts lie back to back: Z9 parts of P/25 x 9 values per (n, t), else Z
  const size_t zpart = fold9 ? (size_t)(g.P / 25) * 9 * g.N * g.T : g.yhat_bytes / sizeof(float);
  dim3 grid((unsigned)((T + 255) / 256), (unsigned)g.N);
  if (g.n == 1)
    hipLaunchKernelGGL(output_xform5<1>, grid, dim3(256), 0, s, Z, y, g.N, g.Ho, g.Wo, g.th, g.tw,
                       T, parts, zpart);
  else if (g.n == 2 && fold9)
    hipLaunchKernelGGL((output_xform5<2, true>), grid, dim3(256), 0, s, Z, y, g.N, g.Ho, g.Wo,
                       g.th, g.tw, T, parts, zpart);
  else if (g.n == 2)
    hipLaunchKernelGGL(output_xform5<2>, grid, dim3(256), 0, s, Z, y, g.N, g.Ho, g.Wo, g.th, g.tw,
                       T, parts, zpart);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// Sum of the fused kernel's partial Z9 buffers into the first one (one
// thread per 4 consecutive values: all of them in flight at once, where the
// output transform alone has one thread per tile and output channel).
__global__ __launch_bounds__(256) void sum_parts_kernel(float* __restrict__ Z, size_t n,
                                                        size_t zpart, int parts) {
  const size_t i = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= n) return;
  if (i + 4 <= n && !(zpart & 3)) {
    float4 a = *reinterpret_cast<const float4*>(Z + i);
    for (int k = 1; k < parts; ++k) {
      const float4 b = *reinterpret_cast<const float4*>(Z + (size_t)k * zpart + i);
      a.x += b.x;
      a.y += b.y;
      a.z += b.z;
      a.w += b.w;
    }
    *reinterpret_cast<float4*>(Z + i) = a;
  } else {
    for (size_t e = i; e < n && e < i + 4; ++e) {
      float a = Z[e];
      for (int k = 1; k < parts; ++k) a += Z[(size_t)k * zpart + e];
      Z[e] = a;
    }
  }
}

hipError_t launch_sum_parts(float* Z, size_t n, int parts, hipStream_t s) {
  if (parts <= 1) return hipSuccess;
  if ((uintptr_t)Z & 15) return hipErrorInvalidValue;
  const size_t blocks = (n + 1023) / 1024;
  if (blocks > 0x7fffffffULL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sum_parts_kernel, dim3((unsigned)blocks), dim3(256), 0, s, Z, n, n, parts);
  return hipGetLastError();
}

hipError_t launch_input_contract5(const nwg_plan_info& g, const float* x, const float* U,
                                  float* Zp, hipStream_t s) {
  if (!input_contract5_applies(g)) return hipErrorInvalidValue;
  const IC5Shape c = ic5_shape(g);
  const long long blocks = (long long)c.nbx * c.nby * g.B;
  if (blocks > 0x7fffffffLL || c.groups > 65535 || c.lds > 160 * 1024) return hipErrorInvalidValue;
  hipLaunchKernelGGL(input_contract5, dim3((unsigned)blocks, (unsigned)c.groups), dim3(320), c.lds,
                     s, x, U, Zp, g.M, g.H, g.W, g.pad, g.th, g.tw, (int)g.T, c.RX, c.RY, c.nbx,
                     c.nby, c.mper, (size_t)(g.P / 25) * 9 * g.N * g.T);
  return hipGetLastError();
}

hipError_t launch_contract_output5(const nwg_plan_info& g, const float* V, const float* U,
                                   float* y, hipStream_t s) {
  if (!contract_output5_applies(g) || g.N > 65535) return hipErrorInvalidValue;
  const int T = (int)g.T;
  dim3 grid((unsigned)((T + 255) / 256), (unsigned)g.N);
#define NWG_CO5(L, MM)                                                                          \
  hipLaunchKernelGGL((contract_output5<L, MM>), grid, dim3(256), 0, s, V, U, y, g.N, g.Ho, g.Wo, \
                     g.th, g.tw, T)
  if (g.n == 1) {
    if (g.M == 1) NWG_CO5(1, 1); else NWG_CO5(1, 2);
  } else {
    if (g.M == 1) NWG_CO5(2, 1); else NWG_CO5(2, 2);
  }
#undef NWG_CO5
  return hipGetLastError();
}

}  // namespace nwg
