// Nested kernel transformation (Sec. III.B, second step; multi-level
// paragraph for depth > 2), run once per weight set; the plan caches U.
//
// The r x r kernel is zero-padded at its end to K_n x K_n (K_n = 2^(n+1)-1).
// Each tap k of an axis sits at one multi-index (k_1..k_n), k_j in {0,1,2},
// with sum_j 2^(j-1) k_j = k: the greedy split, outermost digit first, each
// digit as large as allowed.  Every other entry of the 3^n x 3^n reordered
// kernel is zero.  G of F(2,3) along every axis gives U[p][m][n].
//
// Depth <= 2: one thread per (output channel, input channel).  Depth 3 and
// 4: see kernel_xform_sep below.  Per outer branch the outer levels (3 and
// 4) fold the reordered kernel into a 9 x 9 sub-kernel over the digits
// (k2, k1) of each axis, and the two inner levels (9 -> 16 per axis) run in
// registers.  U is quad-interleaved, U[p/4][m][n][p%4] (p%4 is
// the level-1 column digit), written as float4; consecutive threads take
// consecutive output channels, then input channels, so the writes are
// contiguous.  Depth 0 (r = 1) stores U[m][n] = w[n][m][0][0].
#include "nwg_internal.h"

namespace nwg {
namespace {

// Tap of an axis multi-index (k4, k3, k2, k1) at depth NLEV, or -1 when the
// multi-index is not the greedy split of its tap.
template <int NLEV>
__device__ __forceinline__ int canonical_tap(int k4, int k3, int k2, int k1) {
  const int tap = 8 * k4 + 4 * k3 + 2 * k2 + k1;
  int rem = tap;
  int d[4] = {0, 0, 0, 0};
#pragma unroll
  for (int j = NLEV - 1; j >= 1; --j) {
    int v = rem >> j;
    v = v < 2 ? v : 2;
    d[j] = v;
    rem -= v << j;
  }
  d[0] = rem;
  const bool ok = d[0] == k1 && (NLEV < 2 || d[1] == k2) && (NLEV < 3 || d[2] == k3) &&
                  (NLEV < 4 || d[3] == k4);
  return ok ? tap : -1;
}

template <int NLEV>
__global__ __launch_bounds__(256) void kernel_xform(const float* __restrict__ w,
                                                    float* __restrict__ U, int M, int N, int r,
                                                    long long nthreads) {
  const long long id = (long long)blockIdx.x * 256 + threadIdx.x;
  if (id >= nthreads) return;
  const int nn = (int)(id % N);
  const long long rest = id / N;
  const int m = (int)(rest % M);
  const int branch = (int)(rest / M);
  const float* __restrict__ wk = w + ((size_t)nn * M + m) * r * r;
  const size_t MN = (size_t)M * N;

  if constexpr (NLEV == 0) {
    U[(size_t)m * N + nn] = wk[0];
  } else if constexpr (NLEV == 1) {
    float k[3][3];
#pragma unroll
    for (int u = 0; u < 3; ++u)
#pragma unroll
      for (int v = 0; v < 3; ++v) k[u][v] = (u < r && v < r) ? wk[u * r + v] : 0.0f;
    float rows[3][4];
#pragma unroll
    for (int u = 0; u < 3; ++u) g_one(k[u][0], k[u][1], k[u][2], rows[u]);
    float o[4][4];   // [q1r][q1c]
#pragma unroll
    for (int q1c = 0; q1c < 4; ++q1c) {
      float c[4];
      g_one(rows[0][q1c], rows[1][q1c], rows[2][q1c], c);
#pragma unroll
      for (int q1r = 0; q1r < 4; ++q1r) o[q1r][q1c] = c[q1r];
    }
    float4* U4 = reinterpret_cast<float4*>(U);
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r)
      U4[(size_t)q1r * MN + (size_t)m * N + nn] = make_float4(o[q1r][0], o[q1r][1], o[q1r][2], o[q1r][3]);
  } else {
    // outer branch: (q4r, q4c, q3r, q3c) digits of the branch index
    int qr3 = 0, qc3 = 0, qr4 = 0, qc4 = 0;
    if (NLEV == 3) {
      qr3 = branch >> 2;
      qc3 = branch & 3;
    } else if (NLEV == 4) {
      qr4 = branch >> 6;
      qc4 = (branch >> 4) & 3;
      qr3 = (branch >> 2) & 3;
      qc3 = branch & 3;
    }
    float S[9][9];
#pragma unroll
    for (int i = 0; i < 9; ++i)
#pragma unroll
      for (int j = 0; j < 9; ++j) S[i][j] = 0.0f;
    // outer digits (k4, k3) per axis with their G weights
    const int n4 = NLEV == 4 ? 3 : 1, n3 = NLEV >= 3 ? 3 : 1;
    for (int a4 = 0; a4 < n4; ++a4)
      for (int a3 = 0; a3 < n3; ++a3) {
        float gr = 1.0f;
        if (NLEV >= 3) gr *= g_coef(qr3, a3);
        if (NLEV == 4) gr *= g_coef(qr4, a4);
        if (gr == 0.0f) continue;
        for (int b4 = 0; b4 < n4; ++b4)
          for (int b3 = 0; b3 < n3; ++b3) {
            float gc = gr;
            if (NLEV >= 3) gc *= g_coef(qc3, b3);
            if (NLEV == 4) gc *= g_coef(qc4, b4);
            if (gc == 0.0f) continue;
#pragma unroll
            for (int ir = 0; ir < 9; ++ir) {
              const int tr = canonical_tap<NLEV>(a4, a3, ir / 3, ir % 3);
              if (tr < 0 || tr >= r) continue;
#pragma unroll
              for (int ic = 0; ic < 9; ++ic) {
                const int tc = canonical_tap<NLEV>(b4, b3, ic / 3, ic % 3);
                if (tc < 0 || tc >= r) continue;
                S[ir][ic] += gc * wk[tr * r + tc];
              }
            }
          }
      }
    // two inner levels: rows then columns; 64 quads per branch
    float4* ub = reinterpret_cast<float4*>(U) + (size_t)branch * 64 * MN + (size_t)m * N + nn;
#pragma unroll
    for (int rho = 0; rho < 16; ++rho) {
      // row rho = (q2r, q1r) of G2 applied to the 9 row digits
      const int q2r = rho >> 2, q1r = rho & 3;
      float rowv[9];
#pragma unroll
      for (int ic = 0; ic < 9; ++ic) {
        float s = 0.0f;
#pragma unroll
        for (int ir = 0; ir < 9; ++ir) {
          const float c = g_coef(q2r, ir / 3) * g_coef(q1r, ir % 3);
          if (c != 0.0f) s += c * S[ir][ic];
        }
        rowv[ic] = s;
      }
      float o[16];
      g_inner2(rowv, o);   // index q2c*4 + q1c
#pragma unroll
      for (int q2c = 0; q2c < 4; ++q2c) {
        const int quad = q2r * 16 + q2c * 4 + q1r;
        ub[(size_t)quad * MN] =
            make_float4(o[q2c * 4 + 0], o[q2c * 4 + 1], o[q2c * 4 + 2], o[q2c * 4 + 3]);
      }
    }
  }
}

// ---- depth 3 and 4, separable: rows of the outer levels first -------------
// Work-group (NW wavefronts; NW = 4 at depth 3, where there are 4 column
// branches, and 8 at depth 4, since its LDS allows one work-group per CU):
// 16 output channels of one input channel, their kernels in LDS
// zero-padded to K x K (K = 2^(NLEV+1) - 1, odd, so the 16 channels of a
// quarter-wave sit in different banks).  The outer levels (3, and 4 at depth
// 4) are applied along the rows for 4 outer row branches at a time
// (wavefront w takes branch w % 4 of the batch, so its G coefficients are
// uniform and zero terms are skipped by a scalar branch), leaving
// Rw[branch][channel][inner row digits (k2, k1)][column] in LDS.  Then
// wavefront w takes the outer column branches w, w + NW, ... and its lanes
// (channel, row branch) fold the columns into the 9 x 9 sub-kernel S over the
// inner digits, run the two inner levels in registers and store 64 quads;
// the 16 channels of a quarter-wave store 256 contiguous bytes per quad.
// Every tap index is a compile-time constant.
template <int NLEV, int NW>
__global__ __launch_bounds__(NW * 64) void kernel_xform_sep(const float* __restrict__ w,
                                                        float* __restrict__ U, int M, int N,
                                                        int r) {
  constexpr int K = (2 << NLEV) - 1;        // padded taps per axis
  constexpr int KS = K * K;                 // LDS stride per channel (odd)
  constexpr int RS = 9 * K;                 // Rw stride per (branch, channel) (odd)
  constexpr int NRB = NLEV == 4 ? 16 : 4;   // outer row (and column) branches
  constexpr int NA = NLEV == 4 ? 3 : 1;     // level-4 digits per axis
  extern __shared__ float lds[];
  float* wl = lds;                          // [16][K][K]
  float* Rw = lds + 16 * KS;                // [4][16][9][K]
  const int m = blockIdx.y;
  const int n0 = blockIdx.x * 16;
  for (int e = threadIdx.x; e < 16 * KS; e += NW * 64) {
    const int c = e / KS, k = e - c * KS;
    const int u = k / K, v = k - u * K;
    const int nn = n0 + c;
    wl[e] = (nn < N && u < r && v < r) ? w[((size_t)nn * M + m) * r * r + u * r + v] : 0.0f;
  }
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int cl = lane & 15, rbb = lane >> 4;
  const int nn = n0 + cl;
  const size_t MN = (size_t)M * N;
  for (int rb0 = 0; rb0 < NRB; rb0 += 4) {
    __syncthreads();                        // wl ready / previous batch's Rw read
    // rows: wavefront w takes row branch rb0 + w % 4; the NW / 4 wavefronts
    // of a branch share its (channel, column) elements
    {
      const int rb = rb0 + (wave & 3);
      const int qr3 = rb & 3, qr4 = rb >> 2;
      float* rwb = Rw + (wave & 3) * 16 * RS;
      for (int e = lane + 64 * (wave >> 2); e < 16 * K; e += 64 * (NW / 4)) {
        const int c = e / K, col = e - c * K;
        const float* wc = wl + c * KS + col;
        float acc[9];
#pragma unroll
        for (int i = 0; i < 9; ++i) acc[i] = 0.0f;
#pragma unroll
        for (int a4 = 0; a4 < NA; ++a4)
#pragma unroll
          for (int a3 = 0; a3 < 3; ++a3) {
            const float cf = (NLEV == 4 ? g_coef(qr4, a4) : 1.0f) * g_coef(qr3, a3);
            if (cf == 0.0f) continue;       // uniform: scalar branch
#pragma unroll
            for (int ir = 0; ir < 9; ++ir) {
              const int tap = canonical_tap<NLEV>(a4, a3, ir / 3, ir % 3);
              if (tap >= 0) acc[ir] = fmaf(cf, wc[tap * K], acc[ir]);
            }
          }
#pragma unroll
        for (int ir = 0; ir < 9; ++ir) rwb[c * RS + ir * K + col] = acc[ir];
      }
    }
    __syncthreads();
    // columns: wavefront w takes column branches w, w + NW, ...; lane
    // (channel cl, row branch rb0 + rbb)
    const int rb = rb0 + rbb;
    const int qr3 = rb & 3, qr4 = rb >> 2;
    const float* rwl = Rw + (rbb * 16 + cl) * RS;
    for (int cb = wave; cb < NRB; cb += NW) {
      const int qc3 = cb & 3, qc4 = cb >> 2;
      float S[9][9];
#pragma unroll
      for (int i = 0; i < 9; ++i)
#pragma unroll
        for (int j = 0; j < 9; ++j) S[i][j] = 0.0f;
#pragma unroll
      for (int b4 = 0; b4 < NA; ++b4)
#pragma unroll
        for (int b3 = 0; b3 < 3; ++b3) {
          const float cf = (NLEV == 4 ? g_coef(qc4, b4) : 1.0f) * g_coef(qc3, b3);
          if (cf == 0.0f) continue;         // uniform: scalar branch
#pragma unroll
          for (int ic = 0; ic < 9; ++ic) {
            const int tap = canonical_tap<NLEV>(b4, b3, ic / 3, ic % 3);
            if (tap < 0) continue;
#pragma unroll
            for (int ir = 0; ir < 9; ++ir) S[ir][ic] = fmaf(cf, rwl[ir * K + tap], S[ir][ic]);
          }
        }
      if (nn < N) {
        const int branch = NLEV == 4 ? ((qr4 * 4 + qc4) * 4 + qr3) * 4 + qc3 : qr3 * 4 + qc3;
        float4* ub = reinterpret_cast<float4*>(U) + (size_t)branch * 64 * MN + (size_t)m * N + nn;
#pragma unroll
        for (int rho = 0; rho < 16; ++rho) {
          const int q2r = rho >> 2, q1r = rho & 3;
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
            ub[(size_t)quad * MN] =
                make_float4(o[q2c * 4 + 0], o[q2c * 4 + 1], o[q2c * 4 + 2], o[q2c * 4 + 3]);
          }
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_kernel_xform(const nwg_plan_info& g, const float* w, float* U, hipStream_t s) {
  if (g.n >= 3) {
    if (g.M > 65535) return hipErrorInvalidValue;   // grid.y
    const int K = (2 << g.n) - 1;
    const size_t lds = ((size_t)16 * K * K + (size_t)64 * 9 * K) * sizeof(float);
    dim3 grid((unsigned)((g.N + 15) / 16), (unsigned)g.M);
    const void* fn = g.n == 3 ? reinterpret_cast<const void*>(&kernel_xform_sep<3, 4>)
                              : reinterpret_cast<const void*>(&kernel_xform_sep<4, 8>);
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    if (g.n == 3)
      hipLaunchKernelGGL((kernel_xform_sep<3, 4>), grid, dim3(256), lds, s, w, U, g.M, g.N, g.r);
    else
      hipLaunchKernelGGL((kernel_xform_sep<4, 8>), grid, dim3(512), lds, s, w, U, g.M, g.N, g.r);
    return hipGetLastError();
  }
  const long long nthreads = (long long)g.N * g.M;
  dim3 grid((unsigned)((nthreads + 255) / 256));
  switch (g.n) {
    case 0: hipLaunchKernelGGL(kernel_xform<0>, grid, dim3(256), 0, s, w, U, g.M, g.N, g.r, nthreads); break;
    case 1: hipLaunchKernelGGL(kernel_xform<1>, grid, dim3(256), 0, s, w, U, g.M, g.N, g.r, nthreads); break;
    case 2: hipLaunchKernelGGL(kernel_xform<2>, grid, dim3(256), 0, s, w, U, g.M, g.N, g.r, nthreads); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Linear decomposition (Sec. II.B): one thread per (output channel n,
// decomposed channel mv = (cu c + cv) M + m).  Sub-kernel (cu, cv) is
// w[n][m][3 cu .. 3 cu + 2][3 cv .. 3 cv + 2], zero past r; G of F(2,3) on
// both axes gives 16 values stored as the 4 quads of a depth-1 plan.
__global__ __launch_bounds__(256) void kernel_xform_ld(const float* __restrict__ w,
                                                       float* __restrict__ U, int M, int N, int r,
                                                       int c, long long nthreads) {
  const long long id = (long long)blockIdx.x * 256 + threadIdx.x;
  if (id >= nthreads) return;
  const int nn = (int)(id % N);
  const int mv = (int)(id / N);
  const int m = mv % M, sub = mv / M;
  const int u0 = 3 * (sub / c), v0 = 3 * (sub % c);
  const float* __restrict__ wk = w + ((size_t)nn * M + m) * r * r;
  float k[3][3];
#pragma unroll
  for (int u = 0; u < 3; ++u)
#pragma unroll
    for (int v = 0; v < 3; ++v)
      k[u][v] = (u0 + u < r && v0 + v < r) ? wk[(u0 + u) * r + v0 + v] : 0.0f;
  float rows[3][4];
#pragma unroll
  for (int u = 0; u < 3; ++u) g_one(k[u][0], k[u][1], k[u][2], rows[u]);
  const size_t MN = (size_t)M * c * c * N;
  float4* ub = reinterpret_cast<float4*>(U) + (size_t)mv * N + nn;
  float o[4][4];   // [q1r][q1c]
#pragma unroll
  for (int q1c = 0; q1c < 4; ++q1c) {
    float cc[4];
    g_one(rows[0][q1c], rows[1][q1c], rows[2][q1c], cc);
#pragma unroll
    for (int q1r = 0; q1r < 4; ++q1r) o[q1r][q1c] = cc[q1r];
  }
#pragma unroll
  for (int q1r = 0; q1r < 4; ++q1r)
    ub[(size_t)q1r * MN] = make_float4(o[q1r][0], o[q1r][1], o[q1r][2], o[q1r][3]);
}

hipError_t launch_kernel_xform_ld(const nwg_plan_info& g, const float* w, float* U, hipStream_t s) {
  if (g.ld_c < 1 || ((uintptr_t)U & 15)) return hipErrorInvalidValue;
  const long long nthreads = (long long)g.N * g.M * g.ld_c * g.ld_c;
  const long long blocks = (nthreads + 255) / 256;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kernel_xform_ld, dim3((unsigned)blocks), dim3(256), 0, s, w, U, g.M, g.N,
                     g.r, g.ld_c, nthreads);
  return hipGetLastError();
}

// Split precision: every fp32 value becomes its packed bf16 (hi, lo) pair,
// in place (4 values per thread; n need not be a multiple of 4).
__global__ __launch_bounds__(256) void split_pairs_kernel(float* __restrict__ buf, size_t n) {
  const size_t i = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i + 4 <= n) {
    float4 v = *reinterpret_cast<const float4*>(buf + i);
    *reinterpret_cast<float4*>(buf + i) = store_quad<true>(v.x, v.y, v.z, v.w);
  } else {
    for (size_t e = i; e < n; ++e) buf[e] = __uint_as_float(split_pair(buf[e]));
  }
}

hipError_t launch_split_pairs(float* buf, size_t n, hipStream_t s) {
  if (((uintptr_t)buf & 15) || n == 0) return hipErrorInvalidValue;
  const size_t blocks = (n + 1023) / 1024;
  if (blocks > 0x7fffffffULL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(split_pairs_kernel, dim3((unsigned)blocks), dim3(256), 0, s, buf, n);
  return hipGetLastError();
}

}  // namespace nwg
