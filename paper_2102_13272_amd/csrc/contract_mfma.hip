// Winograd-domain channel contraction: the EWMM of Sec. III.B accumulated
// over the M input channels (Sec. II.B), i.e. for every Winograd point p
//
//     Yhat[p] (N x T) = U[p]^T (N x M) * V[p] (M x T)
//
// a batch of P independent GEMMs, the one dense contraction of the method.
// It runs on fp32 MFMA (v_mfma_f32_16x16x4f32, fp32 accumulate).
//
// Work-group: 256 threads (4 wave64s) own a BM x BN block of one point's
// output; each wave owns a (BM/WM) x (BN/WN) sub-block of 16x16 MFMA tiles.
// The K loop moves BK = 16 channels per step through double-buffered LDS:
// the next step's global loads are issued before the current step's MFMAs
// and written to the other buffer afterwards, so one barrier per step
// suffices.  LDS rows are padded to a stride of 16 or 48 (mod 64) floats so
// that the four 16-lane groups of an MFMA operand read hit disjoint banks.
//
// Operand lane maps of v_mfma_f32_16x16x4f32 (wave64):
//   A (16x4):  lane l holds A[l%16][l/16]
//   B (4x16):  lane l holds B[l/16][l%16]
//   D (16x16): lane l, register v holds D[4*(l/16)+v][l%16]
//
// Work-groups are numbered so that consecutive blocks of the same point land
// on the same XCD (the dispatcher deals work-groups round-robin over the 8
// XCDs), keeping each point's U and V tiles in one L2.
#include "nwg_internal.h"

namespace nwg {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kBK = 16;

__host__ __device__ constexpr int lds_stride(int cols) {
  return ((cols + 16) % 32 == 16) ? cols + 16 : cols + 32;
}

__device__ __forceinline__ long long xcd_remap(long long i, long long G) {
  const long long q = G / 8, rem = G % 8;
  const long long xcd = i % 8, slot = i / 8;
  return xcd < rem ? xcd * (q + 1) + slot : rem * (q + 1) + (xcd - rem) * q + slot;
}

template <int COLS, int SROW>
struct TileLoader {
  // BK x COLS tile of a row-major [K][ld] matrix into LDS [BK][SROW].
  static constexpr int CHUNKS = kBK * COLS / 4;
  static constexpr int PER = (CHUNKS + 255) / 256;
  float4 reg[PER];

  __device__ __forceinline__ void load(const float* __restrict__ src, int ld, int k0, int c0,
                                       int K, int ncols, bool vec) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * 256;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (c < CHUNKS) {
        const int k = c / (COLS / 4);
        const int col = (c % (COLS / 4)) * 4;
        const int gk = k0 + k, gc = c0 + col;
        if (gk < K) {
          const float* p = src + (size_t)gk * ld + gc;
          if (vec) {
            if (gc < ncols) v = *reinterpret_cast<const float4*>(p);
          } else {
            if (gc + 0 < ncols) v.x = p[0];
            if (gc + 1 < ncols) v.y = p[1];
            if (gc + 2 < ncols) v.z = p[2];
            if (gc + 3 < ncols) v.w = p[3];
          }
        }
      }
      reg[i] = v;
    }
  }

  __device__ __forceinline__ void store(float (*dst)[SROW]) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * 256;
      if (c < CHUNKS) {
        const int k = c / (COLS / 4);
        const int col = (c % (COLS / 4)) * 4;
        *reinterpret_cast<float4*>(&dst[k][col]) = reg[i];
      }
    }
  }
};

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void contract_mfma(ContractArgs a, int ntb, int nnb,
                                                     int vecA, int vecB) {
  constexpr int SA = lds_stride(BM), SB = lds_stride(BN);
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  static_assert(WM * WN == 4, "four waves");
  static_assert(FM >= 1 && FN >= 1, "wave tile at least 16x16");
  __shared__ __attribute__((aligned(16))) float As[2][kBK][SA];
  __shared__ __attribute__((aligned(16))) float Bs[2][kBK][SB];

  long long bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tb = (int)(bid % ntb);
  bid /= ntb;
  const int nb = (int)(bid % nnb);
  const long long batch = bid / nnb;
  const float* __restrict__ A = a.A + batch * a.sA;
  const float* __restrict__ B = a.Bm + batch * a.sB;
  float* __restrict__ C = a.C + batch * a.sC;
  const int n0 = nb * BM, c0 = tb * BN;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int lr = lane & 15, lk = lane >> 4;

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  TileLoader<BM, SA> la;
  TileLoader<BN, SB> lb;
  const int nk = (a.K + kBK - 1) / kBK;
  la.load(A, a.ldA, 0, n0, a.K, a.Nrows, vecA);
  lb.load(B, a.ldB, 0, c0, a.K, a.Ncols, vecB);
  la.store(As[0]);
  lb.store(Bs[0]);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(A, a.ldA, (kt + 1) * kBK, n0, a.K, a.Nrows, vecA);
      lb.load(B, a.ldB, (kt + 1) * kBK, c0, a.K, a.Ncols, vecB);
    }
#pragma unroll
    for (int kk = 0; kk < kBK / 4; ++kk) {
      float af[FM], bf[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[i] = As[cur][kk * 4 + lk][wm * WTM + i * 16 + lr];
#pragma unroll
      for (int j = 0; j < FN; ++j) bf[j] = Bs[cur][kk * 4 + lk][wn * WTN + j * 16 + lr];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      la.store(As[cur ^ 1]);
      lb.store(Bs[cur ^ 1]);
    }
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = n0 + wm * WTM + i * 16 + lk * 4 + v;
      if (row >= a.Nrows) continue;
      float* crow = C + (size_t)row * a.ldC;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = c0 + wn * WTN + j * 16 + lr;
        if (col < a.Ncols) crow[col] = acc[i][j][v];
      }
    }
  }
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_tile(const ContractArgs& a, hipStream_t s) {
  const int ntb = (a.Ncols + BN - 1) / BN;
  const int nnb = (a.Nrows + BM - 1) / BM;
  const long long blocks = (long long)ntb * nnb * a.batch;
  if (blocks <= 0 || blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  auto aligned = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  const int vecA = (a.ldA % 4 == 0) && (a.Nrows % 4 == 0) && (a.sA % 4 == 0) && aligned(a.A);
  const int vecB = (a.ldB % 4 == 0) && (a.Ncols % 4 == 0) && (a.sB % 4 == 0) && aligned(a.Bm);
  hipLaunchKernelGGL((contract_mfma<BM, BN, WM, WN>), dim3((unsigned)blocks), dim3(256), 0, s, a,
                     ntb, nnb, vecA, vecB);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_contract(const ContractArgs& a, hipStream_t s) {
  const int N = a.Nrows, T = a.Ncols;
  auto cols_waste = [T](int bn) { return ((T + bn - 1) / bn) * bn; };
  const bool bn64 = cols_waste(64) < cols_waste(128);
  if (N <= 16) return launch_tile<16, 128, 1, 4>(a, s);
  if (N <= 32) return launch_tile<32, 128, 1, 4>(a, s);
  if (N <= 64) return bn64 ? launch_tile<64, 64, 2, 2>(a, s) : launch_tile<64, 128, 2, 2>(a, s);
  return bn64 ? launch_tile<128, 64, 2, 2>(a, s) : launch_tile<128, 128, 2, 2>(a, s);
}

}  // namespace nwg
