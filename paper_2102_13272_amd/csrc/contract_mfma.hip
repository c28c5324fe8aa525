// Winograd-domain channel contraction: the EWMM of Sec. III.B accumulated
// over the M input channels (Sec. II.B), fused with the first (innermost)
// level of the nested output transformation.
//
// For every Winograd point p,   Yhat[p] (N x T) = U[p]^T (N x M) * V[p] (M x T),
// a batch of P independent GEMMs -- the one dense contraction of the method,
// on fp32 MFMA (v_mfma_f32_16x16x4f32, fp32 accumulate).  The 16 points of a
// level-1 group g (digits q1r, q1c) are then reduced by A^T along both axes
// in registers:
//
//     Z[g][n][t][2*i1r + i1c] = sum_{q1r,q1c} A^T[i1r][q1r] A^T[i1c][q1c] Yhat[16g + 4q1r + q1c][n][t]
//
// so the contraction writes P/4 values per (n, t) instead of P.
//
// Layouts (quad-interleaved: the level-1 column digit q1c is innermost):
//   U [P/4][M][N][4],  V [P/4][M][T][4],  Z [P/16][N][T][4].
//
// Work-group: 256 threads (4 wave64s) own a BM x BN block of one group's
// output.  For each q1r the K loop streams the four points q1c = 0..3
// together through LDS as float4 quads; one ds_read_b128 yields the MFMA
// operand of all four points, and four accumulator sets take the four GEMMs.
// After the K loop the four products are folded into the 2x2 level-1
// outputs.  Two pipelines:
//   * deep (64x128 tiles when T is a multiple of 128, else 64x64 with a
//     ragged last column tile; N a multiple of 64, M of 32; 8 or 4 waves):
//     four LDS stages of 8 channels filled by direct global->LDS loads,
//     three chunks in flight;
//   * general (any shape): two LDS stages of 16 channels, direct loads for
//     full tiles, bounds-checked register loads for ragged ones.
// Without global loads the deep kernel reaches 93 % of the fp32 MFMA peak;
// the stages exist to hide HBM latency behind that.
//
// Operand lane maps of v_mfma_f32_16x16x4f32 (wave64):
//   A (16x4):  lane l holds A[l%16][l/16]
//   B (4x16):  lane l holds B[l/16][l%16]
//   D (16x16): lane l, register v holds D[4*(l/16)+v][l%16]
//
// Work-groups are numbered so that the blocks of one group land on the same
// XCD (the dispatcher deals work-groups round-robin over the 8 XCDs),
// keeping the group's U and V tiles in one L2.
//
// Depth 0 (r = 1) has no transform: a plain per-image GEMM kernel below
// takes y[b] = U^T x[b] with the same MFMA tiling.
#include "nwg_internal.h"

#include <cstdlib>
#include <map>
#include <mutex>
#include <utility>

namespace nwg {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kBK = 16;

// ---------------------------------------------------------------------------
// Fused contraction + level-1 output transform (depth >= 1)
// ---------------------------------------------------------------------------

// BK x COLS tile of float4 quads from a [K][ncols] quad matrix into LDS.
// Each thread owns fixed (k, col) slots; the per-chunk part of the address
// (quad and K offset) is uniform.  FULL: every tile is in bounds (no checks).
template <int COLS, bool FULL>
struct QuadLoader {
  static_assert(256 % COLS == 0, "a tile row must split evenly over the threads");
  static constexpr int ELEMS = kBK * COLS;
  static constexpr int PER = ELEMS / 256;     // slots per thread, rows RSTEP apart
  static constexpr int RSTEP = 256 / COLS;
  float4 reg[PER];
  int off0;     // (tid / COLS) * ld + c0 + tid % COLS
  int k0row;    // tid / COLS
  bool colok;   // c0 + tid % COLS < ncols

  __device__ __forceinline__ void init(int ld, int c0, int ncols) {
    const int k = threadIdx.x / COLS, col = threadIdx.x % COLS;
    off0 = k * ld + c0 + col;
    k0row = k;
    colok = c0 + col < ncols;
  }

  // base: uniform pointer of the quad matrix, k0 = first K row of the chunk
  __device__ __forceinline__ void load(const float4* __restrict__ base, int ld, int k0, int K) {
    const float4* __restrict__ p = base + (size_t)k0 * ld + off0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (FULL) {
        reg[i] = p[(size_t)i * RSTEP * ld];
      } else {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (colok && k0row + i * RSTEP < K - k0) v = p[(size_t)i * RSTEP * ld];
        reg[i] = v;
      }
    }
  }

  __device__ __forceinline__ void store(float4 (*dst)[COLS]) const {
    const int k = threadIdx.x / COLS, col = threadIdx.x % COLS;
#pragma unroll
    for (int i = 0; i < PER; ++i) dst[k + i * RSTEP][col] = reg[i];
  }
};

// Full-tile variant: gfx950 direct global->LDS loads (global_load_lds_dwordx4).
// Wave w's j-th load covers flat tile elements [(4j + w) * 64, +64); the
// hardware writes lane l's 16 bytes at the wave's LDS base + 16 l, so the
// data lands in LDS without passing through registers.  The loads are
// asynchronous; the barrier at the end of each step waits for them.
template <int COLS>
struct DirectLoader {
  static_assert(256 % COLS == 0, "a tile row must split evenly over the threads");
  static constexpr int PER = kBK * COLS / 256;
  static constexpr int RSTEP = 256 / COLS;
  int off0;

  __device__ __forceinline__ void init(int ld, int c0) {
    off0 = (threadIdx.x / COLS) * ld + c0 + threadIdx.x % COLS;
  }

  __device__ __forceinline__ void load(const float4* __restrict__ base, int ld, int k0,
                                       float4 (*dst)[COLS]) {
    const float4* p = base + (size_t)k0 * ld + off0;
    float4* flat = &dst[0][0];
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < PER; ++j)
      __builtin_amdgcn_global_load_lds(
          (const void*)(p + (size_t)j * RSTEP * ld),
          (__attribute__((address_space(3))) void*)(flat + j * 256 + wave * 64), 16, 0, 0);
  }
};

// One pipeline step: MFMAs on (Ac, Bc) while the next chunk streams into
// (An, Bn); at the end of a q1r sweep the four products are folded into the
// level-1 outputs.  The buffers are distinct LDS objects so that the
// compiler can see that the asynchronous loads into (An, Bn) never alias
// the reads of (Ac, Bc) and need not be waited for before them.
template <int BM, int BN, int WM, int WN, bool FULL>
struct FusedTile {
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / 16, FN = WTN / 16;
  floatx4 out[4][FM][FN];   // [2*i1r + i1c]
  floatx4 acc[4][FM][FN];   // [q1c]
  QuadLoader<BM, FULL> la;
  QuadLoader<BN, FULL> lb;
  DirectLoader<BM> da;
  DirectLoader<BN> db;

  __device__ __forceinline__ void prefetch(const float4* Ub, const float4* Vb, int N, int T,
                                           int k0, int M, float4 (*An)[BM], float4 (*Bn)[BN]) {
    if (FULL) {
      da.load(Ub, N, k0, An);
      db.load(Vb, T, k0, Bn);
    } else {
      la.load(Ub, N, k0, M);
      lb.load(Vb, T, k0, M);
    }
  }

  __device__ __forceinline__ void commit(float4 (*An)[BM], float4 (*Bn)[BN]) {
    if (!FULL) {
      la.store(An);
      lb.store(Bn);
    }
  }

  __device__ __forceinline__ void compute(const float4 (*Ac)[BM], const float4 (*Bc)[BN], int wm,
                                          int wn, int lr, int lk) {
#pragma unroll
    for (int kk = 0; kk < kBK / 4; ++kk) {
      float4 af[FM], bf[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[i] = Ac[kk * 4 + lk][wm * WTM + i * 16 + lr];
#pragma unroll
      for (int j = 0; j < FN; ++j) bf[j] = Bc[kk * 4 + lk][wn * WTN + j * 16 + lr];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          acc[0][i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].x, bf[j].x, acc[0][i][j], 0, 0, 0);
          acc[1][i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].y, bf[j].y, acc[1][i][j], 0, 0, 0);
          acc[2][i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].z, bf[j].z, acc[2][i][j], 0, 0, 0);
          acc[3][i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].w, bf[j].w, acc[3][i][j], 0, 0, 0);
        }
    }
  }

  // level 1 along columns (q1c -> i1c), then along rows with A^T[i1r][q1r]
  __device__ __forceinline__ void fold(int q1r) {
    const float r0 = at_coef(0, q1r), r1 = at_coef(1, q1r);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const floatx4 z0 = acc[0][i][j] + acc[1][i][j] + acc[2][i][j];
        const floatx4 z1 = acc[1][i][j] - acc[2][i][j] - acc[3][i][j];
        out[0][i][j] += r0 * z0;
        out[1][i][j] += r0 * z1;
        out[2][i][j] += r1 * z0;
        out[3][i][j] += r1 * z1;
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
  }
};

template <int BM, int BN, int WM, int WN, bool FULL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void contract_fused(
    const float4* __restrict__ U, const float4* __restrict__ V, float4* __restrict__ Z, int M,
    int N, int T, int ntb, int nnb, GroupMap gm) {
  using Tile = FusedTile<BM, BN, WM, WN, FULL>;
  constexpr int WTM = Tile::WTM, WTN = Tile::WTN, FM = Tile::FM, FN = Tile::FN;
  static_assert(WM * WN == 4, "four waves");
  static_assert(FM >= 1 && FN >= 1, "wave tile at least 16x16");
  __shared__ float4 A0[kBK][BM], A1[kBK][BM];
  __shared__ float4 B0[kBK][BN], B1[kBK][BN];

  long long bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tb = (int)(bid % ntb);
  bid /= ntb;
  const int nb = (int)(bid % nnb);
  const long long g = live_group(gm, bid / nnb);
  const int n0 = nb * BM, c0 = tb * BN;
  const size_t quadU = (size_t)M * N, quadV = (size_t)M * T;
  const float4* __restrict__ Ug = U + (size_t)(4 * g) * quadU;
  const float4* __restrict__ Vg = V + (size_t)(4 * g) * quadV;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int lr = lane & 15, lk = lane >> 4;

  Tile tile;
#pragma unroll
  for (int o = 0; o < 4; ++o)
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        tile.out[o][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        tile.acc[o][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
  if (FULL) {
    tile.da.init(N, n0);
    tile.db.init(T, c0);
  } else {
    tile.la.init(N, n0, N);
    tile.lb.init(T, c0, T);
  }

  const int nk = (M + kBK - 1) / kBK;
  // (q1r, K chunk) pairs, one pipeline; q1r = 3 is skipped where level-1
  // digit 3 is dead (its U is zero and its V is not written)
  const int total = (gm.q3 ? 3 : 4) * nk;
  tile.prefetch(Ug, Vg, N, T, 0, M, A0, B0);
  tile.commit(A0, B0);
  __syncthreads();
  // chunk it -> (q1r, kt); even chunks live in (A0, B0), odd ones in (A1, B1)
  for (int it = 0; it < total; it += 2) {
    {
      const int q1r = it / nk, kt = it % nk;
      const int nx = it + 1;
      if (nx < total)
        tile.prefetch(Ug + (size_t)(nx / nk) * quadU, Vg + (size_t)(nx / nk) * quadV, N, T,
                      (nx % nk) * kBK, M, A1, B1);
      tile.compute(A0, B0, wm, wn, lr, lk);
      if (kt + 1 == nk) tile.fold(q1r);
      if (nx < total) tile.commit(A1, B1);
      __syncthreads();
    }
    if (it + 1 < total) {
      const int c = it + 1;
      const int q1r = c / nk, kt = c % nk;
      const int nx = c + 1;
      if (nx < total)
        tile.prefetch(Ug + (size_t)(nx / nk) * quadU, Vg + (size_t)(nx / nk) * quadV, N, T,
                      (nx % nk) * kBK, M, A0, B0);
      tile.compute(A1, B1, wm, wn, lr, lk);
      if (kt + 1 == nk) tile.fold(q1r);
      if (nx < total) tile.commit(A0, B0);
      __syncthreads();
    }
  }

  float4* __restrict__ Zg = Z + (size_t)g * N * T;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = n0 + wm * WTM + i * 16 + lk * 4 + v;
      if (!FULL && row >= N) continue;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = c0 + wn * WTN + j * 16 + lr;
        if (FULL || col < T)
          Zg[(size_t)row * T + col] = make_float4(tile.out[0][i][j][v], tile.out[1][i][j][v],
                                                  tile.out[2][i][j][v], tile.out[3][i][j][v]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Deep-pipeline variant for full tiles: STAGES LDS buffers of BKD channels,
// each a distinct LDS object.  Chunk it+STAGES-1 is requested while chunk it
// is multiplied, so STAGES-1 chunks of direct global->LDS loads are in
// flight.  Before the barrier that opens step it, every wave waits only for
// its own loads of chunk it (s_waitcnt vmcnt(k), k = loads issued after
// them); the barrier then also guarantees that nobody still reads the
// buffer the step's new loads overwrite (it was read in step it-1).
// ---------------------------------------------------------------------------

template <int BKD, int COLS, int NT>
struct DeepLoader {
  static_assert(NT % COLS == 0, "a tile row must split evenly over the threads");
  static_assert((BKD * COLS) % NT == 0, "a tile must split evenly over the threads");
  static constexpr int PER = BKD * COLS / NT;   // loads per thread per chunk
  static constexpr int RSTEP = NT / COLS;
  int off0;
  // columns past ncols (a ragged last tile) re-read column ncols - 1; their
  // results are not stored
  __device__ __forceinline__ void init(int ld, int c0, int ncols) {
    const int c = c0 + threadIdx.x % COLS;
    off0 = (threadIdx.x / COLS) * ld + (c < ncols ? c : ncols - 1);
  }
  __device__ __forceinline__ void load(const float4* __restrict__ base, int ld, int k0,
                                       float4 (*dst)[COLS]) {
    const float4* p = base + (size_t)k0 * ld + off0;
    float4* flat = &dst[0][0];
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < PER; ++j)
      __builtin_amdgcn_global_load_lds(
          (const void*)(p + (size_t)j * RSTEP * ld),
          (__attribute__((address_space(3))) void*)(flat + j * NT + wave * 64), 16, 0, 0);
  }
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Q3: level-1 digit 3 is dead (GroupMap::q3): quads q1r = 0..2 only, and
// the fourth point of each quad (q1c = 3, its U zero) is not multiplied.
template <int BM, int BN, int WM, int WN, int BKD, int STAGES, bool SPLIT, bool Q3>
struct DeepTile {
  static constexpr int NQ = Q3 ? 3 : 4;     // quads (q1r) per group
  static constexpr int NT = 64 * WM * WN;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / 16, FN = WTN / 16;
  static constexpr int LPC = DeepLoader<BKD, BM, NT>::PER + DeepLoader<BKD, BN, NT>::PER;
  floatx4 out[4][FM][FN];
  floatx4 acc[4][FM][FN];
  DeepLoader<BKD, BM, NT> da;
  DeepLoader<BKD, BN, NT> db;
  const float4* Ug;
  const float4* Vg;
  size_t quadU, quadV;
  int N, T, nk, total, wm, wn, lr, lk;

  __device__ __forceinline__ void request(int c, float4 (*An)[BM], float4 (*Bn)[BN]) {
    const int q = c / nk, k0 = (c % nk) * BKD;
    da.load(Ug + (size_t)q * quadU, N, k0, An);
    db.load(Vg + (size_t)q * quadV, T, k0, Bn);
  }

  __device__ __forceinline__ void compute(const float4 (*Ac)[BM], const float4 (*Bc)[BN]) {
    if constexpr (SPLIT) {
      compute_split(Ac, Bc);
      return;
    }
#pragma unroll
    for (int kk = 0; kk < BKD / 4; ++kk) {
      float4 af[FM], bf[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[i] = Ac[kk * 4 + lk][wm * WTM + i * 16 + lr];
#pragma unroll
      for (int j = 0; j < FN; ++j) bf[j] = Bc[kk * 4 + lk][wn * WTN + j * 16 + lr];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          acc[0][i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].x, bf[j].x, acc[0][i][j], 0, 0, 0);
          acc[1][i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].y, bf[j].y, acc[1][i][j], 0, 0, 0);
          acc[2][i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].z, bf[j].z, acc[2][i][j], 0, 0, 0);
          if constexpr (!Q3)
            acc[3][i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].w, bf[j].w, acc[3][i][j], 0, 0, 0);
        }
    }
  }

  // Split precision: every LDS word is a packed (hi, lo) bf16 pair.  One
  // v_mfma_f32_16x16x32_bf16 per point takes the chunk's 8 channels: lane
  // group g = l / 16 holds channels 2g and 2g + 1, four K elements each,
  // so that every channel contributes all four partial products:
  //   U side (A): Uhi Ulo Uhi Ulo      (the pair word, twice)
  //   V side (B): Vhi Vlo Vlo Vhi      (the pair word, then its halves swapped)
  // and the sum over K is sum_m (Uhi + Ulo)(Vhi + Vlo), accumulated in fp32.
  __device__ __forceinline__ void compute_split(const float4 (*Ac)[BM], const float4 (*Bc)[BN]) {
    static_assert(BKD == 8, "one bf16 MFMA (K = 32) per 8-channel chunk");
    float4 ua[FM][2], vb[FN][2];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int c = 0; c < 2; ++c) ua[i][c] = Ac[2 * lk + c][wm * WTM + i * 16 + lr];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int c = 0; c < 2; ++c) vb[j][c] = Bc[2 * lk + c][wn * WTN + j * 16 + lr];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const uint32_t w0 = __float_as_uint(reinterpret_cast<const float*>(&ua[i][0])[q]);
        const uint32_t w1 = __float_as_uint(reinterpret_cast<const float*>(&ua[i][1])[q]);
        a[i] = __builtin_bit_cast(bf16x8, u32x4{w0, w0, w1, w1});
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const uint32_t w0 = __float_as_uint(reinterpret_cast<const float*>(&vb[j][0])[q]);
        const uint32_t w1 = __float_as_uint(reinterpret_cast<const float*>(&vb[j][1])[q]);
        b[j] = __builtin_bit_cast(bf16x8, u32x4{w0, __builtin_amdgcn_alignbit(w0, w0, 16), w1,
                                                __builtin_amdgcn_alignbit(w1, w1, 16)});
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[q][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[q][i][j], 0, 0, 0);
    }
  }

  __device__ __forceinline__ void fold(int q1r) {
    const float r0 = at_coef(0, q1r), r1 = at_coef(1, q1r);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const floatx4 z0 = acc[0][i][j] + acc[1][i][j] + acc[2][i][j];
        const floatx4 z1 = Q3 ? acc[1][i][j] - acc[2][i][j]
                              : acc[1][i][j] - acc[2][i][j] - acc[3][i][j];
        out[0][i][j] += r0 * z0;
        out[1][i][j] += r0 * z1;
        out[2][i][j] += r1 * z0;
        out[3][i][j] += r1 * z1;
#pragma unroll
        for (int c = 0; c < NQ; ++c) acc[c][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
  }

  // one pipeline step on buffer (Ac, Bc) for chunk it; chunk it+STAGES-1
  // (clamped to the last chunk, into a buffer that is then never read) is
  // requested into (An, Bn), so every step issues the same loads and exactly
  // STAGES-2 chunks are always requested after chunk it when it is waited for
  __device__ __forceinline__ void step(int it, const float4 (*Ac)[BM], const float4 (*Bc)[BN],
                                       float4 (*An)[BM], float4 (*Bn)[BN]) {
    wait_vmcnt<(STAGES - 2) * LPC>();
    __builtin_amdgcn_s_barrier();
    const int c = it + STAGES - 1;
    request(c < total ? c : total - 1, An, Bn);
    compute(Ac, Bc);
  }
};

// Two wavefronts per SIMD for 32 x 32 wavefront tiles; a 64 x 32 tile (eight
// accumulator sets of 8 floatx4) needs the whole register file, one per SIMD.
template <int BM, int BN, int WM, int WN, int BKD, int STAGES, bool SPLIT, bool Q3>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu((BM / WM) * (BN / WN) > 1024 ? 1 : 2))) void contract_deep(
    const float4* __restrict__ U, const float4* __restrict__ V, float4* __restrict__ Z, int M,
    int N, int T, int ntb, int nnb, int ks, GroupMap gm) {
  using Tile = DeepTile<BM, BN, WM, WN, BKD, STAGES, SPLIT, Q3>;
  constexpr int WTM = Tile::WTM, WTN = Tile::WTN, FM = Tile::FM, FN = Tile::FN;
  static_assert(WM * WN == 4 || WM * WN == 8, "four or eight waves");
  static_assert(STAGES >= 2 && STAGES <= 4, "2 to 4 stages");
  __shared__ float4 A0[BKD][BM], A1[BKD][BM], A2[STAGES > 2 ? BKD : 1][BM],
      A3[STAGES > 3 ? BKD : 1][BM];
  __shared__ float4 B0[BKD][BN], B1[BKD][BN], B2[STAGES > 2 ? BKD : 1][BN],
      B3[STAGES > 3 ? BKD : 1][BN];

  long long bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tb = (int)(bid % ntb);
  bid /= ntb;
  const int nb = (int)(bid % nnb);
  bid /= nnb;
  // K slices (ks > 1): slice sk takes channels [sk M/ks, (sk+1) M/ks) and
  // writes its partial Z to part sk (parts of G N T quads, back to back)
  const int sk = (int)(bid % ks);
  const long long g = live_group(gm, bid / ks);   // ks > 1 only with every group live
  const long long G = (long long)gridDim.x / ((long long)ntb * nnb * ks);
  const int mk = M / ks;
  const int n0 = nb * BM, c0 = tb * BN;

  Tile tile;
  tile.quadU = (size_t)M * N;
  tile.quadV = (size_t)M * T;
  tile.Ug = U + (size_t)(4 * g) * tile.quadU + (size_t)sk * mk * N;
  tile.Vg = V + (size_t)(4 * g) * tile.quadV + (size_t)sk * mk * T;
  tile.N = N;
  tile.T = T;
  tile.nk = mk / BKD;
  tile.total = Tile::NQ * tile.nk;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  tile.wm = wave / WN;
  tile.wn = wave % WN;
  tile.lr = lane & 15;
  tile.lk = lane >> 4;
#pragma unroll
  for (int o = 0; o < 4; ++o)
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        tile.out[o][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
        tile.acc[o][i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
  tile.da.init(N, n0, N);
  tile.db.init(T, c0, T);

  // prologue: chunks 0 .. STAGES-2 (the K loop has nk % STAGES == 0 chunks per q1r)
  tile.request(0, A0, B0);
  if (STAGES > 2) tile.request(1, A1, B1);
  if (STAGES > 3) tile.request(2, A2, B2);
  for (int q1r = 0; q1r < Tile::NQ; ++q1r) {
    for (int kb = 0; kb < tile.nk; kb += STAGES) {
      const int c = q1r * tile.nk + kb;
      if (STAGES == 2) {
        tile.step(c, A0, B0, A1, B1);
        tile.step(c + 1, A1, B1, A0, B0);
      } else if (STAGES == 3) {
        tile.step(c, A0, B0, A2, B2);
        tile.step(c + 1, A1, B1, A0, B0);
        tile.step(c + 2, A2, B2, A1, B1);
      } else {
        tile.step(c, A0, B0, A3, B3);
        tile.step(c + 1, A1, B1, A0, B0);
        tile.step(c + 2, A2, B2, A1, B1);
        tile.step(c + 3, A3, B3, A2, B2);
      }
    }
    tile.fold(q1r);
  }

  float4* __restrict__ Zg = Z + (size_t)(sk * G + g) * N * T;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = n0 + tile.wm * WTM + i * 16 + tile.lk * 4 + v;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = c0 + tile.wn * WTN + j * 16 + tile.lr;
        if (col < T)
          Zg[(size_t)row * T + col] = make_float4(tile.out[0][i][j][v], tile.out[1][i][j][v],
                                                  tile.out[2][i][j][v], tile.out[3][i][j][v]);
      }
    }
  }
}

// Persistent form of contract_deep: one work-group per CU slot walks a list
// of (column tile, row tile, K slice, group) items, and its load pipeline
// runs on across items, so the first chunks of item i+1 stream in while
// item i's last chunks are multiplied and its Z tile is stored (a fresh
// work-group would start with an empty pipeline).  Items are numbered as
// in contract_deep; XCD x takes a contiguous range of them (the split of
// xcd_remap) and its wpx work-groups stride through that range, so the
// tiles that share a group's U and V run together on one L2.
template <int BM, int BN, int WM, int WN, int BKD, int STAGES, bool SPLIT, bool Q3>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu((BM / WM) * (BN / WN) > 1024 ? 1 : 2))) void contract_deep_persist(
    const float4* __restrict__ U, const float4* __restrict__ V, float4* __restrict__ Z, int M,
    int N, int T, int ntb, int nnb, int ks, long long G, int wpx, GroupMap gm) {
  using Tile = DeepTile<BM, BN, WM, WN, BKD, STAGES, SPLIT, Q3>;
  constexpr int WTM = Tile::WTM, WTN = Tile::WTN, FM = Tile::FM, FN = Tile::FN;
  static_assert(WM * WN == 4 || WM * WN == 8, "four or eight waves");
  static_assert(STAGES == 4, "4 stages");
  __shared__ float4 A0[BKD][BM], A1[BKD][BM], A2[BKD][BM], A3[BKD][BM];
  __shared__ float4 B0[BKD][BN], B1[BKD][BN], B2[BKD][BN], B3[BKD][BN];

  // this work-group's items: first + i * wpx, i < mine
  const long long items = (long long)ntb * nnb * ks * G;
  const int xcd = blockIdx.x % 8, j = blockIdx.x / 8;
  const long long q = items / 8, rem = items % 8;
  const long long xstart = xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q;
  const long long xcount = q + (xcd < rem ? 1 : 0);
  const int mine = xcount > j ? (int)((xcount - 1 - j) / wpx + 1) : 0;
  if (mine == 0) return;                    // uniform over the work-group
  const long long first = xstart + j;
  const int mk = M / ks;

  Tile tile;
  tile.quadU = (size_t)M * N;
  tile.quadV = (size_t)M * T;
  tile.N = N;
  tile.T = T;
  tile.nk = mk / BKD;
  tile.total = Tile::NQ * tile.nk;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  tile.wm = wave / WN;
  tile.wn = wave % WN;
  tile.lr = lane & 15;
  tile.lk = lane >> 4;
#pragma unroll
  for (int o = 0; o < 4; ++o)
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int jj = 0; jj < FN; ++jj) {
        tile.out[o][i][jj] = floatx4{0.f, 0.f, 0.f, 0.f};
        tile.acc[o][i][jj] = floatx4{0.f, 0.f, 0.f, 0.f};
      }

  // request cursor: item ri, chunk rc (tile.Ug / tile.Vg and the loaders
  // follow the requested item)
  int ri = 0, rc = 0;
  auto set_req_item = [&](int i) {
    long long b = first + (long long)i * wpx;
    const int tb = (int)(b % ntb);
    b /= ntb;
    const int nb = (int)(b % nnb);
    b /= nnb;
    const int sk = (int)(b % ks);
    const long long g = live_group(gm, b / ks);
    tile.Ug = U + (size_t)(4 * g) * tile.quadU + (size_t)sk * mk * N;
    tile.Vg = V + (size_t)(4 * g) * tile.quadV + (size_t)sk * mk * T;
    tile.da.init(N, nb * BM, N);
    tile.db.init(T, tb * BN, T);
  };
  // past the last item the last chunk is requested again, into a buffer
  // that is never read, so every step issues the same loads
  auto request_next = [&](float4 (*An)[BM], float4 (*Bn)[BN]) {
    tile.request(rc, An, Bn);
    if (rc + 1 < tile.total) {
      ++rc;
    } else if (ri + 1 < mine) {
      ++ri;
      rc = 0;
      set_req_item(ri);
    }
  };
  auto step = [&](const float4 (*Ac)[BM], const float4 (*Bc)[BN], float4 (*An)[BM],
                  float4 (*Bn)[BN]) {
    wait_vmcnt<(STAGES - 2) * Tile::LPC>();
    __builtin_amdgcn_s_barrier();
    request_next(An, Bn);
    tile.compute(Ac, Bc);
  };

  set_req_item(0);
  request_next(A0, B0);
  request_next(A1, B1);
  request_next(A2, B2);
  for (int it = 0; it < mine; ++it) {
    for (int q1r = 0; q1r < Tile::NQ; ++q1r) {
      for (int kb = 0; kb < tile.nk; kb += STAGES) {
        step(A0, B0, A3, B3);
        step(A1, B1, A0, B0);
        step(A2, B2, A1, B1);
        step(A3, B3, A2, B2);
      }
      tile.fold(q1r);
    }
    long long b = first + (long long)it * wpx;
    const int tb = (int)(b % ntb);
    b /= ntb;
    const int nb = (int)(b % nnb);
    b /= nnb;
    const int sk = (int)(b % ks);
    const long long g = live_group(gm, b / ks);
    const int n0 = nb * BM, c0 = tb * BN;
    float4* __restrict__ Zg = Z + (size_t)(sk * G + g) * N * T;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = n0 + tile.wm * WTM + i * 16 + tile.lk * 4 + v;
#pragma unroll
        for (int jj = 0; jj < FN; ++jj) {
          const int col = c0 + tile.wn * WTN + jj * 16 + tile.lr;
          if (col < T)
            Zg[(size_t)row * T + col] = make_float4(tile.out[0][i][jj][v], tile.out[1][i][jj][v],
                                                    tile.out[2][i][jj][v], tile.out[3][i][jj][v]);
        }
      }
    }
#pragma unroll
    for (int o = 0; o < 4; ++o)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int jj = 0; jj < FN; ++jj) tile.out[o][i][jj] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  wait_vmcnt<0>();                          // the clamped tail loads land before exit
}

// ---------------------------------------------------------------------------
// Planar contraction of the mixed nest (nwg_plan_info::mix_planar).  U and V
// hold each live group's 9 live points (3 x 3 level-1 digits, the fourth
// digit dead) as plain matrices, U[i][p][M][N] and V[i][p][M][T], so that
// no dead point is loaded.  An item is a 128 x 64 block of (n, t) of one
// group; four wavefronts of 64 x 32.  A chunk is 32 channels of one point,
// loaded straight to LDS as float4 along n (A) and t (B).  A lane's float4
// of A (n = 4 r + c) feeds four MFMA row blocks c and its float2 of B
// (t = 2 r + b) two column blocks b, so every MFMA block takes every fourth
// row and every second column of the wavefront's tile.  After a point's
// channel sweep its products are folded into the four level-1 outputs with
// A^T[i1r][q1r] A^T[i1c][q1c].  Persistent like contract_deep_persist.
// ---------------------------------------------------------------------------
constexpr int kPlBM = 128, kPlBN = 64, kPlBK = 32;   // n rows, t columns, channels per chunk

struct PlanarTile {
  using LA = DeepLoader<kPlBK, kPlBM / 4, 256>;
  using LB = DeepLoader<kPlBK, kPlBN / 4, 256>;
  static constexpr int LPC = LA::PER + LB::PER;     // loads per thread per chunk
  floatx4 acc[4][2];        // [c][b]: rows 4 r + c, columns 2 r' + b of the wave's tile
  floatx4 out[4][4][2];     // level-1 outputs 2 i1r + i1c
  LA da;
  LB db;
  const float4* Ug;
  const float4* Vg;
  size_t ptU, ptV;          // float4 between points: M N / 4, M T / 4
  int ldU, ldV, nk, total, wm, wn, lr, lk;

  __device__ __forceinline__ void request(int c, float4 (*An)[kPlBM / 4],
                                          float4 (*Bn)[kPlBN / 4]) {
    const int p = c / nk, k0 = (c % nk) * kPlBK;
    da.load(Ug + (size_t)p * ptU, ldU, k0, An);
    db.load(Vg + (size_t)p * ptV, ldV, k0, Bn);
  }

  __device__ __forceinline__ void compute(const float4 (*Ac)[kPlBM / 4],
                                          const float4 (*Bc)[kPlBN / 4]) {
#pragma unroll
    for (int kk = 0; kk < kPlBK / 4; ++kk) {
      const float4 a = Ac[kk * 4 + lk][wm * 16 + lr];
      const float2 b = reinterpret_cast<const float2*>(&Bc[kk * 4 + lk][0])[wn * 16 + lr];
      const float av[4] = {a.x, a.y, a.z, a.w}, bv[2] = {b.x, b.y};
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[c][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[c], bv[j], acc[c][j], 0, 0, 0);
    }
  }

  // point p = 3 q1r + q1c done: out[2 i1r + i1c] += A^T[i1r][q1r] A^T[i1c][q1c] acc
  __device__ __forceinline__ void fold(int p) {
    const int q1r = p / 3, q1c = p - 3 * q1r;
    const float r1 = at_coef(1, q1r), c1 = at_coef(1, q1c);   // A^T[0][q] = 1 for q < 3
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const floatx4 a = acc[c][j];
        out[0][c][j] += a;
        out[1][c][j] += c1 * a;
        out[2][c][j] += r1 * a;
        out[3][c][j] += (r1 * c1) * a;
        acc[c][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
  }
};

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1))) void contract_planar_persist(
    const float4* __restrict__ U, const float4* __restrict__ V, float4* __restrict__ Z, int M,
    int N, int T, int ntb, int nnb, long long G, int wpx, GroupMap gm) {
  constexpr int CA = kPlBM / 4, CB = kPlBN / 4;
  __shared__ float4 A0[kPlBK][CA], A1[kPlBK][CA], A2[kPlBK][CA], A3[kPlBK][CA];
  __shared__ float4 B0[kPlBK][CB], B1[kPlBK][CB], B2[kPlBK][CB], B3[kPlBK][CB];

  // this work-group's items: first + i * wpx, i < mine (as contract_deep_persist)
  const long long items = (long long)ntb * nnb * G;
  const int xcd = blockIdx.x % 8, j = blockIdx.x / 8;
  const long long q = items / 8, rem = items % 8;
  const long long xstart = xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q;
  const long long xcount = q + (xcd < rem ? 1 : 0);
  const int mine = xcount > j ? (int)((xcount - 1 - j) / wpx + 1) : 0;
  if (mine == 0) return;                    // uniform over the work-group
  const long long first = xstart + j;

  PlanarTile tile;
  tile.ptU = (size_t)M * (N / 4);
  tile.ptV = (size_t)M * (T / 4);
  tile.ldU = N / 4;
  tile.ldV = T / 4;
  tile.nk = M / kPlBK;
  tile.total = 9 * tile.nk;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  tile.wm = wave / 2;
  tile.wn = wave % 2;
  tile.lr = lane & 15;
  tile.lk = lane >> 4;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      tile.acc[c][jj] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int o = 0; o < 4; ++o) tile.out[o][c][jj] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

  // request cursor: item ri, chunk rc
  int ri = 0, rc = 0;
  auto set_req_item = [&](int i) {
    long long b = first + (long long)i * wpx;
    const int tb = (int)(b % ntb);
    b /= ntb;
    const int nb = (int)(b % nnb);
    const long long li = b / nnb;             // place in the live list
    tile.Ug = U + (size_t)li * 9 * tile.ptU;
    tile.Vg = V + (size_t)li * 9 * tile.ptV;
    tile.da.init(tile.ldU, nb * CA, tile.ldU);
    tile.db.init(tile.ldV, tb * CB, tile.ldV);
  };
  // past the last item the last chunk is requested again, into a buffer
  // that is never read, so every step issues the same loads
  auto request_next = [&](float4 (*An)[CA], float4 (*Bn)[CB]) {
    tile.request(rc, An, Bn);
    if (rc + 1 < tile.total) {
      ++rc;
    } else if (ri + 1 < mine) {
      ++ri;
      rc = 0;
      set_req_item(ri);
    }
  };
  auto step = [&](const float4 (*Ac)[CA], const float4 (*Bc)[CB], float4 (*An)[CA],
                  float4 (*Bn)[CB]) {
    wait_vmcnt<2 * PlanarTile::LPC>();
    __builtin_amdgcn_s_barrier();
    request_next(An, Bn);
    tile.compute(Ac, Bc);
  };

  set_req_item(0);
  request_next(A0, B0);
  request_next(A1, B1);
  request_next(A2, B2);
  for (int it = 0; it < mine; ++it) {
    for (int p = 0; p < 9; ++p) {
      for (int kb = 0; kb < tile.nk; kb += 4) {
        step(A0, B0, A3, B3);
        step(A1, B1, A0, B0);
        step(A2, B2, A1, B1);
        step(A3, B3, A2, B2);
      }
      tile.fold(p);
    }
    long long b = first + (long long)it * wpx;
    const int tb = (int)(b % ntb);
    b /= ntb;
    const int nb = (int)(b % nnb);
    const long long g = live_group(gm, b / nnb);
    float4* __restrict__ Zg = Z + (size_t)g * N * T;
    const int n0 = nb * kPlBM + tile.wm * 64, t0 = tb * kPlBN + tile.wn * 32;
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = n0 + 4 * (4 * tile.lk + v) + c;
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int col = t0 + 2 * tile.lr + jj;
          Zg[(size_t)row * T + col] = make_float4(tile.out[0][c][jj][v], tile.out[1][c][jj][v],
                                                  tile.out[2][c][jj][v], tile.out[3][c][jj][v]);
        }
      }
#pragma unroll
    for (int o = 0; o < 4; ++o)
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) tile.out[o][c][jj] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  wait_vmcnt<0>();                          // the clamped tail loads land before exit
}

// Work-groups of a persistent kernel that fit on one CU of device dev, asked
// once per (device, kernel) and kept; 0 if the query fails.  Safe to call
// from several threads.
int persist_occupancy(int dev, const void* kernel, int threads) {
  static std::mutex mu;
  static std::map<std::pair<int, const void*>, int> cache;
  std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_pair(dev, kernel);
  const auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int b = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, kernel, threads, 0) != hipSuccess) {
    hipGetLastError();
    b = 0;
  }
  cache[key] = b;
  return b;
}

template <int BM, int BN, int WM, int WN, int BKD, int STAGES, bool SPLIT = false,
          bool Q3 = false>
hipError_t launch_deep(const float* U, const float* V, float* Z, int M, int N, int T,
                       long long G, hipStream_t s, int ks, const GroupMap& gm) {
  // T need not be a multiple of BN: the last column tile is ragged
  const int ntb = (T + BN - 1) / BN, nnb = N / BM;
  const long long blocks = (long long)ntb * nnb * G * ks;
  if (ks < 1 || N % BM || M % (BKD * STAGES * ks) || blocks <= 0 || blocks > 0x7fffffffLL)
    return hipErrorInvalidValue;
  if (((uintptr_t)U | (uintptr_t)V | (uintptr_t)Z) & 15) return hipErrorInvalidValue;
  if ((long long)M * (N > T ? N : T) > 0x7fffffffLL / 4) return hipErrorInvalidValue;
  if (STAGES == 4) {
    // one work-group per CU slot when every slot gets at least 4 items
    int dev = 0, cus = 0;
    const int occ =
        hipGetDevice(&dev) == hipSuccess
            ? persist_occupancy(dev, reinterpret_cast<const void*>(
                                         &contract_deep_persist<BM, BN, WM, WN, BKD, 4, SPLIT, Q3>),
                                64 * WM * WN)
            : 0;
    if (occ > 0 &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus >= 8) {
      const int wpx = cus / 8 * occ;
      if (blocks >= 4LL * 8 * wpx) {
        hipLaunchKernelGGL((contract_deep_persist<BM, BN, WM, WN, BKD, 4, SPLIT, Q3>),
                           dim3((unsigned)(8 * wpx)), dim3(64 * WM * WN), 0, s, (const float4*)U,
                           (const float4*)V, (float4*)Z, M, N, T, ntb, nnb, ks, G, wpx, gm);
        return hipGetLastError();
      }
    }
  }
  hipLaunchKernelGGL((contract_deep<BM, BN, WM, WN, BKD, STAGES, SPLIT, Q3>), dim3((unsigned)blocks),
                     dim3(64 * WM * WN), 0, s, (const float4*)U, (const float4*)V, (float4*)Z,
                     M, N, T, ntb, nnb, ks, gm);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_fused(const float* U, const float* V, float* Z, int M, int N, int T,
                        long long G, hipStream_t s, const GroupMap& gm) {
  const int ntb = (T + BN - 1) / BN;
  const int nnb = (N + BM - 1) / BM;
  const long long blocks = (long long)ntb * nnb * G;
  if (blocks <= 0 || blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  if (((uintptr_t)U | (uintptr_t)V | (uintptr_t)Z) & 15) return hipErrorInvalidValue;
  if ((long long)M * (N > T ? N : T) > 0x7fffffffLL / 4) return hipErrorInvalidValue;
  const bool full = N % BM == 0 && T % BN == 0 && M % kBK == 0;
  if (full)
    hipLaunchKernelGGL((contract_fused<BM, BN, WM, WN, true>), dim3((unsigned)blocks), dim3(256),
                       0, s, (const float4*)U, (const float4*)V, (float4*)Z, M, N, T, ntb, nnb, gm);
  else
    hipLaunchKernelGGL((contract_fused<BM, BN, WM, WN, false>), dim3((unsigned)blocks), dim3(256),
                       0, s, (const float4*)U, (const float4*)V, (float4*)Z, M, N, T, ntb, nnb, gm);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Plain GEMM for depth 0: C[b] (N x HW) = A^T (N x M) * B[b] (M x HW)
// ---------------------------------------------------------------------------

__host__ __device__ constexpr int lds_stride(int cols) {
  return ((cols + 16) % 32 == 16) ? cols + 16 : cols + 32;
}

template <int COLS, int SROW>
struct TileLoader {
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
__global__ __launch_bounds__(256) void gemm_mfma(ContractArgs a, int ntb, int nnb, int vecA,
                                                 int vecB) {
  constexpr int SA = lds_stride(BM), SB = lds_stride(BN);
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  static_assert(WM * WN == 4, "four waves");
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
hipError_t launch_gemm(const ContractArgs& a, hipStream_t s) {
  const int ntb = (a.Ncols + BN - 1) / BN;
  const int nnb = (a.Nrows + BM - 1) / BM;
  const long long blocks = (long long)ntb * nnb * a.batch;
  if (blocks <= 0 || blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  auto aligned = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  const int vecA = (a.ldA % 4 == 0) && (a.Nrows % 4 == 0) && (a.sA % 4 == 0) && aligned(a.A);
  const int vecB = (a.ldB % 4 == 0) && (a.Ncols % 4 == 0) && (a.sB % 4 == 0) && aligned(a.Bm);
  hipLaunchKernelGGL((gemm_mfma<BM, BN, WM, WN>), dim3((unsigned)blocks), dim3(256), 0, s, a,
                     ntb, nnb, vecA, vecB);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_contract_planar(const float* U, const float* V, float* Z, int M, int N, int T,
                                  long long G, const GroupMap& gm, hipStream_t s) {
  if (M <= 0 || N <= 0 || T <= 0 || G <= 0 || gm.np <= 0 || G != (long long)gm.np * gm.np)
    return hipErrorInvalidValue;
  if (M % (4 * kPlBK) || N % kPlBM || T % kPlBN) return hipErrorInvalidValue;
  if (((uintptr_t)U | (uintptr_t)V | (uintptr_t)Z) & 15) return hipErrorInvalidValue;
  const long long items = (long long)(T / kPlBN) * (N / kPlBM) * G;
  if (items > 0x7fffffffLL) return hipErrorInvalidValue;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int occ =
      persist_occupancy(dev, reinterpret_cast<const void*>(&contract_planar_persist), 256);
  if (occ <= 0 || cus < 8) return hipErrorInvalidValue;
  const int wpx = cus / 8 * occ;            // work-groups per XCD, one per CU slot
  hipLaunchKernelGGL(contract_planar_persist, dim3((unsigned)(8 * wpx)), dim3(256), 0, s,
                     (const float4*)U, (const float4*)V, (float4*)Z, M, N, T, T / kPlBN,
                     N / kPlBM, G, wpx, gm);
  return hipGetLastError();
}

hipError_t launch_gemm_depth0(const ContractArgs& a, hipStream_t s) {
  const int N = a.Nrows;
  if (N <= 16) return launch_gemm<16, 128, 1, 4>(a, s);
  if (N <= 32) return launch_gemm<32, 128, 1, 4>(a, s);
  if (N <= 64) return launch_gemm<64, 128, 2, 2>(a, s);
  return launch_gemm<128, 128, 2, 2>(a, s);
}

hipError_t launch_contract_fused(const float* U, const float* V, float* Z, int M, int N, int T,
                                 long long G, hipStream_t s, bool split, int ks,
                                 const GroupMap& gm) {
  // a group list (live groups) needs whole groups per Z part
  if (gm.np != 0 && (ks != 1 || G != (long long)gm.np * gm.np)) return hipErrorInvalidValue;
  if (gm.q3 && (split || ks != 1)) return hipErrorInvalidValue;
  // split precision and K slices: the deep pipeline only (full 64-row
  // tiles, whole sweeps)
  if (split || ks > 1) {
    if (M % (32 * ks) || N % 64 || T < 64) return hipErrorInvalidValue;
    if (split) {
      if (T % 128 == 0) return launch_deep<64, 128, 2, 4, 8, 4, true>(U, V, Z, M, N, T, G, s, ks, gm);
      return launch_deep<64, 64, 2, 2, 8, 4, true>(U, V, Z, M, N, T, G, s, ks, gm);
    }
    if (T % 128 == 0) return launch_deep<64, 128, 2, 4, 8, 4>(U, V, Z, M, N, T, G, s, ks, gm);
    return launch_deep<64, 64, 2, 2, 8, 4>(U, V, Z, M, N, T, G, s, ks, gm);
  }
  // full 64-row tiles and whole 4-stage K sweeps: the deep pipeline; a
  // ragged T takes 64-column tiles (the last one partly recomputed)
  if (M % 32 == 0 && N % 64 == 0) {
    if (gm.q3) {
      if (T % 128 == 0)
        return launch_deep<64, 128, 2, 4, 8, 4, false, true>(U, V, Z, M, N, T, G, s, 1, gm);
      if (T == 64 && N % 128 == 0)
        return launch_deep<128, 64, 2, 2, 8, 4, false, true>(U, V, Z, M, N, T, G, s, 1, gm);
      if (T >= 64)
        return launch_deep<64, 64, 2, 2, 8, 4, false, true>(U, V, Z, M, N, T, G, s, 1, gm);
    }
    if (T % 128 == 0) return launch_deep<64, 128, 2, 4, 8, 4>(U, V, Z, M, N, T, G, s, 1, gm);
    // T = 64 with N a multiple of 128 (e.g. the mixed nest's 31x31 layer):
    // 128 x 64 blocks, so that V is read once per group (3.52 -> 3.44 ms)
    if (T == 64 && N % 128 == 0)   // four wavefronts of 64 x 32 (one per SIMD): 3.43 -> 3.38 ms
      return launch_deep<128, 64, 2, 2, 8, 4>(U, V, Z, M, N, T, G, s, 1, gm);
    // a ragged T: 64-column tiles, the last one partly recomputed (on the
    // 13x13 layer, T = 392, this measured 163 us against 173 us for the whole
    // tiles plus a separate launch of 64 x 16 blocks for the last 8 columns,
    // which re-reads all of U)
    if (T >= 64) return launch_deep<64, 64, 2, 2, 8, 4>(U, V, Z, M, N, T, G, s, 1, gm);
  }
  // small problems (fewer than 256 work-groups with the wide tiles, e.g.
  // 32 channels on 256 tiles at depth 2: 32 work-groups): 16 x 64 tiles
  const long long wide = (long long)((T + 127) / 128) * ((N + 31) / 32) * G;
  if (N <= 32 && wide < 256) return launch_fused<16, 64, 1, 4>(U, V, Z, M, N, T, G, s, gm);
  if (N <= 16) return launch_fused<16, 128, 1, 4>(U, V, Z, M, N, T, G, s, gm);
  if (N <= 32) return launch_fused<32, 128, 1, 4>(U, V, Z, M, N, T, G, s, gm);
  return launch_fused<64, 64, 2, 2>(U, V, Z, M, N, T, G, s, gm);
}

}  // namespace nwg
