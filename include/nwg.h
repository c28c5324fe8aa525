/*
 * nwg.h -- nested-Winograd stride-1 2D convolution on MI355X (gfx950).
 *
 * Operation (Sec. II.A of "Accelerating Large Kernel Convolutions with
 * Nested Winograd Transformation", Jiang, Chen, Tsui): M input maps x of
 * size H x W are correlated with N groups of M-channel r x r kernels w,
 * stride 1, zero padding `pad` on all four sides, giving N output maps y:
 *
 *   y[b][n][i][j] = sum_{m,u,v} xpad[b][m][i+u][j+v] * w[n][m][u][v],
 *   0 <= i < Ho = H + 2 pad - r + 1,  0 <= j < Wo = W + 2 pad - r + 1.
 *
 * Computed by nested Winograd (Sec. III.B) on the fixed base F(2x2, 3x3)
 * (eq. 2.3): the r x r kernel is handled by an n-level nest of the base,
 * n = smallest depth whose padded kernel K_n = 2^(n+1) - 1 >= r
 * (r = 1: n = 0, no transform; r <= 3: n = 1; r <= 7: 2; r <= 15: 3;
 * r <= 31: 4).  Level j works at stride 2^(j-1); each tile produces
 * M_n = 2^n x 2^n outputs from an L_n x L_n input window, L_n = 3*2^n - 2,
 * through P = 4^(2n) Winograd points.
 *
 * Data: all tensors are contiguous fp32 in DEVICE memory.
 *   x [B][M][H][W],  w [N][M][r][r],  y [B][N][Ho][Wo].
 * Winograd-domain buffers (what the stage entry points read and write),
 * "quad-interleaved": the level-1 column digit is the innermost axis, so
 * each (channel, tile) entry is a 16-byte float4 quad:
 *   U [P/4][M][N][4]  transformed kernel, U[p/4][m][n][p%4]
 *   V [P/4][M][T][4]  transformed input,  V[p/4][m][t][p%4]
 *   Z [P/16][N][T][4] channel contraction after the first output level:
 *       Z[g][n][t][2*i1r + i1c] = sum over the 16 points p = 16g + 4 q1r + q1c
 *       of A^T[i1r][q1r] A^T[i1c][q1c] sum_m U[p][m][n] V[p][m][t]
 * with T = B * th * tw tiles, th = ceil(Ho / M_n), tw = ceil(Wo / M_n), and
 * tile t = (b * th + ty) * tw + tx covering outputs [ty*M_n, ty*M_n + M_n) x
 * [tx*M_n, tx*M_n + M_n).  The point index p of a tile is written in base 4
 * with digits (q_n^row, q_n^col, q_{n-1}^row, q_{n-1}^col, ..., q_1^row,
 * q_1^col), most significant first, q_j being the level-j Winograd index.
 * At depth 0 (r = 1) there is no transform: U is [M][N] and the contraction
 * maps x to y directly.  All buffers must be 16-byte aligned.
 * Mixed-nest plans (NWG_TILE_MIX_F23_F33) compute only the points whose
 * transformed kernel can be nonzero (nwg_plan_info live_np, live_prefix,
 * level1_live): the stage calls neither write nor read the dead groups'
 * U, V and Z, nor the quads of a dead level-1 row digit; with mix_planar
 * set, U and V hold only the live points, in the planar layout described
 * at that field.  Z keeps the layout above.  Unfused dense F(2x2,3x3)
 * plans at depth 3 and 4 with live_np > 0 skip their dead groups the same
 * way, keeping the layout above: the kernel transform writes every group
 * of U, the input transform writes only the live groups of V (every group
 * when 256 M T quads of 16 bytes exceed 2^30 bytes), the contraction reads
 * only the live groups of U and V and writes only their Z, and the output
 * transform reads only their Z.
 *
 * Ownership: the caller owns x, w, y, U/V/Z passed to stage calls, and
 * the stream; they must stay valid until the work queued on the stream has
 * finished.  A plan owns its workspace (U, V, Z; workspace_bytes),
 * allocated at creation; V is left out when info.fused_input is set, V and
 * Z when info.fused_conv is set (the stage calls still work on caller
 * buffers).
 * Every call that takes a stream only queues work on it (`stream` is a
 * hipStream_t; NULL is the default stream of the current device) and never
 * synchronises, except nwg_plan_get_timing.  A call that uses a plan's
 * workspace needs the device the plan was created on to be current and the
 * stream to belong to it (NWG_EINVAL otherwise).  A plan is not thread-safe;
 * one call in flight per plan.
 *
 * Errors: functions returning int give NWG_OK (0) or a negative status;
 * functions returning a pointer give NULL.  nwg_last_error() then returns a
 * message, and nwg_last_status() the status (for a NULL pointer: why), for
 * the calling thread.  A launch that fails returns NWG_EHIP; a kernel that
 * fails while it runs is reported by the stream's next synchronising call,
 * or, with the environment variable NWG_DEBUG_SYNC set, by the call that
 * queued it (every call then waits for each kernel it queues: a debugging
 * aid, not for use under stream capture).
 *
 * Limits: each input and output map holds fewer than 2^31 values, and no
 * tensor or workspace buffer more than 1e13 bytes (NWG_EUNSUPPORTED).
 */
#ifndef NWG_H
#define NWG_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nwg_plan nwg_plan;

/* Winograd base of the nest.
 *   NWG_TILE_F2X2_3X3: F(2x2, 3x3) (eq. 2.3), depth 0-4 (r <= 31), the layouts
 *     above.
 *   NWG_TILE_F3X3_3X3: F(3x3, 3x3), dense plans at depth 1-2 only (r <= 9):
 *     strides 1, 3, M_n = K_n = 3^n, L_n = 5 or 17, P = 5^(2n) points with
 *     base-5 digits (q_n^row, q_n^col, ..., q_1^row, q_1^col); Toom-Cook
 *     points 0, 1, -1, 2, infinity.  Plain layouts (no quads):
 *       U [P][M][N], V [P][M][T],
 *       Z [P/25][5][3][N][T], the level-1 output transform along the
 *         columns only: Z[g][q1r][i1c][n][t] = sum over q1c of
 *         A^T[i1c][q1c] Yhat[25g + 5 q1r + q1c][n][t]
 *     (A^T rows [1,1,1,1,0], [0,1,-1,2,0], [0,1,1,4,1]).
 *     Depth 0 (r = 1) is the plain contraction as for F(2x2, 3x3).  With one
 *     output channel at depth 2, nwg_conv2d runs a fused kernel (x -> Z
 *     without V, fused_input = 1; the plan holds U and per input-channel-group
 *     partial sums of Z instead of V and Z) and the output transform; the
 *     stage calls keep the layouts above, and nwg_input_contract is not
 *     available on this tile.  With one or two input channels (and not that
 *     case) the output transform forms the contraction itself from V and U
 *     (fused_output = 1, no Z).  Otherwise fused_input = fused_conv = 0 and
 *     pipeline_parts = 1.
 *   NWG_TILE_AUTO: the plan takes F(3x3,3x3) where it measured faster on
 *     MI355X -- one output channel at depth 2 or one or two input channels
 *     (its fused kernels; unless the F(2x2,3x3) plan runs the layer in one
 *     kernel), or M, N >= 32 and either r = 8..9 (one nesting level fewer)
 *     or r <= 3 --, the mixed nest NWG_TILE_MIX_F23_F33 (below) for dense
 *     plans with r = 16..31 and M, N >= 32 when a roofline model of the two
 *     plans' steps (their algorithmic bytes at 5 TB/s, their MFMA work on
 *     whole 64-column tiles at 100 TFLOP/s) expects it to be faster -- it has
 *     1.6x fewer contraction FLOPs per output but 2.4x the transformed
 *     weights, and few 36 x 36 tiles leave its MFMA tiles mostly empty --,
 *     and F(2x2,3x3) otherwise (always for depthwise plans).  info.tile
 *     reports the tile taken. */
/*   NWG_TILE_LD_F2X2_3X3: the linear decomposition of Sec. II.B (Fig. 2),
 *     the method the paper compares nesting with, on the same F(2x2,3x3)
 *     kernels: the r x r kernel is cut into c x c sub-kernels of 3 x 3
 *     (c = ceil(r/3), zero-padded at the end), sub-kernel (cu, cv) meets the
 *     input window moved by (3 cu, 3 cv), and the Winograd-domain products
 *     of all sub-kernels and input channels are summed before one output
 *     transform.  The plan is a depth-1 plan (n = 1, P = 16, M_n = 2,
 *     K_n = 3c, L_n = 3c + 1, info.ld_c = c) whose contraction runs over
 *     M c^2 channels, channel (cu c + cv) M + m: U [4][M c^2][N][4],
 *     V [4][M c^2][T][4], Z [1][N][T][4].  Dense fp32 plans only. */
/*   NWG_TILE_MIX_F23_F33: a nest with a different base per level (the level
 *     recurrence of Sec. III.B does not need the levels to share a base):
 *     F(2,3) at levels 1 and 2 and F(3,3) (the points above) at the
 *     info.outer33 = n - 2 levels above them, strides 1, 2, 4, 12:
 *       r = 8..15:  n = 3, M_n = 12, K_n = 15, L_n = 26, P = 80^2 = 6400;
 *       r = 16..39: n = 4, M_n = 36, K_n = 39, L_n = 74, P = 400^2 = 160000
 *     (31 x 31: 123 general multiplications per output, 256 with four F(2,3)
 *     levels).  Point digits (q_n^row, q_n^col, ..., q_1^row, q_1^col), most
 *     significant first, radix 5 at the F(3,3) levels and 4 at the F(2,3)
 *     ones, so the quad layouts of F(2x2,3x3) hold unchanged (U [P/4][M][N][4],
 *     V [P/4][M][T][4], Z [P/16][N][T][4]).  At n = 4 the input and the
 *     output transform also use a scratch buffer of max(25*676*M*T,
 *     25*144*N*T) floats (the level-4 blocks of the input windows, the
 *     level-3 blocks of the output tiles) that the plan holds after its Z
 *     (counted in workspace_bytes), also for the stage calls, which therefore
 *     must not overlap on one plan.
 *     Dense fp32 plans; r <= 7 gives the F(2x2,3x3) plan (info.tile reports
 *     it).  No fused paths (fused_input = fused_conv = fused_output = 0). */
enum { NWG_TILE_F2X2_3X3 = 0, NWG_TILE_F3X3_3X3 = 1, NWG_TILE_LD_F2X2_3X3 = 2,
       NWG_TILE_MIX_F23_F33 = 3, NWG_TILE_AUTO = -1 };

enum {
  NWG_OK = 0,
  NWG_EINVAL = -1,       /* bad argument (NULL pointer, bad shape) */
  NWG_ENOMEM = -2,       /* device allocation failed */
  NWG_EHIP = -3,         /* a HIP runtime call or kernel launch failed */
  NWG_EUNSUPPORTED = -4  /* valid request the library does not serve */
};

#define NWG_MAX_DEPTH 4   /* r <= 31 */

/* Arithmetic of the Winograd-domain contraction (nwg_plan_set_precision).
 *   NWG_PRECISION_FP32: fp32 operands, fp32 MFMA (v_mfma_f32_16x16x4f32).
 *   NWG_PRECISION_BF16_SPLIT: every U and V value is stored as a two-term
 *     bf16 split v ~ hi + lo (hi = bf16(v), lo = bf16(v - hi), round to
 *     nearest even; hi + lo keeps 16 significant bits), packed in one 32-bit
 *     word with hi in the low half, so U and V keep their fp32 layouts and
 *     sizes.  The contraction forms all four partial products
 *     (hi + lo)(hi + lo) on bf16 MFMA (v_mfma_f32_16x16x32_bf16) with fp32
 *     accumulation; Z and y stay fp32. */
enum { NWG_PRECISION_FP32 = 0, NWG_PRECISION_BF16_SPLIT = 1 };

/* Plan geometry, as computed by the level recurrence (Sec. III.B). */
typedef struct nwg_plan_info {
  int B, M, N, H, W, r, pad, tile;
  int Ho, Wo;
  int n;                        /* nesting depth, 0..NWG_MAX_DEPTH */
  int m, rb, l;                 /* base F(m, rb), l = m + rb - 1 */
  int strides[NWG_MAX_DEPTH];   /* stride of level 1..n */
  int Mn, Kn, Ln;               /* outputs / padded taps / input per axis per tile */
  int th, tw;                   /* tiles per image */
  long long T;                  /* B * th * tw */
  long long P;                  /* Winograd points per tile, l^(2n) */
  size_t u_bytes, v_bytes, yhat_bytes, workspace_bytes;   /* yhat_bytes: Z */
  long long ewmm_mults;         /* general multiplications per call: P*T*M*N (every
                                   point, dead groups included) */
  double direct_flop;           /* 2*B*N*M*Ho*Wo*r*r */
  double contract_flop;         /* FLOPs of the contraction's nonzero points: 2*P*M*N*T,
                                   or on the mixed nest 2*L^2*live_groups*M*N*T with L
                                   the live level-1 digits (3 or 4; n = 0:
                                   2*B*N*M*Ho*Wo) */
  int fused_input;              /* 1: nwg_conv2d fuses the input transform into the
                                   contraction (F(2x2,3x3): nwg_input_contract, depth 3-4,
                                   N <= 2, or depthwise; F(3x3,3x3): depth 2, N = 1) and
                                   the plan holds no V */
  int depthwise;                /* 1: depthwise plan (see nwg_plan_create_depthwise) */
  int fused_conv;               /* 1: nwg_conv2d runs one kernel x -> y (depth 1 with
                                   M <= 8, N <= 16; depth 2 with M <= 2, M N <= 64;
                                   depthwise at depth 1-2); the plan holds only U */
  int pipeline_parts;           /* 1, or the parts nwg_conv2d splits the input transform
                                   and contraction into (nwg_plan_set_pipeline) */
  int precision;                /* NWG_PRECISION_FP32 (default) or NWG_PRECISION_BF16_SPLIT
                                   (nwg_plan_set_precision) */
  int ld_c;                     /* NWG_TILE_LD_F2X2_3X3: sub-kernels per axis c; else 0 */
  int fused_output;             /* 1: nwg_conv2d forms the contraction inside the output
                                   transform (F(3x3,3x3), M <= 2, not fused_input): input
                                   transform, then one kernel V -> y (timed as the
                                   contraction, index 2); the plan holds no Z */
  int outer33;                  /* NWG_TILE_MIX_F23_F33: F(3,3) levels above the two
                                   F(2,3) levels (1 or 2); else 0 */
  /* Groups that need no work.  A group is the 16 points (4 x 4) sharing their
   * digits above level 1; it is Z's group index g, those digits read as one
   * number (q_n^r, q_n^c, ..., q_2^r, q_2^c, most significant first).
   * On the mixed nest the kernel taps split greedily over the levels leave
   * some digit combinations with no tap (and the padded taps r..Kn-1 are
   * zero), so the transformed kernel of a point is zero for every w when no
   * real tap reaches it.  A group is dead when, along either axis, none of
   * its points is reached; its Z is zero.  The library then neither writes
   * nor reads its U, V and Z, and skips its contraction. */
  int live_np;                  /* live digit prefixes per axis (levels 2..n) on the
                                   mixed nest; 0 when every group is computed */
  unsigned long long live_prefix[2];   /* bit i: prefix i of an axis is live (digits
                                   q_n .. q_2, the outermost most significant) */
  long long live_groups;        /* groups the contraction computes: live_np^2, or P/16 */
  int level1_live;              /* bit q: level-1 digit q is live along each axis (0xf,
                                   or 0x7 on the mixed nest when no tap k < r splits to
                                   level-1 digit 2, i.e. r below the nest's Kn: then the
                                   points with q_1^r = 3 or q_1^c = 3 are zero, quads
                                   q_1^r = 3 are neither written nor read, and the
                                   contraction takes 3 x 3 points per group); 0 on
                                   F(3x3,3x3) and at depth 0 */
  int mix_planar;               /* 1: U and V are in the mixed nest's planar layout (depth
                                   4, level1_live = 0x7, live_np > 0, M % 128 == 0,
                                   N % 128 == 0, T % 64 == 0): only the live groups'
                                   9 live points, U[i][p][M][N] and V[i][p][M][T] with
                                   i the group's place in the live list (row-prefix
                                   rank * live_np + column-prefix rank, ranks among
                                   the live prefixes in prefix order) and
                                   p = 3 q_1^r + q_1^c; u_bytes and v_bytes are those
                                   sizes.  0: the quad layouts described at the stage
                                   calls. */
} nwg_plan_info;

/* Geometry of a convolution without touching any device (host-only): the
 * level recurrence of Sec. III.B (the multi-level nesting paragraph; Alg. 1's
 * expression tree read as a chain of n bases), with level strides
 * s_j = min(M_j, K_j) where the base has m != r.  Writes *out and returns
 * NWG_OK; NWG_EINVAL for a NULL out, a dimension <= 0, pad < 0 or a kernel
 * larger than the padded input; NWG_EUNSUPPORTED for an unknown tile, a
 * kernel beyond the tile's depth (r > 31 on F(2x2,3x3) and AUTO, r > 9 on
 * F(3x3,3x3), r > 39 on the mixed nest) or a size beyond the limits above. */
int nwg_plan_geometry(int B, int M, int N, int H, int W, int r, int pad, int tile,
                      nwg_plan_info* out);

/* Create a plan for the convolution of Sec. II.A ("valid": pad = 0) -- M
 * input maps of H x W, N groups of M-channel r x r kernels, B images --
 * computed by nested Winograd (Sec. III.B) on `tile`, and allocate its
 * workspace on the current device (workspace_bytes; the caller's tensors
 * are not part of it).  NULL on failure, with nwg_last_status():
 * NWG_EINVAL / NWG_EUNSUPPORTED as for nwg_plan_geometry (and r = 1 with
 * pad > 0: NWG_EUNSUPPORTED), NWG_ENOMEM when a device allocation fails
 * (nothing stays allocated), NWG_EHIP when no device is available. */
nwg_plan* nwg_plan_create(int B, int M, int N, int H, int W, int r, int tile);

/* Same with explicit zero padding on all four sides ("same": pad = (r-1)/2;
 * the problem statement of Sec. II.A with the input zero-padded). */
nwg_plan* nwg_plan_create_pad(int B, int M, int N, int H, int W, int r, int pad, int tile);

/* --- Depthwise convolution (Table I's depth-wise row) --------------------
 * Each of C channels is correlated with its own r x r kernel and there is
 * no sum over channels:
 *   y[b][c][i][j] = sum_{u,v} xpad[b][c][i+u][j+v] * w[c][0][u][v],
 * x [B][C][H][W], w [C][1][r][r], y [B][C][Ho][Wo].  The plan's info has
 * M = N = C and depthwise = 1; the Winograd-domain step is the element-wise
 * product Yhat[p][c][t] = U[p][c] V[p][c][t].  U is [P/4][1][C][4] (depth 0:
 * [1][C]); V and Z have the dense layouts with M = N = C.  nwg_conv2d runs,
 * by depth: 0, y = w[c] x (pad must be 0); 1-2, one kernel x -> y (timed as
 * the contraction, index 2); 3-4, nwg_input_contract then
 * nwg_output_transform.  The stage calls take the same buffers as for dense
 * plans; nwg_contract computes the element-wise product (with the level-1
 * output transform) instead of a channel sum.  Errors as for the dense
 * calls. */
int nwg_plan_geometry_depthwise(int B, int C, int H, int W, int r, int pad, int tile,
                                nwg_plan_info* out);
nwg_plan* nwg_plan_create_depthwise(int B, int C, int H, int W, int r, int pad, int tile);

/* Release a plan and its workspace.  NULL is a no-op.  The caller must make
 * sure no work using the plan is still queued. */
void nwg_plan_destroy(nwg_plan* plan);

/* Copy the plan's geometry into *out. */
int nwg_plan_query(const nwg_plan* plan, nwg_plan_info* out);

/* y = conv(x, w), the correlation of Sec. II.A, by the steps of Sec. III.B:
 * the nested kernel transform (only when w differs from the cached weight
 * pointer or after nwg_plan_set_weights), then the nested input transform,
 * the per-point channel contraction (Sec. II.B: the M input channels summed
 * in the Winograd domain) and the nested output transform, all queued on
 * `stream`.  x [B][M][H][W], w [N][M][r][r], y [B][N][Ho][Wo]: contiguous
 * fp32 device buffers of the plan's shape, 16-byte aligned, y not
 * overlapping x or w.  For r = 1 the contraction reads x and writes y
 * directly.  The weight cache is keyed by the pointer only: mutating w in
 * place, or passing a new weight tensor at a freed one's address, requires
 * nwg_plan_set_weights before the next call.  NWG_EINVAL for a NULL
 * argument, NWG_EHIP when a launch fails. */
int nwg_conv2d(nwg_plan* plan, const float* x, const float* w, float* y, void* stream);

/* Re-run the kernel transform of w into the plan's cached U now. */
int nwg_plan_set_weights(nwg_plan* plan, const float* w, void* stream);

/* --- Stage entry points (each is one kernel launch on `stream`) ---------- */

/* Nested kernel transformation (Sec. III.B, 2nd step): w [N][M][r][r] -> U
 * (u_bytes). */
int nwg_kernel_transform(const nwg_plan* plan, const float* w, float* U, void* stream);

/* Nested input transformation (Sec. III.B, 1st step): x -> V (v_bytes).
 * NWG_EINVAL at depth 0 (r = 1), which has no transform. */
int nwg_input_transform(const nwg_plan* plan, const float* x, float* V, void* stream);

/* EWMM accumulated over the M input channels (Sec. II.B, III.B final step),
 * on fp32 MFMA, followed by the first level of the nested output
 * transformation: U, V -> Z (yhat_bytes).  At depth 0, V is x and Z is y
 * (a plain per-image channel GEMM). */
int nwg_contract(const nwg_plan* plan, const float* U, const float* V, float* Z,
                 void* stream);

/* Input transformation, contraction and first output level in one kernel,
 * x, U -> Z (yhat_bytes), with the same result as nwg_input_transform
 * followed by nwg_contract but without forming V.  For layers with one or
 * two output channels, whose contraction is too small to pay for writing
 * and re-reading V, and for depthwise layers.  Depth 3 or 4
 * (8 <= r <= 31) and N <= 2 or a depthwise plan only; NWG_EUNSUPPORTED
 * otherwise. */
int nwg_input_contract(const nwg_plan* plan, const float* x, const float* U, float* Z,
                       void* stream);

/* Nested output transformation (Sec. III.B, final step), levels 2..n:
 * Z -> y, cropped to Ho x Wo.  NWG_EINVAL at depth 0. */
int nwg_output_transform(const nwg_plan* plan, const float* Z, float* y, void* stream);

/* Two-stream pipeline (depth-4 dense plans whose contraction takes full
 * 64-wide tiles: M % 32 == 0, N % 64 == 0, T % 64 == 0; off by default).
 * With parts > 1, nwg_conv2d splits the input
 * transform and the contraction into `parts` pieces over the level-4 branches
 * (contiguous point ranges of V, U and Z) and queues each contraction piece on
 * a stream of the plan's own, after its input piece, so that the next input
 * piece (HBM-bound) overlaps it (MFMA-bound).  The plan's stream waits for
 * the work already queued on the caller's stream first, and the caller's
 * stream waits for the last piece before the output transform: the call
 * stays ordered on the caller's stream.  parts: 1 (off), 2, 4, 8 or 16;
 * NWG_EINVAL for other values, NWG_EUNSUPPORTED for a plan that cannot
 * split.  Timing records each piece (counts then grow by `parts`). */
int nwg_plan_set_pipeline(nwg_plan* plan, int parts);

/* Contraction arithmetic (see NWG_PRECISION_*), for dense F(2x2,3x3) plans at
 * depth 1-4 whose contraction takes full 64-wide tiles (M % 32 == 0,
 * N % 64 == 0, T >= 64) and that are neither fused nor pipelined.  With
 * NWG_PRECISION_BF16_SPLIT, nwg_kernel_transform and nwg_input_transform
 * write U and V as packed (hi, lo) pairs in the fp32 layouts, and
 * nwg_contract reads them so; nwg_output_transform is unchanged.  The cached
 * transformed weights are invalidated: the next nwg_conv2d (or
 * nwg_plan_set_weights) transforms w again.  NWG_EINVAL for an unknown
 * precision, NWG_EUNSUPPORTED for a plan that cannot take it (nothing
 * changes then).  Measured error of the split path on the workloads: see the
 * library's tests; about 1e-5 relative L2 at depth 4 (fp32: about 1e-7). */
int nwg_plan_set_precision(nwg_plan* plan, int precision);

/* --- Per-stage timing ------------------------------------------------------
 * When enabled, nwg_conv2d records HIP events around each of its launches on
 * the caller's stream.  nwg_plan_get_timing waits for the recorded events,
 * adds their durations to ms[4] and launch counts to count[4] (index 0 kernel
 * transform, 1 input transform, 2 contraction, 3 output transform), then
 * forgets them.  A fused nwg_input_contract launch counts as a contraction
 * (index 2) and leaves index 1 untouched. */
int nwg_plan_set_timing(nwg_plan* plan, int enable);
int nwg_plan_get_timing(nwg_plan* plan, double ms[4], long long count[4]);

/* --- Without allocation ----------------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 * nwg_conv2d_noalloc computes what nwg_conv2d computes on a plan created by
 * nwg_plan_create_pad(B, M, N, H, W, r, pad, tile) (dense, fp32, no
 * pipeline), with the same kernels, but takes that plan's workspace (U; V
 * and Z where the plan holds them; each rounded up to 256 bytes) from a
 * static device array of NWG_NOALLOC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends, and transforms w on every
 * call (nothing is cached).  It calls no hipMalloc, hipFree or allocating
 * routine; its first call on a device resolves that device's copy of the
 * array (with that device current).  x, w, y as for nwg_conv2d (contiguous
 * fp32 device buffers, 16-byte aligned).  Returns NWG_OK, queuing the work on
 * `stream`; NWG_EINVAL / NWG_EUNSUPPORTED as nwg_plan_create_pad does for the
 * shape; NWG_EUNSUPPORTED, queuing nothing, when the workspace does not fit
 * (64 MiB: e.g. the 7x7 32->32 64x64 layer needs 11.6 MB, the 13x13 64->64
 * B=8 56x56 layer 581 MB); NWG_EHIP when a launch fails.
 * Every call on a GPU uses that GPU's one array and overwrites it: calls that
 * overlap on one GPU (from two streams or two threads) race, so order them
 * on one stream or serialise them. */
#define NWG_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int nwg_conv2d_noalloc(int B, int M, int N, int H, int W, int r, int pad, int tile,
                       const float* x, const float* w, float* y, void* stream);

/* Message for the last error on the calling thread ("" if none). */
const char* nwg_last_error(void);

/* Status of the last error on the calling thread (NWG_OK if none): for the
 * calls that return NULL, the reason (NWG_EINVAL, NWG_EUNSUPPORTED,
 * NWG_ENOMEM or NWG_EHIP). */
int nwg_last_status(void);

/* Library version string. */
const char* nwg_version(void);

#ifdef __cplusplus
}
#endif

#endif /* NWG_H */
