// Host-only part of the nested-Winograd library (see plan.h): the level
// recurrence of Sec. III.B (Alg. 1's expression tree read as a chain of n
// bases), each tile's geometry, the kernels a plan takes, its workspace, and
// the C entry points that touch no device (nwg_plan_geometry*,
// nwg_last_error, nwg_last_status, nwg_version).
#include "plan.h"

#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>

namespace nwg {
namespace {

thread_local std::string g_last_error;
thread_local int g_last_status = NWG_OK;

// Largest buffer a plan may hold, and largest count it reports: sizes are
// checked in double before any integer product is formed.
constexpr double kMaxBytes = 1e13;
constexpr double kMaxCount = 9e18;

}  // namespace

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  g_last_status = status;
  if (std::getenv("NWG_LOG")) std::fprintf(stderr, "nwg: %s\n", buf);
  return status;
}

void clear_error() {
  g_last_error.clear();
  g_last_status = NWG_OK;
}

// ---- kernels a plan takes ---------------------------------------------------

bool input_contract_applies(const nwg_plan_info& g) {
  return g.tile == NWG_TILE_F2X2_3X3 && g.n >= 3 && g.n <= 4 && (g.depthwise || g.N <= 2);
}

bool small_conv_applies(const nwg_plan_info& g) {
  if (g.depthwise || g.tile != NWG_TILE_F2X2_3X3) return false;
  if (g.n == 1) return g.M <= 8 && g.N <= 16;
  if (g.n == 2) return g.M <= 2 && (long long)g.M * g.N <= 64;
  return false;
}

bool input_contract5_applies(const nwg_plan_info& g) {
  return g.tile == NWG_TILE_F3X3_3X3 && g.n == 2 && g.N == 1 && !g.depthwise;
}

bool contract_output5_applies(const nwg_plan_info& g) {
  return g.tile == NWG_TILE_F3X3_3X3 && (g.n == 1 || g.n == 2) && g.M <= 2 && !g.depthwise &&
         !input_contract5_applies(g);
}

IC5Shape ic5_shape(const nwg_plan_info& g) {
  IC5Shape c;
  c.RX = g.tw < 64 ? g.tw : 64;
  c.RY = 64 / c.RX;
  if (c.RY > g.th) c.RY = g.th;
  c.nbx = (g.tw + c.RX - 1) / c.RX;
  c.nby = (g.th + c.RY - 1) / c.RY;
  // input-channel groups: about 512 work-groups in all, at least 2 channels each
  const long long boxes = (long long)c.nbx * c.nby * g.B;
  long long want = (512 + boxes - 1) / boxes;
  const long long maxg = (g.M + 1LL) / 2;
  if (want > maxg) want = maxg;
  if (want < 1) want = 1;
  c.mper = (int)((g.M + want - 1) / want);
  c.groups = (int)((g.M + (long long)c.mper - 1) / c.mper);
  c.lds = (size_t)(((c.RY - 1) * 9 + 17) * ((c.RX - 1) * 9 + 17) + 625) * sizeof(float);
  return c;
}

int input_contract5_parts(const nwg_plan_info& g) { return ic5_shape(g).groups; }

size_t input_contract5_zbytes(const nwg_plan_info& g) {
  return (size_t)ic5_shape(g).groups * (size_t)(g.P / 25) * 9 * g.N * g.T * sizeof(float);
}

int mix_outer_levels(const nwg_plan_info& g) {
  return g.tile == NWG_TILE_MIX_F23_F33 ? g.n - 2 : 0;
}

size_t mix_scratch_bytes(const nwg_plan_info& g) {
  if (mix_outer_levels(g) != 2) return 0;
  const size_t z3 = (size_t)25 * 144 * g.N * g.T * sizeof(float);
  const size_t x4 = (size_t)25 * g.M * g.T * kMixL3 * kMixL3 * sizeof(float);
  return z3 > x4 ? z3 : x4;
}

// K slices of a linear-decomposition plan's contraction: its grid has one
// level-1 group, so with few tiles the M c^2 channels are split (a divisor
// of M c^2 / 32, up to 64 slices) until there are about 1024 work-groups.
int ld_kslices(const nwg_plan_info& g) {
  if (g.ld_c <= 0) return 1;
  const long long mk = (long long)g.M * g.ld_c * g.ld_c;
  if (mk % 32 || g.N % 64 || g.T < 64) return 1;
  const long long ntb = g.T % 128 == 0 ? g.T / 128 : (g.T + 63) / 64;
  const long long wgs = ntb * (g.N / 64);
  const long long units = mk / 32;
  int best = 1;
  for (int sl = 1; sl <= 64 && sl <= units; ++sl) {
    if (units % sl) continue;
    best = sl;
    if (wgs * sl >= 1024) break;
  }
  return best;
}

// bytes of the plan's Z buffer: the stage-call Z, the fused F(3,3) kernel's
// partial Z9 buffers, a linear-decomposition plan's K-slice parts, or the
// mixed nest's Z followed by the scratch of its depth-4 transforms
size_t zalloc_bytes(const nwg_plan_info& g) {
  if (g.fused_input && g.tile == NWG_TILE_F3X3_3X3) return input_contract5_zbytes(g);
  if (g.ld_c > 0) return (size_t)ld_kslices(g) * g.yhat_bytes;
  if (g.tile == NWG_TILE_MIX_F23_F33) return g.yhat_bytes + mix_scratch_bytes(g);
  return g.yhat_bytes;
}

bool plan_holds_v(const nwg_plan_info& g) {
  return g.n > 0 && !(g.fused_input || g.depthwise || g.fused_conv);
}

bool plan_holds_z(const nwg_plan_info& g) {
  return g.n > 0 && !(g.fused_conv || g.fused_output);
}

// Depth-4 dense plans whose contraction takes the full-tile path can split
// the input transform and the contraction into parts over the level-4
// branches (contiguous ranges of points) and overlap them on two streams.
bool pipeline_allowed(const nwg_plan_info& g) {
  return g.tile == NWG_TILE_F2X2_3X3 && g.precision == NWG_PRECISION_FP32 && g.n == 4 &&
         !g.depthwise && !g.fused_input && g.M % 32 == 0 && g.N % 64 == 0 && g.T % 64 == 0;
}

bool split_allowed(const nwg_plan_info& g) {
  return g.tile == NWG_TILE_F2X2_3X3 && g.n >= 1 && !g.depthwise && !g.fused_input &&
         !g.fused_conv && g.pipeline_parts <= 1 && g.M % 32 == 0 && g.N % 64 == 0 && g.T >= 64;
}

GroupMap group_map(const nwg_plan_info& g) {
  GroupMap m{};
  const bool mix = g.tile == NWG_TILE_MIX_F23_F33;
  if ((!mix && g.tile != NWG_TILE_F2X2_3X3) || g.depthwise || g.n < 3 || g.n - 1 > 3) return m;
  m.q3 = g.level1_live == 0x7 ? 1 : 0;
  if (g.live_np <= 0) return m;
  m.np = g.live_np;
  m.nd = g.n - 1;
  m.mask0 = g.live_prefix[0];
  m.mask1 = g.live_prefix[1];
  // groups are ordered by (q_n^r, q_n^c, ..., q_2^r, q_2^c), each radix l_j
  int wc = 1;
  for (int d = 0; d < m.nd; ++d) {
    m.rad[d] = mix && d > 0 ? 5 : 4;                 // F(2,3) digits; the mixed nest's F(3,3) above q_2
    m.wc[d] = wc;
    m.wr[d] = wc * m.rad[d];
    wc = m.wr[d] * m.rad[d];
  }
  return m;
}

namespace {

// Output size and the limits every tile shares: each map (input and output)
// must hold fewer than 2^31 values, and no buffer more than 1e13 bytes.
int output_size(int B, int M, int N, int H, int W, int r, int pad, long long* Ho,
                long long* Wo) {
  *Ho = (long long)H + 2LL * pad - r + 1;
  *Wo = (long long)W + 2LL * pad - r + 1;
  if (*Ho <= 0 || *Wo <= 0)
    return fail(NWG_EINVAL, "kernel %d larger than padded input %dx%d (pad %d)", r, H, W, pad);
  if ((double)H * W >= 2147483648.0 || (double)*Ho * *Wo >= 2147483648.0)
    return fail(NWG_EUNSUPPORTED, "maps of 2^31 or more values (%dx%d -> %lldx%lld)", H, W,
                *Ho, *Wo);
  const double x = 4.0 * B * M * H * W, y = 4.0 * B * N * (double)*Ho * (double)*Wo;
  if (x > kMaxBytes || y > kMaxBytes)
    return fail(NWG_EUNSUPPORTED, "input or output larger than 1e13 bytes");
  return NWG_OK;
}

// Linear decomposition (Sec. II.B) on F(2,3): a depth-1 plan over M c^2
// contraction channels, c = ceil(r/3) sub-kernels per axis.
int ld_geometry(int B, int M, int N, int H, int W, int r, int pad, int depthwise,
                nwg_plan_info* g) {
  if (depthwise) return fail(NWG_EUNSUPPORTED, "the linear-decomposition tile serves dense plans");
  long long Ho, Wo;
  const int rc = output_size(B, M, N, H, W, r, pad, &Ho, &Wo);
  if (rc != NWG_OK) return rc;
  // sub-kernels per axis; more than 65535 decomposed channels is refused below
  const long long cl = (r + 2LL) / 3;
  if (cl > 256)
    return fail(NWG_EUNSUPPORTED, "kernel size %d: too many sub-kernels for the decomposition", r);
  const int c = (int)cl;
  const double th = (double)((Ho + 1) / 2), tw = (double)((Wo + 1) / 2);
  const double T = B * th * tw;
  const double mk = (double)M * c * c, f = (double)sizeof(float);
  const double u = f * 16 * mk * N, v = f * 16 * mk * T, yh = f * 4 * N * T;
  if (u > kMaxBytes || v > kMaxBytes || yh > kMaxBytes || T > 0x7fffffffLL / 64 || mk > 65535 ||
      16 * T * mk * N > kMaxCount)
    return fail(NWG_EUNSUPPORTED, "workspace too large (or more than 65535 decomposed channels)");
  g->B = B; g->M = M; g->N = N; g->H = H; g->W = W; g->r = r; g->pad = pad;
  g->tile = NWG_TILE_LD_F2X2_3X3;
  g->Ho = (int)Ho;
  g->Wo = (int)Wo;
  g->n = 1;
  g->m = 2; g->rb = 3; g->l = 4;
  g->strides[0] = 1;
  g->Mn = 2;
  g->Kn = 3 * c;
  g->Ln = 3 * c + 1;
  g->th = (int)th;
  g->tw = (int)tw;
  g->T = (long long)T;
  g->P = 16;
  g->ld_c = c;
  g->u_bytes = (size_t)u;
  g->v_bytes = (size_t)v;
  g->yhat_bytes = (size_t)yh;
  g->direct_flop = 2.0 * B * N * (double)M * Ho * Wo * r * r;
  g->ewmm_mults = (long long)(16 * T * mk * N);
  g->contract_flop = 2.0 * 16 * mk * N * T;
  g->pipeline_parts = 1;
  g->precision = NWG_PRECISION_FP32;
  g->workspace_bytes = g->u_bytes + g->v_bytes + zalloc_bytes(*g);
  return NWG_OK;
}

// Digits k_j of a tap's row in a level's kernel transform that the row of
// point q reaches (bit k): G of F(2,3) (points 0, 1, -1, infinity) and of
// F(3,3) (points 0, 1, -1, 2, infinity) has one nonzero entry in its first
// and last rows and three in the others.
unsigned g_row_digits(int l, int q) { return q == 0 ? 1u : q == l - 1 ? 4u : 7u; }

// Which digit prefixes (q_n .. q_2) of an axis have a point whose
// transformed kernel can be nonzero, and which level-1 digits q_1 any point
// has that for (the mixed nest, mix = true, or a chain of F(2,3) levels).
// Tap k < r reaches point (q_n .. q_1) when each digit of its greedy split
// (outermost first, each at most 2, as the kernel transform splits it) is
// one that the point's G row reaches.
void nest_liveness(nwg_plan_info* g, bool mix) {
  const int n = g->n;
  int l[NWG_MAX_DEPTH];
  for (int j = 0; j < n; ++j) l[j] = mix && j >= 2 ? 5 : 4;   // level j + 1
  int npref = 1;
  for (int j = 1; j < n; ++j) npref *= l[j];
  if (npref > 128) return;                            // beyond the masks: all groups live
  int live = 0;
  unsigned q1mask = 0;
  unsigned long long mask[2] = {0, 0};
  for (int pf = 0; pf < npref; ++pf) {
    int q[NWG_MAX_DEPTH] = {0};
    int rest = pf;
    for (int j = 1; j < n; ++j) {                     // q_2 least significant
      q[j] = rest % l[j];
      rest /= l[j];
    }
    unsigned reached = 0;                             // bit q_1
    for (int q1 = 0; q1 < l[0]; ++q1) {
      q[0] = q1;
      for (int k = 0; k < g->r && !((reached >> q1) & 1u); ++k) {
        int rem = k;
        bool ok = true;
        for (int j = n - 1; j >= 1 && ok; --j) {
          const int d = rem / g->strides[j] < 2 ? rem / g->strides[j] : 2;
          rem -= d * g->strides[j];
          ok = (g_row_digits(l[j], q[j]) >> d) & 1u;
        }
        if (ok && rem <= 2 && ((g_row_digits(l[0], q[0]) >> rem) & 1u)) reached |= 1u << q1;
      }
    }
    if (reached) {
      mask[pf >> 6] |= 1ULL << (pf & 63);
      ++live;
      q1mask |= reached;
    }
  }
  // the mixed nest's kernels skip level-1 digit 3 (the F(2,3) row that
  // reaches tap digit 2 alone: no tap k < r has it when r is below the
  // nest's taps); F(2,3) chains keep every level-1 digit and skip groups only
  if (mix) g->level1_live = q1mask == 0x7u ? 0x7 : 0xf;
  const int lq = g->level1_live == 0x7 ? 3 : 4;
  if (live < npref) {
    g->live_np = live;
    g->live_prefix[0] = mask[0];
    g->live_prefix[1] = mask[1];
    g->live_groups = (long long)live * live;
  }
  g->contract_flop = 2.0 * lq * lq * g->live_groups * g->M * g->N * g->T;
}

// Depth-4 mixed plans with dead groups and level-1 digit 3 dead, on shapes
// the planar contraction tiles evenly (128 x 64 blocks of (n, t), 128-deep
// channel sweeps): U and V hold only the live groups' 3 x 3 live points,
// point by point.  The transforms address a level-4 row block (20 row
// prefixes) of groups through one buffer resource, which must stay below
// 2 GiB.
void mix_layout(nwg_plan_info* g) {
  if (g->n != 4 || g->level1_live != 0x7 || g->live_np <= 0) return;
  if (g->M % 128 || g->N % 128 || g->T % 64) return;
  const double span = 20.0 * g->live_np * 9 * g->M * (double)(g->N > g->T ? g->N : g->T) * 4;
  if (span >= 2147483648.0) return;
  g->mix_planar = 1;
  g->u_bytes = (size_t)9 * g->live_groups * g->M * g->N * sizeof(float);
  g->v_bytes = (size_t)9 * g->live_groups * g->M * g->T * sizeof(float);
}

// Level recurrence on the base F(m, rb): s_0 = 1, M_1 = m, K_1 = rb,
// s_j = min(M_j, K_j), M_{j+1} = M_j + s_j (m_{j+1} - 1),
// K_{j+1} = K_j + s_j (rb - 1); n is the smallest depth with K_n >= r, and
// r = 1 needs no level.  The mixed nest takes m = 3 above level 2.
int geometry_tile(int B, int M, int N, int H, int W, int r, int pad, int tile, int depthwise,
                  nwg_plan_info* g) {
  std::memset(g, 0, sizeof *g);
  if (B <= 0 || M <= 0 || N <= 0 || H <= 0 || W <= 0 || r <= 0 || pad < 0)
    return fail(NWG_EINVAL, "invalid shape B=%d M=%d N=%d H=%d W=%d r=%d pad=%d", B, M, N, H, W,
                r, pad);
  if (tile != NWG_TILE_F2X2_3X3 && tile != NWG_TILE_F3X3_3X3 && tile != NWG_TILE_LD_F2X2_3X3 &&
      tile != NWG_TILE_MIX_F23_F33)
    return fail(NWG_EUNSUPPORTED, "unsupported tile %d", tile);
  if (tile == NWG_TILE_LD_F2X2_3X3) return ld_geometry(B, M, N, H, W, r, pad, depthwise, g);
  const bool mix = tile == NWG_TILE_MIX_F23_F33;
  if (mix && depthwise)
    return fail(NWG_EUNSUPPORTED, "the mixed F(2,3)/F(3,3) nest serves dense plans");
  // up to 7 taps the mixed nest has only its two F(2,3) levels
  if (mix && r <= 7)
    return geometry_tile(B, M, N, H, W, r, pad, NWG_TILE_F2X2_3X3, 0, g);
  if (mix && r > 39)
    return fail(NWG_EUNSUPPORTED, "kernel size %d exceeds the mixed nest's 39 taps", r);
  const bool f33 = tile == NWG_TILE_F3X3_3X3;
  if (f33 && depthwise)
    return fail(NWG_EUNSUPPORTED, "depthwise plans use the F(2x2,3x3) tile");
  long long Ho, Wo;
  const int rc = output_size(B, M, N, H, W, r, pad, &Ho, &Wo);
  if (rc != NWG_OK) return rc;
  // base F(m, rb): F(2,3) or F(3,3); F(3,3) is kept to depth 2 (r <= 9),
  // where its fp32 error stays near 1e-6 (the mixed nest: F(2,3) at levels
  // 1-2, F(3,3) above)
  const int m = f33 ? 3 : 2, rb = 3, l = m + rb - 1;
  const int max_depth = f33 ? 2 : NWG_MAX_DEPTH;
  auto level_m = [&](int j) { return mix && j >= 2 ? 3 : m; };   // level j + 1
  int n = 0, Mn = 1, Kn = 1;
  int strides[NWG_MAX_DEPTH + 1] = {0};
  long long P1 = 1;   // Winograd points per axis
  if (r > 1) {
    strides[0] = 1;
    n = 1;
    Mn = m;
    Kn = rb;
    P1 = l;
    while (Kn < r) {
      const int s = Mn < Kn ? Mn : Kn;
      if (n >= max_depth)
        return fail(NWG_EUNSUPPORTED,
                    "kernel size %d needs nesting depth > %d (r <= %d supported on this tile)", r,
                    max_depth, f33 ? 9 : 31);
      const int mj = level_m(n);
      strides[n] = s;
      Mn += s * (mj - 1);
      Kn += s * (rb - 1);
      P1 *= mj + rb - 1;
      ++n;
    }
  }
  // the kernel transform sees Mk input channels: 1 for a depthwise layer
  const int Mk = depthwise ? 1 : M;
  const double th = (double)((Ho + Mn - 1) / Mn), tw = (double)((Wo + Mn - 1) / Mn);
  const double T = B * th * tw;
  const double P = (double)P1 * P1;
  const double f = (double)sizeof(float);
  double u, v, yh, mults, cflop;
  if (n == 0) {
    u = f * Mk * N;
    v = yh = 0.0;
    mults = (double)B * N * Mk * Ho * Wo;
    cflop = 2.0 * mults;
  } else {
    // the contraction writes Yhat after (part of) the level-1 output
    // transform: per (n, t) P/4 values for F(2,3) (both axes), 3 P/5 for
    // F(3,3) (columns only)
    const double zpts = f33 ? (P / 5) * 3 : P / 4;
    u = f * P * Mk * N;
    v = f * P * M * T;
    yh = f * zpts * N * T;
    mults = P * T * Mk * N;
    cflop = 2.0 * mults;
  }
  if (u > kMaxBytes || v > kMaxBytes || yh > kMaxBytes || mults > kMaxCount ||
      (n > 0 && T > 0x7fffffffLL / 64) || T > kMaxCount)
    return fail(NWG_EUNSUPPORTED, "workspace too large");
  g->B = B; g->M = M; g->N = N; g->H = H; g->W = W; g->r = r; g->pad = pad; g->tile = tile;
  g->depthwise = depthwise ? 1 : 0;
  g->Ho = (int)Ho;
  g->Wo = (int)Wo;
  g->n = n;
  g->m = m; g->rb = rb; g->l = l;
  for (int j = 0; j < n; ++j) g->strides[j] = strides[j];
  g->Mn = Mn;
  g->Kn = Kn;
  g->Ln = n == 0 ? 1 : Mn + Kn - 1;
  g->th = (int)th;
  g->tw = (int)tw;
  g->T = (long long)T;
  g->P = P1 * P1;
  g->outer33 = mix ? n - 2 : 0;
  g->direct_flop = 2.0 * B * N * (double)Mk * Ho * Wo * r * r;
  g->u_bytes = (size_t)u;
  g->v_bytes = (size_t)v;
  g->yhat_bytes = (size_t)yh;
  g->ewmm_mults = (long long)mults;
  g->contract_flop = cflop;
  // one or two output channels (or depthwise) at depth 3-4: the fused kernel
  // never forms V.  Few channels (or depthwise) at depth 1-2: one kernel
  // x -> y, neither V nor Z.
  g->fused_input = (f33 ? input_contract5_applies(*g) : input_contract_applies(*g)) ? 1 : 0;
  g->fused_conv = !f33 && !mix && (small_conv_applies(*g) || (depthwise && (n == 1 || n == 2)))
                      ? 1 : 0;
  g->fused_output = contract_output5_applies(*g) ? 1 : 0;
  g->pipeline_parts = 1;
  g->precision = NWG_PRECISION_FP32;
  g->workspace_bytes = g->u_bytes + (plan_holds_v(*g) ? g->v_bytes : 0) +
                       (plan_holds_z(*g) ? zalloc_bytes(*g) : 0);
  g->live_groups = f33 || n == 0 ? 0 : g->P / 16;
  g->level1_live = f33 || n == 0 ? 0 : 0xf;
  if (mix && n >= 3) {
    nest_liveness(g, true);
    mix_layout(g);
    g->workspace_bytes = g->u_bytes + g->v_bytes + zalloc_bytes(*g);
  } else if (!mix && !f33 && !depthwise && n >= 3 && !g->fused_input && !g->fused_conv &&
             !g->fused_output) {
    // unfused dense F(2,3) chains: the contraction and the output transform
    // skip the groups no tap reaches (their U is zero for every weight)
    nest_liveness(g, false);
  }
  return NWG_OK;
}

}  // namespace

namespace {

// Step time of an unfused dense plan on MI355X, in seconds, from the bytes
// and FLOPs its kernels move and compute, at the rates they sustain at depth
// 4 (about 5 TB/s of HBM traffic, 100 TFLOP/s of fp32 MFMA): the transforms
// move x + V and Z + y (and the mixed nest's depth-4 scratch both ways); the
// contraction takes the longer of its U + V + Z traffic and its MFMA work on
// whole 64-column tiles and 64-row / 32-deep channel blocks.  On the mixed
// nest only the live groups count, and of them the live points (planar
// layout) or quads (quad layout).  Its kernels fall short of these rates
// more than the F(2,3) ones do: its estimate is scaled by 1.47 at depth 4
// and 1.3 at depth 3, the factors that order the two nests as measured on
// the fifteen layers of the automatic-choice test (ties within 3 % either
// way).  Used only to choose between nests.
double unfused_step_seconds(const nwg_plan_info& g) {
  constexpr double kBw = 5.0e12, kMfma = 100e12;
  auto up = [](double v, double q) { return std::ceil(v / q) * q; };
  double pts = (double)g.P, U = (double)g.u_bytes, V = (double)g.v_bytes,
         Z = (double)g.yhat_bytes, scratch = 0.0, scale = 1.0;
  double Vc = V;                                      // V as the contraction reads it
  if (g.tile == NWG_TILE_F2X2_3X3 && g.live_np > 0) {
    // the contraction and the output transform visit the live groups only.
    // The input transform writes only their V too, but the model charges it
    // every group's: on 32- and 64-channel layers the F(2,3) kernels run
    // about 1.5x below the model's rates, and with the live write counted no
    // single factor below orders all the measured layers
    const double live = (double)g.live_groups / (double)(g.P / 16);
    pts *= live;
    U *= live;
    Vc *= live;
    Z *= live;
  }
  if (g.tile == NWG_TILE_MIX_F23_F33 && g.n >= 3) {
    const double G = (double)(g.P / 16), live = (double)g.live_groups;
    const bool q3 = g.level1_live == 0x7;
    pts = live * (q3 ? 9.0 : 16.0);
    if (!g.mix_planar) {
      U = U / G * live * (q3 ? 0.75 : 1.0);
      V = V / G * live * (q3 ? 0.75 : 1.0);
    }
    Vc = V;
    Z = Z / G * live;
    if (g.n == 4)   // X4 (level-4 input blocks) and Z3 (level-3 output blocks), each written and read
      scratch = 2.0 * 4.0 * 25.0 * (double)g.T * ((double)kMixL3 * kMixL3 * g.M + 144.0 * g.N);
    scale = g.n == 4 ? 1.47 : 1.22;
  }
  const double flop = 2.0 * pts * up(g.M, 32) * up(g.N, 64) * up((double)g.T, 64);
  const double x = 4.0 * g.B * g.M * g.H * g.W, y = 4.0 * g.B * g.N * (double)g.Ho * g.Wo;
  const double cb = U + Vc + Z;
  const double tc = flop / kMfma > cb / kBw ? flop / kMfma : cb / kBw;
  return scale * (tc + (x + V) / kBw + (Z + y) / kBw + scratch / kBw);
}

}  // namespace

// NWG_TILE_AUTO: F(3x3,3x3) where it measured faster than F(2x2,3x3) --
// the fused one-output-channel kernel at depth 2 (unless F(2,3) runs the
// layer in one kernel), or both channel counts >= 32 and either a nesting
// level saved (r = 8, 9) or depth 1 (r <= 3); the mixed nest for dense
// layers at depth 3 (r = 10..15) or 4 with both channel counts >= 32 when
// the step model above expects it to be faster (with its dead groups and
// points skipped it has 2.5x to 5.6x fewer contraction FLOPs per output,
// but its 12 x 12 and 36 x 36 tiles leave few tiles on small images, and
// its transformed weights are up to 2x larger); F(2x2,3x3) otherwise.
int compute_geometry(int B, int M, int N, int H, int W, int r, int pad, int tile, int depthwise,
                     nwg_plan_info* g) {
  if (!g) return fail(NWG_EINVAL, "output pointer is NULL");
  if (tile != NWG_TILE_AUTO) return geometry_tile(B, M, N, H, W, r, pad, tile, depthwise, g);
  nwg_plan_info a, b;
  const int ra = geometry_tile(B, M, N, H, W, r, pad, NWG_TILE_F2X2_3X3, depthwise, &a);
  if (ra == NWG_OK && !depthwise && (a.n == 4 || (a.n == 3 && r > 9)) && M >= 32 && N >= 32) {
    if (geometry_tile(B, M, N, H, W, r, pad, NWG_TILE_MIX_F23_F33, 0, &b) == NWG_OK) {
      *g = unfused_step_seconds(b) < unfused_step_seconds(a) ? b : a;
      return NWG_OK;
    }
    clear_error();
  }
  if (ra != NWG_OK || depthwise || r > 9 || r == 1) {
    *g = a;
    return ra;
  }
  if (geometry_tile(B, M, N, H, W, r, pad, NWG_TILE_F3X3_3X3, 0, &b) != NWG_OK) {
    clear_error();
    *g = a;
    return NWG_OK;
  }
  const bool big = M >= 32 && N >= 32;
  const bool pick = ((b.fused_input || b.fused_output) && !a.fused_conv) ||
                    (big && a.n > b.n) || (big && a.n == 1 && !a.fused_conv);
  *g = pick ? b : a;
  return NWG_OK;
}

int check_plan_request(const nwg_plan_info& g) {
  if (g.n == 0 && g.pad != 0)
    return fail(NWG_EUNSUPPORTED,
                "1x1 kernels with padding are not supported (pad must be 0 for r = 1)");
  return NWG_OK;
}

}  // namespace nwg

extern "C" {

const char* nwg_version(void) {
  return "nwg 0.4 (nested F(2x2,3x3), F(3x3,3x3) and mixed F(2,3)/F(3,3), gfx950)";
}

const char* nwg_last_error(void) { return nwg::g_last_error.c_str(); }

int nwg_last_status(void) { return nwg::g_last_status; }

int nwg_plan_geometry(int B, int M, int N, int H, int W, int r, int pad, int tile,
                      nwg_plan_info* out) {
  return nwg::compute_geometry(B, M, N, H, W, r, pad, tile, 0, out);
}

int nwg_plan_geometry_depthwise(int B, int C, int H, int W, int r, int pad, int tile,
                                nwg_plan_info* out) {
  return nwg::compute_geometry(B, C, C, H, W, r, pad, tile, 1, out);
}

}  // extern "C"
