// Host side of the nested-Winograd library: the plan (level recurrence of
// Sec. III.B and Alg. 1, read as a chain of n identical F(2,3) bases), the
// workspace, the weight cache, the C ABI of include/nwg.h and per-stage
// timing.  All device work is queued on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "nwg_internal.h"

namespace {

thread_local std::string g_last_error;

void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  if (std::getenv("NWG_LOG")) std::fprintf(stderr, "nwg: %s\n", buf);
}

struct TimingRecord {
  int stage;
  hipEvent_t start, stop;
};

}  // namespace

struct nwg_plan {
  nwg_plan_info info;
  int device = 0;
  float* U = nullptr;
  float* V = nullptr;
  float* Yh = nullptr;
  const float* cached_w = nullptr;
  bool weights_valid = false;
  bool timing = false;
  std::vector<TimingRecord> pending;
  std::vector<hipEvent_t> event_pool;
  // two-stream pipeline (depth 4, dense): the input transform of part k+1
  // runs on the caller's stream while the contraction of part k runs on
  // `side`; created on first use, default priority
  hipStream_t side = nullptr;
  hipEvent_t ev_start = nullptr, ev_join = nullptr;
  std::vector<hipEvent_t> ev_part;
};

namespace {

// Level recurrence on the base F(m, rb): s_0 = 1, M_1 = m, K_1 = rb,
// s_j = min(M_j, K_j), M_{j+1} = M_j + s_j (m-1), K_{j+1} = K_j + s_j (rb-1);
// n is the smallest depth with K_n >= r, and r = 1 needs no level.
// Depth-4 dense plans whose contraction takes the full-tile path can split
// the input transform and the contraction into parts over the level-4
// branches (contiguous ranges of points) and overlap them on two streams.
// Off by default: on the 31x31 layer (B = 16, 128 -> 128) the overlapped
// contraction lost more (4.73 -> 5.6-6.6 ms over its parts) than the hidden
// input transform saved; every part count from 2 to 16 made the step slower.
bool pipeline_allowed(const nwg_plan_info& g) {
  return g.tile == NWG_TILE_F2X2_3X3 && g.precision == NWG_PRECISION_FP32 && g.n == 4 &&
         !g.depthwise && !g.fused_input &&
         g.M % 32 == 0 && g.N % 64 == 0 && g.T % 64 == 0;
}

// depthwise: M = N = C channels, one r x r kernel each, no channel sum.
// K slices of a linear-decomposition plan's contraction: its grid has one
// level-1 group, so with few tiles the M c^2 channels are split (a divisor
// of M c^2 / 32, up to 64 slices) until there are about 1024 work-groups
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
// partial Z9 buffers, or a linear-decomposition plan's K-slice parts
size_t zalloc_bytes(const nwg_plan_info& g) {
  if (g.fused_input && g.tile == NWG_TILE_F3X3_3X3) return nwg::input_contract5_zbytes(g);
  if (g.ld_c > 0) return (size_t)ld_kslices(g) * g.yhat_bytes;
  // mixed nest at depth 4: Z, then the scratch of its transforms
  if (g.tile == NWG_TILE_MIX_F23_F33) return g.yhat_bytes + nwg::mix_scratch_bytes(g);
  return g.yhat_bytes;
}

int compute_geometry_tile(int B, int M, int N, int H, int W, int r, int pad, int tile,
                          int depthwise, nwg_plan_info* g);

// Linear decomposition (Sec. II.B) on F(2,3): a depth-1 plan over M c^2
// contraction channels, c = ceil(r/3) sub-kernels per axis.
int ld_geometry(int B, int M, int N, int H, int W, int r, int pad, int depthwise,
                nwg_plan_info* g) {
  if (depthwise) {
    set_error("the linear-decomposition tile serves dense plans");
    return NWG_EUNSUPPORTED;
  }
  const long long Ho = (long long)H + 2LL * pad - r + 1, Wo = (long long)W + 2LL * pad - r + 1;
  if (Ho <= 0 || Wo <= 0) {
    set_error("kernel %d larger than padded input %dx%d (pad %d)", r, H, W, pad);
    return NWG_EINVAL;
  }
  const int c = (r + 2) / 3;
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
  g->th = (int)((Ho + 1) / 2);
  g->tw = (int)((Wo + 1) / 2);
  g->T = (long long)B * g->th * g->tw;
  g->P = 16;
  g->ld_c = c;
  const double mk = (double)M * c * c, f = (double)sizeof(float);
  const double u = f * 16 * mk * N, v = f * 16 * mk * g->T, yh = f * 4 * N * (double)g->T;
  if (u > 1e13 || v > 1e13 || g->T > 0x7fffffffLL / 64 || mk > 65535) {
    set_error("workspace too large (or more than 65535 decomposed channels)");
    return NWG_EUNSUPPORTED;
  }
  g->u_bytes = (size_t)u;
  g->v_bytes = (size_t)v;
  g->yhat_bytes = (size_t)yh;
  g->direct_flop = 2.0 * B * N * (double)M * Ho * Wo * r * r;
  g->ewmm_mults = (long long)(16 * (double)g->T * mk * N);
  g->contract_flop = 2.0 * 16 * mk * N * (double)g->T;
  g->pipeline_parts = 1;
  g->precision = NWG_PRECISION_FP32;
  g->workspace_bytes = g->u_bytes + g->v_bytes + zalloc_bytes(*g);
  return NWG_OK;
}

// NWG_TILE_AUTO: F(3x3,3x3) where it measured faster than F(2x2,3x3) --
// the fused one-output-channel kernel at depth 2 (unless F(2,3) runs the
// layer in one kernel), or both channel counts >= 32 and either a nesting
// level saved (r = 8, 9) or depth 1 (r <= 3); the mixed nest for dense
// layers with r = 16..31 and both channel counts >= 32 (on the 31x31
// 128 -> 128 layer: 1.64x fewer contraction FLOPs, 294 against 231
// TFLOP/s); F(2x2,3x3) otherwise.
int compute_geometry(int B, int M, int N, int H, int W, int r, int pad, int tile, int depthwise,
                     nwg_plan_info* g) {
  if (tile != NWG_TILE_AUTO)
    return compute_geometry_tile(B, M, N, H, W, r, pad, tile, depthwise, g);
  nwg_plan_info a, b;
  const int ra = compute_geometry_tile(B, M, N, H, W, r, pad, NWG_TILE_F2X2_3X3, depthwise, &a);
  if (ra == NWG_OK && !depthwise && a.n == 4 && M >= 32 && N >= 32) {
    if (compute_geometry_tile(B, M, N, H, W, r, pad, NWG_TILE_MIX_F23_F33, 0, &b) == NWG_OK) {
      *g = b;
      return NWG_OK;
    }
    set_error("");
  }
  if (ra != NWG_OK || depthwise || r > 9 || r == 1) {
    if (g) *g = a;
    return ra;
  }
  if (compute_geometry_tile(B, M, N, H, W, r, pad, NWG_TILE_F3X3_3X3, 0, &b) != NWG_OK) {
    set_error("");
    *g = a;
    return NWG_OK;
  }
  const bool big = M >= 32 && N >= 32;
  const bool pick = ((b.fused_input || b.fused_output) && !a.fused_conv) ||
                    (big && a.n > b.n) || (big && a.n == 1 && !a.fused_conv);
  *g = pick ? b : a;
  return NWG_OK;
}

int compute_geometry_tile(int B, int M, int N, int H, int W, int r, int pad, int tile,
                          int depthwise, nwg_plan_info* g) {
  if (!g) {
    set_error("output pointer is NULL");
    return NWG_EINVAL;
  }
  std::memset(g, 0, sizeof *g);
  if (B <= 0 || M <= 0 || N <= 0 || H <= 0 || W <= 0 || r <= 0 || pad < 0) {
    set_error("invalid shape B=%d M=%d N=%d H=%d W=%d r=%d pad=%d", B, M, N, H, W, r, pad);
    return NWG_EINVAL;
  }
  if (tile != NWG_TILE_F2X2_3X3 && tile != NWG_TILE_F3X3_3X3 && tile != NWG_TILE_LD_F2X2_3X3 &&
      tile != NWG_TILE_MIX_F23_F33) {
    set_error("unsupported tile %d", tile);
    return NWG_EUNSUPPORTED;
  }
  if (tile == NWG_TILE_LD_F2X2_3X3) return ld_geometry(B, M, N, H, W, r, pad, depthwise, g);
  const bool mix = tile == NWG_TILE_MIX_F23_F33;
  if (mix && depthwise) {
    set_error("the mixed F(2,3)/F(3,3) nest serves dense plans");
    return NWG_EUNSUPPORTED;
  }
  // up to 7 taps the mixed nest has only its two F(2,3) levels
  if (mix && r <= 7)
    return compute_geometry_tile(B, M, N, H, W, r, pad, NWG_TILE_F2X2_3X3, 0, g);
  if (mix && r > 39) {
    set_error("kernel size %d exceeds the mixed nest's 39 taps", r);
    return NWG_EUNSUPPORTED;
  }
  const bool f33 = tile == NWG_TILE_F3X3_3X3;
  if (f33 && depthwise) {
    set_error("depthwise plans use the F(2x2,3x3) tile");
    return NWG_EUNSUPPORTED;
  }
  const long long Ho = (long long)H + 2LL * pad - r + 1, Wo = (long long)W + 2LL * pad - r + 1;
  if (Ho <= 0 || Wo <= 0) {
    set_error("kernel %d larger than padded input %dx%d (pad %d)", r, H, W, pad);
    return NWG_EINVAL;
  }
  // base F(m, rb): F(2,3) or F(3,3); F(3,3) is kept to depth 2 (r <= 9),
  // where its fp32 error stays near 1e-6
  // (the mixed nest: F(2,3) at levels 1-2, F(3,3) above)
  const int m = f33 ? 3 : nwg::kOut, rb = nwg::kTaps, l = m + rb - 1;
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
      if (n >= max_depth) {
        set_error("kernel size %d needs nesting depth > %d (r <= %d supported on this tile)", r,
                  max_depth, f33 ? 9 : 31);
        return NWG_EUNSUPPORTED;
      }
      const int mj = level_m(n);
      strides[n] = s;
      Mn += s * (mj - 1);
      Kn += s * (rb - 1);
      P1 *= mj + rb - 1;
      ++n;
    }
  }
  g->B = B; g->M = M; g->N = N; g->H = H; g->W = W; g->r = r; g->pad = pad; g->tile = tile;
  g->depthwise = depthwise ? 1 : 0;
  // the kernel transform sees M_k input channels: 1 for a depthwise layer
  const int Mk = depthwise ? 1 : M;
  g->Ho = (int)Ho;
  g->Wo = (int)Wo;
  g->n = n;
  g->m = m; g->rb = rb; g->l = l;
  for (int j = 0; j < n; ++j) g->strides[j] = strides[j];
  g->Mn = Mn;
  g->Kn = Kn;
  g->Ln = n == 0 ? 1 : Mn + Kn - 1;
  g->th = (int)((Ho + Mn - 1) / Mn);
  g->tw = (int)((Wo + Mn - 1) / Mn);
  g->T = (long long)B * g->th * g->tw;
  const long long P = P1 * P1;
  g->P = P;
  g->outer33 = mix ? n - 2 : 0;
  const double f = (double)sizeof(float);
  g->direct_flop = 2.0 * B * N * (double)Mk * Ho * Wo * r * r;
  if (n == 0) {
    g->u_bytes = (size_t)Mk * N * sizeof(float);
    g->v_bytes = 0;
    g->yhat_bytes = 0;
    g->ewmm_mults = (long long)B * N * Mk * Ho * Wo;
    g->contract_flop = 2.0 * B * N * (double)Mk * Ho * Wo;
  } else {
    // the contraction writes Yhat after (part of) the level-1 output
    // transform: per (n, t) P/4 values for F(2,3) (both axes), 3 P/5 for
    // F(3,3) (columns only)
    const double zpts = f33 ? (double)(P / 5) * 3 : (double)(P / 4);
    const double u = f * P * Mk * N, v = f * P * M * g->T, yh = f * zpts * N * g->T;
    if (u > 1e13 || v > 1e13 || yh > 1e13 || g->T > 0x7fffffffLL / 64) {
      set_error("workspace too large");
      return NWG_EUNSUPPORTED;
    }
    g->u_bytes = (size_t)u;
    g->v_bytes = (size_t)v;
    g->yhat_bytes = (size_t)yh;
    g->ewmm_mults = P * g->T * Mk * (long long)N;
    g->contract_flop = 2.0 * P * (double)Mk * N * g->T;
  }
  // one or two output channels (or depthwise) at depth 3-4: the fused kernel
  // never forms V.  Few channels (or depthwise) at depth 1-2: one kernel
  // x -> y, neither V nor Z.
  g->fused_input = (f33 ? nwg::input_contract5_applies(*g) : nwg::input_contract_applies(*g)) ? 1 : 0;
  g->fused_conv =
      !f33 && !mix && (nwg::small_conv_applies(*g) || (depthwise && (n == 1 || n == 2))) ? 1 : 0;
  g->fused_output = nwg::contract_output5_applies(*g) ? 1 : 0;
  const bool no_v = g->fused_input || depthwise || g->fused_conv;
  const bool no_z = g->fused_conv || g->fused_output;
  g->workspace_bytes = g->u_bytes + (no_v ? 0 : g->v_bytes) + (no_z ? 0 : zalloc_bytes(*g));
  g->pipeline_parts = 1;
  g->precision = NWG_PRECISION_FP32;
  return NWG_OK;
}

int check_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return NWG_OK;
  set_error("%s: %s", what, hipGetErrorString(e));
  return NWG_EHIP;
}

hipEvent_t take_event(nwg_plan* p) {
  if (!p->event_pool.empty()) {
    hipEvent_t e = p->event_pool.back();
    p->event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Runs `launch` on stream s, bracketed by timing events when enabled.
template <typename F>
int timed(nwg_plan* p, int stage, hipStream_t s, const char* what, F&& launch) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (p && p->timing) {
    e0 = take_event(p);
    e1 = take_event(p);
  }
  // a launch whose events cannot be recorded runs untimed
  bool timed_ok = e0 && e1 && hipEventRecord(e0, s) == hipSuccess;
  const int rc = check_hip(launch(), what);
  timed_ok = timed_ok && hipEventRecord(e1, s) == hipSuccess;
  if (timed_ok) {
    p->pending.push_back({stage, e0, e1});
  } else {
    if (e0) p->event_pool.push_back(e0);
    if (e1) p->event_pool.push_back(e1);
  }
  return rc;
}

// Depth 0 (r = 1, pad = 0): per image, y[b] (N x HW) = U^T (N x M) * x[b] (M x HW).
nwg::ContractArgs depth0_args(const nwg_plan_info& g, const float* U, const float* x, float* y) {
  nwg::ContractArgs a{};
  const int hw = g.Ho * g.Wo;
  a.A = U;
  a.Bm = x;
  a.C = y;
  a.Nrows = g.N;
  a.K = g.M;
  a.ldA = g.N;
  a.Ncols = hw;
  a.ldB = hw;
  a.ldC = hw;
  a.sA = 0;
  a.sB = (long long)g.M * g.H * g.W;
  a.sC = (long long)g.N * hw;
  a.batch = g.B;
  return a;
}

// geometry seen by the kernel transform: one input channel when depthwise
nwg_plan_info kernel_geometry(const nwg_plan_info& g) {
  nwg_plan_info k = g;
  if (g.depthwise) k.M = 1;
  return k;
}

// ks > 1 (linear-decomposition plans, nwg_conv2d only): K slices writing
// partial Z buffers that launch_sum_parts adds
hipError_t launch_contract(const nwg_plan_info& g, const float* U, const float* V, float* Z,
                           hipStream_t s, int ks = 1) {
  if (g.depthwise)
    return g.n == 0 ? nwg::launch_dw_scale(g, V, U, Z, s) : nwg::launch_dw_contract(g, U, V, Z, s);
  if (g.n == 0) return nwg::launch_gemm_depth0(depth0_args(g, U, V, Z), s);
  if (g.tile == NWG_TILE_F3X3_3X3) return nwg::launch_contract5(g, U, V, Z, s);
  // linear decomposition: the contraction runs over M c^2 channels
  const int mk = g.ld_c > 0 ? g.M * g.ld_c * g.ld_c : g.M;
  const hipError_t e = nwg::launch_contract_fused(U, V, Z, mk, g.N, (int)g.T, g.P / 16, s,
                                                  g.precision == NWG_PRECISION_BF16_SPLIT, ks);
  if (e != hipSuccess || ks == 1) return e;
  return nwg::launch_sum_parts(Z, (size_t)(g.P / 4) * g.N * g.T, ks, s);
}

// stage launchers by tile (depth >= 1)
hipError_t launch_kxform(const nwg_plan_info& g, const float* w, float* U, hipStream_t s) {
  if (g.tile == NWG_TILE_F3X3_3X3 && g.n > 0) return nwg::launch_kernel_xform5(g, w, U, s);
  if (g.tile == NWG_TILE_MIX_F23_F33) return nwg::launch_kernel_xform_mix(g, w, U, s);
  if (g.tile == NWG_TILE_LD_F2X2_3X3) return nwg::launch_kernel_xform_ld(g, w, U, s);
  const hipError_t e = nwg::launch_kernel_xform(kernel_geometry(g), w, U, s);
  if (e != hipSuccess || g.precision != NWG_PRECISION_BF16_SPLIT) return e;
  // split precision: the fp32 U just written becomes its (hi, lo) pairs
  return nwg::launch_split_pairs(U, g.u_bytes / sizeof(float), s);
}
hipError_t launch_ixform(const nwg_plan_info& g, const float* x, float* V, float* scratch,
                         hipStream_t s) {
  if (g.tile == NWG_TILE_F3X3_3X3) return nwg::launch_input_xform5(g, x, V, s);
  if (g.tile == NWG_TILE_MIX_F23_F33) return nwg::launch_input_xform_mix(g, x, V, scratch, s);
  return nwg::launch_input_xform(g, x, V, s);
}
// Z3 (and X4 above): the mixed nest's depth-4 scratch (the plan's, after its Z)
hipError_t launch_oxform(const nwg_plan_info& g, const float* Z, float* y, float* Z3,
                         hipStream_t s) {
  if (g.tile == NWG_TILE_F3X3_3X3) return nwg::launch_output_xform5(g, Z, y, s);
  if (g.tile == NWG_TILE_MIX_F23_F33) return nwg::launch_output_xform_mix(g, Z, y, Z3, s);
  return nwg::launch_output_xform(g, Z, y, s);
}
float* mix_scratch(const nwg_plan* p) {
  return p->Yh && nwg::mix_scratch_bytes(p->info) ? p->Yh + p->info.yhat_bytes / sizeof(float)
                                                   : nullptr;
}

// Input transform and contraction in `parts` pieces on two streams: part k's
// contraction (on the plan's side stream) waits only for part k's input
// transform, so part k+1's input transform (HBM-bound) overlaps it
// (MFMA-bound).  The side stream starts after the work already queued on s
// and s continues only after the last contraction.
int run_pipelined(nwg_plan* p, const float* x, hipStream_t s) {
  const nwg_plan_info& g = p->info;
  const int np = g.pipeline_parts;
  if (!p->side) {
    int rc = check_hip(hipStreamCreateWithFlags(&p->side, hipStreamNonBlocking), "side stream");
    if (rc == NWG_OK)
      rc = check_hip(hipEventCreateWithFlags(&p->ev_start, hipEventDisableTiming), "event");
    if (rc == NWG_OK)
      rc = check_hip(hipEventCreateWithFlags(&p->ev_join, hipEventDisableTiming), "event");
    if (rc != NWG_OK) return rc;
  }
  while ((int)p->ev_part.size() < np) {
    hipEvent_t e = nullptr;
    const int rc = check_hip(hipEventCreateWithFlags(&e, hipEventDisableTiming), "event");
    if (rc != NWG_OK) return rc;
    p->ev_part.push_back(e);
  }
  int rc = check_hip(hipEventRecord(p->ev_start, s), "event record");
  if (rc == NWG_OK) rc = check_hip(hipStreamWaitEvent(p->side, p->ev_start, 0), "stream wait");
  if (rc != NWG_OK) return rc;
  const long long G = g.P / 16, Gp = G / np;
  const size_t M = g.M, N = g.N, T = g.T;
  for (int k = 0; k < np && rc == NWG_OK; ++k) {
    rc = timed(p, 1, s, "input transform launch",
               [&] { return nwg::launch_input_xform(g, x, p->V, s, k, np); });
    if (rc == NWG_OK) rc = check_hip(hipEventRecord(p->ev_part[k], s), "event record");
    if (rc == NWG_OK) rc = check_hip(hipStreamWaitEvent(p->side, p->ev_part[k], 0), "stream wait");
    if (rc != NWG_OK) break;
    const size_t g0 = (size_t)k * Gp;
    rc = timed(p, 2, p->side, "contraction launch", [&] {
      return nwg::launch_contract_fused(p->U + 16 * g0 * M * N, p->V + 16 * g0 * M * T,
                                        p->Yh + 4 * g0 * N * T, g.M, g.N, (int)g.T, Gp, p->side);
    });
  }
  // join even after an error, so that s never runs ahead of the side stream
  const int rj = check_hip(hipEventRecord(p->ev_join, p->side), "event record");
  const int rw = rj == NWG_OK ? check_hip(hipStreamWaitEvent(s, p->ev_join, 0), "stream wait") : rj;
  return rc != NWG_OK ? rc : rw;
}

int run_kernel_transform(nwg_plan* p, const nwg_plan_info& g, const float* w, float* U,
                         hipStream_t s) {
  return timed(p, 0, s, "kernel transform launch",
               [&] { return launch_kxform(g, w, U, s); });
}

}  // namespace

extern "C" {

const char* nwg_version(void) {
  return "nwg 0.3 (nested F(2x2,3x3), F(3x3,3x3) and mixed F(2,3)/F(3,3), gfx950)";
}

const char* nwg_last_error(void) { return g_last_error.c_str(); }

int nwg_plan_geometry(int B, int M, int N, int H, int W, int r, int pad, int tile,
                      nwg_plan_info* out) {
  return compute_geometry(B, M, N, H, W, r, pad, tile, 0, out);
}

int nwg_plan_geometry_depthwise(int B, int C, int H, int W, int r, int pad, int tile,
                                nwg_plan_info* out) {
  return compute_geometry(B, C, C, H, W, r, pad, tile, 1, out);
}

}  // extern "C"

namespace {

nwg_plan* create_plan(const nwg_plan_info& g) {
  if (g.n == 0 && g.pad != 0) {
    set_error("1x1 kernels with padding are not supported (pad must be 0 for r = 1)");
    return nullptr;
  }
  nwg_plan* p = new (std::nothrow) nwg_plan;
  if (!p) {
    set_error("host allocation failed");
    return nullptr;
  }
  p->info = g;
  if (hipGetDevice(&p->device) != hipSuccess) {
    set_error("no HIP device available");
    delete p;
    return nullptr;
  }
  auto alloc = [&](float** ptr, size_t bytes, const char* what) {
    if (bytes == 0) return true;
    hipError_t e = hipMalloc((void**)ptr, bytes);
    if (e != hipSuccess) {
      hipGetLastError();
      set_error("hipMalloc of %s (%zu bytes) failed: %s", what, bytes, hipGetErrorString(e));
      return false;
    }
    return true;
  };
  const bool no_v = g.fused_input || g.depthwise || g.fused_conv;
  const bool no_z = g.fused_conv || g.fused_output;
  if (!alloc(&p->U, g.u_bytes, "U") || !alloc(&p->V, no_v ? 0 : g.v_bytes, "V") ||
      !alloc(&p->Yh, no_z ? 0 : zalloc_bytes(g), "Yhat")) {
    nwg_plan_destroy(p);
    // keep the allocation message
    return nullptr;
  }
  return p;
}

}  // namespace

extern "C" {

nwg_plan* nwg_plan_create_pad(int B, int M, int N, int H, int W, int r, int pad, int tile) {
  nwg_plan_info g;
  if (compute_geometry(B, M, N, H, W, r, pad, tile, 0, &g) != NWG_OK) return nullptr;
  return create_plan(g);
}

nwg_plan* nwg_plan_create_depthwise(int B, int C, int H, int W, int r, int pad, int tile) {
  nwg_plan_info g;
  if (compute_geometry(B, C, C, H, W, r, pad, tile, 1, &g) != NWG_OK) return nullptr;
  return create_plan(g);
}

nwg_plan* nwg_plan_create(int B, int M, int N, int H, int W, int r, int tile) {
  return nwg_plan_create_pad(B, M, N, H, W, r, 0, tile);
}

void nwg_plan_destroy(nwg_plan* p) {
  if (!p) return;
  if (p->U) hipFree(p->U);
  if (p->V) hipFree(p->V);
  if (p->Yh) hipFree(p->Yh);
  for (auto& r : p->pending) {
    hipEventDestroy(r.start);
    hipEventDestroy(r.stop);
  }
  for (auto e : p->event_pool) hipEventDestroy(e);
  for (auto e : p->ev_part) hipEventDestroy(e);
  if (p->ev_start) hipEventDestroy(p->ev_start);
  if (p->ev_join) hipEventDestroy(p->ev_join);
  if (p->side) hipStreamDestroy(p->side);
  delete p;
}

int nwg_plan_query(const nwg_plan* p, nwg_plan_info* out) {
  if (!p || !out) {
    set_error("NULL plan or output");
    return NWG_EINVAL;
  }
  *out = p->info;
  return NWG_OK;
}

int nwg_kernel_transform(const nwg_plan* p, const float* w, float* U, void* stream) {
  if (!p || !w || !U) {
    set_error("NULL argument to nwg_kernel_transform");
    return NWG_EINVAL;
  }
  return check_hip(launch_kxform(p->info, w, U, (hipStream_t)stream), "kernel transform launch");
}

int nwg_input_transform(const nwg_plan* p, const float* x, float* V, void* stream) {
  if (!p || !x || !V) {
    set_error("NULL argument to nwg_input_transform");
    return NWG_EINVAL;
  }
  if (p->info.n == 0) {
    set_error("depth 0 (r = 1) has no input transform");
    return NWG_EINVAL;
  }
  return check_hip(launch_ixform(p->info, x, V, mix_scratch(p), (hipStream_t)stream),
                   "input transform launch");
}

int nwg_contract(const nwg_plan* p, const float* U, const float* V, float* Yh, void* stream) {
  if (!p || !U || !V || !Yh) {
    set_error("NULL argument to nwg_contract");
    return NWG_EINVAL;
  }
  return check_hip(launch_contract(p->info, U, V, Yh, (hipStream_t)stream),
                   "contraction launch");
}

int nwg_input_contract(const nwg_plan* p, const float* x, const float* U, float* Yh,
                       void* stream) {
  if (!p || !x || !U || !Yh) {
    set_error("NULL argument to nwg_input_contract");
    return NWG_EINVAL;
  }
  if (p->info.tile != NWG_TILE_F2X2_3X3 || !nwg::input_contract_applies(p->info)) {
    set_error("fused input transform + contraction needs the F(2x2,3x3) tile, depth 3 or 4 "
              "and N <= 2 or a "
              "depthwise plan (depth %d, N = %d)", p->info.n, p->info.N);
    return NWG_EUNSUPPORTED;
  }
  return check_hip(nwg::launch_input_contract(p->info, x, U, Yh, (hipStream_t)stream),
                   "fused input transform + contraction launch");
}

int nwg_output_transform(const nwg_plan* p, const float* Yh, float* y, void* stream) {
  if (!p || !Yh || !y) {
    set_error("NULL argument to nwg_output_transform");
    return NWG_EINVAL;
  }
  if (p->info.n == 0) {
    set_error("depth 0 (r = 1) has no output transform");
    return NWG_EINVAL;
  }
  return check_hip(launch_oxform(p->info, Yh, y, mix_scratch(p), (hipStream_t)stream),
                   "output transform launch");
}

int nwg_plan_set_weights(nwg_plan* p, const float* w, void* stream) {
  if (!p || !w) {
    set_error("NULL argument to nwg_plan_set_weights");
    return NWG_EINVAL;
  }
  const int rc = run_kernel_transform(p, p->info, w, p->U, (hipStream_t)stream);
  if (rc == NWG_OK) {
    p->cached_w = w;
    p->weights_valid = true;
  } else {
    p->weights_valid = false;
  }
  return rc;
}

int nwg_conv2d(nwg_plan* p, const float* x, const float* w, float* y, void* stream) {
  if (!p || !x || !w || !y) {
    set_error("NULL argument to nwg_conv2d");
    return NWG_EINVAL;
  }
  hipStream_t s = (hipStream_t)stream;
  const nwg_plan_info& g = p->info;
  if (!p->weights_valid || p->cached_w != w) {
    const int rc = nwg_plan_set_weights(p, w, stream);
    if (rc != NWG_OK) return rc;
  }
  if (g.n == 0) {
    return timed(p, 2, s, "contraction launch",
                 [&] { return launch_contract(g, p->U, x, y, s); });
  }
  if (g.fused_conv) {
    // input transform, channel sum (or product) and output transform in one kernel
    return timed(p, 2, s, "single-kernel convolution launch", [&] {
      return g.depthwise ? nwg::launch_dw_small(g, x, p->U, y, s)
                         : nwg::launch_small_conv(g, x, p->U, y, s);
    });
  }
  int rc;
  if (g.fused_input && g.tile == NWG_TILE_F3X3_3X3) {
    // partial Z9 per input-channel group, summed by the output transform
    const int parts = nwg::input_contract5_parts(g);
    rc = timed(p, 2, s, "fused input transform + contraction launch", [&] {
      const hipError_t e = nwg::launch_input_contract5(g, x, p->U, p->Yh, s);
      if (e != hipSuccess) return e;
      return nwg::launch_sum_parts(p->Yh, (size_t)(g.P / 25) * 9 * g.N * g.T, parts, s);
    });
    if (rc != NWG_OK) return rc;
    return timed(p, 3, s, "output transform launch",
                 [&] { return nwg::launch_output_xform5(g, p->Yh, y, s, 1, true); });
  } else if (g.fused_input) {
    rc = timed(p, 2, s, "fused input transform + contraction launch",
               [&] { return nwg::launch_input_contract(g, x, p->U, p->Yh, s); });
  } else if (g.pipeline_parts > 1) {
    rc = run_pipelined(p, x, s);
  } else {
    rc = timed(p, 1, s, "input transform launch",
               [&] { return launch_ixform(g, x, p->V, mix_scratch(p), s); });
    if (rc != NWG_OK) return rc;
    if (g.fused_output)
      return timed(p, 2, s, "contraction + output transform launch",
                   [&] { return nwg::launch_contract_output5(g, p->V, p->U, y, s); });
    rc = timed(p, 2, s, "contraction launch",
               [&] { return launch_contract(g, p->U, p->V, p->Yh, s, ld_kslices(g)); });
  }
  if (rc != NWG_OK) return rc;
  return timed(p, 3, s, "output transform launch",
               [&] { return launch_oxform(g, p->Yh, y, mix_scratch(p), s); });
}

int nwg_plan_set_precision(nwg_plan* p, int precision) {
  if (!p) {
    set_error("NULL plan");
    return NWG_EINVAL;
  }
  if (precision != NWG_PRECISION_FP32 && precision != NWG_PRECISION_BF16_SPLIT) {
    set_error("unknown precision %d", precision);
    return NWG_EINVAL;
  }
  const nwg_plan_info& g = p->info;
  if (precision == NWG_PRECISION_BF16_SPLIT &&
      (g.tile != NWG_TILE_F2X2_3X3 || g.n < 1 || g.depthwise || g.fused_input || g.fused_conv ||
       g.pipeline_parts > 1 || g.M % 32 || g.N % 64 || g.T < 64)) {
    set_error("split precision needs a dense, unfused, unpipelined F(2x2,3x3) plan at depth "
              ">= 1 with M %% 32 == 0, N %% 64 == 0 and T >= 64 (M = %d, N = %d, T = %lld)",
              g.M, g.N, g.T);
    return NWG_EUNSUPPORTED;
  }
  if (precision != g.precision) {
    p->info.precision = precision;
    p->weights_valid = false;
  }
  return NWG_OK;
}

int nwg_plan_set_pipeline(nwg_plan* p, int parts) {
  if (!p) {
    set_error("NULL plan");
    return NWG_EINVAL;
  }
  if (parts == 1) {
    p->info.pipeline_parts = 1;
    return NWG_OK;
  }
  if (parts != 2 && parts != 4 && parts != 8 && parts != 16) {
    set_error("pipeline parts must be 1, 2, 4, 8 or 16 (got %d)", parts);
    return NWG_EINVAL;
  }
  if (!pipeline_allowed(p->info)) {
    set_error("the two-stream pipeline needs a dense depth-4 plan with M %% 32 == 0, "
              "N %% 64 == 0 and T %% 64 == 0");
    return NWG_EUNSUPPORTED;
  }
  p->info.pipeline_parts = parts;
  return NWG_OK;
}

int nwg_plan_set_timing(nwg_plan* p, int enable) {
  if (!p) {
    set_error("NULL plan");
    return NWG_EINVAL;
  }
  p->timing = enable != 0;
  return NWG_OK;
}

int nwg_plan_get_timing(nwg_plan* p, double ms[4], long long count[4]) {
  if (!p || !ms || !count) {
    set_error("NULL argument to nwg_plan_get_timing");
    return NWG_EINVAL;
  }
  int rc = NWG_OK;
  for (auto& r : p->pending) {
    float t = 0.0f;
    if (rc == NWG_OK) rc = check_hip(hipEventSynchronize(r.stop), "timing event sync");
    if (rc == NWG_OK) rc = check_hip(hipEventElapsedTime(&t, r.start, r.stop), "elapsed time");
    if (rc == NWG_OK) {
      ms[r.stage] += t;
      count[r.stage] += 1;
    }
    p->event_pool.push_back(r.start);
    p->event_pool.push_back(r.stop);
  }
  p->pending.clear();
  return rc;
}

}  // extern "C"
