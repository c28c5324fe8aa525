// Device side of the nested-Winograd plan: its workspace, the weight cache,
// the C ABI of include/nwg.h that queues work (the geometry, level
// recurrence and error state are in plan.cpp) and per-stage timing.  All
// device work is queued on the caller's stream.
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

using nwg::fail;

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

// NWG_DEBUG_SYNC set in the environment: every call waits for each kernel it
// queues and reports a failure there, naming the kernel (not for use under
// stream capture).
bool debug_sync() {
  static const bool on = std::getenv("NWG_DEBUG_SYNC") != nullptr;
  return on;
}

int check_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return NWG_OK;
  return fail(NWG_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// A launch's status; with NWG_DEBUG_SYNC also its completion on stream s.
int check_launch(hipError_t e, const char* what, hipStream_t s) {
  int rc = check_hip(e, what);
  if (rc == NWG_OK && debug_sync()) {
    const hipError_t es = hipStreamSynchronize(s);
    if (es != hipSuccess) rc = fail(NWG_EHIP, "%s (completion): %s", what, hipGetErrorString(es));
  }
  return rc;
}

// The device a stream's work runs on: its own for a created stream, the
// current device for the NULL stream.
int stream_device(hipStream_t s, int* dev) {
  const hipError_t e = s ? hipStreamGetDevice(s, dev) : hipGetDevice(dev);
  if (e != hipSuccess) {
    hipGetLastError();
    return fail(NWG_EHIP, "device of the stream: %s", hipGetErrorString(e));
  }
  return NWG_OK;
}

// Work that touches a plan's workspace must run on the device that holds it,
// with that device current (the plan's side stream and events are created
// on the current device).
int check_plan_device(const nwg_plan* p, hipStream_t s) {
  int dev = -1, cur = -1;
  int rc = stream_device(s, &dev);
  if (rc == NWG_OK) rc = stream_device(nullptr, &cur);
  if (rc != NWG_OK) return rc;
  if (dev != p->device || cur != p->device)
    return fail(NWG_EINVAL,
                "the plan's workspace is on device %d; the stream runs on device %d and "
                "device %d is current", p->device, dev, cur);
  return NWG_OK;
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
  const hipError_t el = launch();
  timed_ok = timed_ok && hipEventRecord(e1, s) == hipSuccess;
  const int rc = check_launch(el, what, s);
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
  // the mixed nest contracts its live groups only (the others' Z is zero)
  const nwg::GroupMap gm = nwg::group_map(g);
  if (g.mix_planar)
    return nwg::launch_contract_planar(U, V, Z, g.M, g.N, (int)g.T, g.live_groups, gm, s);
  const long long G = gm.np > 0 ? g.live_groups : g.P / 16;
  const hipError_t e = nwg::launch_contract_fused(U, V, Z, mk, g.N, (int)g.T, G, s,
                                                  g.precision == NWG_PRECISION_BF16_SPLIT, ks, gm);
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

// A plan's buffers: U (transformed weights), V and Z (with the partial sums
// or the mixed nest's scratch after it); NULL where the plan holds none.
struct Workspace {
  const float* U;
  float* V;
  float* Yh;
};

float* mix_scratch_of(const nwg_plan_info& g, float* Yh) {
  return Yh && nwg::mix_scratch_bytes(g) ? Yh + g.yhat_bytes / sizeof(float) : nullptr;
}

// Everything nwg_conv2d queues after the kernel transform: the kernels the
// plan's geometry selects, on stream s.  p supplies the timing records and
// the two-stream pipeline; NULL runs untimed (and needs pipeline_parts = 1).
int run_steps(nwg_plan* p, const nwg_plan_info& g, const Workspace& ws, const float* x,
              float* y, hipStream_t s) {
  const float* U = ws.U;
  if (g.n == 0) {
    return timed(p, 2, s, "contraction launch", [&] { return launch_contract(g, U, x, y, s); });
  }
  if (g.fused_conv) {
    // input transform, channel sum (or product) and output transform in one kernel
    return timed(p, 2, s, "single-kernel convolution launch", [&] {
      return g.depthwise ? nwg::launch_dw_small(g, x, U, y, s)
                         : nwg::launch_small_conv(g, x, U, y, s);
    });
  }
  int rc;
  if (g.fused_input && g.tile == NWG_TILE_F3X3_3X3) {
    // partial Z9 per input-channel group, summed by the output transform
    const int parts = nwg::input_contract5_parts(g);
    rc = timed(p, 2, s, "fused input transform + contraction launch", [&] {
      const hipError_t e = nwg::launch_input_contract5(g, x, U, ws.Yh, s);
      if (e != hipSuccess) return e;
      return nwg::launch_sum_parts(ws.Yh, (size_t)(g.P / 25) * 9 * g.N * g.T, parts, s);
    });
    if (rc != NWG_OK) return rc;
    return timed(p, 3, s, "output transform launch",
                 [&] { return nwg::launch_output_xform5(g, ws.Yh, y, s, 1, true); });
  } else if (g.fused_input) {
    rc = timed(p, 2, s, "fused input transform + contraction launch",
               [&] { return nwg::launch_input_contract(g, x, U, ws.Yh, s); });
  } else if (g.pipeline_parts > 1) {
    if (!p) return fail(NWG_EUNSUPPORTED, "the two-stream pipeline needs a plan");
    rc = run_pipelined(p, x, s);
  } else {
    rc = timed(p, 1, s, "input transform launch",
               [&] { return launch_ixform(g, x, ws.V, mix_scratch_of(g, ws.Yh), s); });
    if (rc != NWG_OK) return rc;
    if (g.fused_output)
      return timed(p, 2, s, "contraction + output transform launch",
                   [&] { return nwg::launch_contract_output5(g, ws.V, U, y, s); });
    rc = timed(p, 2, s, "contraction launch",
               [&] { return launch_contract(g, U, ws.V, ws.Yh, s, nwg::ld_kslices(g)); });
  }
  if (rc != NWG_OK) return rc;
  return timed(p, 3, s, "output transform launch",
               [&] { return launch_oxform(g, ws.Yh, y, mix_scratch_of(g, ws.Yh), s); });
}

}  // namespace


namespace {

nwg_plan* create_plan(const nwg_plan_info& g) {
  if (nwg::check_plan_request(g) != NWG_OK) return nullptr;
  nwg_plan* p = new (std::nothrow) nwg_plan;
  if (!p) {
    fail(NWG_ENOMEM, "host allocation of the plan failed");
    return nullptr;
  }
  p->info = g;
  if (hipGetDevice(&p->device) != hipSuccess) {
    hipGetLastError();
    fail(NWG_EHIP, "no HIP device available");
    delete p;
    return nullptr;
  }
  // a failed hipMalloc is an allocation failure (NWG_ENOMEM), whatever the
  // runtime's code for it; the plan is released with what it holds
  auto alloc = [&](float** ptr, size_t bytes, const char* what) {
    if (bytes == 0) return true;
    const hipError_t e = hipMalloc((void**)ptr, bytes);
    if (e != hipSuccess) {
      *ptr = nullptr;
      hipGetLastError();
      fail(NWG_ENOMEM, "hipMalloc of %s (%zu bytes) failed: %s", what, bytes,
           hipGetErrorString(e));
      return false;
    }
    return true;
  };
  const size_t vb = nwg::plan_holds_v(g) ? g.v_bytes : 0;
  const size_t zb = nwg::plan_holds_z(g) ? nwg::zalloc_bytes(g) : 0;
  if (!alloc(&p->U, g.u_bytes, "U") || !alloc(&p->V, vb, "V") || !alloc(&p->Yh, zb, "Yhat")) {
    nwg_plan_destroy(p);    // frees nothing it did not allocate; keeps the message
    return nullptr;
  }
  return p;
}

}  // namespace

// The launch sequence of nwg_conv2d on caller-provided workspace, for entry
// points that hold no plan (untimed, one stream).
namespace nwg {

int kernel_transform_into(const nwg_plan_info& g, const float* w, float* U, hipStream_t s) {
  return check_launch(launch_kxform(g, w, U, s), "kernel transform launch", s);
}

int conv_steps(const nwg_plan_info& g, const float* U, float* V, float* Yh, const float* x,
               float* y, hipStream_t s) {
  return run_steps(nullptr, g, {U, V, Yh}, x, y, s);
}

}  // namespace nwg

extern "C" {

nwg_plan* nwg_plan_create_pad(int B, int M, int N, int H, int W, int r, int pad, int tile) {
  nwg_plan_info g;
  if (nwg::compute_geometry(B, M, N, H, W, r, pad, tile, 0, &g) != NWG_OK) return nullptr;
  return create_plan(g);
}

nwg_plan* nwg_plan_create_depthwise(int B, int C, int H, int W, int r, int pad, int tile) {
  nwg_plan_info g;
  if (nwg::compute_geometry(B, C, C, H, W, r, pad, tile, 1, &g) != NWG_OK) return nullptr;
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
  if (!p || !out) return fail(NWG_EINVAL, "NULL plan or output");
  *out = p->info;
  return NWG_OK;
}

int nwg_kernel_transform(const nwg_plan* p, const float* w, float* U, void* stream) {
  if (!p || !w || !U)
    return fail(NWG_EINVAL, "NULL argument to nwg_kernel_transform");
  hipStream_t s = (hipStream_t)stream;
  return check_launch(launch_kxform(p->info, w, U, s), "kernel transform launch", s);
}

int nwg_input_transform(const nwg_plan* p, const float* x, float* V, void* stream) {
  if (!p || !x || !V)
    return fail(NWG_EINVAL, "NULL argument to nwg_input_transform");
  if (p->info.n == 0)
    return fail(NWG_EINVAL, "depth 0 (r = 1) has no input transform");
  hipStream_t s = (hipStream_t)stream;
  if (mix_scratch(p)) {   // the plan's scratch is part of this call
    const int rd = check_plan_device(p, s);
    if (rd != NWG_OK) return rd;
  }
  return check_launch(launch_ixform(p->info, x, V, mix_scratch(p), s), "input transform launch", s);
}

int nwg_contract(const nwg_plan* p, const float* U, const float* V, float* Yh, void* stream) {
  if (!p || !U || !V || !Yh)
    return fail(NWG_EINVAL, "NULL argument to nwg_contract");
  hipStream_t s = (hipStream_t)stream;
  return check_launch(launch_contract(p->info, U, V, Yh, s), "contraction launch", s);
}

int nwg_input_contract(const nwg_plan* p, const float* x, const float* U, float* Yh,
                       void* stream) {
  if (!p || !x || !U || !Yh)
    return fail(NWG_EINVAL, "NULL argument to nwg_input_contract");
  if (p->info.tile != NWG_TILE_F2X2_3X3 || !nwg::input_contract_applies(p->info))
    return fail(NWG_EUNSUPPORTED,
                "fused input transform + contraction needs the F(2x2,3x3) tile, depth 3 or 4 "
                "and N <= 2 or a depthwise plan (depth %d, N = %d)", p->info.n, p->info.N);
  return check_launch(nwg::launch_input_contract(p->info, x, U, Yh, (hipStream_t)stream),
                      "fused input transform + contraction launch", (hipStream_t)stream);
}

int nwg_output_transform(const nwg_plan* p, const float* Yh, float* y, void* stream) {
  if (!p || !Yh || !y)
    return fail(NWG_EINVAL, "NULL argument to nwg_output_transform");
  if (p->info.n == 0)
    return fail(NWG_EINVAL, "depth 0 (r = 1) has no output transform");
  hipStream_t s = (hipStream_t)stream;
  if (mix_scratch(p)) {   // the plan's scratch is part of this call
    const int rd = check_plan_device(p, s);
    if (rd != NWG_OK) return rd;
  }
  return check_launch(launch_oxform(p->info, Yh, y, mix_scratch(p), s), "output transform launch",
                      s);
}

int nwg_plan_set_weights(nwg_plan* p, const float* w, void* stream) {
  if (!p || !w)
    return fail(NWG_EINVAL, "NULL argument to nwg_plan_set_weights");
  const int rd = check_plan_device(p, (hipStream_t)stream);
  if (rd != NWG_OK) return rd;
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
  if (!p || !x || !w || !y)
    return fail(NWG_EINVAL, "NULL argument to nwg_conv2d");
  const int rd = check_plan_device(p, (hipStream_t)stream);
  if (rd != NWG_OK) return rd;
  if (!p->weights_valid || p->cached_w != w) {
    const int rc = nwg_plan_set_weights(p, w, stream);
    if (rc != NWG_OK) return rc;
  }
  return run_steps(p, p->info, {p->U, p->V, p->Yh}, x, y, (hipStream_t)stream);
}

int nwg_plan_set_precision(nwg_plan* p, int precision) {
  if (!p)
    return fail(NWG_EINVAL, "NULL plan");
  if (precision != NWG_PRECISION_FP32 && precision != NWG_PRECISION_BF16_SPLIT)
    return fail(NWG_EINVAL, "unknown precision %d", precision);
  const nwg_plan_info& g = p->info;
  if (precision == NWG_PRECISION_BF16_SPLIT && !nwg::split_allowed(g))
    return fail(NWG_EUNSUPPORTED,
                "split precision needs a dense, unfused, unpipelined F(2x2,3x3) plan at depth "
                ">= 1 with M %% 32 == 0, N %% 64 == 0 and T >= 64 (M = %d, N = %d, T = %lld)",
                g.M, g.N, g.T);
  if (precision != g.precision) {
    p->info.precision = precision;
    p->weights_valid = false;
  }
  return NWG_OK;
}

int nwg_plan_set_pipeline(nwg_plan* p, int parts) {
  if (!p)
    return fail(NWG_EINVAL, "NULL plan");
  if (parts == 1) {
    p->info.pipeline_parts = 1;
    return NWG_OK;
  }
  if (parts != 2 && parts != 4 && parts != 8 && parts != 16)
    return fail(NWG_EINVAL, "pipeline parts must be 1, 2, 4, 8 or 16 (got %d)", parts);
  if (!nwg::pipeline_allowed(p->info))
    return fail(NWG_EUNSUPPORTED,
                "the two-stream pipeline needs a dense depth-4 plan with M %% 32 == 0, "
                "N %% 64 == 0 and T %% 64 == 0");
  p->info.pipeline_parts = parts;
  return NWG_OK;
}

int nwg_plan_set_timing(nwg_plan* p, int enable) {
  if (!p)
    return fail(NWG_EINVAL, "NULL plan");
  p->timing = enable != 0;
  return NWG_OK;
}

int nwg_plan_get_timing(nwg_plan* p, double ms[4], long long count[4]) {
  if (!p || !ms || !count)
    return fail(NWG_EINVAL, "NULL argument to nwg_plan_get_timing");
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
