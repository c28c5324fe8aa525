// Host-only part of the nested-Winograd library: the plan geometry (the
// level recurrence of Sec. III.B), the choice of kernels a plan takes, its
// workspace, and the per-thread error state.  Plain C++: no HIP header, so
// that it also builds for the CPU alone (and under the address and
// undefined-behaviour sanitizers, which the library's tests do).
#pragma once

#include <cstddef>

#include "../../include/nwg.h"

namespace nwg {

// Per-thread error state behind nwg_last_error / nwg_last_status: `fail`
// records a status and a message and returns the status.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Geometry of a dense (depthwise = 0) or depthwise plan on `tile`, including
// NWG_TILE_AUTO's choice.  NWG_OK, or a status with a message.
int compute_geometry(int B, int M, int N, int H, int W, int r, int pad, int tile, int depthwise,
                     nwg_plan_info* g);

// Arguments nwg_plan_create* takes beyond the geometry (r = 1 has no padding).
int check_plan_request(const nwg_plan_info& g);

// Which kernels a plan runs (by its geometry).
// F(2x2,3x3), depth 3-4, N <= 2 or depthwise: x, U -> Z without V.
bool input_contract_applies(const nwg_plan_info& g);
// F(2x2,3x3), few channels at depth 1-2: x -> y in one kernel.
bool small_conv_applies(const nwg_plan_info& g);
// F(3x3,3x3), depth 2, one output channel: x -> partial Z9 without V.
bool input_contract5_applies(const nwg_plan_info& g);
// F(3x3,3x3), one or two input channels (not the case above): V -> y.
bool contract_output5_applies(const nwg_plan_info& g);

// The fused F(3x3,3x3) kernel's work split: a box of RX x RY tiles of one
// image per work-group, `groups` input-channel groups of `mper` channels,
// `lds` bytes of LDS.
struct IC5Shape {
  int RX, RY, nbx, nby, groups, mper;
  size_t lds;
};
IC5Shape ic5_shape(const nwg_plan_info& g);
int input_contract5_parts(const nwg_plan_info& g);
size_t input_contract5_zbytes(const nwg_plan_info& g);

// Mixed nest: the F(3,3) levels above the two F(2,3) levels (0 on other
// tiles) and the bytes of the depth-4 scratch its transforms use.
constexpr int kMixL3 = 26;                  // window side left for levels 1..3
int mix_outer_levels(const nwg_plan_info& g);
size_t mix_scratch_bytes(const nwg_plan_info& g);

// K slices of a linear-decomposition plan's contraction (1 otherwise).
int ld_kslices(const nwg_plan_info& g);
// Bytes of the plan's Z buffer (with the partial sums or scratch it holds).
size_t zalloc_bytes(const nwg_plan_info& g);
// Whether V / Z are part of the plan's workspace.
bool plan_holds_v(const nwg_plan_info& g);
bool plan_holds_z(const nwg_plan_info& g);
// Plans that nwg_plan_set_pipeline can split over two streams.
bool pipeline_allowed(const nwg_plan_info& g);
// Plans that can take NWG_PRECISION_BF16_SPLIT.
bool split_allowed(const nwg_plan_info& g);

// The contraction's list of groups (nwg_plan_info::live_np): entry i is the
// group with row prefix p_r = the (i / np)-th live prefix and column prefix
// p_c = the (i % np)-th, at g = sum_d digit_d(p_r) wr[d] + digit_d(p_c) wc[d]
// (digit d = q_{d+2}, the least significant first).  np = 0: entry i is
// group i.
struct GroupMap {
  int np;                       // live prefixes per axis; 0: every group
  int nd;                       // digits of a prefix (levels 2..n), at most 3
  unsigned long long mask0, mask1;   // live prefixes (bit i: prefix i)
  int rad[3], wr[3], wc[3];     // radix of digit d, its weight in g for rows and columns
  int q3;                       // 1: level-1 digit 3 is dead (nwg_plan_info::level1_live
                                // = 0x7): quads q1r = 0..2 of a group only
};
GroupMap group_map(const nwg_plan_info& g);

}  // namespace nwg
