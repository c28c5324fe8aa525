// Exercises the library's host-only plan code (csrc/plan.cpp) on the CPU,
// built with the address and undefined-behaviour sanitizers by
// tests/test_host_sanitize_cpu.py: a seeded sweep over shapes, tiles and
// extreme values (INT_MAX, 0, negatives, NULL outputs), checking on every
// accepted plan the identities of the level recurrence (Sec. III.B) and
// the bookkeeping the rest of the library relies on.  Prints one line per
// named shape for the Python side to compare with the GPU build's answers.
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "../../paper_2102_13272_amd/csrc/plan.h"

namespace {

int failures = 0;

void expect(bool ok, const char* what, const nwg_plan_info& g) {
  if (ok) return;
  ++failures;
  std::fprintf(stderr, "FAIL %s: B=%d M=%d N=%d H=%d W=%d r=%d pad=%d tile=%d dw=%d\n", what, g.B,
               g.M, g.N, g.H, g.W, g.r, g.pad, g.tile, g.depthwise);
}

// identities every accepted plan satisfies
void check_plan(const nwg_plan_info& g) {
  expect(g.Ho == (long long)g.H + 2LL * g.pad - g.r + 1, "Ho", g);
  expect(g.Wo == (long long)g.W + 2LL * g.pad - g.r + 1, "Wo", g);
  expect(g.n >= 0 && g.n <= NWG_MAX_DEPTH, "depth", g);
  expect(g.Kn >= g.r, "K_n covers r", g);
  expect(g.n == 0 || g.Ln == g.Mn + g.Kn - 1, "L_n", g);
  expect((long long)g.th * g.Mn >= g.Ho && (long long)(g.th - 1) * g.Mn < g.Ho, "th", g);
  expect((long long)g.tw * g.Mn >= g.Wo && (long long)(g.tw - 1) * g.Mn < g.Wo, "tw", g);
  expect(g.T == (long long)g.B * g.th * g.tw, "T", g);
  if (g.tile != NWG_TILE_LD_F2X2_3X3) {
    // P = prod over levels of l_j^2; strides follow s_j = min(M_j, K_j)
    long long P1 = 1;
    int Mj = 1, Kj = 1;
    for (int j = 0; j < g.n; ++j) {
      const int mj = (g.tile == NWG_TILE_MIX_F23_F33 && j >= 2) || g.tile == NWG_TILE_F3X3_3X3
                         ? 3 : 2;
      const int s = j == 0 ? 1 : (Mj < Kj ? Mj : Kj);
      expect(g.strides[j] == s, "stride", g);
      if (j == 0) {
        Mj = mj;
        Kj = 3;
      } else {
        Mj += s * (mj - 1);
        Kj += s * 2;
      }
      P1 *= mj + 2;
    }
    expect(g.n == 0 || (Mj == g.Mn && Kj == g.Kn), "M_n, K_n", g);
    expect(g.P == P1 * P1, "P", g);
    const int Mk = g.depthwise ? 1 : g.M;
    if (g.n > 0 && g.mix_planar) {
      // planar mixed layout: the 9 live points of each live group
      expect(g.tile == NWG_TILE_MIX_F23_F33 && g.n == 4 && g.level1_live == 0x7 &&
                 g.live_np > 0 && g.live_groups == (long long)g.live_np * g.live_np,
             "planar conditions", g);
      expect(g.u_bytes == (size_t)(36.0 * (double)g.live_groups * Mk * g.N), "u_bytes", g);
      expect(g.v_bytes == (size_t)(36.0 * (double)g.live_groups * g.M * (double)g.T),
             "v_bytes", g);
    } else if (g.n > 0) {
      expect(g.u_bytes == (size_t)(4.0 * (double)g.P * Mk * g.N), "u_bytes", g);
      expect(g.v_bytes == (size_t)(4.0 * (double)g.P * g.M * (double)g.T), "v_bytes", g);
    }
  }
  size_t ws = g.u_bytes;
  if (nwg::plan_holds_v(g)) ws += g.v_bytes;
  if (nwg::plan_holds_z(g)) ws += nwg::zalloc_bytes(g);
  expect(ws == g.workspace_bytes, "workspace", g);
  expect(nwg::ld_kslices(g) >= 1, "K slices", g);
  if (g.fused_input && g.tile == NWG_TILE_F3X3_3X3) {
    const nwg::IC5Shape c = nwg::ic5_shape(g);
    expect(c.groups >= 1 && c.mper >= 1 && (long long)c.groups * c.mper >= g.M, "ic5", g);
  }
  (void)nwg::pipeline_allowed(g);
  (void)nwg::split_allowed(g);
  (void)nwg::mix_scratch_bytes(g);
}

uint64_t state = 0x9e3779b97f4a7c15ull;
uint64_t next() {
  state ^= state << 13;
  state ^= state >> 7;
  state ^= state << 17;
  return state;
}
int pick(const int* v, int n) { return v[next() % (uint64_t)n]; }

}  // namespace

int main(int argc, char** argv) {
  const int tiles[] = {NWG_TILE_F2X2_3X3, NWG_TILE_F3X3_3X3, NWG_TILE_LD_F2X2_3X3,
                       NWG_TILE_MIX_F23_F33, NWG_TILE_AUTO, 7, -2};
  const int ints[] = {INT_MIN, -1, 0, 1, 2, 3, 5, 16, 32, 33, 56, 64, 128, 1000, 65535, 65536,
                      1 << 20, INT_MAX - 1, INT_MAX};
  const int rs[] = {INT_MIN, -1, 0, 1, 2, 3, 4, 5, 7, 8, 9, 10, 13, 15, 16, 17, 23, 31, 32, 39,
                    40, 63, INT_MAX};
  const long sweep = argc > 1 ? std::atol(argv[1]) : 200000;
  long accepted = 0;
  nwg_plan_info g;
  for (long it = 0; it < sweep; ++it) {
    const int B = pick(ints, 19), M = pick(ints, 19), N = pick(ints, 19);
    const int H = pick(ints, 19), W = pick(ints, 19), r = pick(rs, 23);
    const int pad = (next() & 1) ? pick(ints, 19) : (r > 0 ? (r - 1) / 2 : 0);
    const int tile = pick(tiles, 7);
    std::memset(&g, 0xa5, sizeof g);
    const int rc = (next() & 3) == 0 ? nwg_plan_geometry_depthwise(B, M, H, W, r, pad, tile, &g)
                                     : nwg_plan_geometry(B, M, N, H, W, r, pad, tile, &g);
    if (rc == NWG_OK) {
      ++accepted;
      check_plan(g);
    } else if (rc != NWG_EINVAL && rc != NWG_EUNSUPPORTED) {
      ++failures;
      std::fprintf(stderr, "FAIL status %d\n", rc);
    } else if (nwg_last_status() != rc || nwg_last_error()[0] == '\0') {
      ++failures;
      std::fprintf(stderr, "FAIL error state for status %d\n", rc);
    }
  }
  // NULL output on every tile, both entry points
  for (int tile : tiles) {
    if (nwg_plan_geometry(1, 4, 4, 16, 16, 4, 0, tile, nullptr) != NWG_EINVAL ||
        nwg_plan_geometry_depthwise(1, 4, 16, 16, 4, 0, tile, nullptr) != NWG_EINVAL) {
      ++failures;
      std::fprintf(stderr, "FAIL NULL output accepted on tile %d\n", tile);
    }
  }
  // the named shapes: one line each for the Python side
  const int named[][9] = {
      {1, 4, 4, 16, 16, 4, 0, NWG_TILE_F2X2_3X3, 0},  {1, 32, 32, 64, 64, 7, 3, NWG_TILE_AUTO, 0},
      {8, 64, 64, 56, 56, 13, 6, NWG_TILE_AUTO, 0},   {16, 128, 128, 56, 56, 31, 15, NWG_TILE_AUTO, 0},
      {16, 128, 128, 56, 56, 31, 15, NWG_TILE_F2X2_3X3, 0},
      {4, 32, 1, 256, 256, 9, 4, NWG_TILE_AUTO, 0},   {4, 1, 32, 256, 256, 5, 2, NWG_TILE_AUTO, 0},
      {4, 5, 5, 256, 256, 3, 1, NWG_TILE_AUTO, 0},    {4, 32, 5, 256, 256, 1, 0, NWG_TILE_AUTO, 0},
      {8, 54, 54, 83, 83, 7, 3, NWG_TILE_AUTO, 1},    {8, 64, 64, 56, 56, 13, 6, NWG_TILE_LD_F2X2_3X3, 0},
      {2, 33, 20, 40, 40, 23, 11, NWG_TILE_MIX_F23_F33, 0},
      {1, 64, 1, 256, 256, 9, 4, NWG_TILE_F3X3_3X3, 0}};
  for (const auto& c : named) {
    const int rc = c[8] ? nwg_plan_geometry_depthwise(c[0], c[1], c[3], c[4], c[5], c[6], c[7], &g)
                        : nwg_plan_geometry(c[0], c[1], c[2], c[3], c[4], c[5], c[6], c[7], &g);
    if (rc != NWG_OK) {
      ++failures;
      std::fprintf(stderr, "FAIL named shape rejected: %s\n", nwg_last_error());
      continue;
    }
    check_plan(g);
    std::printf("%d %d %d %d %d %d %d %d %d -> tile %d n %d Mn %d Kn %d Ln %d th %d tw %d T %lld "
                "P %lld u %zu v %zu z %zu ws %zu fi %d fc %d fo %d o33 %d ldc %d\n",
                c[0], c[1], c[2], c[3], c[4], c[5], c[6], c[7], c[8], g.tile, g.n, g.Mn, g.Kn,
                g.Ln, g.th, g.tw, g.T, g.P, g.u_bytes, g.v_bytes, g.yhat_bytes,
                g.workspace_bytes, g.fused_input, g.fused_conv, g.fused_output, g.outer33,
                g.ld_c);
  }
  std::printf("swept %ld, accepted %ld, failures %d\n", sweep, accepted, failures);
  return failures ? 1 : 0;
}
