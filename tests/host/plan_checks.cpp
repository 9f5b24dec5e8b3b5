// Host-side checks of the planner (csrc/plan.cpp), built with g++ under
// AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_host_sanitize.py.
// No device is involved: the planner's compute-unit query is answered here.
// Prints one line per check; exits non-zero on the first failure (the
// sanitizers abort on any overflow or bad access first).
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "plan.hpp"
#include "wino.h"

namespace wino {
// 256 compute units in 8 XCDs, as on one MI355X.
int device_cu_count() { return 256; }
}  // namespace wino

#define CHECK(cond, what)                                           \
  do {                                                              \
    if (!(cond)) {                                                  \
      std::fprintf(stderr, "FAIL: %s (line %d)\n", what, __LINE__); \
      return 1;                                                     \
    }                                                               \
    std::printf("ok: %s\n", what);                                  \
  } while (0)

static wino_status plan_status(int N, int m, int r, int64_t C, int64_t K, const int64_t* dims, int pad,
                               wino_plan_t** keep = nullptr) {
  wino_opts o{};
  for (int i = 0; i < 3; ++i) o.pad[i] = pad;
  wino_plan_t* p = nullptr;
  const wino_status st = wino_plan(N, m, r, int(C), int(K), dims, &o, &p);
  if (st == WINO_OK) {
    wino_plan_desc d{};
    if (wino_plan_describe(p, &d) != WINO_OK) std::abort();
    (void)wino_filter_bytes(p);
    (void)wino_workspace_bytes(p);
    (void)wino_weight_gradient_workspace_bytes(p);
    wino_plan_t* a = nullptr;
    if (wino_plan_adjoint(p, &a) == WINO_OK) wino_destroy(a);
    if (keep) *keep = p;
    else wino_destroy(p);
  } else if (p != nullptr) {
    std::abort();   // a failed plan leaves *out untouched
  }
  return st;
}

int main() {
  const int64_t big = 0x7fffffff;
  // the five workloads and the paper's 2-D benchmark layer plan
  {
    const int64_t c1[4] = {1, 16, 16, 16}, c2[4] = {8, 16, 56, 56}, c3[3] = {64, 56, 56},
                  c4[4] = {1, 128, 128, 128}, c5[4] = {4, 16, 112, 112}, f4[3] = {200, 224, 224};
    CHECK(plan_status(3, 2, 3, 16, 16, c1, 0) == WINO_OK, "config 1");
    wino_plan_t* p = nullptr;
    CHECK(plan_status(3, 2, 3, 64, 128, c2, 1, &p) == WINO_OK, "config 2");
    wino_plan_desc d{};
    CHECK(wino_plan_describe(p, &d) == WINO_OK && d.T == 50176, "config 2 tiles");
    // 1568 blocks of 64 x 64 over 8 XCDs of 32 CUs (64 resident work-groups):
    // 196 per XCD, 4 past the last full round, each split into 8 parts
    CHECK(d.gemm_tail_blocks == 32 && d.gemm_parts == 8, "config 2 tail split");
    CHECK(wino_workspace_bytes(p) == size_t(4) * 64 * 64 * 50176 + size_t(4) * 32 * 8 * 8 * 64 * 64,
          "config 2 workspace = V + partial outputs");
    wino_destroy(p);
    CHECK(plan_status(2, 4, 3, 256, 256, c3, 1) == WINO_OK, "config 3");
    CHECK(plan_status(3, 4, 3, 32, 32, c4, 1) == WINO_OK, "config 4");
    CHECK(plan_status(3, 2, 3, 3, 64, c5, 1) == WINO_OK, "C3D conv1");
    CHECK(plan_status(2, 5, 4, 32, 32, f4, 0) == WINO_OK, "F(5,4) benchmark layer");
  }
  // channel and kernel counts past 2^20, and the 32-bit extremes
  {
    const int64_t dims[4] = {1, 8, 8, 8};
    CHECK(plan_status(3, 2, 3, big, 16, dims, 1) == WINO_EINVAL, "C = 2^31 - 1");
    CHECK(plan_status(3, 2, 3, 16, big, dims, 1) == WINO_EINVAL, "K = 2^31 - 1");
    CHECK(plan_status(3, 2, 3, big, big, dims, 1) == WINO_EINVAL, "C = K = 2^31 - 1");
    CHECK(plan_status(3, 4, 3, 16, big - 39, dims, 1) == WINO_EINVAL, "K = 2^31 - 40");
    CHECK(plan_status(2, 4, 3, (1 << 20) + 1, 4, dims, 1) == WINO_EINVAL, "C = 2^20 + 1");
    CHECK(plan_status(2, 4, 3, 1 << 20, 4, dims, 1) == WINO_OK, "C = 2^20");
    CHECK(plan_status(3, 2, 3, 1 << 20, 1 << 20, dims, 1) == WINO_EINVAL, "C = K = 2^20: filter grid too big");
    CHECK(plan_status(3, 2, 3, 16384, 16384, dims, 1) == WINO_OK, "C = K = 2^14");
    // the 3-D alpha = 8 sizes: eight filter threads per (channel, kernel)
    CHECK(plan_status(3, 5, 4, 8192, 8192, dims, 1) == WINO_OK, "F(5^3,4^3) C = K = 2^13");
    CHECK(plan_status(3, 5, 4, 1 << 20, 1 << 20, dims, 1) == WINO_EINVAL, "F(5^3,4^3) C = K = 2^20");
    CHECK(plan_status(3, 4, 5, big, 4, dims, 2) == WINO_EINVAL, "F(4^3,5^3) C = 2^31 - 1");
    CHECK(plan_status(3, 3, 6, 4, 4, dims, 2) == WINO_OK, "F(3^3,6^3)");
    CHECK(plan_status(3, 3, 2, 4, 4, dims, 1) == WINO_OK, "F(3^3,2^3)");
  }
  // extents: tile counts, byte counts and grids past their ranges
  {
    const int64_t d1[4] = {big, big, big, big};
    CHECK(plan_status(3, 2, 3, 4, 4, d1, 1) == WINO_EINVAL, "every extent 2^31 - 1");
    const int64_t d2[4] = {1, 3, 3, int64_t(1) << 26};
    CHECK(plan_status(3, 2, 3, 4, 4, d2, 0) == WINO_OK, "one long axis");
    const int64_t d3[4] = {big, 1, 1, 4};
    CHECK(plan_status(3, 2, 3, 4, 4, d3, 1) == WINO_EINVAL, "batch 2^31 - 1: tiles past 2^31");
    const int64_t d4[4] = {1 << 20, 8, 8, 8};
    CHECK(plan_status(3, 2, 3, 1 << 20, 64, d4, 1) == WINO_EINVAL, "x of 2^50 floats: grids too big");
    const int64_t d5[4] = {0, 8, 8, 8}, d6[4] = {1, 8, -1, 8}, d7[4] = {1, 8, big + 1, 8};
    CHECK(plan_status(3, 2, 3, 4, 4, d5, 1) == WINO_EINVAL, "batch 0");
    CHECK(plan_status(3, 2, 3, 4, 4, d6, 1) == WINO_EINVAL, "negative extent");
    CHECK(plan_status(3, 2, 3, 4, 4, d7, 1) == WINO_EINVAL, "extent 2^31");
    const int64_t d8[4] = {1, 4, 4, 4};
    CHECK(plan_status(3, 2, 3, 4, 4, d8, 1 << 20) == WINO_EINVAL, "pad 2^20: tiles past 2^31");
    CHECK(plan_status(3, 2, 3, 4, 4, d8, (1 << 20) + 1) == WINO_EINVAL, "pad 2^20 + 1");
    CHECK(plan_status(2, 4, 3, 4, 4, d8, 1 << 20) == WINO_EINVAL, "2-D pad 2^20: tiles past 2^31");
    const int64_t d9[3] = {1, 4, 4};
    CHECK(plan_status(2, 2, 3, 4, 4, d9, 3000) == WINO_OK, "2-D pad 3000");
    CHECK(plan_status(2, 2, 3, 4, 4, d9, 30000) == WINO_EINVAL, "2-D pad 30000: input grid past 2^32 work-items");
  }
  // options
  {
    const int64_t dims[4] = {1, 8, 8, 8};
    wino_opts o{};
    wino_plan_t* p = nullptr;
    o.flags = WINO_RELU | WINO_LEAKY_RELU;
    CHECK(wino_plan(3, 2, 3, 4, 4, dims, &o, &p) == WINO_EINVAL && p == nullptr, "two activations");
    o.flags = WINO_LEAKY_RELU;
    o.slope = NAN;
    CHECK(wino_plan(3, 2, 3, 4, 4, dims, &o, &p) == WINO_EINVAL, "NaN slope");
    o.slope = 0.2f;
    CHECK(wino_plan(3, 2, 3, 4, 4, dims, &o, &p) == WINO_OK, "leaky ReLU");
    wino_destroy(p);
    const double pts[3] = {0.0, 1.0, 1e300};
    o = wino_opts{};
    o.points = pts;
    o.n_points = 3;
    p = nullptr;
    CHECK(wino_plan(3, 2, 3, 4, 4, dims, &o, &p) == WINO_EINVAL && p == nullptr, "huge point");
    const double pts2[3] = {0.0, 1.0 / 3.0, -1.0 / 3.0};
    o.points = pts2;
    CHECK(wino_plan(3, 2, 3, 4, 4, dims, &o, &p) == WINO_OK, "points 0, 1/3, -1/3");
    wino_destroy(p);
    CHECK(wino_plan(3, 2, 3, 4, 4, nullptr, nullptr, &p) == WINO_EINVAL, "NULL dims");
    CHECK(wino_plan(3, 2, 3, 4, 4, dims, nullptr, nullptr) == WINO_EINVAL, "NULL out");
    CHECK(wino_plan(3, 5, 3, 4, 4, dims, nullptr, &p) == WINO_EUNSUPPORTED, "unsupported size");
    CHECK(wino_plan(3, 7, 3, 4, 4, dims, nullptr, &p) == WINO_EUNSUPPORTED, "alpha 9");
    wino_destroy(nullptr);
  }
  // per-axis tiles (eq. 4 with one transform triple per axis)
  {
    const int64_t dims[4] = {4, 8, 28, 28};
    wino_opts o{};
    o.pad[0] = o.pad[1] = o.pad[2] = 1;
    o.tile[0] = 2;
    wino_plan_t* p = nullptr;
    CHECK(wino_plan(3, 4, 3, 256, 256, dims, &o, &p) == WINO_OK, "tiles (2, 4, 4)");
    wino_plan_desc d{};
    CHECK(wino_plan_describe(p, &d) == WINO_OK && d.n_xi == 144 && d.T == 4 * 4 * 7 * 7 && d.fused == 0,
          "tiles (2, 4, 4) described");
    CHECK(wino_weight_gradient_workspace_bytes(p) == 0, "no weight gradient for per-axis tiles");
    wino_plan_t* a = nullptr;
    CHECK(wino_plan_adjoint(p, &a) == WINO_OK, "adjoint of per-axis tiles");
    wino_destroy(a);
    wino_destroy(p);
    o.tile[0] = 4; o.tile[1] = 2; o.tile[2] = 2;
    CHECK(wino_plan(3, 2, 3, 3, 64, dims, &o, &p) == WINO_OK, "tiles (4, 2, 2)");
    wino_destroy(p);
    o.tile[2] = 4;
    CHECK(wino_plan(3, 2, 3, 3, 64, dims, &o, &p) == WINO_EUNSUPPORTED, "tiles (4, 2, 4)");
    o.tile[0] = 0; o.tile[1] = 0; o.tile[2] = int32_t(1) << 30;
    CHECK(wino_plan(3, 2, 3, 3, 64, dims, &o, &p) == WINO_EINVAL, "tile 2^30");
    const int64_t big[4] = {0x7fffffff, 3, 3, 0x7fffffff};
    o.tile[0] = 2; o.tile[1] = 4; o.tile[2] = 4;
    CHECK(wino_plan(3, 4, 3, 4, 4, big, &o, &p) == WINO_EINVAL, "per-axis tiles, tiles past 2^31");
  }
  // max-pool geometry
  {
    using wino::PoolGeom;
    PoolGeom g{};
    const int64_t ok[4] = {4 * 512, 2, 7, 7};
    const int32_t w222[3] = {2, 2, 2};
    CHECK(wino::pool_geometry(ok, w222, &g) == WINO_OK && g.total == 4 * 512 * 9 && !g.pair, "last pool");
    const int64_t pr[4] = {4 * 64, 16, 112, 112};
    const int32_t w122[3] = {1, 2, 2};
    CHECK(wino::pool_geometry(pr, w122, &g) == WINO_OK && g.pair && g.grid == (4 * 64 * 16 * 56 * 56 / 2 + 255) / 256,
          "pool 1 (pairs)");
    const int64_t huge[4] = {int64_t(1) << 62, 2, 2, 2};
    CHECK(wino::pool_geometry(huge, w222, &g) == WINO_EINVAL, "lead 2^62");
    const int64_t over[4] = {int64_t(1) << 40, big, big, big};
    CHECK(wino::pool_geometry(over, w222, &g) == WINO_EINVAL, "lead x X overflows int64");
    const int64_t grid[4] = {int64_t(1) << 34, 2, 2, 2};
    CHECK(wino::pool_geometry(grid, w222, &g) == WINO_EINVAL, "grid past 2^31");
    const int64_t neg[4] = {-1, 2, 2, 2};
    CHECK(wino::pool_geometry(neg, w222, &g) == WINO_EINVAL, "negative lead");
    const int32_t w0[3] = {0, 2, 2}, w3[3] = {3, 2, 2};
    CHECK(wino::pool_geometry(ok, w0, &g) == WINO_EINVAL, "window 0");
    CHECK(wino::pool_geometry(ok, w3, &g) == WINO_EINVAL, "window past the extent");
  }
  // accuracy queries
  {
    double pts[7] = {0}, g = 0.0, gd = 0.0;
    CHECK(wino_search_points(3, 4, 3, pts, &g) == WINO_OK, "point search F(4,3)");
    CHECK(wino_points_error_growth(3, 4, 3, nullptr, 0, &gd) == WINO_OK && g <= gd, "searched <= default");
    CHECK(wino_search_points(2, 5, 4, pts, &g) == WINO_OK, "point search F(5,4)");
    const double bad[5] = {0.0, 1.0, 1.0, 2.0, -2.0};
    CHECK(wino_points_error_growth(3, 4, 3, bad, 5, &g) == WINO_EINVAL, "coincident points");
  }
  std::printf("all planner checks ok\n");
  return 0;
}
