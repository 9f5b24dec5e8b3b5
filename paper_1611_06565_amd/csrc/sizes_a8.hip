// Kernel instances and launches of the alpha = 8 sizes of Table 1 in 3-D:
// F(5^3, 4^3), F(4^3, 5^3), F(3^3, 6^3) (a8.hpp).  No weight gradient.
#include <cstdint>

#include "a8.hpp"
#include "launch.hpp"

namespace wino {

namespace {

template <int MM, int R, bool CONST>
struct LaunchA8 {
  using S = A8Shape<MM, R>;

  static wino_status filter(const wino_plan_s& p, const float* w, float* U, bool adjoint, hipStream_t s) {
    FilterArgs a{};
    a.uplane = int64_t(p.C_pad) * p.K_pad;
    a.C = p.C; a.K = p.K; a.C_pad = p.C_pad; a.K_pad = p.K_pad;
    a.adjoint = adjoint ? 1 : 0;
    hipLaunchKernelGGL((k_filter_a8<MM, R, CONST>), dim3(p.grid_filter), dim3(64), 0, s, w, U, a, p.fm);
    return launch_status();
  }

  static wino_status input(const wino_plan_s& p, const float* x, float* V, hipStream_t s) {
    InputArgs a{};
    a.xstride_c = p.X[0] * p.X[1] * p.X[2];
    a.C = p.C; a.C_pad = p.C_pad;
    a.T = int32_t(p.T); a.T_pad = int32_t(p.T_pad);
    for (int i = 0; i < 3; ++i) {
      a.X[i] = int32_t(p.X[i]); a.tiles[i] = int32_t(p.tiles[i]); a.pad[i] = p.pad[i];
    }
    a.ntb = int32_t(p.T_pad / S::BLK);
    a.nblocks = int32_t(p.grid_input);
    hipLaunchKernelGGL((k_input_a8<MM, R, CONST>), dim3(p.grid_input), dim3(256), 0, s, x, V, a, p.fm);
    return launch_status();
  }

  static wino_status gemm(const wino_plan_s& p, const float* V, float*, const float* U, const float* bias,
                          float* y, hipStream_t s) {
    GemmArgs g{};
    g.uplane = int64_t(p.C_pad) * p.K_pad;
    g.ystride_k = p.Y[0] * p.Y[1] * p.Y[2];
    g.T = int32_t(p.T); g.T_pad = int32_t(p.T_pad);
    g.C_pad = p.C_pad; g.K = p.K; g.K_pad = p.K_pad;
    g.nkb = p.gemm_nkb;
    g.nblocks = int32_t(p.grid_gemm);
    for (int i = 0; i < 3; ++i) { g.tiles[i] = int32_t(p.tiles[i]); g.Y[i] = int32_t(p.Y[i]); }
    g.act = act_kind(p);
    g.slope = p.slope;
    g.bias = bias;
    hipLaunchKernelGGL((k_gemm_a8<MM, R, CONST>), dim3(p.grid_gemm), dim3(S::NT), 0, s, V, U, y, g, p.fm);
    return launch_status();
  }

  static constexpr SizeOps ops() { return SizeOps{&filter, &input, &gemm, nullptr, nullptr}; }
};

template <int MM, int R>
const SizeOps* table(bool const_mats) {
  static const SizeOps with = LaunchA8<MM, R, true>::ops();
  static const SizeOps without = LaunchA8<MM, R, false>::ops();
  return const_mats ? &with : &without;
}

}  // namespace

const SizeOps* size_ops_a8(int m, int r, bool const_mats) {
  if (m == 5 && r == 4) return table<5, 4>(const_mats);
  if (m == 4 && r == 5) return table<4, 5>(const_mats);
  if (m == 3 && r == 6) return table<3, 6>(const_mats);
  return nullptr;
}

}  // namespace wino
