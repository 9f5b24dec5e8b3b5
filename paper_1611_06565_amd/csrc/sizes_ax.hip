// Kernel instances of the 3-D layers with per-axis tiles: F(2,3) on axis 0
// and F(4,3) on axes 1 and 2, and the reverse (aniso.hpp).
#include "aniso.hpp"
#include "launch.hpp"

namespace wino {

namespace {

template <int M0, int M1, int R>
struct LaunchAx {
  using S = AxShape<M0, M1, R>;

  static wino_status filter(const wino_plan_s& p, const float* w, float* U, bool adjoint, hipStream_t s) {
    FilterArgs a{};
    a.uplane = int64_t(p.C_pad) * p.K_pad;
    a.C = p.C; a.K = p.K; a.C_pad = p.C_pad; a.K_pad = p.K_pad;
    a.adjoint = adjoint ? 1 : 0;
    hipLaunchKernelGGL((k_filter_ax<M0, M1, R>), dim3(p.grid_filter), dim3(64), 0, s, w, U, a);
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
    hipLaunchKernelGGL((k_input_ax<M0, M1, R>), dim3(p.grid_input), dim3(S::A0 * 64), 0, s, x, V, a);
    return launch_status();
  }

  static wino_status gemm(const wino_plan_s& p, const float* V, float*, const float* U, const float* bias, float* y,
                          hipStream_t s) {
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
    hipLaunchKernelGGL((k_gemm_ax<M0, M1, R>), dim3(p.grid_gemm), dim3(S::NT), 0, s, V, U, y, g);
    return launch_status();
  }

  static wino_status wgrad(const wino_plan_s&, const float*, const float*, float*, float*, hipStream_t) {
    return WINO_EUNSUPPORTED;
  }
};

template <int M0, int M1, int R>
constexpr SizeOps make_ops_ax() {
  using L = LaunchAx<M0, M1, R>;
  return SizeOps{&L::filter, &L::input, &L::gemm, &L::wgrad, nullptr};
}

}  // namespace

const SizeOps* size_ops_ax(int m0, int m1) {
  static const SizeOps a24 = make_ops_ax<2, 4, 3>();
  static const SizeOps a42 = make_ops_ax<4, 2, 3>();
  if (m0 == 2 && m1 == 4) return &a24;
  if (m0 == 4 && m1 == 2) return &a42;
  return nullptr;
}

}  // namespace wino
