// Kernel dispatch of one compiled size (N, m, r): the launches behind the
// device entry points, with the plan's geometry.  Each sizes_*.hip
// translation unit instantiates it for its sizes and publishes a SizeOps
// table; the entry points (wino.hip) pick the table of a plan.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "gemm_acc.hpp"
#include "gemm_acc4.hpp"
#include "kernels.hpp"
#include "plan.hpp"
#include "synth.hpp"
#include "wgrad.hpp"
#include "wino.h"

namespace wino {

inline wino_status launch_status() {
  return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EDEVICE;
}

inline int32_t act_kind(const wino_plan_s& p) {
  return (p.flags & WINO_RELU) ? 1 : ((p.flags & WINO_LEAKY_RELU) ? 2 : 0);
}

// k_fused43 (F(4^3) with the input transform inside the product), defined in
// fused_f43.hip.
// pool: 0 none, 1 max-pool window (1, 2, 2), 2 window (2, 2, 2) (y pooled).
wino_status launch_fused43(const wino_plan_s& p, bool const_mats, const float* x, const float* U,
                           const float* bias, float* y, hipStream_t s, int pool = 0);

// The launches of one size, as plain function pointers.
struct SizeOps {
  wino_status (*filter)(const wino_plan_s&, const float* w, float* U, bool adjoint, hipStream_t);
  wino_status (*input)(const wino_plan_s&, const float* x, float* V, hipStream_t);
  wino_status (*gemm)(const wino_plan_s&, const float* V, float* part, const float* U, const float* bias,
                      float* y, hipStream_t);
  wino_status (*wgrad)(const wino_plan_s&, const float* x, const float* dy, float* dw, float* ws, hipStream_t);
  // the forward with the input transform inside the product (null for sizes without one)
  wino_status (*fused)(const wino_plan_s&, const float* x, const float* U, const float* bias, float* y,
                       hipStream_t);
  // the product with the max-pool in its epilogue (pool 1: window (1, 2, 2),
  // 2: (2, 2, 2); y pooled), null for sizes without one; part as for gemm
  wino_status (*gemm_pool)(const wino_plan_s&, const float* V, float* part, const float* U, const float* bias,
                           float* y, int pool, hipStream_t);
};

template <int N, int MM, int R, bool CONST>
struct Launch {
  static constexpr int A = MM + R - 1;
  static constexpr int NXI = ipow(A, N);
  static constexpr int BLK = Blocking<N, MM, R>::BLK;
  static constexpr int CG = Blocking<N, MM, R>::CG;
  static constexpr int CGU = Blocking<N, MM, R>::CGU;
  // k_gemm_inv work-group shape: F(4^3): 12 waves x three alpha-rows (18
  // elements); F(3^3, 2^3): 8 waves x two alpha-rows (8 elements); 2-D sizes:
  // alpha waves x one alpha-row (alpha elements).  The last
  // axis is reduced in registers, 16-byte operand loads, no register ring
  // (the other waves of the SIMD hide the load latency).
  static constexpr int NW = (N == 3 && A == 6) ? 12 : (N == 3 && A == 4) ? 8 : ipow(A, N - 1);
  static constexpr int LOC = 1;
  static constexpr int VEC = Blocking<N, MM, R>::VEC;
  static constexpr int DEPTH = 1;

  static wino_status filter(const wino_plan_s& p, const float* w, float* U, bool adjoint, hipStream_t s) {
    FilterArgs a{};
    a.uplane = int64_t(p.C_pad) * p.K_pad;
    a.C = p.C; a.K = p.K; a.C_pad = p.C_pad; a.K_pad = p.K_pad;
    a.adjoint = adjoint ? 1 : 0;
    // one thread per (channel, kernel): small work-groups spread the few
    // threads of a layer (8192 for C = 64, K = 128) over more CUs
    hipLaunchKernelGGL((k_filter<N, MM, R, CONST>), dim3(p.grid_filter), dim3(64), 0, s, w, U, a, p.fm);
    return launch_status();
  }

  static wino_status input(const wino_plan_s& p, const float* x, float* V, hipStream_t s) {
    InputArgs a{};
    a.xstride_c = 1;
    for (int i = 0; i < N; ++i) a.xstride_c *= p.X[i];
    a.C = p.C; a.C_pad = p.C_pad;
    a.T = int32_t(p.T); a.T_pad = int32_t(p.T_pad);
    for (int i = 0; i < 3; ++i) {
      a.X[i] = int32_t(p.X[i]); a.tiles[i] = int32_t(p.tiles[i]); a.pad[i] = p.pad[i];
    }
    a.ntb = int32_t(p.T_pad / BLK);
    a.nblocks = int32_t(p.grid_input);
    if constexpr (Blocking<N, MM, R>::NXI > 64) {
      // large windows: A threads per (tile, channel), one V block (BLK tiles
      // x one channel group) per work-group.  Row-aligned loads when every
      // block is BLK tiles of one input row, rows are whole 16-byte units and
      // a window starts at most 2 values left of its tile.
      constexpr int A = Blocking<N, MM, R>::A;
      static_assert(BLK * CG == 64, "one pair per lane");
      // (x is 16-byte aligned: the entry points check it)
      a.rowfast = (p.tiles[N - 1] % BLK == 0 && p.X[N - 1] % 4 == 0 && p.pad[N - 1] <= 2) ? 1 : 0;
      hipLaunchKernelGGL((k_input_split<N, MM, R, CONST>), dim3(p.grid_input), dim3(A * 64), 0, s, x, V, a,
                         p.fm);
    } else {
      // m = 2: aligned pairs plus neighbouring lanes when the last axis has
      // pad 1 and an even length (x is 16-byte aligned: the entry points check it)
      a.rowfast = (MM == 2 && p.pad[N - 1] == 1 && p.X[N - 1] % 2 == 0) ? 1 : 0;
      hipLaunchKernelGGL((k_input<N, MM, R, CONST>), dim3(p.grid_input), dim3(256), 0, s, x, V, a, p.fm);
    }
    return launch_status();
  }

  // Weight gradient (wgrad.hpp): V by the forward's input transform, D by
  // k_dy, partial products over tile-block ranges, then their sum and A'^T.
  static wino_status wgrad(const wino_plan_s& p, const float* x, const float* dy, float* dw, float* ws,
                           hipStream_t s) {
    if constexpr ((BLK != 64 && BLK != 16) || CG != 4) {
      return WINO_EUNSUPPORTED;
    } else {
      float* V = ws;
      float* D = ws + p.v_floats;
      float* part = D + p.wg_d_floats;
      wino_status st = input(p, x, V, s);
      if (st != WINO_OK) return st;
      WgArgs a{};
      a.ystride_k = 1;
      for (int i = 0; i < N; ++i) a.ystride_k *= p.Y[i];
      a.T = int32_t(p.T); a.ntb = int32_t((p.T_pad + 63) / 64); a.nvb = int32_t(p.T_pad / BLK);
      a.K = p.K; a.K_pad4 = p.wg_kpad4; a.C = p.C; a.C_pad = p.C_pad;
      a.nkb = (p.wg_kpad4 + 63) / 64; a.ncb = (p.C_pad + 63) / 64;
      a.nsplit = p.wg_nsplit;
      for (int i = 0; i < 3; ++i) { a.tiles[i] = int32_t(p.tiles[i]); a.Y[i] = int32_t(p.Y[i]); }
      a.nblocks = int32_t(p.grid_wgemm);
      hipLaunchKernelGGL((k_dy<N, MM, R, CONST>), dim3(p.grid_dy), dim3(256), 0, s, dy, D, a, p.fmw);
      hipLaunchKernelGGL((k_wgrad_gemm<BLK>), dim3(p.grid_wgemm), dim3(256), 0, s, V, D, part, a, int32_t(NXI));
      hipLaunchKernelGGL(k_wgrad_sum, dim3(p.grid_wsum), dim3(256), 0, s, part, a, int32_t(NXI));
      hipLaunchKernelGGL((k_wgrad_finish<N, MM, R, CONST>), dim3(p.grid_wfin), dim3(256), 0, s, part, dw, a,
                         p.fmw);
      return launch_status();
    }
  }

  // Arguments of a pass-accumulating product (k_gemm_acc, k_gemm_acc4): the
  // per-XCD work ranges and tail split fixed by the planner.
  static void acc_args(const wino_plan_s& p, AccArgs& a, int TB, const float* bias, float* part) {
    a.vblock = int64_t(p.nxi) * p.C_pad * TB;
    a.uplane = int64_t(p.C_pad) * p.K_pad;
    a.ystride_k = 1;
    for (int i = 0; i < N; ++i) a.ystride_k *= p.Y[i];
    a.T = int32_t(p.T); a.C_pad = p.C_pad; a.K = p.K; a.K_pad = p.K_pad;
    a.nkb = p.gemm_nkb;
    for (int i = 0; i < 3; ++i) { a.tiles[i] = int32_t(p.tiles[i]); a.Y[i] = int32_t(p.Y[i]); }
    a.act = act_kind(p);
    a.slope = p.slope;
    a.bias = bias;
    a.nparts = p.nparts;
    a.part = part;
    for (int x = 0; x < 8; ++x) {
      a.xb0[x] = p.acc_xb0[x]; a.xn[x] = p.acc_xn[x]; a.xs[x] = p.acc_xs[x]; a.xt0[x] = p.acc_xt0[x];
    }
  }

  // F(4^3): the input transform inside the product (fused43.hpp, launched
  // from its own unit); no workspace.
  static wino_status fused(const wino_plan_s& p, const float* x, const float* U, const float* bias, float* y,
                           hipStream_t s) {
    if constexpr (N == 3 && MM == 4 && R == 3) return launch_fused43(p, CONST, x, U, bias, y, s);
    else return WINO_EUNSUPPORTED;
  }

  static wino_status gemm(const wino_plan_s& p, const float* V, float* part, const float* U, const float* bias,
                          float* y, hipStream_t s) {
    constexpr int KIND = Blocking<N, MM, R>::KIND;
    if constexpr (KIND == 0) {
      using G = AccGeom<N, MM, R>;
      AccArgs a{};
      // tail blocks: passes split over p.nparts units, whose partial outputs
      // (after V in the workspace) are summed in order
      acc_args(p, a, G::TB, bias, part);
      hipLaunchKernelGGL((k_gemm_acc<N, MM, R, CONST>), dim3(p.grid_gemm), dim3(G::NT), 0, s, V, U, y, a, p.fm);
      if (p.nparts > 1)
        hipLaunchKernelGGL((k_part_reduce<N, MM, G::TB, G::KB>), dim3(p.grid_reduce), dim3(256), 0, s, y, a,
                           int32_t(p.ntail));
      return launch_status();
    } else if constexpr (KIND == 1) {
      using G = Acc4Geom<N, MM, R>;
      AccArgs a{};
      acc_args(p, a, G::TB, bias, part);
      hipLaunchKernelGGL((k_gemm_acc4<N, MM, R, CONST>), dim3(p.grid_gemm), dim3(G::NT), 0, s, V, U, y, a, p.fm);
      if (p.nparts > 1)
        hipLaunchKernelGGL((k_part_reduce<N, MM, G::TB, G::KB>), dim3(p.grid_reduce), dim3(256), 0, s, y, a,
                           int32_t(p.ntail));
      return launch_status();
    } else {
      using Geo = GemmGeom<N, MM, R, BLK, NW, LOC>;
      static_assert(Geo::NT <= 768, "the planner sizes k_gemm_inv grids for at most 768 threads");
      const GemmArgs g = gemm_args(p, bias, 0);
      hipLaunchKernelGGL((k_gemm_inv<N, MM, R, CONST, BLK, NW, LOC, VEC, DEPTH>), dim3(p.grid_gemm),
                         dim3(Geo::NT), 0, s, V, U, y, g, p.fm);
      return launch_status();
    }
  }

  // Arguments of k_gemm_inv; pool > 0 adds the pooled extents (floor rounding).
  static GemmArgs gemm_args(const wino_plan_s& p, const float* bias, int pool) {
    GemmArgs g{};
    g.uplane = int64_t(p.C_pad) * p.K_pad;
    g.ystride_k = 1;
    for (int i = 0; i < N; ++i) g.ystride_k *= p.Y[i];
    g.T = int32_t(p.T); g.T_pad = int32_t(p.T_pad);
    g.C_pad = p.C_pad; g.K = p.K; g.K_pad = p.K_pad;
    g.nkb = p.gemm_nkb;
    g.nblocks = int32_t(p.grid_gemm);
    for (int i = 0; i < 3; ++i) { g.tiles[i] = int32_t(p.tiles[i]); g.Y[i] = int32_t(p.Y[i]); }
    g.act = act_kind(p);
    g.slope = p.slope;
    g.bias = bias;
    if (pool > 0) {
      g.Yp[0] = int32_t(p.Y[0] / (pool == 2 ? 2 : 1));
      g.Yp[1] = int32_t(p.Y[1] / 2);
      g.Yp[2] = int32_t(p.Y[2] / 2);
      g.ystride_p = int64_t(g.Yp[0]) * g.Yp[1] * g.Yp[2];
    }
    return g;
  }

  // The product with the max-pool in its epilogue: F(4^3) two-stage
  // (windows (1, 2, 2) and (2, 2, 2)) and F(2^3) (window (2, 2, 2), one tile).
  static wino_status gemm_pool(const wino_plan_s& p, const float* V, float* part, const float* U,
                               const float* bias, float* y, int pool, hipStream_t s) {
    constexpr int KIND = Blocking<N, MM, R>::KIND;
    if constexpr (N == 3 && MM == 2 && KIND == 0) {
      if (pool != 2) return WINO_EUNSUPPORTED;
      using G = AccGeom<N, MM, R>;
      AccArgs a{};
      acc_args(p, a, G::TB, bias, part);
      for (int i = 0; i < 3; ++i) a.Yp[i] = int32_t(p.Y[i] / 2);
      a.ystride_p = int64_t(a.Yp[0]) * a.Yp[1] * a.Yp[2];
      hipLaunchKernelGGL((k_gemm_acc<N, MM, R, CONST, 1>), dim3(p.grid_gemm), dim3(G::NT), 0, s, V, U, y, a,
                         p.fm);
      if (p.nparts > 1)
        hipLaunchKernelGGL((k_part_reduce_pool<N, MM, G::TB, G::KB>), dim3(p.grid_reduce / G::NOUT), dim3(256),
                           0, s, y, a, int32_t(p.ntail));
      return launch_status();
    } else if constexpr (N == 3 && MM == 4 && R == 3 && KIND == 2 && LOC == 1) {
      using Geo = GemmGeom<N, MM, R, BLK, NW, LOC>;
      const GemmArgs g = gemm_args(p, bias, pool);
      if (pool == 1)
        hipLaunchKernelGGL((k_gemm_inv<N, MM, R, CONST, BLK, NW, LOC, VEC, DEPTH, 1>), dim3(p.grid_gemm),
                           dim3(Geo::NT), 0, s, V, U, y, g, p.fm);
      else
        hipLaunchKernelGGL((k_gemm_inv<N, MM, R, CONST, BLK, NW, LOC, VEC, DEPTH, 2>), dim3(p.grid_gemm),
                           dim3(Geo::NT), 0, s, V, U, y, g, p.fm);
      return launch_status();
    } else {
      return WINO_EUNSUPPORTED;
    }
  }
};


template <int N, int MM, int R, bool CONST>
constexpr SizeOps make_ops() {
  using L = Launch<N, MM, R, CONST>;
  if constexpr (N == 3 && MM == 4 && R == 3)
    return SizeOps{&L::filter, &L::input, &L::gemm, &L::wgrad, &L::fused, &L::gemm_pool};
  else if constexpr (N == 3 && MM == 2)
    return SizeOps{&L::filter, &L::input, &L::gemm, &L::wgrad, nullptr, &L::gemm_pool};
  else
    return SizeOps{&L::filter, &L::input, &L::gemm, &L::wgrad, nullptr};
}

// Per-axis tiles (aniso.hpp): F(M0, R) on axis 0, F(M1, R) on axes 1 and 2;
// instances in sizes_ax.hip.
const SizeOps* size_ops_ax(int m0, int m1);

// 3-D sizes with alpha = 8 (a8.hpp): F(5^3, 4^3), F(4^3, 5^3), F(3^3, 6^3);
// instances in sizes_a8.hip.
const SizeOps* size_ops_a8(int m, int r, bool const_mats);

// The tables, one per size of WINO_SIZES (defined in the sizes_*.hip units);
// const_mats selects the instances with the default points compiled in.
#define WINO_DECLARE_OPS(N_, M_, R_) const SizeOps* size_ops_##N_##_##M_##_##R_(bool const_mats);
WINO_SIZES(WINO_DECLARE_OPS)
#undef WINO_DECLARE_OPS
#define WINO_DEFINE_OPS(N_, M_, R_)                                            \
  const SizeOps* size_ops_##N_##_##M_##_##R_(bool const_mats) {                \
    static const SizeOps with = make_ops<N_, M_, R_, true>();                  \
    static const SizeOps without = make_ops<N_, M_, R_, false>();              \
    return const_mats ? &with : &without;                                      \
  }

}  // namespace wino
