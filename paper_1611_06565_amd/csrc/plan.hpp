// The plan of one layer: sizes, transform matrices and launch geometry,
// fixed by wino_plan on the host.  Plain C++ (no HIP): plan.cpp builds with
// any C++20 compiler, so its size and grid arithmetic can run under host
// sanitizers.
#pragma once

#include <cstdint>

#include "synth.hpp"
#include "wino.h"

struct wino_plan_s {
  int N, m, r, alpha, nxi, C, K;
  int C_pad, K_pad;
  int64_t batch;
  int64_t X[3], Y[3], tiles[3];
  int32_t pad[3];
  int64_t T, T_pad;
  int blk, kblk, cg, cgu, kind;
  // per-axis output tiles (eq. 4's own transform triple per axis): mv[i] is
  // the tile extent of axis i (1 on unused axes); aniso when they differ
  // (then axis 0 uses F(mv[0], r) and axes 1, 2 F(mv[1], r), default points)
  int mv[3], av[3];
  bool aniso;
  int32_t n_user_pts;     // the caller's points (0: default set), kept for wino_plan_adjoint
  double user_pts[wino::kMaxAlpha];
  // weight gradient: F(r, m) on the same points (its B^T is the forward's)
  bool wgrad_ok;
  wino::FMats fmw;
  int32_t wg_nsplit, wg_kpad4;
  int64_t wg_d_floats, wg_part_floats;
  // pass-accumulating product (m = 2, F(4^2)) tail split, fixed at plan time
  // from the device's compute units: the last xtail[x] blocks of XCD x are
  // done in nparts parts each
  int nparts;             // 1: no split
  int32_t xtail[8];
  int64_t ntail;          // sum of xtail
  int64_t v_floats;       // V in the workspace (rounded up to 256 bytes)
  int64_t part_floats;    // partial outputs after V when nparts > 1
  uint32_t flags;
  float slope;            // slope of the activation below zero (WINO_LEAKY_RELU)
  bool const_mats;
  double AT[wino::kMaxAlpha][wino::kMaxAlpha], BT[wino::kMaxAlpha][wino::kMaxAlpha],
      G[wino::kMaxAlpha][wino::kMaxAlpha];
  wino::FMats fm;
  // Launch geometry, each grid checked against the 32-bit limits of a launch.
  uint32_t grid_filter;   // k_filter (64 threads)
  uint32_t grid_input;    // k_input (256) or k_input_split (384)
  uint32_t grid_gemm;     // product kernel
  uint32_t grid_reduce;   // k_part_reduce (256), 0 when nparts == 1
  // pass-accumulating products: XCD x owns blocks acc_xb0[x] .. + acc_xn[x];
  // its last acc_xs[x] are tail blocks, the first of which is tail block
  // acc_xt0[x] overall
  int32_t acc_xb0[8], acc_xn[8], acc_xs[8], acc_xt0[8];
  int32_t gemm_nkb;       // kernel blocks of the product
  uint32_t grid_dy, grid_wgemm, grid_wsum, grid_wfin;   // weight gradient
  // F(4^3): the forward runs the input transform inside the product
  // (k_fused43, one work-group per 16 tiles x 16 kernels) and needs no workspace
  bool fused;
  uint32_t grid_fused;
};

namespace wino {

// Compute units of the current device, or 0 if unknown.  Defined by the
// device library; a host-only build links its own stand-in.
int device_cu_count();

// Max-pool geometry over the trailing 3 axes of [lead][X_1][X_2][X_3].
struct PoolGeom {
  int64_t lead;
  int32_t X[3], Y[3], p[3];
  int64_t total;          // lead * prod Y
  bool pair;              // the paired kernel (window 2 on rows of a multiple of 4)
  uint32_t grid;          // work-groups of 256 threads
};

// Validate a max-pool call and fill its geometry; WINO_EINVAL on bad sizes
// or a grid past the launch limits.
wino_status pool_geometry(const int64_t* dims, const int32_t* window, PoolGeom* g);

}  // namespace wino
