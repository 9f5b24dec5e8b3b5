// Kernel instances and launch of k_fused43: F(4^3, 3^3) with the input
// transform inside the product.
#include <algorithm>
#include <cstdint>

#include "fused43.hpp"
#include "launch.hpp"

namespace wino {

namespace {

template <int POOL>
void launch_pool(bool kloop, bool const_mats, dim3 grid, const float* x, const float* U, float* y,
                 const FusedArgs& a, const FMats& fm, hipStream_t s) {
  const dim3 nt(Fused43Geom::NT);
  if (kloop && a.C <= 4)
    hipLaunchKernelGGL((k_fused43<true, true, POOL, true>), grid, nt, 0, s, x, U, y, a, fm);
  else if (kloop)
    hipLaunchKernelGGL((k_fused43<true, true, POOL>), grid, nt, 0, s, x, U, y, a, fm);
  else if (const_mats)
    hipLaunchKernelGGL((k_fused43<true, false, POOL>), grid, nt, 0, s, x, U, y, a, fm);
  else
    hipLaunchKernelGGL((k_fused43<false, false, POOL>), grid, nt, 0, s, x, U, y, a, fm);
}

}  // namespace

wino_status launch_fused43(const wino_plan_s& p, bool const_mats, const float* x, const float* U,
                           const float* bias, float* y, hipStream_t s, int pool) {
  FusedArgs a{};
  a.xstride_c = p.X[0] * p.X[1] * p.X[2];
  a.uplane = int64_t(p.C_pad) * p.K_pad;
  a.ystride_k = p.Y[0] * p.Y[1] * p.Y[2];
  a.C = p.C; a.C_pad = p.C_pad; a.K = p.K; a.K_pad = p.K_pad;
  a.T = int32_t(p.T);
  a.nkb = p.K_pad / Fused43Geom::BLK;
  for (int i = 0; i < 3; ++i) {
    a.X[i] = int32_t(p.X[i]); a.tiles[i] = int32_t(p.tiles[i]); a.pad[i] = p.pad[i]; a.Y[i] = int32_t(p.Y[i]);
  }
  // whole 16-tile blocks along input rows of a multiple of 4 values (x is
  // 16-byte aligned: the entry points check it)
  a.rowfast = (p.tiles[2] % Fused43Geom::BLK == 0 && p.X[2] % 4 == 0 && p.pad[2] <= 2) ? 1 : 0;
  // every output row a whole number of 4-wide tiles, y 16-byte aligned:
  // the epilogue stores rows of four as one 16-byte store
  a.vec_store = (p.Y[2] % 4 == 0 && (reinterpret_cast<uintptr_t>(y) & 15) == 0) ? 1 : 0;
  // one chunk of channels (C <= 8) and several kernel blocks, default points:
  // every kernel block of a tile block in one work-group (the planes formed
  // once), one work-group per tile block
  const bool kloop = const_mats && p.C <= Fused43Geom::CH && a.nkb > 1;
  uint32_t grid = p.grid_fused;
  if (kloop) {
    // tile blocks in contiguous ranges per XCD (one work-group per CU, 1/8 of
    // the CUs per XCD); the blocks past an XCD's last full round are split into
    // one unit per kernel block when those units fit in one round
    const int nb = int(p.grid_fused / uint32_t(a.nkb));
    const int slots = device_cu_count() / 8;
    int units = 0;
    for (int xc = 0; xc < 8; ++xc) {
      a.xn[xc] = nb / 8 + (xc < nb % 8 ? 1 : 0);
      a.xb0[xc] = xc * (nb / 8) + (xc < nb % 8 ? xc : nb % 8);
      const int xs = slots > 0 ? a.xn[xc] % slots : 0;
      a.xs[xc] = (xs * a.nkb <= slots) ? xs : 0;
      units = std::max(units, a.xn[xc] - a.xs[xc] + a.xs[xc] * a.nkb);
    }
    grid = uint32_t(units) * 8u;
  }
  a.nblocks = int32_t(grid);
  a.act = act_kind(p);
  a.slope = p.slope;
  a.bias = bias;
  // the max-pool's output extents (floor rounding) and per-kernel stride
  const int w0 = pool == 2 ? 2 : 1, w12 = pool > 0 ? 2 : 1;
  a.Yp[0] = int32_t(p.Y[0] / w0);
  a.Yp[1] = int32_t(p.Y[1] / w12);
  a.Yp[2] = int32_t(p.Y[2] / w12);
  a.ystride_p = int64_t(a.Yp[0]) * a.Yp[1] * a.Yp[2];
  if (pool == 1) launch_pool<1>(kloop, const_mats, dim3(grid), x, U, y, a, p.fm, s);
  else if (pool == 2) launch_pool<2>(kloop, const_mats, dim3(grid), x, U, y, a, p.fm, s);
  else launch_pool<0>(kloop, const_mats, dim3(grid), x, U, y, a, p.fm, s);
  return launch_status();
}

}  // namespace wino
