// 3-D layers with a different output tile on the first axis: eq. (4) with
// its own transform triple per axis, F(m0, r) on axis 0 and F(m1, r) on axes
// 1 and 2 (for example m0 = 2 on a short temporal axis and m1 = 4 on the
// spatial ones).  Tiles are alpha0 x alpha1 x alpha1 input windows stepping
// by (m0, m1, m1); every axis uses the default points of its own F(m, r).
//
//   k_filter_ax  U = g x_0 G_0 x_1 G_1 x_2 G_1
//   k_input_ax   V = d x_0 B_0^T x_1 B_1^T x_2 B_1^T, split over alpha0
//                threads per (tile, channel) as k_input_split is
//   k_gemm_ax    M_xi = V_xi U_xi on fp32 MFMA with all alpha0 alpha1^2
//                elements of a 16-tile x 16-kernel block resident, then
//                y = M x_0 A_0^T x_1 A_1^T x_2 A_1^T, stitched, cropped, with
//                bias and activation
//
// Layouts are those of F(4^3): V[T_pad/16][C_pad/4][alpha^N][16][4],
// U[alpha^N][C_pad/4][K_pad][4] with alpha^N = alpha0 alpha1^2.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "kernels.hpp"
#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

template <int M0, int M1, int R>
struct AxShape {
  static constexpr int A0 = M0 + R - 1, A1 = M1 + R - 1;
  static constexpr int PL = A1 * A1;                // values of a first-axis plane
  static constexpr int NXI = A0 * PL;
  static constexpr int NOUT = M0 * M1 * M1;
  static constexpr int BLK = 16, CG = 4;
  static constexpr int NW = 12, NT = NW * 64;       // product work-group
  static constexpr int XPW = NXI / NW;              // elements per wave
  static constexpr int UPW = XPW / A1;              // last-axis rows per wave
  static constexpr int NUNIT = A0 * A1;             // last-axis rows of a block
  static constexpr int PLS = BLK * BLK + 8;         // epilogue plane stride (bank spread)
  static constexpr int LDS_FLOATS = NUNIT * M1 * PLS;
  static_assert(NXI % NW == 0 && XPW % A1 == 0, "waves own whole rows of the last axis");
  using BT0 = MatRef<Which::BT, true, M0, R>;
  using BT1 = MatRef<Which::BT, true, M1, R>;
  using G0 = MatRef<Which::G, true, M0, R>;
  using G1 = MatRef<Which::G, true, M1, R>;
  using AT0 = MatRef<Which::AT, true, M0, R>;
  using AT1 = MatRef<Which::AT, true, M1, R>;
};

// ------------------------------------------------------------ filter
// One thread per (channel, kernel), lanes over the channel group fastest (as
// k_filter).  adjoint: w is [C][K][r^3] and is read transposed and reversed.
template <int M0, int M1, int R>
__global__ void __launch_bounds__(64) k_filter_ax(const float* __restrict__ w, float* __restrict__ U,
                                                   FilterArgs a) {
  using S = AxShape<M0, M1, R>;
  constexpr int NXI = S::NXI, CG = S::CG, RN = R * R * R;
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int cl = int(idx % CG);
  const int k = int((idx / CG) % a.K_pad);
  const int cg = int(idx / (int64_t(CG) * a.K_pad));
  const int c = cg * CG + cl;
  if (c >= a.C_pad) return;
  float u[NXI];
  if (c < a.C && k < a.K) {
    float g[RN];
    if (a.adjoint) {
      const float* src = w + (int64_t(c) * a.K + k) * RN;
#pragma unroll
      for (int i = 0; i < RN; ++i) g[i] = src[RN - 1 - i];
    } else {
      const float* src = w + (int64_t(k) * a.C + c) * RN;
#pragma unroll
      for (int i = 0; i < RN; ++i) g[i] = src[i];
    }
    transform3_axes<R, S::A0, R, S::A1, R, S::A1>(g, u, typename S::G0{nullptr}, typename S::G1{nullptr},
                                                  typename S::G1{nullptr});
  } else {
#pragma unroll
    for (int i = 0; i < NXI; ++i) u[i] = 0.0f;
  }
  float* dst = U + (int64_t(cg) * a.K_pad + k) * CG + cl;
#pragma unroll
  for (int xi = 0; xi < NXI; ++xi) dst[int64_t(xi) * a.uplane] = u[xi];
}

// ------------------------------------------------------------- input
// A work-group covers one V block (16 tiles x 4 channels) with alpha0 waves:
// wave i0 gathers plane i0 of every (tile, channel) window (alpha1 rows of
// alpha1 values, zero outside the input, each row one load from a start
// clamped into the input row and shifted in registers) and transforms it
// along axes 1 and 2; the planes meet in LDS; wave x0 then forms output
// plane x0 = sum_i0 B_0^T[x0][i0] plane_i0 and stores it, 16 bytes (the 4
// channels of a tile) per lane.
template <int M0, int M1, int R>
__global__ void __launch_bounds__((M0 + R - 1) * 64) k_input_ax(const float* __restrict__ x,
                                                              float* __restrict__ V, InputArgs a) {
  using S = AxShape<M0, M1, R>;
  constexpr int A0 = S::A0, A1 = S::A1, PL = S::PL, NXI = S::NXI, BLK = S::BLK, CG = S::CG;
  constexpr int NQ = BLK * CG;
  __shared__ float4 planes[A0][PL][BLK];   // [plane][value][tile] -> the 4 channels

  const int lane = int(threadIdx.x) & 63;
  const int i0 = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int L = xcd_remap(int(blockIdx.x), a.nblocks);
  const int tb = L % a.ntb, cg = L / a.ntb;
  const int tl = lane % BLK, cl = lane / BLK;
  const int c = cg * CG + cl;
  const int t = tb * BLK + tl;
  const int XL = a.X[2];
  const bool live = t < a.T && c < a.C;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<3>(live ? t : 0, a.tiles, ti);
  const float* xn = x + (int64_t(n) * a.C + min(c, a.C - 1)) * a.xstride_c;
  const int o0 = ti[0] * M0 - a.pad[0], o1 = ti[1] * M1 - a.pad[1], oL = ti[2] * M1 - a.pad[2];
  const bool wide = XL >= A1;
  const int sL = wide ? min(max(oL, 0), XL - A1) : 0;
  const int delta = oL - sL;
  const int q0 = o0 + i0;
  const bool valid0 = live && (unsigned)q0 < (unsigned)a.X[0];
  const int64_t off0 = min(max(q0, 0), a.X[0] - 1);
  float d[PL];
#pragma unroll
  for (int i1 = 0; i1 < A1; ++i1) {
    const int q1 = o1 + i1;
    const bool valid = valid0 && (unsigned)q1 < (unsigned)a.X[1];
    const float* xr = xn + (off0 * a.X[1] + min(max(q1, 0), a.X[1] - 1)) * XL;
    float* dr = d + i1 * A1;
    if (wide) {
      float ld[A1];
      __builtin_memcpy(ld, xr + sL, sizeof(ld));
#pragma unroll
      for (int i = 0; i < A1; ++i) {
        float v = 0.0f;
#pragma unroll
        for (int j = 0; j < A1; ++j) v = (j == i + delta) ? ld[j] : v;
        dr[i] = valid ? v : 0.0f;
      }
    } else {
#pragma unroll
      for (int i = 0; i < A1; ++i) {
        const int qq = oL + i;
        const bool in = valid && (unsigned)qq < (unsigned)XL;
        const float v = xr[min(max(qq, 0), XL - 1)];
        dr[i] = in ? v : 0.0f;
      }
    }
  }
  float p2[PL];
  transform_nd<2, A1, A1>(d, p2, typename S::BT1{nullptr});   // axes 1 and 2 of the plane
  float* pl = reinterpret_cast<float*>(&planes[i0][0][tl]) + cl;
#pragma unroll
  for (int j = 0; j < PL; ++j) pl[j * BLK * CG] = p2[j];
  __syncthreads();

  // output plane x0 = i0 of this wave: lane (sj, tile) stores values j = sj + 4 k
  const int x0 = i0;
  const int sj = lane / BLK;
  float* dst = V + (int64_t(tb) * a.C_pad + int64_t(cg) * CG) * NXI * BLK + int64_t(x0) * PL * NQ + tl * CG;
  auto combine = [&](auto X0) {
    constexpr int xr = decltype(X0)::value;
#pragma unroll
    for (int k = 0; k < (PL + 3) / 4; ++k) {
      const int j = sj + 4 * k;
      if (j < PL) {
        float4 col[A0];
#pragma unroll
        for (int i = 0; i < A0; ++i) col[i] = planes[i][j][tl];
        const float* cf = reinterpret_cast<const float*>(col);
        f32x4 out;
        out[0] = row_dot<A0, xr>(typename S::BT0{nullptr}, cf + 0, 4);
        out[1] = row_dot<A0, xr>(typename S::BT0{nullptr}, cf + 1, 4);
        out[2] = row_dot<A0, xr>(typename S::BT0{nullptr}, cf + 2, 4);
        out[3] = row_dot<A0, xr>(typename S::BT0{nullptr}, cf + 3, 4);
        __builtin_nontemporal_store(out, reinterpret_cast<f32x4*>(dst + j * NQ));
      }
    }
  };
  switch (x0) {
    case 0: combine(std::integral_constant<int, 0>{}); break;
    case 1: combine(std::integral_constant<int, 1>{}); break;
    case 2: combine(std::integral_constant<int, 2>{}); break;
    case 3: combine(std::integral_constant<int, 3>{}); break;
    case 4: if constexpr (A0 > 4) combine(std::integral_constant<int, (A0 > 4 ? 4 : 0)>{}); break;
    default: if constexpr (A0 > 5) combine(std::integral_constant<int, (A0 > 5 ? 5 : 0)>{}); break;
  }
}

// ----------------------------------------------------------- product
// Work-group = 16 tiles x 16 kernels x all alpha^N elements; 12 waves split
// the elements, whole rows of the last axis each, and keep one 16 x 16
// accumulator per element on v_mfma_f32_16x16x4f32.  Operands stream from
// global memory as in k_gemm_inv: a lane loads 16 bytes (4 channels) of V
// and of U per element and 16-channel stage, feeding four k-steps.
// Epilogue: A_1^T along the last axis in registers; the m1 results of every
// last-axis row go to LDS; then item (output of the last axis, kernel, tile)
// applies A_0^T along axis 0 and A_1^T along axis 1, adds the bias, applies
// the activation, crops and stores.
template <int M0, int M1, int R>
__global__ void __launch_bounds__(768) k_gemm_ax(const float* __restrict__ V, const float* __restrict__ U,
                                                 float* __restrict__ y, GemmArgs g) {
  using S = AxShape<M0, M1, R>;
  using MS = MfmaShape<16>;
  constexpr int A0 = S::A0, A1 = S::A1, NXI = S::NXI, BLK = S::BLK, CG = S::CG, XPW = S::XPW;
  constexpr int UPW = S::UPW, NUNIT = S::NUNIT, PLS = S::PLS;
  constexpr int VEC = 4, SC = MS::KSTEP * VEC;      // 16 channels per stage
  __shared__ float sm[S::LDS_FLOATS];
  __shared__ float bsm[BLK];

  const int lane = int(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int L = xcd_remap(int(blockIdx.x), g.nblocks);
  const int tb = L / g.nkb, kb = L % g.nkb;
  const int col = lane % BLK, kr = lane / BLK;

  // operands through buffer resources, as in k_gemm_inv: wave-uniform stage
  // bases, the lane's byte offset, each element's offset as the scalar one
  // (the planner keeps a wave's U offsets below 2^32 bytes)
  const int64_t vxi = int64_t(BLK) * CG, uxi = g.uplane;
  const int c0 = VEC * kr;
  const float* vnext = V + int64_t(tb) * NXI * g.C_pad * BLK + int64_t(wave) * XPW * vxi;
  const float* unext = U + int64_t(wave) * XPW * uxi + int64_t(kb) * BLK * CG;
  const int vlane = ((c0 / CG) * NXI * BLK * CG + col * CG + c0 % CG) * 4;
  const int ulane = (((c0 / CG) * g.K_pad + col) * CG + c0 % CG) * 4;
  const int64_t vgstep = int64_t(NXI) * BLK * SC, ugstep = int64_t(g.K_pad) * SC;
  const int nstages = g.C_pad / SC;

  typename MS::acc_t acc[XPW];
#pragma unroll
  for (int e = 0; e < XPW; ++e) acc[e] = typename MS::acc_t{};
  for (int s = 0; s < nstages; ++s) {
    float4 ra[XPW], rb[XPW];
    const __amdgpu_buffer_rsrc_t rv = raw_rsrc(vnext), ru = raw_rsrc(unext);
#pragma unroll
    for (int e = 0; e < XPW; ++e) {
      ra[e] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rv, vlane, int(e * vxi * 4), 0));
      rb[e] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(ru, ulane, int(e * uxi * 4), 0));
    }
    vnext += vgstep;
    unext += ugstep;
#pragma unroll
    for (int j = 0; j < VEC; ++j)
#pragma unroll
      for (int e = 0; e < XPW; ++e)
        acc[e] = MS::mma(reinterpret_cast<const float*>(&ra[e])[j], reinterpret_cast<const float*>(&rb[e])[j],
                         acc[e]);
  }

  // Part 1: A_1^T along the last axis; plane (row, o2) at [k][t ^ k]
  if (g.bias != nullptr && int(threadIdx.x) < BLK) {
    const int kg = kb * BLK + int(threadIdx.x);
    bsm[threadIdx.x] = kg < g.K ? g.bias[kg] : 0.0f;
  }
#pragma unroll
  for (int r = 0; r < MS::NACC; ++r) {
    const int t = MS::acc_row(lane, r);
#pragma unroll
    for (int u = 0; u < UPW; ++u) {
      float sv[A1];
#pragma unroll
      for (int e = 0; e < A1; ++e) sv[e] = acc[u * A1 + e][r];
      float o[M1];
      apply_vec<A1, M1>(typename S::AT1{nullptr}, sv, 1, o, 1);
      float* dst = sm + ((wave * UPW + u) * M1) * PLS + col * BLK + (t ^ col);
#pragma unroll
      for (int q = 0; q < M1; ++q) dst[q * PLS] = o[q];
    }
  }
  __syncthreads();

  // Part 2: item (o2, k, t), last-axis output fastest, then the tile, so that
  // neighbouring lanes store neighbouring outputs of a row
  constexpr int NT = S::NT;
  constexpr int NTE = (NT / (M1 * BLK)) * (M1 * BLK);
  const int tid = int(threadIdx.x);
  if (tid >= NTE) return;
  const int o2 = tid % M1;
  const int tl = (tid / M1) % BLK;
  const int t = tb * BLK + tl;
  if (t >= g.T) return;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<3>(t, g.tiles, ti);
  const int y2 = ti[2] * M1 + o2;
  if (y2 >= g.Y[2]) return;
  constexpr int ITEMS = M1 * BLK * BLK;
  for (int i = tid; i < ITEMS; i += NTE) {
    const int k_l = (i / (M1 * BLK)) % BLK;
    const int kg = kb * BLK + k_l;
    if (kg >= g.K) continue;
    float v[NUNIT];
#pragma unroll
    for (int uu = 0; uu < NUNIT; ++uu) v[uu] = sm[(uu * M1 + o2) * PLS + k_l * BLK + (tl ^ k_l)];
    float tmp[M0 * A1], out[M0 * M1];
    apply_axis<1, A0, M0, A1>(v, tmp, typename S::AT0{nullptr});   // axis 0
    apply_axis<M0, A1, M1, 1>(tmp, out, typename S::AT1{nullptr}); // axis 1
    float* yk = y + (int64_t(n) * g.K + kg) * g.ystride_k;
    const float bk = g.bias != nullptr ? bsm[k_l] : 0.0f;
#pragma unroll
    for (int q0 = 0; q0 < M0; ++q0) {
      const int y0 = ti[0] * M0 + q0;
#pragma unroll
      for (int q1 = 0; q1 < M1; ++q1) {
        const int y1 = ti[1] * M1 + q1;
        if (y0 >= g.Y[0] || y1 >= g.Y[1]) continue;
        float val = out[q0 * M1 + q1] + bk;
        val = activate(val, g.act, g.slope);
        yk[(int64_t(y0) * g.Y[1] + y1) * g.Y[2] + y2] = val;
      }
    }
  }
}

}  // namespace wino
