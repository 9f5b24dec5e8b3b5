// F(4^3, 3^3) with the input transform fused into the batched product:
// V never reaches memory.
//
// One work-group owns a block of 16 tiles x 16 kernels and keeps the 216
// per-element products M_xi = sum_c V_xi U_xi of that block in MFMA
// accumulators (as k_gemm_inv does), but it forms V itself, 8 channels at a
// time, from the input x:
//
//   produce  thread (tile, channel, plane i0) loads plane i0 of its tile's
//            6 x 6 x 6 input window (zero outside the padded input) and
//            transforms it along the last two axes: P_i0 = d_i0 x_1 B^T x_2 B^T
//            (eq. 4); the 36 values go to LDS.
//   consume  the wave of element xi = (xi0, xi1, xi2) finishes the transform
//            along the first axis while it loads its MFMA operand,
//            V_xi = sum_i0 B^T[xi0][i0] P_i0[xi1][xi2] (only the non-zero
//            entries of B^T's row are read), and multiplies it with U_xi on
//            v_mfma_f32_16x16x4f32 (two k-steps per 8-channel chunk).
//
// This is the GPU counterpart of the paper's blocking of a thread's tiles to
// its cache with the data reshuffle counted (§4.1, §4.3): the transformed
// data of a tile block lives only in LDS.  After the last chunk the inverse
// transform, bias, activation, crop and store run as k_gemm_inv's epilogue.
//
// The transform is recomputed for every block of 16 kernels of a tile block
// (its two kernel blocks run on the same XCD and share the input windows in
// L2), which pays while K is small: the planner picks this kernel for
// F(4^3) layers with at most 64 kernels.
//
// Channel mapping of a chunk (8 channels): MFMA lane group kr holds channels
// 2kr and 2kr + 1 (k-steps 0 and 1), so a lane reads its A operand as one
// 8-byte LDS read per term and its U operand as one 8-byte global read
// (U[xi][c/4][k][c%4]: channels 2kr, 2kr + 1 sit in group kr/2 at 2(kr%2)).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "kernels.hpp"
#include "layout.hpp"
#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

struct FusedArgs {
  int64_t xstride_c;   // prod X_i
  int64_t uplane;      // C_pad * K_pad
  int64_t ystride_k;   // prod Y_i
  int32_t C, C_pad, K, K_pad;
  int32_t T, nkb, nblocks;
  int32_t X[3], tiles[3], pad[3], Y[3];
  int32_t rowfast;     // every 16-tile block is 16 tiles of one input row (rows of a multiple of 4, pad <= 2)
  int32_t act;         // activation f of eq. (2): 0 none, 1 ReLU, 2 leaky ReLU
  float slope;
  const float* bias;   // [K] or null
};

struct Fused43Geom {
  static constexpr int A = 6, NXI = 216, BLK = 16, NW = 12, NT = NW * 64, LOC = 1;
  static constexpr int CH = 8;                       // channels per chunk
  static constexpr int PL = A * A;                   // values of a plane after two axes
  static constexpr int XPW = NXI / NW;               // elements per wave (18: three alpha-rows)
  static constexpr int P_FLOATS = A * PL * CH * BLK; // 27648: the chunk's planes
  using Epi = GemmGeom<3, 4, 3, BLK, NW, LOC>;
  static constexpr int LDS_FLOATS = Epi::LDS_FLOATS > P_FLOATS ? Epi::LDS_FLOATS : P_FLOATS;
  static_assert(XPW == 18 && NW * 4 == CH * A, "a wave is 4 (channel, plane) rows of 16 tiles");
};

// P layout in LDS: P[i0][j][pair][tile][2] (j < 36 the plane value, pair =
// channel / 2): lane (kr, col) of an MFMA operand reads 8 bytes at
// ((i0 * 36 + j) * 4 + kr) * 32 + 2 * col, 512 contiguous bytes per wave.
__device__ __forceinline__ int p_index(int i0, int j, int ch, int tl) {
  return ((i0 * Fused43Geom::PL + j) * (Fused43Geom::CH / 2) + (ch >> 1)) * 32 + tl * 2 + (ch & 1);
}

template <bool CONST>
__global__ void __launch_bounds__(768, 1) k_fused43(const float* __restrict__ x, const float* __restrict__ U,
                                                    float* __restrict__ y, FusedArgs a, FMats fm) {
  using G = Fused43Geom;
  constexpr int N = 3, MM = 4, R = 3, A = G::A, BLK = G::BLK, CH = G::CH, PL = G::PL, XPW = G::XPW;
  using S = MfmaShape<16>;
  __shared__ float sm[G::LDS_FLOATS];

  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  // consecutive logical blocks (the kernel blocks of one tile block, then the
  // next tile block) run on one XCD and share the input windows in its L2
  const int L = xcd_remap(int(blockIdx.x), a.nblocks);
  const int tb = L / a.nkb, kb = L % a.nkb;
  const MatRef<Which::BT, CONST, MM, R> BT{&fm};

  // ---- producer role: lane = tile of the block, 16-lane row = (channel, plane)
  const int tl = lane & 15;
  const int q = wave * 4 + (lane >> 4);      // 0..47
  const int pch = q % CH, i0 = q / CH;
  const int XL = a.X[N - 1];
  // rowfast: the block's 16 tiles share the sample and leading tile coordinates
  int ti_b[3] = {0, 0, 0};
  const int n_b = split_tile<N>(tb * BLK, a.tiles, ti_b);
  // gather path: this lane's own tile
  const int t = tb * BLK + tl;
  const bool tlive = t < a.T;
  int ti_t[3] = {0, 0, 0};
  const int n_t = split_tile<N>(tlive ? t : 0, a.tiles, ti_t);

  auto produce = [&](int chunk) {
    // an opaque zero, new every chunk: the window addresses below depend on
    // it, so the compiler recomputes them per chunk instead of keeping them
    // live across the loop (where they would spill)
    int z;
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
    const int c = chunk * CH + pch + z;
    const bool clive = c < a.C;
    const float* xc = x + int64_t(clive ? c : 0) * a.xstride_c;
    float d[PL];   // the plane's rows, each transformed along the last axis
    if (a.rowfast) {
      const float* xn = xc + int64_t(n_b) * a.C * a.xstride_c;
      const int tW = ti_b[2] + tl;
      const int q0 = ti_b[0] * MM - a.pad[0] + i0 + z;
      const bool valid0 = clive && (unsigned)q0 < (unsigned)a.X[0];
      const int wo = min(MM * tW, XL - 4);
      const bool own_in = MM * tW < XL;
      // row ends: lanes 0..7 fetch the two values left of the block, 8..15 the two right of it
      const int wl = MM * ti_b[2] - 2, wr = MM * ti_b[2] + MM * BLK;
      const bool left = tl < BLK / 2;
      const int wh = left ? max(wl, 0) : min(wr, XL - 2);
      const bool h_in = left ? wl >= 0 : wr < XL;
      // the twelve loads of the six rows are issued before any is used
      float4 o[A];
      float2 h[A];
      bool rv[A];
#pragma unroll
      for (int i1 = 0; i1 < A; ++i1) {
        const int q1 = ti_b[1] * MM - a.pad[1] + i1;
        rv[i1] = valid0 && (unsigned)q1 < (unsigned)a.X[1];
        // 32-bit offsets inside one channel's volume (the planner bounds it below 2^31)
        const int roff = (min(max(q0, 0), a.X[0] - 1) * a.X[1] + min(max(q1, 0), a.X[1] - 1)) * XL;
        o[i1] = *reinterpret_cast<const float4*>(xn + roff + wo);
        h[i1] = *reinterpret_cast<const float2*>(xn + roff + wh);
      }
      auto rows = [&](auto PP) {
        constexpr int P = decltype(PP)::value;
#pragma unroll
        for (int i1 = 0; i1 < A; ++i1) {
          // the 16 lanes of a DPP row share channel, plane and row, hence validity
          const float4 ov = (own_in && rv[i1]) ? o[i1] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
          const float2 hv = (h_in && rv[i1]) ? h[i1] : make_float2(0.0f, 0.0f);
          float e[8];   // offsets -2 .. 5 from 4 * tW
          e[0] = dpp_from_prev(hv.x, ov.z);
          e[1] = dpp_from_prev(hv.y, ov.w);
          e[2] = ov.x; e[3] = ov.y; e[4] = ov.z; e[5] = ov.w;
          e[6] = dpp_from_next(hv.x, ov.x);
          e[7] = dpp_from_next(hv.y, ov.y);
          float w6[A];
#pragma unroll
          for (int i = 0; i < A; ++i) w6[i] = e[i + 2 - P];
          apply_vec<A, A>(BT, w6, 1, d + i1 * A, 1);   // B^T along the row (the window's last axis)
        }
      };
      switch (a.pad[2]) {
        case 0: rows(std::integral_constant<int, 0>{}); break;
        case 1: rows(std::integral_constant<int, 1>{}); break;
        default: rows(std::integral_constant<int, 2>{}); break;
      }
    } else {
      const bool live = tlive && clive;
      const float* xn = xc + int64_t(n_t) * a.C * a.xstride_c;
      int o[3];
#pragma unroll
      for (int ax = 0; ax < N; ++ax) o[ax] = ti_t[ax] * MM - a.pad[ax] + z;
      const int oL = o[N - 1];
      const bool wide = XL >= A;
      const int sL = wide ? min(max(oL, 0), XL - A) : 0;
      const int delta = oL - sL;
      const int q0 = o[0] + i0;
      const bool valid0 = live && (unsigned)q0 < (unsigned)a.X[0];
      const int off0 = min(max(q0, 0), a.X[0] - 1);
#pragma unroll
      for (int i1 = 0; i1 < A; ++i1) {
        const int q1 = o[1] + i1;
        const bool valid = valid0 && (unsigned)q1 < (unsigned)a.X[1];
        const float* xr = xn + (off0 * a.X[1] + min(max(q1, 0), a.X[1] - 1)) * XL;   // 32-bit, as above
        float w6[A];
        if (wide) {
          float ld[A];
          __builtin_memcpy(ld, xr + sL, sizeof(ld));
#pragma unroll
          for (int i = 0; i < A; ++i) {
            float v = 0.0f;
#pragma unroll
            for (int j = 0; j < A; ++j) v = (j == i + delta) ? ld[j] : v;
            w6[i] = valid ? v : 0.0f;
          }
        } else {
#pragma unroll
          for (int i = 0; i < A; ++i) {
            const int qq = oL + i;
            const bool in = valid && (unsigned)qq < (unsigned)XL;
            const float v = xr[min(max(qq, 0), XL - 1)];
            w6[i] = in ? v : 0.0f;
          }
        }
        apply_vec<A, A>(BT, w6, 1, d + i1 * A, 1);     // B^T along the row
      }
    }
    // B^T along the columns (the window's middle axis), each column's six
    // values stored as they are formed: P_i0[xi1][xi2] at j = 6 xi1 + xi2
#pragma unroll
    for (int i2 = 0; i2 < A; ++i2) {
      float cv[A];
      apply_vec<A, A>(BT, d + i2, A, cv, 1);
#pragma unroll
      for (int j1 = 0; j1 < A; ++j1) sm[p_index(i0, j1 * A + i2, pch, tl)] = cv[j1];
    }
  };

  // ---- consumer role: MFMA lane (kr, col); wave owns elements wave * 18 ..
  const int col = lane & 15, kr = lane >> 4;
  const int x0 = wave >> 1;                      // first-axis index of the wave's elements
  const int j0 = (wave & 1) * XPW;               // first plane value of the wave: 18 * (wave % 2)
  typename S::acc_t acc[XPW];
#pragma unroll
  for (int e = 0; e < XPW; ++e) acc[e] = typename S::acc_t{};
  const float2* P2 = reinterpret_cast<const float2*>(sm);
  // U[xi][c/4][k][c%4]: lane (kr, col) reads channels 2kr, 2kr + 1 of the chunk
  // 32-bit offsets into U (the planner bounds U below 2^31 floats)
  const int uplane = int(a.uplane);
  const float* ubase = U + wave * XPW * uplane + ((kr >> 1) * a.K_pad + kb * BLK + col) * 4 +
                       2 * (kr & 1);

  // the chunk's 18 U operands, loaded together before the chunk's barrier
  // so that their latency overlaps the other waves' producing
  float2 ur[XPW];
  auto load_u = [&](int chunk) {
    const float* uc = ubase + chunk * 8 * a.K_pad;
#pragma unroll
    for (int e = 0; e < XPW; ++e) ur[e] = *reinterpret_cast<const float2*>(uc + e * uplane);
  };
  auto consume = [&](auto X0) {
    constexpr int xr = decltype(X0)::value;
    // the P values an element needs: one 8-byte read per first-axis plane
    // whose B^T coefficient is not zero (a compile-time test for the default
    // points); element e + 1's reads are issued before element e's products
    auto fetch = [&](float2* pv, int e) {
#pragma unroll
      for (int i = 0; i < A; ++i)
        if (BT(xr, i) != 0.0f) pv[i] = P2[((i * PL + j0 + e) * 4 + kr) * 16 + col];
    };
    auto product = [&](const float2* pv, int e) {
      float2 v = make_float2(0.0f, 0.0f);
      bool first = true;
#pragma unroll
      for (int i = 0; i < A; ++i) {
        const float cf = BT(xr, i);
        if (cf == 0.0f) continue;
        if (first) {
          v.x = cf * pv[i].x; v.y = cf * pv[i].y;
          first = false;
        } else {
          v.x = __builtin_fmaf(cf, pv[i].x, v.x);
          v.y = __builtin_fmaf(cf, pv[i].y, v.y);
        }
      }
      acc[e] = S::mma(v.x, ur[e].x, acc[e]);
      acc[e] = S::mma(v.y, ur[e].y, acc[e]);
    };
    float2 pa[A], pb[A];
    fetch(pa, 0);
#pragma unroll
    for (int e = 0; e < XPW; e += 2) {
      fetch(pb, e + 1);
      product(pa, e);
      if (e + 2 < XPW) fetch(pa, e + 2);
      product(pb, e + 1);
    }
  };

  // chunks past the last real channel hold only zero padding (x and U are
  // zero there): they are skipped
  const int nchunks = (a.C + CH - 1) / CH;
  for (int chunk = 0; chunk < nchunks; ++chunk) {
    if (chunk > 0) __syncthreads();             // the previous chunk's planes are read
    produce(chunk);
    load_u(chunk);
    __syncthreads();
    switch (x0) {
      case 0: consume(std::integral_constant<int, 0>{}); break;
      case 1: consume(std::integral_constant<int, 1>{}); break;
      case 2: consume(std::integral_constant<int, 2>{}); break;
      case 3: consume(std::integral_constant<int, 3>{}); break;
      case 4: consume(std::integral_constant<int, 4>{}); break;
      default: consume(std::integral_constant<int, 5>{}); break;
    }
  }
  __syncthreads();                              // the planes' LDS is reused by the epilogue

  EpiArgs e{y, a.K, a.ystride_k, {a.Y[0], a.Y[1], a.Y[2]}, a.act, a.slope, a.bias};
  auto tile_of = [&](int tl2, int* ti) -> int {
    const int t2 = tb * BLK + tl2;
    if (t2 >= a.T) return -1;
    return split_tile<N>(t2, a.tiles, ti);
  };
  if (a.bias != nullptr) gemm_epilogue<N, MM, R, CONST, BLK, G::NW, G::LOC, true>(acc, sm, kb, e, fm, tile_of);
  else gemm_epilogue<N, MM, R, CONST, BLK, G::NW, G::LOC, false>(acc, sm, kb, e, fm, tile_of);
}

}  // namespace wino
