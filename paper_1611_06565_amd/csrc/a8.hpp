// 3-D layers on the alpha = 8 sizes of Table 1: F(5^3, 4^3), F(4^3, 5^3) and
// F(3^3, 6^3) (m + r - 1 = 8, alpha^3 = 512 transformed values per tile).
//
// 512 elements are too many for any of the other product kernels: all 512
// accumulators of a 16 x 16 (tile, kernel) block fill the register file, and
// a thread cannot hold a 512-value window.  So:
//
//   k_filter_a8  one thread per (channel, kernel, xi0) forms one xi0-plane
//                of U = g x_0 G x_1 G x_2 G (64 values);
//   k_input_a8   a work-group forms half a V block (8 tiles x 4 channels):
//                each half wave transforms plane i0 of each window along the
//                last two axes into LDS, then each half wave combines the
//                eight planes along the first axis for one xi0 and stores
//                V[.][xi0 * 64 + j];
//   k_gemm_a8    a work-group owns 16 tiles x 16 kernels and walks the first
//                axis: pass xi0 accumulates M_xi = sum_c V_xi U_xi for the 64
//                elements of plane xi0 (16 waves, half an alpha-row each),
//                applies A^T along the last axis in registers and along the
//                middle axis through LDS, and adds A^T[o0][xi0] times the
//                result into the m^3 outputs of each (tile, kernel), kept in
//                the registers of the thread that stores them (eq. 4 is
//                linear, so the inverse transform splits over xi0).
//
// Layouts are those of F(4^3): V[T_pad/16][C_pad/4][512][16][4],
// U[512][C_pad/4][K_pad][4].
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "kernels.hpp"
#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

template <int MM, int R>
struct A8Shape {
  static constexpr int A = MM + R - 1;
  static constexpr int PL = A * A;                  // values of a first-axis plane (64)
  static constexpr int NXI = A * PL;                // 512
  static constexpr int BLK = 16, CG = 4;
  static_assert(A == 8, "alpha = 8");
  // product: 16 waves, wave w owns the half alpha-row (xi1 = w / 2,
  // xi2 = 4 (w % 2) .. + 3) of the current plane
  static constexpr int NW = 16, NT = NW * 64;
  static constexpr int EW = A / 2;                  // elements per wave and pass
  static constexpr int SC = 16;                     // channels per operand stage (4 groups)
  static constexpr int EPL = BLK * BLK + 8;         // LDS plane stride (bank spread)
  static constexpr int NPLANE = A * 2 * MM;         // (xi1, half, o2) planes
  static constexpr int NOUT3 = MM * MM * MM;        // outputs of a (tile, kernel)
  static constexpr int TROW = BLK * MM + 1;         // store stage row: 16 tiles x m values (+1 bank spread)
  static constexpr int STORE_FLOATS = BLK * MM * MM * TROW;   // [kernel][o0][o1] rows
  static constexpr int LDS_FLOATS = NPLANE * EPL > STORE_FLOATS ? NPLANE * EPL : STORE_FLOATS;
  static constexpr int ITEMS = MM * BLK * BLK;      // (o2, kernel, tile) output columns
  static constexpr int IPT = (ITEMS + NT - 1) / NT; // columns per thread
  static constexpr int NOUT = MM * MM;              // outputs (o0, o1) of a column
};

// ------------------------------------------------------------ filter
// idx = ((xi0 * C_pad/4 + cg) * K_pad + k) * 4 + cl: a 64-thread work-group
// shares xi0 (C_pad * K_pad is a multiple of 256).  adjoint: w is [C][K][r^3]
// and is read transposed and reversed.
template <int MM, int R, bool CONST>
__global__ void __launch_bounds__(64) k_filter_a8(const float* __restrict__ w, float* __restrict__ U,
                                                   FilterArgs a, FMats fm) {
  using S = A8Shape<MM, R>;
  constexpr int A = S::A, CG = S::CG;
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int cl = int(idx % CG);
  const int k = int((idx / CG) % a.K_pad);
  const int64_t rest = idx / (int64_t(CG) * a.K_pad);
  const int ncg = a.C_pad / CG;
  const int cg = int(rest % ncg);
  const int xi0 = __builtin_amdgcn_readfirstlane(int(rest / ncg));
  if (xi0 >= A) return;
  const int c = cg * CG + cl;
  const MatRef<Which::G, CONST, MM, R> G{&fm};
  float u[S::PL];
  if (c < a.C && k < a.K) {
    constexpr int RR = R * R;
    float h[RR];   // the kernel contracted with row xi0 of G along the first axis
#pragma unroll
    for (int i = 0; i < RR; ++i) h[i] = 0.0f;
    for (int i0 = 0; i0 < R; ++i0) {
      const float gc = G(xi0, i0);
#pragma unroll
      for (int i = 0; i < RR; ++i) {
        const int flat = i0 * RR + i;
        const float v = a.adjoint ? w[(int64_t(c) * a.K + k) * (R * RR) + (R * RR - 1 - flat)]
                                  : w[(int64_t(k) * a.C + c) * (R * RR) + flat];
        h[i] = __builtin_fmaf(gc, v, h[i]);
      }
    }
    transform_nd<2, R, A>(h, u, G);
  } else {
#pragma unroll
    for (int i = 0; i < S::PL; ++i) u[i] = 0.0f;
  }
  float* dst = U + (int64_t(cg) * a.K_pad + k) * CG + cl + int64_t(xi0) * S::PL * a.uplane;
#pragma unroll
  for (int j = 0; j < S::PL; ++j) dst[int64_t(j) * a.uplane] = u[j];
}

// ------------------------------------------------------------- input
// One work-group per half V block (8 of its 16 tiles x one group of 4
// channels), 4 waves.  The 64 plane values j go through LDS in two halves
// (32 KB), the second half held in registers meanwhile, so that four
// work-groups share a CU.
// Phase 1: lane (plane i0 = 2 * wave + lane / 32, channel cl, tile tl) loads
// plane i0 of its tile's 8 x 8 x 8 window (zero outside the padded input and
// for channels past C) and transforms it along the last two axes.  A window
// whose rows lie inside the input row is read as one 32-byte load per row;
// one that crosses an end of the row (the first and last tiles of a row)
// value by value, clamped and masked.
// Phase 2, once per half of the plane values: the lanes write their half to
// P[i0][j][tl][cl]; item (j, tl, cl) reads P[0..7][j], applies B^T along the
// first axis (one matrix application for all eight xi0) and stores
// V[xi0 * 64 + j] for every xi0; a half wave covers the half block's 128
// contiguous bytes of one j.
template <int MM, int R, bool CONST>
__global__ void __launch_bounds__(256) k_input_a8(const float* __restrict__ x, float* __restrict__ V,
                                                  InputArgs a, FMats fm) {
  using S = A8Shape<MM, R>;
  constexpr int A = S::A, PL = S::PL, BLK = S::BLK, CG = S::CG;
  constexpr int HB = BLK / 2;              // tiles of a half block
  constexpr int HQ = HB * CG;              // (tile, channel) pairs of a half block (32)
  constexpr int NT = 256;
  constexpr int PH = PL / 2;               // plane values per half
  __shared__ float P[A * PH * HQ];         // 32 KB: one half of the planes
  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ncg = a.C_pad / CG;
  // logical block (channel group, tile block, half), halves and tile blocks
  // fastest, in contiguous ranges per XCD: an XCD walks consecutive windows of
  // one channel group, whose overlaps then hit its L2
  const int L = xcd_remap(int(blockIdx.x), a.nblocks);
  const int hb = L & 1;
  const int tb = (L >> 1) % a.ntb, cg = (L >> 1) / a.ntb;
  const MatRef<Which::BT, CONST, MM, R> BT{&fm};
  float d[PL];   // plane i0 of the window, then of its transform
  {
    const int i0 = 2 * wave + (lane >> 5), tl = lane & (HB - 1), cl = (lane & 31) / HB;
    const int t = tb * BLK + hb * HB + tl;
    const int c = cg * CG + cl;
    const bool live = t < a.T && c < a.C;
    int ti[3] = {0, 0, 0};
    const int n = split_tile<3>(live ? t : 0, a.tiles, ti);
    const float* xc = x + (int64_t(n) * a.C + (live ? c : 0)) * a.xstride_c;
    const int q0 = ti[0] * MM - a.pad[0] + i0;
    const bool v0 = live && (unsigned)q0 < (unsigned)a.X[0];
    const int64_t off0 = int64_t(min(max(q0, 0), a.X[0] - 1)) * a.X[1];
    const int XL = a.X[2];
    const int s2 = ti[2] * MM - a.pad[2];
    if (s2 >= 0 && s2 + A <= XL) {
#pragma unroll
      for (int i1 = 0; i1 < A; ++i1) {
        const int q1 = ti[1] * MM - a.pad[1] + i1;
        const bool v1 = v0 && (unsigned)q1 < (unsigned)a.X[1];
        const float* xr = xc + (off0 + min(max(q1, 0), a.X[1] - 1)) * XL;
        float ld[A];
        __builtin_memcpy(ld, xr + s2, sizeof(ld));
#pragma unroll
        for (int i2 = 0; i2 < A; ++i2) d[i1 * A + i2] = v1 ? ld[i2] : 0.0f;
      }
    } else {
#pragma unroll
      for (int i1 = 0; i1 < A; ++i1) {
        const int q1 = ti[1] * MM - a.pad[1] + i1;
        const bool v1 = v0 && (unsigned)q1 < (unsigned)a.X[1];
        const float* xr = xc + (off0 + min(max(q1, 0), a.X[1] - 1)) * XL;
#pragma unroll
        for (int i2 = 0; i2 < A; ++i2) {
          const int q2 = s2 + i2;
          const float v = xr[min(max(q2, 0), XL - 1)];
          d[i1 * A + i2] = (v1 && (unsigned)q2 < (unsigned)XL) ? v : 0.0f;
        }
      }
    }
#pragma unroll
    for (int i1 = 0; i1 < A; ++i1) {
      float row[A];
      apply_vec<A, A>(BT, d + i1 * A, 1, row, 1);   // B^T along the row (last axis)
#pragma unroll
      for (int i2 = 0; i2 < A; ++i2) d[i1 * A + i2] = row[i2];
    }
#pragma unroll
    for (int i2 = 0; i2 < A; ++i2) {
      float cv[A];
      apply_vec<A, A>(BT, d + i2, A, cv, 1);          // B^T along the columns (middle axis)
#pragma unroll
      for (int j1 = 0; j1 < A; ++j1) d[j1 * A + i2] = cv[j1];   // d[j] = plane value j
    }
  }
  float* const dst = V + (int64_t(tb) * ncg + cg) * S::NXI * (BLK * CG) + hb * HQ;
  const int pidx = ((2 * wave + (lane >> 5)) * PH) * HQ + (lane & (HB - 1)) * CG + (lane & 31) / HB;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (h == 1) __syncthreads();                  // the first half has been read
#pragma unroll
    for (int jj = 0; jj < PH; ++jj) P[pidx + jj * HQ] = d[h * PH + jj];
    __syncthreads();
#pragma unroll 2
    for (int i = tid; i < PH * HQ; i += NT) {
      const int q = i % HQ, jj = i / HQ, j = h * PH + jj;
      float pv[A], vo[A];
#pragma unroll
      for (int i0 = 0; i0 < A; ++i0) pv[i0] = P[(i0 * PH + jj) * HQ + q];
      apply_vec<A, A>(BT, pv, 1, vo, 1);
#pragma unroll
      for (int xi0 = 0; xi0 < A; ++xi0)
        __builtin_nontemporal_store(vo[xi0], dst + (xi0 * PL + j) * (BLK * CG) + q);
    }
  }
}

// ------------------------------------------------------------- product
// One work-group per (tile block, kernel block); see the top of the file.
// Operands: lane (kr, col) loads 16 bytes per element and stage, channels
// 4 (4 s + kr) .. + 3 of V row `col` and of U column `col`; k-step j of the
// stage uses the j-th of them, so the four k-steps contract 16 channels.
template <int MM, int R, bool CONST>
__global__ void __launch_bounds__(1024) k_gemm_a8(const float* __restrict__ V, const float* __restrict__ U,
                                                  float* __restrict__ y, GemmArgs g, FMats fm) {
  using S = A8Shape<MM, R>;
  using F = MfmaShape<16>;
  constexpr int A = S::A, PL = S::PL, BLK = S::BLK, CG = S::CG, EW = S::EW, EPL = S::EPL;
  constexpr int IPT = S::IPT, NOUT = S::NOUT;
  __shared__ float sm[S::LDS_FLOATS];
  __shared__ float bsm[BLK];
  __shared__ int tsm[BLK][4];   // per tile of the block: sample (-1 past T), output origin on each axis

  const int lane = int(threadIdx.x) & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int L = xcd_remap(int(blockIdx.x), g.nblocks);
  const int tb = L / g.nkb, kb = L % g.nkb;
  const int col = lane & 15, kr = lane >> 4;
  const int xi1 = wave >> 1, half = wave & 1;
  const int ncg = g.C_pad / CG;
  const int nstage = g.C_pad / S::SC;
  const MatRef<Which::AT, CONST, MM, R> AT{&fm};

  if (g.bias != nullptr && int(threadIdx.x) < BLK) {
    const int kg = kb * BLK + int(threadIdx.x);
    bsm[threadIdx.x] = kg < g.K ? g.bias[kg] : 0.0f;
  }
  if (int(threadIdx.x) < BLK) {
    const int t = tb * BLK + int(threadIdx.x);
    int ti[3] = {0, 0, 0};
    const int n = split_tile<3>(t < g.T ? t : 0, g.tiles, ti);
    tsm[threadIdx.x][0] = t < g.T ? n : -1;
    for (int ax = 0; ax < 3; ++ax) tsm[threadIdx.x][1 + ax] = ti[ax] * MM;
  }

  // the thread's output columns: item i = tid + NT q -> (o2, kernel, tile)
  float out[IPT][NOUT];
#pragma unroll
  for (int q = 0; q < IPT; ++q)
#pragma unroll
    for (int o = 0; o < NOUT; ++o) out[q][o] = 0.0f;

  // operand rows of lane (kr, col): V[tb][cg][xi][col][.], U[xi][cg][kb*16+col][.],
  // read through buffer resources: wave-uniform bases per step (scalar
  // registers), the lane's byte offset as the vector offset and each
  // element's offset as the scalar one, so the loads need no per-lane 64-bit
  // address arithmetic (the planner keeps 4 U planes below 2^32 bytes)
  const float* vbase = V + int64_t(tb) * ncg * S::NXI * (BLK * CG);
  const float* ubase = U + int64_t(kb) * BLK * CG;
  const int vlane = (kr * S::NXI * (BLK * CG) + col * CG) * 4;
  const int ulane = (kr * g.K_pad * CG + col * CG) * 4;
  // the EW operands of V and of U of element run xb (the wave's) at channel stage st
  auto load_ops = [&](float4* av, float4* uv, int xb, int st) {
    const __amdgpu_buffer_rsrc_t rv = raw_rsrc(vbase + (int64_t(st) * 4 * S::NXI + xb) * (BLK * CG));
    const __amdgpu_buffer_rsrc_t ru = raw_rsrc(ubase + int64_t(xb) * g.uplane + int64_t(st) * 4 * g.K_pad * CG);
#pragma unroll
    for (int e = 0; e < EW; ++e) {
      av[e] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rv, vlane, e * (BLK * CG) * 4, 0));
      uv[e] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(ru, ulane, int(e * g.uplane * 4), 0));
    }
  };

  if constexpr (MM == 4 && CONST) {
    // F(4^3, 5^3): the next step's operands load while this step multiplies
    // and, at the end of a pass, while the pass's inverse transform runs
    // (two operand buffers).  Measured against the plain loop below on one
    // box: 961 -> 874 us; slower for m = 5 and m = 3, which keep the loop.
    typename F::acc_t acc[EW];
    // the end of pass xi0: A^T along the last axis over this wave's half row
    // (partial sums of the m outputs o2; the other half row's wave adds the
    // rest) to LDS plane (xi1, half, o2) at [kernel][tile ^ (kernel / 4)], then
    // A^T along the middle axis and A^T[o0][xi0] into the outputs
    auto pass_end = [&](int xi0) {
  #pragma unroll
      for (int r = 0; r < F::NACC; ++r) {
        const int t = F::acc_row(lane, r);
  #pragma unroll
        for (int o2 = 0; o2 < MM; ++o2) {
          float v = 0.0f;
  #pragma unroll
          for (int e = 0; e < EW; ++e) v = __builtin_fmaf(AT(o2, half * EW + e), acc[e][r], v);
          sm[((xi1 * 2 + half) * MM + o2) * EPL + col * BLK + (t ^ (col >> 2))] = v;
        }
      }
      __syncthreads();
  #pragma unroll
      for (int q = 0; q < IPT; ++q) {
        const int i = int(threadIdx.x) + S::NT * q;
        if (i < S::ITEMS) {
          const int tl = i % BLK, kl = (i / BLK) % BLK, o2 = i / (BLK * BLK);
          float v[A], w1[MM];
  #pragma unroll
          for (int x1 = 0; x1 < A; ++x1) {
            const int base = kl * BLK + (tl ^ (kl >> 2));
            v[x1] = sm[((x1 * 2 + 0) * MM + o2) * EPL + base] + sm[((x1 * 2 + 1) * MM + o2) * EPL + base];
          }
          apply_vec<A, MM>(AT, v, 1, w1, 1);
  #pragma unroll
          for (int o0 = 0; o0 < MM; ++o0) {
            const float c0 = AT(o0, xi0);
  #pragma unroll
            for (int o1 = 0; o1 < MM; ++o1) out[q][o0 * MM + o1] = __builtin_fmaf(c0, w1[o1], out[q][o0 * MM + o1]);
          }
        }
      }
      __syncthreads();   // the planes are rewritten by the next pass
    };
    // operands of step gs = (pass xi0, channel stage s): 16 bytes of V row
    // `col` and of U column `col` per element
    float4 av[2][EW], uv[2][EW];
    auto load = [&](auto B, int gs) {
      constexpr int b = decltype(B)::value;
      const int x0 = gs / nstage, st = gs % nstage;
      const int xb = x0 * PL + xi1 * A + half * EW;   // first element of the wave
      load_ops(av[b], uv[b], xb, st);
    };
    auto mma = [&](auto B) {
      constexpr int b = decltype(B)::value;
  #pragma unroll
      for (int e = 0; e < EW; ++e) {
        acc[e] = F::mma(av[b][e].x, uv[b][e].x, acc[e]);
        acc[e] = F::mma(av[b][e].y, uv[b][e].y, acc[e]);
        acc[e] = F::mma(av[b][e].z, uv[b][e].z, acc[e]);
        acc[e] = F::mma(av[b][e].w, uv[b][e].w, acc[e]);
      }
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    const int total = A * nstage;
    auto step = [&](auto B, int gs) {
      constexpr int b = decltype(B)::value;
      if (gs % nstage == 0) {
#pragma unroll
        for (int e = 0; e < EW; ++e) acc[e] = typename F::acc_t{};
      }
      if (gs + 1 < total) load(std::integral_constant<int, b ^ 1>{}, gs + 1);
      mma(B);
      if (gs % nstage == nstage - 1) pass_end(gs / nstage);
    };
    load(I0{}, 0);
    for (int gs = 0; gs < total; gs += 2) {
      step(I0{}, gs);
      if (gs + 1 < total) step(I1{}, gs + 1);
    }
  } else {
    for (int xi0 = 0; xi0 < A; ++xi0) {
      typename F::acc_t acc[EW];
  #pragma unroll
      for (int e = 0; e < EW; ++e) acc[e] = typename F::acc_t{};
      const int xb = xi0 * PL + xi1 * A + half * EW;   // first element of the wave
      for (int s = 0; s < nstage; ++s) {
        float4 av[EW], uv[EW];
        load_ops(av, uv, xb, s);
  #pragma unroll
        for (int e = 0; e < EW; ++e) {
          acc[e] = F::mma(av[e].x, uv[e].x, acc[e]);
          acc[e] = F::mma(av[e].y, uv[e].y, acc[e]);
          acc[e] = F::mma(av[e].z, uv[e].z, acc[e]);
          acc[e] = F::mma(av[e].w, uv[e].w, acc[e]);
        }
      }
      // A^T along the last axis over this wave's half row: partial sums of the
      // m outputs o2 (the other half row's wave adds the rest), to LDS plane
      // (xi1, half, o2) at [kernel][tile ^ (kernel / 4)]
  #pragma unroll
      for (int r = 0; r < F::NACC; ++r) {
        const int t = F::acc_row(lane, r);
  #pragma unroll
        for (int o2 = 0; o2 < MM; ++o2) {
          float v = 0.0f;
  #pragma unroll
          for (int e = 0; e < EW; ++e) v = __builtin_fmaf(AT(o2, half * EW + e), acc[e][r], v);
          sm[((xi1 * 2 + half) * MM + o2) * EPL + col * BLK + (t ^ (col >> 2))] = v;
        }
      }
      __syncthreads();
      // A^T along the middle axis, then A^T[o0][xi0] into the outputs
  #pragma unroll
      for (int q = 0; q < IPT; ++q) {
        const int i = int(threadIdx.x) + S::NT * q;
        if (i < S::ITEMS) {
          const int tl = i % BLK, kl = (i / BLK) % BLK, o2 = i / (BLK * BLK);
          float v[A], w1[MM];
  #pragma unroll
          for (int x1 = 0; x1 < A; ++x1) {
            const int base = kl * BLK + (tl ^ (kl >> 2));
            v[x1] = sm[((x1 * 2 + 0) * MM + o2) * EPL + base] + sm[((x1 * 2 + 1) * MM + o2) * EPL + base];
          }
          apply_vec<A, MM>(AT, v, 1, w1, 1);
  #pragma unroll
          for (int o0 = 0; o0 < MM; ++o0) {
            const float c0 = AT(o0, xi0);
  #pragma unroll
            for (int o1 = 0; o1 < MM; ++o1) out[q][o0 * MM + o1] = __builtin_fmaf(c0, w1[o1], out[q][o0 * MM + o1]);
          }
        }
      }
      __syncthreads();   // the planes are rewritten by the next pass
    }

  }

  // bias and activation, then through LDS into rows [kernel][o0][o1][tile][o2]
  // (the planes are free: the last pass ended with a barrier), so that the
  // stores below write each output row's runs contiguously
#pragma unroll
  for (int q = 0; q < IPT; ++q) {
    const int i = int(threadIdx.x) + S::NT * q;
    if (i >= S::ITEMS) continue;
    const int tl = i % BLK, kl = (i / BLK) % BLK, o2 = i / (BLK * BLK);
    const float bk = g.bias != nullptr ? bsm[kl] : 0.0f;
#pragma unroll
    for (int o = 0; o < NOUT; ++o)
      sm[(kl * NOUT + o) * S::TROW + tl * MM + o2] = activate(out[q][o] + bk, g.act, g.slope);
  }
  __syncthreads();
  // crop and store: item (kernel, o0, o1, value of the 16-tile row), the
  // row's values fastest, so a wave writes runs of consecutive outputs
  constexpr int RV = BLK * MM;                      // values of a stage row
  for (int i = int(threadIdx.x); i < BLK * NOUT * RV; i += S::NT) {
    const int v = i % RV, row = i / RV;             // row = kl * NOUT + o0 * MM + o1
    const int kl = row / NOUT, o01 = row % NOUT;
    const int o0 = o01 / MM, o1 = o01 % MM;
    const int tl = v / MM, o2 = v % MM;
    const int n = tsm[tl][0], kg = kb * BLK + kl;
    if (n < 0 || kg >= g.K) continue;
    const int y0 = tsm[tl][1] + o0, y1 = tsm[tl][2] + o1, y2 = tsm[tl][3] + o2;
    if (y0 >= g.Y[0] || y1 >= g.Y[1] || y2 >= g.Y[2]) continue;
    y[(int64_t(n) * g.K + kg) * g.ystride_k + (int64_t(y0) * g.Y[1] + y1) * g.Y[2] + y2] =
        sm[row * S::TROW + v];
  }
}

}  // namespace wino
