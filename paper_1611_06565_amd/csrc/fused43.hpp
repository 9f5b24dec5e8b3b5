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
  int32_t vec_store;   // output rows a multiple of 4 long and y 16-byte aligned: rows of 4 stored as float4
  int32_t act;         // activation f of eq. (2): 0 none, 1 ReLU, 2 leaky ReLU
  float slope;
  const float* bias;   // [K] or null
  // Kernel-block loop only.  Work-group b runs on XCD b % 8 as its unit
  // b / 8; XCD x owns tile blocks xb0[x] .. xb0[x] + xn[x] - 1.  Its last
  // xs[x] blocks (those past its last full round of work-groups) are tail
  // blocks, each split into nkb units of one kernel block, so that the last
  // round is short.  Surplus units exit at once.
  int32_t xb0[8], xn[8], xs[8];
  // Max-pool of the activated outputs (POOL > 0): window = stride (1, 2, 2)
  // (POOL 1) or (2, 2, 2) (POOL 2), floor rounding: y is [n][K][Yp] with
  // Yp_i = Y_i / window_i, and ystride_p = prod Yp_i.
  int32_t Yp[3];
  int64_t ystride_p;
};

struct Fused43Geom {
  static constexpr int A = 6, MM = 4, NXI = 216, BLK = 16, NW = 12, NT = NW * 64;
  static constexpr int CH = 8;                       // channels per chunk
  static constexpr int PL = A * A;                   // values of a plane after two axes
  static constexpr int XPW = NXI / NW;               // elements per wave (18)
  static constexpr int NPOS = PL / NW;               // plane positions per wave (3, all six xi0 each)
  static constexpr int P_FLOATS = A * PL * CH * BLK; // 27648: the chunk's planes
  static constexpr int EPL = BLK * BLK + 8;          // epilogue plane stride (bank spread)
  static constexpr int E_FLOATS = PL * MM * EPL;     // 38016: (position, o0) planes
  static constexpr int LDS_FLOATS = E_FLOATS > P_FLOATS ? E_FLOATS : P_FLOATS;
  static_assert(XPW == NPOS * A && NW * 4 == CH * A, "a wave is 4 (channel, plane) rows of 16 tiles");
};

// P layout in LDS: P[i0][j][pair][tile][2] (j < 36 the plane value, pair =
// channel / 2): lane (kr, col) of an MFMA operand reads 8 bytes at
// ((i0 * 36 + j) * 4 + kr) * 32 + 2 * col, 512 contiguous bytes per wave.
__device__ __forceinline__ int p_index(int i0, int j, int ch, int tl) {
  return ((i0 * Fused43Geom::PL + j) * (Fused43Geom::CH / 2) + (ch >> 1)) * 32 + tl * 2 + (ch & 1);
}

// Work-group barrier that waits for this wave's LDS accesses only (lgkmcnt(0)),
// not for its global loads (__syncthreads() would wait for those too, vmcnt(0)).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);             // lgkmcnt(0); vmcnt and expcnt untouched
  asm volatile("s_barrier" ::: "memory");
}

template <bool CONST, bool KLOOP, int POOL = 0, bool NARROW = false>
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
  int tb, kb = 0;          // tile block, and kernel block outside the loop
  int kbs = 0, kbe = 0;    // the loop's kernel blocks kbs .. kbe - 1
  if constexpr (KLOOP) {
    const int xcd = int(blockIdx.x) & 7, j = int(blockIdx.x) >> 3;
    const int xs = a.xs[xcd], nwhole = a.xn[xcd] - xs;
    if (j >= nwhole + xs * a.nkb) return;        // surplus unit: the whole work-group leaves
    const int u = j - nwhole;
    tb = a.xb0[xcd] + (u < 0 ? j : nwhole + u / a.nkb);
    kbs = u < 0 ? 0 : u % a.nkb;
    kbe = u < 0 ? a.nkb : kbs + 1;
  } else {
    const int L = xcd_remap(int(blockIdx.x), a.nblocks);
    tb = L / a.nkb;
    kb = L % a.nkb;
  }
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

  // ---- consumer role: MFMA lane (kr, col).  Wave w owns the plane
  // positions j = 3w .. 3w + 2 (j = 6 xi1 + xi2) for all six first-axis
  // indices xi0: it reads each P_i0[j] once and forms the six elements
  // V_(xi0, j) = sum_i0 B^T[xi0][i0] P_i0[j] from them (eq. 4 along the
  // first axis, the shared sub-expressions of B^T's rows computed once).
  // acc[p * 6 + xi0] is the 16 x 16 product block of element (xi0, 3w + p).
  const int jw = __builtin_amdgcn_readfirstlane(wave) * G::NPOS;   // wave-uniform
  const int col = lane & 15, kr = lane >> 4;
  typename S::acc_t acc[XPW];
#pragma unroll
  for (int e = 0; e < XPW; ++e) acc[e] = typename S::acc_t{};
  // U[xi][c/4][k][c%4]: lane (kr, col) reads channels 2kr, 2kr + 1 of the
  // chunk; 32-bit offsets (the planner bounds U below 2^31 floats).  The
  // chunk's 18 operands are loaded together after its producing.
  const int uplane = int(a.uplane);
  // Loaded through a buffer resource: the wave-uniform base at element
  // (0, jw) of the chunk (and of the kernel block) in scalar registers, the
  // lane's byte offset as the vector offset and each element's offset as the
  // scalar one (the planner keeps them below 2^32 bytes), so the loads need
  // no per-lane 64-bit address arithmetic.
  const float* ubase = U + jw * uplane + (KLOOP ? 0 : kb * BLK * 4);
  const int ulane = (((kr >> 1) * a.K_pad + col) * 4 + 2 * (kr & 1)) * 4;
  float2 ur[XPW];
  auto load_u = [&](int chunk, int kbx) {
    const __amdgpu_buffer_rsrc_t ru = raw_rsrc(ubase + chunk * 8 * a.K_pad + (KLOOP ? kbx * (BLK * 4) : 0));
#pragma unroll
    for (int p = 0; p < G::NPOS; ++p)
#pragma unroll
      for (int x0 = 0; x0 < A; ++x0)
        ur[p * A + x0] =
            __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(ru, ulane, (x0 * PL + p) * uplane * 4, 0));
  };
  const float2* P2 = reinterpret_cast<const float2*>(sm);
  auto fetch = [&](float2* pv, int p) {
#pragma unroll
    for (int i = 0; i < A; ++i) pv[i] = P2[((i * PL + jw + p) * 4 + kr) * 16 + col];
  };
  auto product = [&](const float2* pv, int p) {
    float vx[A], vy[A], ox[A], oy[A];
#pragma unroll
    for (int i = 0; i < A; ++i) {
      vx[i] = pv[i].x;
      vy[i] = pv[i].y;
    }
    apply_vec<A, A>(BT, vx, 1, ox, 1);
    apply_vec<A, A>(BT, vy, 1, oy, 1);
#pragma unroll
    for (int x0 = 0; x0 < A; ++x0) acc[p * A + x0] = S::mma(ox[x0], ur[p * A + x0].x, acc[p * A + x0]);
#pragma unroll
    for (int x0 = 0; x0 < A; ++x0) acc[p * A + x0] = S::mma(oy[x0], ur[p * A + x0].y, acc[p * A + x0]);
  };
  auto consume = [&]() {
    float2 pa[A], pb[A];
    fetch(pa, 0);
    fetch(pb, 1);
    product(pa, 0);
    fetch(pa, 2);
    product(pb, 1);
    product(pa, 2);
  };
  static_assert(G::NPOS == 3, "three plane positions per wave");

  // chunks past the last real channel hold only zero padding (x and U are
  // zero there): they are skipped
  const int nchunks = (a.C + CH - 1) / CH;
  if constexpr (!KLOOP) {
    for (int chunk = 0; chunk < nchunks; ++chunk) {
      if (chunk > 0) __syncthreads();           // the previous chunk's planes are read
      produce(chunk);
      load_u(chunk, kb);
      __syncthreads();
      consume();
    }
  }

  // One chunk (C <= 8, the kernel-block loop): the planes are formed once,
  // each wave turns them into its 18 elements of V in registers, and the
  // work-group multiplies them with every kernel block's U in turn; the LDS
  // is then free for each block's epilogue.  Each block's U operands are
  // loaded ahead: the first block's before the barrier after the producing
  // (the barrier waits for LDS traffic only, so they arrive during the
  // elements' formation), the next block's during the epilogue's second part.
  //
  // With at most 4 channels (narrow) one MFMA k-step per element suffices:
  // lane group kr takes channel kr (element value and U operand in .x), and
  // the planes of channels 4..7 (the odd waves' producing) are not formed.
  [[maybe_unused]] float2 vv[XPW];
  static_assert(!NARROW || KLOOP, "the narrow form is a kernel-block loop");
  constexpr bool narrow = NARROW;
  auto load_u_narrow = [&](int kbx) {
    const __amdgpu_buffer_rsrc_t ru = raw_rsrc(U + jw * uplane + kbx * BLK * 4);
#pragma unroll
    for (int p = 0; p < G::NPOS; ++p)
#pragma unroll
      for (int x0 = 0; x0 < A; ++x0)
        ur[p * A + x0].x = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(ru, (col * 4 + kr) * 4, (x0 * PL + p) * uplane * 4, 0));
  };
  auto load_u_block = [&](int kbx) {
    if constexpr (narrow) load_u_narrow(kbx);
    else load_u(0, kbx);
  };
  if constexpr (KLOOP) {
  if (!narrow || pch < 4) produce(0);           // pch < 4: the even waves
  load_u_block(kbs);
  lds_barrier();
#pragma unroll
  for (int p = 0; p < G::NPOS; ++p) {
    float vx[A], vy[A], ox[A], oy[A];
    if constexpr (narrow) {
#pragma unroll
      for (int i = 0; i < A; ++i) vx[i] = sm[p_index(i, jw + p, kr, col)];
      apply_vec<A, A>(BT, vx, 1, ox, 1);
#pragma unroll
      for (int x0 = 0; x0 < A; ++x0) vv[p * A + x0].x = ox[x0];
    } else {
      float2 pv[A];
      fetch(pv, p);
#pragma unroll
      for (int i = 0; i < A; ++i) {
        vx[i] = pv[i].x;
        vy[i] = pv[i].y;
      }
      apply_vec<A, A>(BT, vx, 1, ox, 1);
      apply_vec<A, A>(BT, vy, 1, oy, 1);
#pragma unroll
      for (int x0 = 0; x0 < A; ++x0) vv[p * A + x0] = make_float2(ox[x0], oy[x0]);
    }
  }
  }
  // ---- epilogue of kernel block kbx (eq. 4 inverted): A^T along the first
  // axis in registers, then along the last two axes, bias, activation, crop
  // and store.  Part 1: wave w writes, for each of its positions j and
  // output o0, the 16 x 16 (tile, kernel) block to LDS plane (j, o0) at
  // [k][t ^ k].
  const MatRef<Which::AT, CONST, MM, R> AT{&fm};
  __shared__ float bsm[BLK];
  // the kernel blocks of this work-group: its own, or those of the loop
  const int kb0 = KLOOP ? kbs : kb, kb1 = KLOOP ? kbe : kb + 1;
  for (int kbx = kb0; kbx < kb1; ++kbx) {
  if constexpr (KLOOP) {
    if (kbx > kb0) __syncthreads();             // the previous block's stores have read the LDS
    if constexpr (narrow) {
#pragma unroll
      for (int e = 0; e < XPW; ++e) acc[e] = S::mma(vv[e].x, ur[e].x, typename S::acc_t{});
    } else {
#pragma unroll
      for (int e = 0; e < XPW; ++e) {
        acc[e] = typename S::acc_t{};
        acc[e] = S::mma(vv[e].x, ur[e].x, acc[e]);
        acc[e] = S::mma(vv[e].y, ur[e].y, acc[e]);
      }
    }
  }
  if (a.bias != nullptr && int(threadIdx.x) < BLK) {
    const int kg = kbx * BLK + int(threadIdx.x);
    bsm[threadIdx.x] = kg < a.K ? a.bias[kg] : 0.0f;
  }
  __syncthreads();                              // the planes' LDS is reused below
#pragma unroll
  for (int r = 0; r < S::NACC; ++r) {
    const int tr = S::acc_row(lane, r);
#pragma unroll
    for (int p = 0; p < G::NPOS; ++p) {
      float sv[A], o[MM];
#pragma unroll
      for (int x0 = 0; x0 < A; ++x0) sv[x0] = acc[p * A + x0][r];
      apply_vec<A, MM>(AT, sv, 1, o, 1);
      float* dst = sm + (jw + p) * MM * G::EPL + col * BLK + (tr ^ col);
#pragma unroll
      for (int o0 = 0; o0 < MM; ++o0) dst[o0 * G::EPL] = o[o0];
    }
  }
  __syncthreads();
  if constexpr (KLOOP) {
    if (kbx + 1 < kb1) load_u_block(kbx + 1);   // the accumulators are in LDS: U for the next block
  }

  if constexpr (POOL == 0) {
    // Part 2: item (o0, kernel, tile), tiles fastest, reads the 36 values of
    // its plane, applies A^T along the last two axes and stores 4 x 4 outputs,
    // each row of 4 as one 16-byte store when every row of the output is a
    // whole number of aligned tiles (a.vec_store)
    constexpr int ITEMS = MM * BLK * BLK;
    for (int i = int(threadIdx.x); i < ITEMS; i += G::NT) {
      const int tl2 = i % BLK, kl = (i / BLK) % BLK, o0 = i / (BLK * BLK);
      const int t2 = tb * BLK + tl2;
      const int kg = kbx * BLK + kl;
      if (t2 >= a.T || kg >= a.K) continue;
      int ti[3] = {0, 0, 0};
      const int n = split_tile<N>(t2, a.tiles, ti);
      const int y0 = ti[0] * MM + o0;
      if (y0 >= a.Y[0]) continue;
      float v[PL], out[MM * MM];
  #pragma unroll
      for (int j = 0; j < PL; ++j) v[j] = sm[(j * MM + o0) * G::EPL + kl * BLK + (tl2 ^ kl)];
      transform_nd<2, A, MM>(v, out, AT);
      const float bk = a.bias != nullptr ? bsm[kl] : 0.0f;
  #pragma unroll
      for (int q2 = 0; q2 < MM * MM; ++q2) out[q2] = activate(out[q2] + bk, a.act, a.slope);
      float* yk = y + (int64_t(n) * a.K + kg) * a.ystride_k + int64_t(y0) * a.Y[1] * a.Y[2];
      const int y2 = ti[2] * MM;
  #pragma unroll
      for (int o1 = 0; o1 < MM; ++o1) {
        const int y1 = ti[1] * MM + o1;
        if (y1 >= a.Y[1]) continue;
        float* row = yk + int64_t(y1) * a.Y[2] + y2;
        if (a.vec_store) {
          const f32x4 v4 = {out[o1 * MM], out[o1 * MM + 1], out[o1 * MM + 2], out[o1 * MM + 3]};
          __builtin_nontemporal_store(v4, reinterpret_cast<f32x4*>(row));
        } else {
  #pragma unroll
          for (int o2 = 0; o2 < MM; ++o2)
            if (y2 + o2 < a.Y[2]) row[o2] = out[o1 * MM + o2];
        }
      }
    }
  } else {
    // Part 2 with the max-pool: item (o0 group, kernel, tile) reads the 36
    // values of each plane of its group (one o0 for window (1, 2, 2), the
    // pair 2h, 2h + 1 for (2, 2, 2)), applies A^T along the last two axes,
    // bias and activation, and stores the maximum over each window of the
    // tile (a tile of 4 holds whole windows of 2 along every axis).  The
    // window is scanned first axis slowest with a strict comparison from
    // -inf, as the stand-alone max-pool does, so both give the same bits.
    constexpr int P0 = POOL == 2 ? 2 : 1;       // window along the first axis
    constexpr int NG0 = MM / P0;                // o0 groups per tile
    constexpr int ITEMS = NG0 * BLK * BLK;
    for (int i = int(threadIdx.x); i < ITEMS; i += G::NT) {
      const int tl2 = i % BLK, kl = (i / BLK) % BLK, h0 = i / (BLK * BLK);
      const int t2 = tb * BLK + tl2;
      const int kg = kbx * BLK + kl;
      if (t2 >= a.T || kg >= a.K) continue;
      int ti[3] = {0, 0, 0};
      const int n = split_tile<N>(t2, a.tiles, ti);
      const int p0 = ti[0] * NG0 + h0;          // pooled index along the first axis
      if (p0 >= a.Yp[0]) continue;
      const float bk = a.bias != nullptr ? bsm[kl] : 0.0f;
      float out[P0][MM * MM];
#pragma unroll
      for (int g0 = 0; g0 < P0; ++g0) {
        const int o0 = h0 * P0 + g0;
        float v[PL];
#pragma unroll
        for (int j = 0; j < PL; ++j) v[j] = sm[(j * MM + o0) * G::EPL + kl * BLK + (tl2 ^ kl)];
        transform_nd<2, A, MM>(v, out[g0], AT);
#pragma unroll
        for (int q2 = 0; q2 < MM * MM; ++q2) out[g0][q2] = activate(out[g0][q2] + bk, a.act, a.slope);
      }
      float* yk = y + (int64_t(n) * a.K + kg) * a.ystride_p + int64_t(p0) * a.Yp[1] * a.Yp[2];
#pragma unroll
      for (int w1 = 0; w1 < MM / 2; ++w1) {
        const int p1 = ti[1] * (MM / 2) + w1;
        if (p1 >= a.Yp[1]) continue;
#pragma unroll
        for (int w2 = 0; w2 < MM / 2; ++w2) {
          const int p2 = ti[2] * (MM / 2) + w2;
          if (p2 >= a.Yp[2]) continue;
          float best = -__builtin_inff();
#pragma unroll
          for (int g0 = 0; g0 < P0; ++g0)
#pragma unroll
            for (int i1 = 0; i1 < 2; ++i1)
#pragma unroll
              for (int i2 = 0; i2 < 2; ++i2) {
                const float vv = out[g0][(2 * w1 + i1) * MM + 2 * w2 + i2];
                best = vv > best ? vv : best;
              }
          yk[int64_t(p1) * a.Yp[2] + p2] = best;
        }
      }
    }
  }
  }
}

}  // namespace wino
