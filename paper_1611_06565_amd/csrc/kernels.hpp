// gfx950 kernels of the N-D Winograd forward.
//
//   k_filter       U[xi][c][k]  = (w[k][c] x_n G)[xi]            eq. (4), kernel side
//   k_input        V[xi][c][t]  = (d_{t,c} x_n B^T)[xi]          eq. (4), data side
//   k_input_split  the same for alpha^N = 216, split over A threads per (t, c)
//   k_gemm_inv     M_xi = V_xi . U_xi on fp32 MFMA (eq. 5), then
//                  y tile = M[:, t, k] x_n A^T, stitched and cropped (eq. 4);
//                  F(4^3) and the 2-D sizes F(3,2), F(5,4), F(4,5), F(3,6)
//                  (m = 2 uses k_gemm_acc in gemm_acc.hpp, F(4^2)
//                  k_gemm_acc4 in gemm_acc4.hpp)
//   k_maxpool3d    pooling for the C3D stack (not part of the method)
//
// Layouts (float32, zero padding rows/columns):
//   x [batch][C][X_1..X_N]     w [K][C][r^N]      y [batch][K][Y_1..Y_N]
//   U [alpha^N][C_pad/CGU][K_pad][CGU]
//   V [T_pad/BLK][C_pad/CG][alpha^N][BLK][CG]
// T counts tiles over the whole batch (tiles of every sample form the rows of
// one GEMM, §4.1 and §4.4: the method is batch-size agnostic).  BLK is the
// GEMM block of tiles and CG the channel group (see Blocking): interleaving
// channel groups innermost lets every lane fetch VEC k-steps of an MFMA
// operand with one load; storing V tile-block major keeps all of one
// GEMM work-group's operand rows in one contiguous region, and putting the
// elements inside the channel group makes the input transform of one (tile
// block, channel group) write one contiguous run.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "layout.hpp"
#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- arguments
struct FilterArgs {
  int64_t uplane;  // C_pad * K_pad
  int32_t C, K, C_pad, K_pad;
  int32_t adjoint;  // w is [C][K][r^N]; use w[c][k] with every axis reversed
};

struct InputArgs {
  int64_t xstride_c;  // prod X_i
  int32_t C, C_pad;
  int32_t T, T_pad;
  int32_t ntb, nblocks;  // tile blocks; work-groups in the grid
  int32_t X[3], tiles[3], pad[3];
  int32_t rowfast;       // k_input_split: every tile block is 16 tiles of one row (see there)
};

struct GemmArgs {
  int64_t uplane;     // C_pad * K_pad
  int64_t ystride_k;  // prod Y_i
  int32_t T, T_pad, C_pad, K, K_pad;
  int32_t nkb;        // K_pad / BLK
  int32_t nblocks;    // work-groups in the grid
  int32_t tiles[3], Y[3];
  int32_t act;        // activation f of eq. (2): 0 none, 1 ReLU, 2 leaky ReLU
  float slope;        // leaky ReLU: f(v) = slope * v for v <= 0
  const float* bias;  // [K] or null: b_k of eq. (2), added before the activation
  // max-pool in the epilogue (k_gemm_inv with POOL > 0): pooled extents
  // Y_i / window_i and their product
  int32_t Yp[3];
  int64_t ystride_p;
};

// Tile t (linear over batch and the tile grid, last axis fastest) -> sample
// and per-axis tile coordinates.
template <int N>
__device__ __forceinline__ int split_tile(int t, const int32_t* tiles, int* ti) {
#pragma unroll
  for (int a = N - 1; a >= 0; --a) {
    ti[a] = t % tiles[a];
    t /= tiles[a];
  }
  return t;
}

// Work-groups are dispatched round-robin over the 8 XCDs.  Renumber them so
// that consecutive logical blocks (in the GEMM the K-blocks of one tile block,
// which read the same V rows) land on the same XCD and share its L2.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  constexpr int NX = 8;
  const int xcd = b % NX, j = b / NX;
  const int per = nb / NX, rem = nb % NX;
  return xcd < rem ? xcd * (per + 1) + j : rem * (per + 1) + (xcd - rem) * per + j;
}

// The activation f of eq. (2) applied in the output epilogues after the bias:
// kind 0 identity, 1 ReLU max(0, v), 2 leaky ReLU (v for v > 0, slope * v
// otherwise).  kind is uniform over a launch.
__device__ __forceinline__ float activate(float v, int32_t kind, float slope) {
  if (kind == 1) return v > 0.0f ? v : 0.0f;
  if (kind == 2) return v > 0.0f ? v : v * slope;
  return v;
}

// ------------------------------------------------------------ filter (a2)
// One thread per (channel, kernel); lanes run over the channel group fastest
// so each plane store is contiguous.
template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(64) k_filter(const float* __restrict__ w, float* __restrict__ U,
                                                FilterArgs a, FMats fm) {
  using B = Blocking<N, MM, R>;
  constexpr int A = B::A, NXI = B::NXI, CG = B::CGU;
  constexpr int RN = ipow(R, N);
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
      // reversing every axis of a C-order r^N array reverses its flat index
      const float* src = w + (int64_t(c) * a.K + k) * RN;
#pragma unroll
      for (int i = 0; i < RN; ++i) g[i] = src[RN - 1 - i];
    } else {
      const float* src = w + (int64_t(k) * a.C + c) * RN;
#pragma unroll
      for (int i = 0; i < RN; ++i) g[i] = src[i];
    }
    transform_nd<N, R, A>(g, u, MatRef<Which::G, CONST, MM, R>{&fm});
  } else {
#pragma unroll
    for (int i = 0; i < NXI; ++i) u[i] = 0.0f;
  }
  float* dst = U + (int64_t(cg) * a.K_pad + k) * CG + cl;
#pragma unroll
  for (int xi = 0; xi < NXI; ++xi) dst[int64_t(xi) * a.uplane] = u[xi];
}

// ------------------------------------------------------------- input (a3)
// One thread per (tile, channel): gather the alpha^N window (zero outside the
// input), transform along every axis (eq. 4, B^T on the data side), and write
// the alpha^N values to V.
//
// A work-group covers one GEMM tile block (BLK tiles) and 256 / (BLK * CG)
// channel groups.  Each window row (A values along the last axis) is a single
// wide load from a start clamped into the input row, shifted and zero-masked
// in registers; a row whose leading coordinates fall outside the input loads
// a clamped row and is masked to zero.  A wave whose windows all lie inside
// the input loads the rows as they are and skips the shifts and masks (a
// wave-uniform branch).
//
// m = 2: lanes run over the tiles fastest (a wave is 64 consecutive tiles of
// one channel).  With pad 1 on the last axis and an even row length (rowfast)
// a lane's window row x[2t - 1 .. 2t + 2] is its own aligned pair
// x[2t .. 2t + 1], the last value of the previous lane's pair and the first of
// the next lane's (DPP wave shifts); lanes 0 and 63 load the missing end.  A
// neighbour whose tile lies in another row of tiles only supplies positions
// outside the input, which are masked.  Other m: lanes run over the channels
// of a group fastest, then tiles.
//
// Outputs go through LDS so that each lane stores 16 bytes (4 channels of a
// tile) and a wave writes 1 KB contiguous per store.
__device__ __forceinline__ float dpp_wave_prev(float old, float v) {
  // lane i takes lane i-1's v (wave_shr:1); lane 0 keeps old
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), 0x138, 0xf, 0xf, false));
}
__device__ __forceinline__ float dpp_wave_next(float old, float v) {
  // lane i takes lane i+1's v (wave_shl:1); lane 63 keeps old
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), 0x130, 0xf, 0xf, false));
}

template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(256) k_input(const float* __restrict__ x, float* __restrict__ V,
                                               InputArgs a, FMats fm) {
  using B = Blocking<N, MM, R>;
  constexpr int A = B::A, NXI = B::NXI, BLK = B::BLK, CG = B::CG;
  constexpr int GPW = 256 / (BLK * CG);   // channel groups per work-group
  constexpr int NROW = NXI / A;           // window rows (leading indices)
  constexpr int XCH = NXI % 16 == 0 ? 16 : 12;   // planes staged through LDS at a time
  constexpr bool TILEFAST = MM == 2;      // lanes over tiles fastest
  static_assert(GPW * BLK * CG == 256, "work-group shape");
  static_assert(CG % 4 == 0 && NXI % XCH == 0 && XCH % 4 == 0, "store rounds of 4 planes");
  static_assert(!TILEFAST || (BLK == 64 && A == 4), "m = 2: a wave is 64 tiles of one channel");
  const int tid = int(threadIdx.x);
  const int cl = TILEFAST ? (tid / BLK) % CG : tid % CG;
  const int tl = TILEFAST ? tid % BLK : (tid / CG) % BLK;
  const int gl = tid / (CG * BLK);
  // consecutive tile blocks of one channel group run on the same XCD, so the
  // input windows they share (neighbouring tiles overlap by r - 1) hit its L2
  const int L = xcd_remap(int(blockIdx.x), a.nblocks);
  const int tb = L % a.ntb;
  const int cg = (L / a.ntb) * GPW + gl;
  const int c = cg * CG + cl;
  const int t = tb * BLK + tl;
  const bool live = t < a.T && c < a.C;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<N>(live ? t : 0, a.tiles, ti);
  int o[3];
#pragma unroll
  for (int ax = 0; ax < N; ++ax) o[ax] = ti[ax] * MM - a.pad[ax];
  const int XL = a.X[N - 1];
  // last axis: the window [oL, oL + A) is read as [sL, sL + A) inside the row
  const int oL = o[N - 1];
  const bool wide = XL >= A;              // uniform over the launch
  const int sL = wide ? min(max(oL, 0), XL - A) : 0;
  const int delta = oL - sL;              // window element i is loaded element i + delta
  // a wave whose windows all lie inside the input skips the shift and masks
  bool inner = wide && delta == 0;
#pragma unroll
  for (int ax = 0; ax < N - 1; ++ax) inner = inner && o[ax] >= 0 && o[ax] + A <= a.X[ax];
  const bool plain = __all(!live || inner);
  const float* xc = x + (int64_t(n) * a.C + min(c, a.C - 1)) * a.xstride_c;
  float d[NXI];
  // leading coordinates of window row `row`: offset of the clamped input row
  // and whether it lies inside the input
  auto row_at = [&](int row, int64_t& off) {
    int lead[2] = {0, 0};
    int rem = row;
#pragma unroll
    for (int ax = N - 2; ax >= 0; --ax) {
      lead[ax] = rem % A;
      rem /= A;
    }
    off = 0;
    bool valid = live;
#pragma unroll
    for (int ax = 0; ax < N - 1; ++ax) {
      const int q = o[ax] + lead[ax];
      valid = valid && (unsigned)q < (unsigned)a.X[ax];
      off = off * a.X[ax] + min(max(q, 0), a.X[ax] - 1);
    }
    return valid;
  };
  auto gather = [&](auto PLAIN) {
    constexpr bool P = decltype(PLAIN)::value;
#pragma unroll
    for (int row = 0; row < NROW; ++row) {
      int64_t off;
      const bool valid = row_at(row, off);
      const float* xr = xc + off * XL;
      float* dr = d + row * A;
      if constexpr (P) {
        __builtin_memcpy(dr, xr + oL, A * sizeof(float));
      } else if (wide) {
        float ld[A];
        __builtin_memcpy(ld, xr + sL, sizeof(ld));
#pragma unroll
        for (int i = 0; i < A; ++i) {
          float v = 0.0f;
#pragma unroll
          for (int j = 0; j < A; ++j) v = (j == i + delta) ? ld[j] : v;
          dr[i] = valid ? v : 0.0f;
        }
      } else {
#pragma unroll
        for (int i = 0; i < A; ++i) {
          const int q = oL + i;
          const bool in = valid && (unsigned)q < (unsigned)XL;
          const float v = xr[min(max(q, 0), XL - 1)];
          dr[i] = in ? v : 0.0f;
        }
      }
    }
  };
  if constexpr (TILEFAST) {
    if (a.rowfast) {
      // window row (pad 1) = x[2tW - 1], x[2tW], x[2tW + 1], x[2tW + 2]
      const int lane = tid & 63;
      const int tW = ti[N - 1];
      const bool own_in = 2 * tW < XL;            // the pair lies inside the row (XL even)
      const bool prev_in = tW > 0;
      const bool next_in = 2 * tW + 2 < XL;
      const int wo = min(2 * tW, XL - 2);
#pragma unroll
      for (int row = 0; row < NROW; ++row) {
        int64_t off;
        const bool valid = row_at(row, off);
        const float* xr = xc + off * XL;
        float2 pr = *reinterpret_cast<const float2*>(xr + wo);
        if (!(valid && own_in)) pr = make_float2(0.0f, 0.0f);
        // the wave's two ends: lane 0's left value, lane 63's right value
        float h = 0.0f;
        if (lane == 0 && valid && prev_in) h = xr[2 * tW - 1];
        if (lane == 63 && valid && next_in) h = xr[2 * tW + 2];
        const float lv = dpp_wave_prev(h, pr.y);
        const float rv = dpp_wave_next(h, pr.x);
        float* dr = d + row * A;
        dr[0] = (valid && prev_in) ? lv : 0.0f;
        dr[1] = pr.x;
        dr[2] = pr.y;
        dr[3] = (valid && next_in) ? rv : 0.0f;
      }
    } else {
      gather(std::false_type{});
    }
  } else {
    if (live) {
      if (plain) gather(std::true_type{});
      else gather(std::false_type{});
    } else {
#pragma unroll
      for (int i = 0; i < NXI; ++i) d[i] = 0.0f;
    }
  }
  float v[NXI];
  transform_nd<N, A, A>(d, v, MatRef<Which::BT, CONST, MM, R>{&fm});
  // V[tb][cg][xi][tl][cl]: the work-group's NXI planes of each of its channel
  // groups are one contiguous run.  The values go through LDS XCH planes at a
  // time; a plane holds the work-group's 256 values as [group][tile][channel]
  // (TILEFAST: [group][channel][tile], so that the lanes of a wave write
  // consecutive words).
  __shared__ float stage[XCH][256];
  float* const gbase = V + (int64_t(tb) * a.C_pad + int64_t(cg - gl) * CG) * NXI * BLK;
  constexpr int C4 = CG / 4;              // float4s per tile row of a group
  const int pr4 = tid >> 6, f = tid & 63; // plane within a round of 4; float4 = (group, tile, quarter)
  const int g = f / (BLK * C4), ft = (f / C4) % BLK, f4 = f % C4;
  const bool store = (cg - gl + g) * CG < a.C_pad;
  const int widx = TILEFAST ? (gl * CG + cl) * BLK + tl : (gl * BLK + tl) * CG + cl;
#pragma unroll
  for (int x0 = 0; x0 < NXI; x0 += XCH) {
    if (x0 > 0) __syncthreads();          // previous planes stored
#pragma unroll
    for (int i = 0; i < XCH; ++i) stage[i][widx] = v[x0 + i];
    __syncthreads();
    if (store) {
#pragma unroll
      for (int i = 0; i < XCH; i += 4) {
        // non-temporal: V streams to HBM without evicting the input windows
        // that neighbouring work-groups still read from L2
        float4 val;
        if constexpr (TILEFAST) {
          const float* sp = stage[i + pr4] + (g * CG + f4 * 4) * BLK + ft;
          val = make_float4(sp[0], sp[BLK], sp[2 * BLK], sp[3 * BLK]);
        } else {
          val = reinterpret_cast<const float4*>(stage[i + pr4])[((g * BLK + ft) * CG) / 4 + f4];
        }
        float* p = gbase + (int64_t(g) * NXI + x0 + i + pr4) * (BLK * CG) + ft * CG + f4 * 4;
        __builtin_nontemporal_store(val.x, p + 0);
        __builtin_nontemporal_store(val.y, p + 1);
        __builtin_nontemporal_store(val.z, p + 2);
        __builtin_nontemporal_store(val.w, p + 3);
      }
    }
  }
}

// Input transform for large windows (alpha^N = 216, F(4^3, 3^3)): one
// (tile, channel)'s window is too big for one thread's registers at a useful
// occupancy, so it is split over A threads along axis 0.  Thread (i0, q)
// loads plane i0 of the window of pair q (A rows of A values) and transforms
// it along the other two axes; the planes meet in LDS; then the wave of
// output plane x0 forms sum_i0 B^T[x0][i0] * plane_i0 (axis 0 of eq. 4) and
// writes its A^2 values.
//
// A work-group covers one V block: 16 tiles x one group of 4 channels.  On
// the loading side lanes run over the tiles fastest (lane = 16 * channel +
// tile), so when the 16 tiles are consecutive along the last axis of one
// input row (rowfast: the plan checks it once) every lane fetches the four
// inputs at 4 * its tile coordinate with one aligned 16-byte load, the two
// values on each side of its window come from the neighbouring lanes of its
// 16-lane row (DPP row shifts), and the two row ends of the block from one
// extra 8-byte load.  Otherwise each lane gathers its own window rows as in
// k_input.  On the storing side lane (j, tile) writes the 4 channels of one
// tile as 16 bytes, so a wave writes 4 runs of 256 contiguous bytes of V.
__device__ __forceinline__ float dpp_from_prev(float old, float v) {
  // lane i of each 16-lane row takes lane i-1's v; lane 0 keeps old
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), 0x111, 0xf, 0xf, false));
}
__device__ __forceinline__ float dpp_from_next(float old, float v) {
  // lane i of each 16-lane row takes lane i+1's v; lane 15 keeps old
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), 0x101, 0xf, 0xf, false));
}

template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(384) k_input_split(const float* __restrict__ x, float* __restrict__ V, InputArgs a, FMats fm) {
  using B = Blocking<N, MM, R>;
  constexpr int A = B::A, NXI = B::NXI, BLK = B::BLK, CG = B::CG;
  constexpr int NQ = BLK * CG;            // (tile, channel) pairs per work-group: one V block
  constexpr int PL = NXI / A;             // values per plane
  static_assert(N == 3 && MM == 4 && A == 6 && BLK == 16 && CG == 4 && NQ == 64, "one wave per plane, six planes");
  constexpr int HALF = PL / 2;            // the planes meet in LDS in two halves (occupancy)
  static_assert(PL % 2 == 0, "even plane size");
  __shared__ float4 planes[A][HALF][BLK];   // [plane][value][tile] -> the CG channels

  const int lane = int(threadIdx.x) & 63;
  const int i0 = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);   // plane of this wave
  const int L = xcd_remap(int(blockIdx.x), a.nblocks);
  const int tb = L % a.ntb, cg = L / a.ntb;
  const int tl = lane % BLK, cl = lane / BLK;
  const int c = cg * CG + cl;
  const int t = tb * BLK + tl;
  const int XL = a.X[N - 1];
  const int cc = min(c, a.C - 1);
  const float* xc = x + int64_t(cc) * a.xstride_c;          // channel c of sample 0
  float d[PL];

  if (a.rowfast) {
    // the 16 tiles share sample and leading tile coordinates; lane tl's
    // window row starts at 4 * (tW0 + tl) - pad
    int ti[3] = {0, 0, 0};
    const int n = split_tile<N>(tb * BLK, a.tiles, ti);
    const float* xn = xc + int64_t(n) * a.C * a.xstride_c;
    const int tW = ti[2] + tl;
    const int q0 = ti[0] * MM - a.pad[0] + i0;
    const bool valid0 = c < a.C && (unsigned)q0 < (unsigned)a.X[0];
    const int wo = min(MM * tW, XL - 4);
    const bool own_in = MM * tW < XL;
    // row ends: lanes 0..7 fetch the two values left of the block, 8..15 the
    // two right of it
    const int wl = MM * ti[2] - 2, wr = MM * ti[2] + MM * BLK;
    const bool left = tl < BLK / 2;
    const int wh = left ? max(wl, 0) : min(wr, XL - 2);
    const bool h_in = left ? wl >= 0 : wr < XL;
    // the rows of one pad (window value i sits at offset i - P from 4 * tW)
    auto rows = [&](auto PP) {
      constexpr int P = decltype(PP)::value;
#pragma unroll
      for (int i1 = 0; i1 < A; ++i1) {
        const int q1 = ti[1] * MM - a.pad[1] + i1;
        const bool valid = valid0 && (unsigned)q1 < (unsigned)a.X[1];
        const float* xr = xn + (int64_t(min(max(q0, 0), a.X[0] - 1)) * a.X[1] + min(max(q1, 0), a.X[1] - 1)) * XL;
        float4 o = *reinterpret_cast<const float4*>(xr + wo);
        float2 h = *reinterpret_cast<const float2*>(xr + wh);
        // the lanes of a DPP row share the channel, hence the row's validity
        if (!(own_in && valid)) o = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (!(h_in && valid)) h = make_float2(0.0f, 0.0f);
        // e = offset from 4 * tW: -2, -1 from the previous lane, 0..3 own, 4, 5 from the next
        float e[8];
        e[0] = dpp_from_prev(h.x, o.z);
        e[1] = dpp_from_prev(h.y, o.w);
        e[2] = o.x; e[3] = o.y; e[4] = o.z; e[5] = o.w;
        e[6] = dpp_from_next(h.x, o.x);
        e[7] = dpp_from_next(h.y, o.y);
#pragma unroll
        for (int i = 0; i < A; ++i) d[i1 * A + i] = e[i + 2 - P];
      }
    };
    switch (a.pad[2]) {
      case 0: rows(std::integral_constant<int, 0>{}); break;
      case 1: rows(std::integral_constant<int, 1>{}); break;
      default: rows(std::integral_constant<int, 2>{}); break;
    }
  } else {
    const bool live = t < a.T && c < a.C;
    int ti[3] = {0, 0, 0};
    const int n = split_tile<N>(live ? t : 0, a.tiles, ti);
    const float* xn = xc + int64_t(n) * a.C * a.xstride_c;
    int o[3];
#pragma unroll
    for (int ax = 0; ax < N; ++ax) o[ax] = ti[ax] * MM - a.pad[ax];
    const int oL = o[N - 1];
    const bool wide = XL >= A;
    const int sL = wide ? min(max(oL, 0), XL - A) : 0;
    const int delta = oL - sL;
    const int q0 = o[0] + i0;
    const bool valid0 = live && (unsigned)q0 < (unsigned)a.X[0];
    const int64_t off0 = min(max(q0, 0), a.X[0] - 1);
#pragma unroll
    for (int i1 = 0; i1 < A; ++i1) {
      const int q1 = o[1] + i1;
      const bool valid = valid0 && (unsigned)q1 < (unsigned)a.X[1];
      const float* xr = xn + (off0 * a.X[1] + min(max(q1, 0), a.X[1] - 1)) * XL;
      float* dr = d + i1 * A;
      if (wide) {
        float ld[A];
        __builtin_memcpy(ld, xr + sL, sizeof(ld));
#pragma unroll
        for (int i = 0; i < A; ++i) {
          float v = 0.0f;
#pragma unroll
          for (int j = 0; j < A; ++j) v = (j == i + delta) ? ld[j] : v;
          dr[i] = valid ? v : 0.0f;
        }
      } else {
#pragma unroll
        for (int i = 0; i < A; ++i) {
          const int qq = oL + i;
          const bool in = valid && (unsigned)qq < (unsigned)XL;
          const float v = xr[min(max(qq, 0), XL - 1)];
          dr[i] = in ? v : 0.0f;
        }
      }
    }
  }
  const MatRef<Which::BT, CONST, MM, R> BT{&fm};
  float p2[PL];
  transform_nd<2, A, A>(d, p2, BT);       // axes 1 and 2 of the plane

  // output plane x0 = i0 of this wave: V[tb][cg][xi][tile][CG], xi = x0 * PL + j
  const int x0 = i0;
  const int sj = lane / BLK;              // storing lane: value j = sj + 4 * k of the half, tile tl
  float* dst = V + (int64_t(tb) * a.C_pad + int64_t(cg) * CG) * NXI * BLK + int64_t(x0) * PL * NQ + tl * CG;
  auto combine = [&](auto X0, int h) {
    constexpr int xr = decltype(X0)::value;
#pragma unroll
    for (int k = 0; k < (HALF + 3) / 4; ++k) {
      const int j = sj + 4 * k;
      if (j < HALF) {
        float4 col[A];
#pragma unroll
        for (int i = 0; i < A; ++i) col[i] = planes[i][j][tl];
        const float* cf = reinterpret_cast<const float*>(col);
        f32x4 out;
        out[0] = row_dot<A, xr>(BT, cf + 0, 4);
        out[1] = row_dot<A, xr>(BT, cf + 1, 4);
        out[2] = row_dot<A, xr>(BT, cf + 2, 4);
        out[3] = row_dot<A, xr>(BT, cf + 3, 4);
        __builtin_nontemporal_store(out, reinterpret_cast<f32x4*>(dst + (h * HALF + j) * NQ));
      }
    }
  };
  static_assert(A == 6, "six output planes");
  float* pl = reinterpret_cast<float*>(&planes[i0][0][tl]) + cl;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (h > 0) __syncthreads();           // the first half has been read
#pragma unroll
    for (int j = 0; j < HALF; ++j) pl[j * BLK * CG] = p2[h * HALF + j];
    __syncthreads();
    switch (x0) {
      case 0: combine(std::integral_constant<int, 0>{}, h); break;
      case 1: combine(std::integral_constant<int, 1>{}, h); break;
      case 2: combine(std::integral_constant<int, 2>{}, h); break;
      case 3: combine(std::integral_constant<int, 3>{}, h); break;
      case 4: combine(std::integral_constant<int, 4>{}, h); break;
      default: combine(std::integral_constant<int, 5>{}, h); break;
    }
  }
}

// ------------------------------------------------- batched GEMM (a4 + a5)
// (F(4^3) and the other 2-D sizes; m = 2 uses k_gemm_acc, F(4^2)
// k_gemm_acc4.)  Work-group = BLK tiles x BLK kernels x all
// alpha^N elements.  The NW waves split the elements evenly in whole units of
// the LOC trailing axes (alpha^LOC consecutive elements) and keep one BLK x
// BLK fp32 MFMA accumulator per element for the whole channel reduction.
// MFMA operands stream straight from global memory (V from HBM/L2, U from L2)
// through a DEPTH-stage register ring, DEPTH-1 channel steps ahead.
//
// Epilogue (eq. 4's inverse transform, separable): each lane holds, for every
// (tile, kernel) of its accumulator registers, all elements of its wave's
// units, so A^T is applied along the LOC trailing axes in registers; the
// partial results go through LDS, and A^T along the leading axes is done by
// threads laid out so that neighbouring lanes write neighbouring outputs of
// a row.
template <int BLK> struct MfmaShape;
template <> struct MfmaShape<32> {
  static constexpr int KSTEP = 2, NACC = 16;
  using acc_t = f32x16;
  __device__ static __forceinline__ acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  // accumulator register r of a lane holds row 8*(r/4) + 4*(lane/32) + r%4, column lane%32
  __device__ static __forceinline__ int acc_row(int lane, int r) {
    return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
};
template <> struct MfmaShape<16> {
  static constexpr int KSTEP = 4, NACC = 4;
  using acc_t = f32x4;
  __device__ static __forceinline__ acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  // accumulator register r of a lane holds row 4*(lane/16) + r, column lane%16
  __device__ static __forceinline__ int acc_row(int lane, int r) { return 4 * (lane >> 4) + r; }
};

// Shape of one GEMM work-group.  NW waves split the alpha^N elements evenly;
// each wave's share is made of whole "units" of the LOC trailing axes
// (alpha^LOC consecutive elements), which is what lets the epilogue reduce
// those axes in registers.
template <int N, int MM, int R, int BLK, int NW, int LOC>
struct GemmGeom {
  static constexpr int A = MM + R - 1;
  static constexpr int NXI = ipow(A, N);
  static constexpr int NT = NW * 64;
  static constexpr int XPW = NXI / NW;               // elements per wave
  static constexpr int UNIT = ipow(A, LOC);          // elements per register-reduced unit
  static constexpr int UPW = XPW / UNIT;             // units per wave
  static constexpr int NUNIT = NXI / UNIT;           // units in the work-group = alpha^(N-LOC)
  static constexpr int OLOC = ipow(MM, LOC);         // outputs per unit after the reduction
  static constexpr int PLANES = NUNIT * OLOC;        // LDS planes of BLK x BLK partial results
  static constexpr int PL = BLK * BLK + 32 / MM;     // plane stride, padded against bank conflicts
  static constexpr int LDS_FLOATS = PLANES * PL;
  static_assert(NXI % NW == 0 && XPW % UNIT == 0, "waves must own whole units");
  static_assert(LOC >= 1 && LOC < N, "at least one axis is reduced in registers, one across waves");
};

// Value of the neighbouring lane of the pair (lanes 2i and 2i + 1 swap).
__device__ __forceinline__ float dpp_swap_pair(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0xb1, 0xf, 0xf, false));
}

struct EpiArgs {
  float* y;
  int32_t K;
  int64_t ystride_k;  // prod Y_i
  int32_t Y[3];
  int32_t act;
  float slope;
  const float* bias;  // [K] or null
  int32_t Yp[3];      // POOL > 0: pooled extents, y is [n][K][Yp]
  int64_t ystride_p;  // prod Yp_i
};

// Inverse transform of a work-group's accumulators (eq. 4), stitched into y.
// acc[x] is the BLK x BLK (tile, kernel) block of element wave*XPW + x.
// tile_of(tl, ti) maps a local tile row to its sample (return value, -1 if
// the row is padding) and per-axis tile coordinates ti.
//
// Part 1: A^T along the LOC trailing axes in registers; the m^LOC results of
// every unit go to LDS plane (unit, o_loc) at [k][t ^ k].
// Part 2: A^T along the N-LOC leading axes, ReLU, crop, store.  Item
// (o_loc, k, t) runs with the last-axis output fastest, then the tile, so
// neighbouring lanes write neighbouring outputs of a row.
template <int N, int MM, int R, bool CONST, int BLK, int NW, int LOC, bool BIAS, int POOL = 0, class AccT,
          class TileFn>
__device__ __forceinline__ void gemm_epilogue(const AccT* acc, float* sm, int kb, const EpiArgs& g,
                                              const FMats& fm, TileFn tile_of) {
  using S = MfmaShape<BLK>;
  using Geo = GemmGeom<N, MM, R, BLK, NW, LOC>;
  constexpr int A = Geo::A, NT = Geo::NT;
  constexpr int UPW = Geo::UPW, UNIT = Geo::UNIT, OLOC = Geo::OLOC, PL = Geo::PL;
  constexpr int NUNIT = Geo::NUNIT;
  // Part 2 runs on the first NTE threads, a whole number of (output of the
  // last axis, tile) rows
  constexpr int NTE = (NT / (MM * BLK)) * (MM * BLK);
  static_assert(NTE > 0, "at least one row of output lanes");
  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  const int col = lane % BLK;
  const MatRef<Which::AT, CONST, MM, R> AT{&fm};
  // BIAS (a separate instance, so that layers without a bias run the same
  // code as before it existed): the block's bias values go through LDS, as a
  // global load inside the store loop would make its stores wait for each
  // other (vmcnt counts both)
  __shared__ float bsm[BLK];
  if constexpr (BIAS) {
    if (int(threadIdx.x) < BLK) {
      const int kg = kb * BLK + int(threadIdx.x);
      bsm[threadIdx.x] = kg < g.K ? g.bias[kg] : 0.0f;
    }
  }
#pragma unroll
  for (int r = 0; r < S::NACC; ++r) {
    const int t = S::acc_row(lane, r);
#pragma unroll
    for (int u = 0; u < UPW; ++u) {
      float sv[UNIT];
#pragma unroll
      for (int e = 0; e < UNIT; ++e) sv[e] = acc[u * UNIT + e][r];
      float o[OLOC];
      transform_nd<LOC, A, MM>(sv, o, AT);
      float* dst = sm + ((wave * UPW + u) * OLOC) * PL + col * BLK + (t ^ col);
#pragma unroll
      for (int j = 0; j < OLOC; ++j) dst[j * PL] = o[j];
    }
  }
  __syncthreads();

  const int tid = int(threadIdx.x);
  if (tid >= NTE) return;
  const int o_last = tid % MM;
  const int tl = (tid / MM) % BLK;
  int ti[3] = {0, 0, 0};
  const int n = tile_of(tl, ti);
  if (n < 0) return;
  const int y_last = ti[N - 1] * MM + o_last;
  if (y_last >= g.Y[N - 1]) return;
  constexpr int ITEMS = OLOC * BLK * BLK;
  constexpr int LEAD = N - LOC;
  constexpr int OLEAD = ipow(MM, LEAD);
  for (int i = tid; i < ITEMS; i += NTE) {
    const int k_l = (i / (MM * BLK)) % BLK;
    const int o_rest = i / (MM * BLK * BLK);
    const int kg = kb * BLK + k_l;
    if (kg >= g.K) continue;
    const int jj = o_rest * MM + o_last;
    int yc[3] = {0, 0, 0};
    bool ok = true;
    {
      int rem = o_rest;
#pragma unroll
      for (int ax = N - 2; ax >= LEAD; --ax) {
        const int oa = rem % MM;
        rem /= MM;
        yc[ax] = ti[ax] * MM + oa;
        ok = ok && yc[ax] < g.Y[ax];
      }
      yc[N - 1] = y_last;
    }
    if (!ok) continue;
    float v[NUNIT];
#pragma unroll
    for (int uu = 0; uu < NUNIT; ++uu) v[uu] = sm[(uu * OLOC + jj) * PL + k_l * BLK + (tl ^ k_l)];
    float out[OLEAD];
    transform_nd<LEAD, A, MM>(v, out, AT);
    if constexpr (POOL == 0) {
      float* yk = g.y + (int64_t(n) * g.K + kg) * g.ystride_k;
      if constexpr (BIAS) {
        const float bk = bsm[k_l];
#pragma unroll
        for (int q = 0; q < OLEAD; ++q) out[q] += bk;
      }
#pragma unroll
      for (int q = 0; q < OLEAD; ++q) {
        int rem = q;
        bool in = true;
#pragma unroll
        for (int ax = LEAD - 1; ax >= 0; --ax) {
          const int oa = rem % MM;
          rem /= MM;
          yc[ax] = ti[ax] * MM + oa;
          in = in && yc[ax] < g.Y[ax];
        }
        if (!in) continue;
        int64_t off = yc[0];
#pragma unroll
        for (int ax = 1; ax < N; ++ax) off = off * g.Y[ax] + yc[ax];
        float val = out[q];
        val = activate(val, g.act, g.slope);
        yk[off] = val;
      }
    } else {
      // Max-pool with window (1, 2, 2) (POOL 1) or (2, 2, 2) (POOL 2), floor
      // rounding, after the activation.  Neighbouring lanes hold the last-axis
      // outputs 2w and 2w + 1 of the same (tile, kernel): the even lane takes
      // its partner's values by a DPP swap and scans each window first axis
      // slowest, last axis fastest, with a strict comparison from -inf, as
      // the stand-alone max-pool does (same bits).  A pooled output whose
      // window reaches past Y is dropped, so the even lane only reads a
      // partner that is live.
      static_assert(N == 3 && LOC == 1 && MM == 4, "pooling: F(4^3), last axis reduced in registers");
      constexpr int W0 = POOL == 2 ? 2 : 1;
      if constexpr (BIAS) {
        const float bk = bsm[k_l];
#pragma unroll
        for (int q = 0; q < OLEAD; ++q) out[q] += bk;
      }
#pragma unroll
      for (int q = 0; q < OLEAD; ++q) out[q] = activate(out[q], g.act, g.slope);
      float other[OLEAD];
#pragma unroll
      for (int q = 0; q < OLEAD; ++q) other[q] = dpp_swap_pair(out[q]);
      const int p2 = y_last >> 1;
      if ((o_last & 1) == 0 && p2 < g.Yp[2]) {
        float* yk = g.y + (int64_t(n) * g.K + kg) * g.ystride_p + p2;
#pragma unroll
        for (int g0 = 0; g0 < MM / W0; ++g0) {
          const int p0 = ti[0] * (MM / W0) + g0;
          if (p0 >= g.Yp[0]) continue;
#pragma unroll
          for (int w1 = 0; w1 < MM / 2; ++w1) {
            const int p1 = ti[1] * (MM / 2) + w1;
            if (p1 >= g.Yp[1]) continue;
            float best = -__builtin_inff();
#pragma unroll
            for (int i0 = 0; i0 < W0; ++i0)
#pragma unroll
              for (int i1 = 0; i1 < 2; ++i1) {
                const int q = (g0 * W0 + i0) * MM + 2 * w1 + i1;
                best = out[q] > best ? out[q] : best;
                best = other[q] > best ? other[q] : best;
              }
            yk[(int64_t(p0) * g.Yp[1] + p1) * g.Yp[2]] = best;
          }
        }
      }
    }
  }
}

// Raw buffer resource covering the 4 GiB that follow a wave-uniform base
// (num_records 2^32 - 1 bytes, stride 0; the fourth word is the gfx9
// family's raw 32-bit format).  Loads through it add a 32-bit vector offset
// and a 32-bit scalar offset to the base.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const float* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), 0, -1, 0x00020000);
}

// VEC = floats per operand load (one load feeds VEC MFMA k-steps).  DEPTH =
// stages in the register ring (DEPTH-1 stages in flight while one is
// consumed).
template <int N, int MM, int R, bool CONST, int BLK, int NW, int LOC, int VEC, int DEPTH, int POOL = 0>
__global__ void __launch_bounds__(NW * 64) k_gemm_inv(const float* __restrict__ V,
                                                      const float* __restrict__ U,
                                                      float* __restrict__ y, GemmArgs g, FMats fm) {
  using S = MfmaShape<BLK>;
  using Geo = GemmGeom<N, MM, R, BLK, NW, LOC>;
  constexpr int NXI = Geo::NXI, XPW = Geo::XPW;
  static_assert(VEC == 4, "16-byte operand loads");

  __shared__ float sm[Geo::LDS_FLOATS];

  const int lane = int(threadIdx.x) & 63;
  // uniform for the buffer bases of the 3-D sizes (the 2-D sizes keep the
  // form their per-lane pointers were tuned with)
  const int wave = N == 3 ? __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6) : int(threadIdx.x) >> 6;
  const int L = xcd_remap(int(blockIdx.x), g.nblocks);
  const int tb = L / g.nkb, kb = L % g.nkb;
  const int col = lane % BLK, kr = lane / BLK;

  // Operand rows: V[tb][cg][xi][t][CG] and U[xi][cg][k][CG].  A "stage" is
  // SC = KSTEP * VEC channels: lane (kr, col) owns channels VEC*kr ..
  // VEC*kr+VEC-1 of every stage (channel c0 = SC*s + VEC*kr of stage s sits
  // in group c0 / CG at offset c0 % CG); MFMA k-step j of the stage uses
  // channel c0 + j, so the VEC steps cover all SC channels.
  constexpr int SC = S::KSTEP * VEC;
  constexpr int CG = Blocking<N, MM, R>::CG;
  static_assert(Blocking<N, MM, R>::CGU == CG && Blocking<N, MM, R>::STAGE == SC, "U and V share the groups");
  static_assert(SC % CG == 0 && CG % VEC == 0, "a stage holds whole groups; a load stays in one group");
  const int64_t vxi = int64_t(BLK) * CG;                           // V element stride (floats)
  const int64_t uxi = g.uplane;                                    // U plane stride (floats)
  const int c0 = VEC * kr;                                         // this lane's channel in a stage
  // 3-D: the operands of a stage are read through buffer resources, the
  // wave's stage bases (uniform, in scalar registers), the lane's byte offset
  // as the vector offset and each element's offset as the scalar one, so the
  // loads need no per-lane 64-bit address arithmetic (the planner keeps the
  // offsets of a wave's U elements below 2^32 bytes).  On the C3D stack's
  // conv2-4: 272 / 142 / 258 -> 237 / 125 / 239 us.  The 2-D sizes keep
  // per-lane pointers (the buffer form made the Fig. 4 layers 2% slower).
  constexpr bool BUF = N == 3;
  const float* vnext;
  const float* unext;
  int vlane = 0, ulane = 0;
  if constexpr (BUF) {
    vnext = V + int64_t(tb) * NXI * g.C_pad * BLK + int64_t(wave) * XPW * vxi;
    unext = U + int64_t(wave) * XPW * uxi + int64_t(kb) * BLK * CG;
    vlane = ((c0 / CG) * NXI * BLK * CG + col * CG + c0 % CG) * 4;
    ulane = (((c0 / CG) * g.K_pad + col) * CG + c0 % CG) * 4;
  } else {
    vnext = V + int64_t(tb) * NXI * g.C_pad * BLK + int64_t(c0 / CG) * NXI * BLK * CG + int64_t(wave) * XPW * vxi +
            col * CG + c0 % CG;
    unext = U + int64_t(wave) * XPW * uxi + (int64_t(c0 / CG) * g.K_pad + int64_t(kb) * BLK + col) * CG + c0 % CG;
  }
  const int64_t vgstep = int64_t(NXI) * BLK * SC, ugstep = int64_t(g.K_pad) * SC;
  const int nstages = g.C_pad / SC;

  typename S::acc_t acc[XPW];
#pragma unroll
  for (int x = 0; x < XPW; ++x) acc[x] = typename S::acc_t{};

  using vec_t = typename std::conditional<VEC == 4, float4,
                typename std::conditional<VEC == 2, float2, float>::type>::type;
  vec_t ra[DEPTH][XPW], rb[DEPTH][XPW];
  auto fetch = [&](vec_t* a2, vec_t* b2) {
    if constexpr (BUF) {
      const __amdgpu_buffer_rsrc_t rv = raw_rsrc(vnext), ru = raw_rsrc(unext);
#pragma unroll
      for (int x = 0; x < XPW; ++x) {
        a2[x] = __builtin_bit_cast(vec_t, __builtin_amdgcn_raw_buffer_load_b128(rv, vlane, int(x * vxi * 4), 0));
        b2[x] = __builtin_bit_cast(vec_t, __builtin_amdgcn_raw_buffer_load_b128(ru, ulane, int(x * uxi * 4), 0));
      }
    } else {
#pragma unroll
      for (int x = 0; x < XPW; ++x) {
        a2[x] = *reinterpret_cast<const vec_t*>(vnext + x * vxi);
        b2[x] = *reinterpret_cast<const vec_t*>(unext + x * uxi);
      }
    }
    vnext += vgstep;
    unext += ugstep;
  };
  auto consume = [&](const vec_t* a2, const vec_t* b2) {
    const float* af = reinterpret_cast<const float*>(a2);
    const float* bf = reinterpret_cast<const float*>(b2);
#pragma unroll
    for (int j = 0; j < VEC; ++j)
#pragma unroll
      for (int x = 0; x < XPW; ++x) acc[x] = S::mma(af[x * VEC + j], bf[x * VEC + j], acc[x]);
  };
  // Prologue: DEPTH-1 stages in flight.
#pragma unroll
  for (int d = 0; d < DEPTH - 1; ++d)
    if (d < nstages) fetch(ra[d], rb[d]);
  // Steady state: every iteration issues DEPTH fetches and consumes DEPTH
  // stages with no branches in between, so the wait counts the compiler
  // inserts only ever wait for the stage being consumed.
  int s = 0;
  for (; s + 2 * DEPTH - 1 <= nstages; s += DEPTH) {
#pragma unroll
    for (int j = 0; j < DEPTH; ++j) {
      fetch(ra[(j + DEPTH - 1) % DEPTH], rb[(j + DEPTH - 1) % DEPTH]);
      consume(ra[j], rb[j]);
    }
  }
  // Tail: the last (at most 2*DEPTH-2) stages.
#pragma unroll
  for (int j = 0; j < 2 * DEPTH - 2; ++j) {
    if (s + j < nstages) {
      if (s + j + DEPTH - 1 < nstages)
        fetch(ra[(j + DEPTH - 1) % DEPTH], rb[(j + DEPTH - 1) % DEPTH]);
      consume(ra[j % DEPTH], rb[j % DEPTH]);
    }
  }

  EpiArgs e{y, g.K, g.ystride_k, {g.Y[0], g.Y[1], g.Y[2]}, g.act, g.slope, g.bias,
            {g.Yp[0], g.Yp[1], g.Yp[2]}, g.ystride_p};
  auto tile_of = [&](int tl, int* ti) -> int {
    const int t = tb * BLK + tl;
    if (t >= g.T) return -1;
    return split_tile<N>(t, g.tiles, ti);
  };
  if (g.bias != nullptr) gemm_epilogue<N, MM, R, CONST, BLK, NW, LOC, true, POOL>(acc, sm, kb, e, fm, tile_of);
  else gemm_epilogue<N, MM, R, CONST, BLK, NW, LOC, false, POOL>(acc, sm, kb, e, fm, tile_of);
}

// ------------------------------------------------------------ max-pool (a6)
struct PoolArgs {
  int64_t lead;
  int32_t X[3], Y[3], p[3];
  int64_t total;  // lead * prod Y
};

static __global__ void __launch_bounds__(256) k_maxpool3d(const float* __restrict__ x, float* __restrict__ y,
                                                   PoolArgs a) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= a.total) return;
  int64_t r = i;
  const int y2 = int(r % a.Y[2]); r /= a.Y[2];
  const int y1 = int(r % a.Y[1]); r /= a.Y[1];
  const int y0 = int(r % a.Y[0]); r /= a.Y[0];
  const float* src = x + r * (int64_t(a.X[0]) * a.X[1] * a.X[2]);
  float best = -__builtin_inff();
  for (int i0 = 0; i0 < a.p[0]; ++i0)
    for (int i1 = 0; i1 < a.p[1]; ++i1)
      for (int i2 = 0; i2 < a.p[2]; ++i2) {
        const float v = src[(int64_t(y0 * a.p[0] + i0) * a.X[1] + (y1 * a.p[1] + i1)) * a.X[2] +
                            (y2 * a.p[2] + i2)];
        best = v > best ? v : best;
      }
  y[i] = best;
}

// The same for a last-axis window of 2 on rows of a multiple of 4 values:
// one thread per pair of neighbouring outputs reads each window row as one
// aligned 16-byte load and writes the pair as 8 bytes.
static __global__ void __launch_bounds__(256) k_maxpool3d_pair(const float* __restrict__ x, float* __restrict__ y,
                                                        PoolArgs a) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;   // output pair
  if (i >= a.total / 2) return;
  int64_t r = i;
  const int h = int(r % (a.Y[2] / 2)); r /= a.Y[2] / 2;
  const int y1 = int(r % a.Y[1]); r /= a.Y[1];
  const int y0 = int(r % a.Y[0]); r /= a.Y[0];
  const float* src = x + r * (int64_t(a.X[0]) * a.X[1] * a.X[2]) + 4 * h;
  float b0 = -__builtin_inff(), b1 = -__builtin_inff();
  for (int i0 = 0; i0 < a.p[0]; ++i0)
    for (int i1 = 0; i1 < a.p[1]; ++i1) {
      const float4 v = *reinterpret_cast<const float4*>(
          src + (int64_t(y0 * a.p[0] + i0) * a.X[1] + (y1 * a.p[1] + i1)) * a.X[2]);
      // the one-output kernel's comparisons, in its order
      b0 = v.x > b0 ? v.x : b0;
      b0 = v.y > b0 ? v.y : b0;
      b1 = v.z > b1 ? v.z : b1;
      b1 = v.w > b1 ? v.w : b1;
    }
  *reinterpret_cast<float2*>(y + 2 * i) = make_float2(b0, b1);
}

}  // namespace wino
