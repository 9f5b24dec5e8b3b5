// gfx950 kernels of the N-D Winograd forward.
//
//   k_filter     U[xi][c][k]  = (w[k][c] x_n G)[xi]            eq. (4), kernel side
//   k_input      V[xi][c][t]  = (d_{t,c} x_n B^T)[xi]          eq. (4), data side
//   k_gemm_inv   M_xi = V_xi . U_xi on fp32 MFMA (eq. 5), then
//                y tile = M[:, t, k] x_n A^T, stitched and cropped (eq. 4)
//   k_maxpool3d  pooling for the C3D stack (not part of the method)
//
// Layouts (float32, zero padding rows/columns):
//   x [batch][C][X_1..X_N]     w [K][C][r^N]      y [batch][K][Y_1..Y_N]
//   U [alpha^N][C_pad][K_pad]  V [alpha^N][C_pad][T_pad]
// T counts tiles over the whole batch (tiles of every sample form the rows of
// one GEMM, §4.1 and §4.4: the method is batch-size agnostic).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- arguments
struct FilterArgs {
  int64_t uplane;  // C_pad * K_pad
  int32_t C, K, C_pad, K_pad;
};

struct InputArgs {
  int64_t vplane;  // C_pad * T_pad
  int64_t xstride_c;  // prod X_i
  int32_t C, C_pad;
  int32_t T, T_pad;
  int32_t X[3], tiles[3], pad[3];
};

struct GemmArgs {
  int64_t vplane, uplane;
  int64_t ystride_k;  // prod Y_i
  int32_t T, T_pad, C_pad, K, K_pad;
  int32_t nkb;        // K_pad / BLK
  int32_t nblocks;    // work-groups in the grid
  int32_t tiles[3], Y[3];
  int32_t relu;
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

// ------------------------------------------------------------ filter (a2)
template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(256) k_filter(const float* __restrict__ w, float* __restrict__ U,
                                                FilterArgs a, FMats fm) {
  constexpr int A = MM + R - 1;
  constexpr int NXI = ipow(A, N);
  constexpr int RN = ipow(R, N);
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int k = int(idx % a.K_pad);
  const int c = int(idx / a.K_pad);
  if (c >= a.C_pad) return;
  float u[NXI];
  if (c < a.C && k < a.K) {
    float g[RN];
    const float* src = w + (int64_t(k) * a.C + c) * RN;
#pragma unroll
    for (int i = 0; i < RN; ++i) g[i] = src[i];
    transform_nd<N, R, A>(g, u, MatRef<Which::G, CONST, MM, R>{&fm});
  } else {
#pragma unroll
    for (int i = 0; i < NXI; ++i) u[i] = 0.0f;
  }
  float* dst = U + int64_t(c) * a.K_pad + k;
#pragma unroll
  for (int xi = 0; xi < NXI; ++xi) dst[int64_t(xi) * a.uplane] = u[xi];
}

// ------------------------------------------------------------- input (a3)
// One thread per (tile, channel): gather the alpha^N window (zero outside the
// input), transform along every axis, scatter to the alpha^N planes of V.
// Consecutive threads take consecutive tiles, so every plane store is a
// contiguous run.
template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(256) k_input(const float* __restrict__ x, float* __restrict__ V,
                                               InputArgs a, FMats fm) {
  constexpr int A = MM + R - 1;
  constexpr int NXI = ipow(A, N);
  const int t = int(blockIdx.x) * 256 + int(threadIdx.x);
  const int c = int(blockIdx.y);
  if (t >= a.T_pad) return;
  float d[NXI];
  if (t < a.T && c < a.C) {
    int ti[3] = {0, 0, 0};
    const int n = split_tile<N>(t, a.tiles, ti);
    int o[3];
    bool in[3][A];
#pragma unroll
    for (int ax = 0; ax < N; ++ax) {
      o[ax] = ti[ax] * MM - a.pad[ax];
#pragma unroll
      for (int i = 0; i < A; ++i) in[ax][i] = (unsigned)(o[ax] + i) < (unsigned)a.X[ax];
    }
    const float* xc = x + (int64_t(n) * a.C + c) * a.xstride_c;
    if constexpr (N == 2) {
#pragma unroll
      for (int i0 = 0; i0 < A; ++i0)
#pragma unroll
        for (int i1 = 0; i1 < A; ++i1)
          d[i0 * A + i1] = (in[0][i0] && in[1][i1])
                               ? xc[int64_t(o[0] + i0) * a.X[1] + (o[1] + i1)] : 0.0f;
    } else {
#pragma unroll
      for (int i0 = 0; i0 < A; ++i0)
#pragma unroll
        for (int i1 = 0; i1 < A; ++i1)
#pragma unroll
          for (int i2 = 0; i2 < A; ++i2)
            d[(i0 * A + i1) * A + i2] =
                (in[0][i0] && in[1][i1] && in[2][i2])
                    ? xc[(int64_t(o[0] + i0) * a.X[1] + (o[1] + i1)) * a.X[2] + (o[2] + i2)]
                    : 0.0f;
    }
  } else {
#pragma unroll
    for (int i = 0; i < NXI; ++i) d[i] = 0.0f;
  }
  float v[NXI];
  transform_nd<N, A, A>(d, v, MatRef<Which::BT, CONST, MM, R>{&fm});
  float* dst = V + int64_t(c) * a.T_pad + t;
#pragma unroll
  for (int xi = 0; xi < NXI; ++xi) dst[int64_t(xi) * a.vplane] = v[xi];
}

// ------------------------------------------------- batched GEMM (a4 + a5)
// Work-group = BLK tiles x BLK kernels x all alpha^N elements; wave w owns
// XPW = alpha^N / NW consecutive elements and keeps one BLK x BLK fp32 MFMA
// accumulator per element for the whole channel reduction.  MFMA operands
// stream straight from global memory (V from HBM/L2, U from L2) one channel
// step ahead; the inverse transform needs every element of a (tile, kernel)
// pair, so the epilogue exchanges accumulators through LDS in row slices.
template <int BLK> struct MfmaShape;
template <> struct MfmaShape<32> {
  static constexpr int KSTEP = 2, NACC = 16, ROWS = 8;
  using acc_t = f32x16;
  __device__ static __forceinline__ acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  // Output element of accumulator register `reg` in round q (regs 4q..4q+3):
  // row 8*(reg/4) + 4*(lane/32) + reg%4, column lane%32.
  static constexpr int ROUNDS = 4, REGS_PER_ROUND = 4;
  __device__ static __forceinline__ int row_local(int lane, int j) { return 4 * (lane >> 5) + j; }
  __device__ static __forceinline__ int row_global(int rl, int q) { return 8 * q + rl; }
  __device__ static __forceinline__ int reg(int q, int j) { return 4 * q + j; }
  __device__ static __forceinline__ int swz(int rl, int col) { return col ^ (rl << 2); }
};
template <> struct MfmaShape<16> {
  static constexpr int KSTEP = 4, NACC = 4, ROWS = 4;
  using acc_t = f32x4;
  __device__ static __forceinline__ acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  // Register `reg` holds row 4*(lane/16) + reg, column lane%16.
  static constexpr int ROUNDS = 4, REGS_PER_ROUND = 1;
  __device__ static __forceinline__ int row_local(int lane, int) { return lane >> 4; }
  __device__ static __forceinline__ int row_global(int rl, int q) { return 4 * rl + q; }
  __device__ static __forceinline__ int reg(int q, int) { return q; }
  __device__ static __forceinline__ int swz(int rl, int col) { return col ^ ((rl >> 1) << 3); }
};

// Work-groups are dispatched round-robin over the 8 XCDs.  Renumber them so
// that consecutive logical blocks (the K-blocks of one tile block, which read
// the same V rows) land on the same XCD and share its L2.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  constexpr int NX = 8;
  const int xcd = b % NX, j = b / NX;
  const int per = nb / NX, rem = nb % NX;
  return xcd < rem ? xcd * (per + 1) + j : rem * (per + 1) + (xcd - rem) * per + j;
}

template <int N, int MM, int R, bool CONST, int BLK, int NW>
__global__ void __launch_bounds__(NW * 64) k_gemm_inv(const float* __restrict__ V,
                                                      const float* __restrict__ U,
                                                      float* __restrict__ y, GemmArgs g, FMats fm) {
  using S = MfmaShape<BLK>;
  constexpr int A = MM + R - 1;
  constexpr int NXI = ipow(A, N);
  constexpr int XPW = NXI / NW;
  static_assert(NXI % NW == 0, "elements must split evenly over waves");
  constexpr int NT = NW * 64;
  constexpr int P = S::ROWS * BLK;          // (tile, kernel) pairs per round
  constexpr int TPP = NT / P;               // threads per pair
  static_assert(TPP >= 1 && NT % P == 0, "pairs must cover the work-group");
  constexpr int AR = ipow(A, N - 1);

  __shared__ float sm[NXI * S::ROWS * BLK];

  const int lane = int(threadIdx.x) & 63;
  const int wave = int(threadIdx.x) >> 6;
  const int L = xcd_remap(int(blockIdx.x), g.nblocks);
  const int tb = L / g.nkb, kb = L % g.nkb;
  const int xi0 = wave * XPW;
  const int col = lane % BLK, kr = lane / BLK;

  const float* vp = V + int64_t(xi0) * g.vplane + int64_t(kr) * g.T_pad + int64_t(tb) * BLK + col;
  const float* up = U + int64_t(xi0) * g.uplane + int64_t(kr) * g.K_pad + int64_t(kb) * BLK + col;
  const int64_t vstep = int64_t(S::KSTEP) * g.T_pad, ustep = int64_t(S::KSTEP) * g.K_pad;

  typename S::acc_t acc[XPW];
#pragma unroll
  for (int x = 0; x < XPW; ++x) acc[x] = typename S::acc_t{};

  float an[XPW], bn[XPW];
#pragma unroll
  for (int x = 0; x < XPW; ++x) {
    an[x] = vp[int64_t(x) * g.vplane];
    bn[x] = up[int64_t(x) * g.uplane];
  }
  for (int c0 = 0; c0 < g.C_pad; c0 += S::KSTEP) {
    float ac[XPW], bc[XPW];
#pragma unroll
    for (int x = 0; x < XPW; ++x) { ac[x] = an[x]; bc[x] = bn[x]; }
    if (c0 + S::KSTEP < g.C_pad) {
      vp += vstep;
      up += ustep;
#pragma unroll
      for (int x = 0; x < XPW; ++x) {
        an[x] = vp[int64_t(x) * g.vplane];
        bn[x] = up[int64_t(x) * g.uplane];
      }
    }
#pragma unroll
    for (int x = 0; x < XPW; ++x) acc[x] = S::mma(ac[x], bc[x], acc[x]);
  }

  // ---- epilogue: inverse transform along every axis, stitch, crop.
  const MatRef<Which::AT, CONST, MM, R> AT{&fm};
  const int tid = int(threadIdx.x);
  const int p = tid % P, part = tid / P;
  const int rl_c = p % S::ROWS, kl_c = p / S::ROWS;
  const int kglob = kb * BLK + kl_c;
#pragma unroll
  for (int q = 0; q < S::ROUNDS; ++q) {
    if (q) __syncthreads();
#pragma unroll
    for (int j = 0; j < S::REGS_PER_ROUND; ++j) {
      const int rl = S::row_local(lane, j);
      float* dst = sm + rl * BLK + S::swz(rl, col);
#pragma unroll
      for (int x = 0; x < XPW; ++x) dst[(xi0 + x) * (S::ROWS * BLK)] = acc[x][S::reg(q, j)];
    }
    __syncthreads();
    const int t = tb * BLK + S::row_global(rl_c, q);
    if (t < g.T && kglob < g.K) {
      int ti[3] = {0, 0, 0};
      const int n = split_tile<N>(t, g.tiles, ti);
      const float* src = sm + rl_c * BLK + S::swz(rl_c, kl_c);
      float* yk = y + (int64_t(n) * g.K + kglob) * g.ystride_k;
      for (int o0 = part; o0 < MM; o0 += TPP) {
        const int y0 = ti[0] * MM + o0;
        if (y0 >= g.Y[0]) break;
        // contract axis 0 while streaming the alpha^N values from LDS
        float s[AR];
        bool first = true;
#pragma unroll
        for (int x0 = 0; x0 < A; ++x0) {
          const float cf = AT(o0, x0);
          if (cf == 0.0f) continue;
#pragma unroll
          for (int rr = 0; rr < AR; ++rr) {
            const float v = src[(x0 * AR + rr) * (S::ROWS * BLK)];
            if (first) s[rr] = (cf == 1.0f) ? v : (cf == -1.0f ? -v : cf * v);
            else if (cf == 1.0f) s[rr] += v;
            else if (cf == -1.0f) s[rr] -= v;
            else s[rr] = __builtin_fmaf(cf, v, s[rr]);
          }
          first = false;
        }
        if constexpr (N == 2) {
          float o[MM];
          apply_axis<1, A, MM, 1>(s, o, AT);
#pragma unroll
          for (int o1 = 0; o1 < MM; ++o1) {
            const int y1 = ti[1] * MM + o1;
            if (y1 < g.Y[1]) {
              float v = o[o1];
              if (g.relu) v = v > 0.0f ? v : 0.0f;
              yk[int64_t(y0) * g.Y[1] + y1] = v;
            }
          }
        } else {
          float t1[MM * A];
          float o[MM * MM];
          apply_axis<1, A, MM, A>(s, t1, AT);
          apply_axis<MM, A, MM, 1>(t1, o, AT);
#pragma unroll
          for (int o1 = 0; o1 < MM; ++o1) {
            const int y1 = ti[1] * MM + o1;
            if (y1 >= g.Y[1]) continue;
            float* row = yk + (int64_t(y0) * g.Y[1] + y1) * g.Y[2];
#pragma unroll
            for (int o2 = 0; o2 < MM; ++o2) {
              const int y2 = ti[2] * MM + o2;
              if (y2 < g.Y[2]) {
                float v = o[o1 * MM + o2];
                if (g.relu) v = v > 0.0f ? v : 0.0f;
                row[y2] = v;
              }
            }
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------ max-pool (a6)
struct PoolArgs {
  int64_t lead;
  int32_t X[3], Y[3], p[3];
  int64_t total;  // lead * prod Y
};

__global__ void __launch_bounds__(256) k_maxpool3d(const float* __restrict__ x, float* __restrict__ y,
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

}  // namespace wino
