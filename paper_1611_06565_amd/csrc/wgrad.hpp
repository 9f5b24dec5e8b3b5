// Weight gradient of a layer (the backward pass on the kernel side; the paper
// measures forward passes only).
//
// Per axis, the gradient of the r kernel taps over one output tile is a
// correlation of the tile's m output gradients with the alpha-value input
// window: dw_t[p] = sum_{o<m} dy_t[o] d_t[o + p], p < r.  That is the
// minimal filtering algorithm F(r, m) of §2.2 with the roles of kernel and
// output swapped, and over N axes (eq. 3-4)
//
//   dw_t = A'^T [ (dy_t x_n G') (.) (d_t x_n B'^T) ]
//
// with (A'^T, G', B'^T) the triple of F(r, m) on the forward's points.  B'^T
// equals the forward's B^T (both come from the same points; the plan checks
// it exactly), so d_t x_n B'^T is the forward's V.  Summed over the tiles of
// the whole batch, the inverse transform comes out of the sum, and the sum
// per element is a product (eq. 5 read the other way):
//
//   M_xi [K x C] = sum_t D_xi[k][t] V_xi[c][t],   dw = M x_n A'^T.
//
//   k_dy          D[xi][k][t] = (dy_t[k] x_n G')[xi], layout of V
//   k_wgrad_gemm  partial M_xi over a range of tile blocks, fp32 MFMA
//   k_wgrad_sum     sum of the partials (fixed order)
//   k_wgrad_finish  A'^T, one output tap per thread
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.hpp"
#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

struct WgArgs {
  int64_t ystride_k;    // prod Y_i (dy per kernel)
  int32_t T, ntb;       // tiles; 64-tile steps (D is stored in 64-tile blocks)
  int32_t nvb;          // V's tile blocks (of VB tiles)
  int32_t K, K_pad4;    // kernels, rounded up to 4 (D's channel groups)
  int32_t C, C_pad;     // channels (V's C_pad, a multiple of 4)
  int32_t nkb, ncb;     // 64-blocks of kernels and channels in M
  int32_t nsplit;       // tile-block ranges summed separately
  int32_t nblocks;      // work-groups of k_wgrad_gemm
  int32_t tiles[3], Y[3];
};

// One thread per (tile, kernel) of a (tile block, kernel group): lane = tile,
// wave = kernel % 4, so a wave reads one kernel's output gradients at 64
// consecutive tiles (neighbouring lanes, neighbouring outputs).  The values
// then cross an LDS stage (tiles padded to 5 floats, conflict-free writes) so
// that every element's 64 x 4 values are stored as one contiguous 1 KB run.
// Outputs past Y (partial tiles) and padding tiles and kernels read as zero.
// For alpha^N > 64 (F(4^3)) a work-group produces one plane i0 of the first
// axis only (blockIdx = block * alpha + i0): its threads take the tile's m^N
// values one first-axis plane o0 at a time, transform each along the other
// axes and accumulate G'[i0][o0] times it, so no thread holds alpha^N values.
// CONST: the forward's points are the default set, which is also F(r, m)'s
// default (the same first alpha - 1 points), so G' is compiled in.
template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(256) k_dy(const float* __restrict__ dy, float* __restrict__ D, WgArgs a,
                                            FMats fw) {
  constexpr int A = MM + R - 1, NXI = ipow(A, N), NIN = ipow(MM, N);
  constexpr bool PLANES = NXI > 64;
  constexpr int NV = PLANES ? NXI / A : NXI;       // values of this thread
  constexpr int XR = NV < 16 ? NV : 16;            // values per LDS round
  constexpr int TP = 5;                            // padded tile stride in the stage
  __shared__ float stage[XR][64 * TP];
  // the A planes of a block are neighbours in the grid, so they run together
  // and read the block's output gradients from L2 rather than from HBM A times
  const int i0 = PLANES ? int(blockIdx.x) % A : 0;
  const int bid = PLANES ? int(blockIdx.x) / A : int(blockIdx.x);
  const int tb = bid / (a.K_pad4 / 4), kg = bid % (a.K_pad4 / 4);
  const int tl = int(threadIdx.x) & 63, kl = int(threadIdx.x) >> 6;
  const int t = tb * 64 + tl, k = kg * 4 + kl;
  const bool live = t < a.T && k < a.K;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<N>(live ? t : 0, a.tiles, ti);
  const float* src = dy + (int64_t(n) * a.K + (live ? k : 0)) * a.ystride_k;
  // output gradient i of the tile (last axis fastest), zero past Y
  auto load = [&](int i) {
    int64_t off = 0, mul = 1;
    bool in = live;
    int rem = i;
#pragma unroll
    for (int ax = N - 1; ax >= 0; --ax) {
      const int yc = ti[ax] * MM + rem % MM;
      rem /= MM;
      in = in && yc < a.Y[ax];
      off += int64_t(yc) * mul;
      mul *= a.Y[ax];
    }
    return in ? src[off] : 0.0f;
  };
  const MatRef<Which::G, CONST, R, MM> Gp{&fw};    // G' of F(r, m): alpha x m
  float u[NV];
  if constexpr (PLANES) {
    constexpr int NP = NIN / MM;                   // values of one first-axis plane
#pragma unroll
    for (int j = 0; j < NV; ++j) u[j] = 0.0f;
#pragma unroll
    for (int o0 = 0; o0 < MM; ++o0) {
      const float c = Gp(i0, o0);
      if (c == 0.0f) continue;
      float g[NP], q[NV];
      if (N == 3 && MM == 4 && a.Y[2] % 4 == 0) {
        // whole tiles on the last axis: each row of the plane is one aligned
        // 16-byte load (4 * ti[2] and the row starts are multiples of 4)
        const int y0 = ti[0] * MM + o0;
#pragma unroll
        for (int rr = 0; rr < MM; ++rr) {
          const int y1 = ti[1] * MM + rr;
          const bool in = live && y0 < a.Y[0] && y1 < a.Y[1];
          const int64_t off = (int64_t(in ? y0 : 0) * a.Y[1] + (in ? y1 : 0)) * a.Y[2] + ti[2] * MM;
          const float4 v = in ? *reinterpret_cast<const float4*>(src + off) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
          g[rr * 4 + 0] = v.x; g[rr * 4 + 1] = v.y; g[rr * 4 + 2] = v.z; g[rr * 4 + 3] = v.w;
        }
      } else {
#pragma unroll
        for (int i = 0; i < NP; ++i) g[i] = load(o0 * NP + i);
      }
      transform_nd<N - 1, MM, A>(g, q, Gp);
#pragma unroll
      for (int j = 0; j < NV; ++j) u[j] = __builtin_fmaf(c, q[j], u[j]);
    }
  } else {
    float g[NIN];
#pragma unroll
    for (int i = 0; i < NIN; ++i) g[i] = load(i);
    transform_nd<N, MM, A>(g, u, Gp);
  }
  float* dst = D + (int64_t(tb) * (a.K_pad4 / 4) + kg) * NXI * 256 + int64_t(i0) * NV * 256 + threadIdx.x;
  const int rd = (int(threadIdx.x) >> 2) * TP + (int(threadIdx.x) & 3);   // (tile, kernel) of the store
#pragma unroll
  for (int x0 = 0; x0 < NV; x0 += XR) {
    if (x0 > 0) __syncthreads();                   // the previous round has been read
#pragma unroll
    for (int j = 0; j < XR; ++j)
      if (x0 + j < NV) stage[j][tl * TP + kl] = u[x0 + j];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < XR; ++j)
      if (x0 + j < NV) __builtin_nontemporal_store(stage[j][rd], dst + (x0 + j) * 256);
  }
}

// Partial M_xi over tile blocks [tb0, tb1) for one 64-kernel x 64-channel
// block: work-group = four waves, each a 32 x 32 quadrant on
// v_mfma_f32_32x32x2f32 with the tiles as the contraction.  A step stages
// the 16 D chunks and 16 V chunks (1 KB each: 64 tiles x 4 kernels or
// channels) of one tile block through LDS; chunks are padded by 4 floats so
// that the 32 lanes of an operand read hit 32 banks.  The next step's chunks
// are loaded into registers while this step multiplies.  VB is V's tile block:
// 64 (one chunk per step) or 16 (a V chunk of the step is four 256-byte runs
// of consecutive 16-tile blocks; blocks past V's end read as zero).
template <int VB>
__global__ void __launch_bounds__(256) k_wgrad_gemm(const float* __restrict__ V, const float* __restrict__ D,
                                                    float* __restrict__ part, WgArgs a, int32_t nxi) {
  static_assert(VB == 64 || VB == 16, "V tile blocks of 64 or 16");
  using S = MfmaShape<32>;
  constexpr int CP = 260;                          // padded chunk stride (floats)
  __shared__ __attribute__((aligned(16))) float Ds[16 * CP];
  __shared__ __attribute__((aligned(16))) float Vs[16 * CP];
  // wave index uniform (scalar): the chunk choice, its bounds test and the
  // source address of every load are then scalar work, the lane adds 16 bytes
  const int lane = int(threadIdx.x) & 63, wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
  const int L = xcd_remap(int(blockIdx.x), a.nblocks);
  const int cb = L % a.ncb, kb = (L / a.ncb) % a.nkb;
  const int xi = (L / (a.ncb * a.nkb)) % nxi, sp = L / (a.ncb * a.nkb * nxi);
  const int tb0 = int(int64_t(sp) * a.ntb / a.nsplit), tb1 = int(int64_t(sp + 1) * a.ntb / a.nsplit);
  const int kgroups = a.K_pad4 / 4, cgroups = a.C_pad / 4;

  // loads of one step: chunk j * 4 + wave (j < 4: D kernel groups, else V
  // channel groups), lane l takes floats 4l .. 4l + 3
  f32x4 reg[8];
  auto load = [&](int tb) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int ch = (j & 3) * 4 + wave;
      const bool isd = j < 4;
      const int g = (isd ? kb : cb) * 16 + ch;
      bool ok = g < (isd ? kgroups : cgroups);
      const float* src;
      if (isd || VB == 64) {
        src = (isd ? D + ((int64_t(tb) * kgroups + g) * nxi + xi) * 256
                   : V + ((int64_t(tb) * cgroups + g) * nxi + xi) * 256) + 4 * lane;
      } else {
        const int vb = tb * 4 + lane / 16;               // lane's 16-tile block of V
        ok = ok && vb < a.nvb;
        src = V + ((int64_t(vb) * cgroups + g) * nxi + xi) * 64 + 4 * (lane % 16);
      }
      reg[j] = ok ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src)) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
  };
  const int kq = wave >> 1, cq = wave & 1;
  const int i = lane & 31, kk = lane >> 5;
  // operand reads: D row k = 32 kq + i, V column c = 32 cq + i, tile 2 s + kk
  const float* da = Ds + (kq * 8 + i / 4) * CP + kk * 4 + (i & 3);
  const float* vb = Vs + (cq * 8 + i / 4) * CP + kk * 4 + (i & 3);
  S::acc_t acc = S::acc_t{};
  if (tb0 < tb1) load(tb0);
  for (int tb = tb0; tb < tb1; ++tb) {
    __syncthreads();                               // the previous step's reads are done
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float* dst = (j < 4 ? Ds : Vs) + ((j & 3) * 4 + wave) * CP + lane * 4;
      *reinterpret_cast<f32x4*>(dst) = reg[j];
    }
    __syncthreads();
    if (tb + 1 < tb1) load(tb + 1);
#pragma unroll
    for (int s = 0; s < 32; ++s) acc = S::mma(da[s * 8], vb[s * 8], acc);
  }
  // part[sp][xi][k][c] over the 64-padded kernel and channel ranges
  const int64_t kp = int64_t(a.nkb) * 64, cpn = int64_t(a.ncb) * 64;
  float* pp = part + (int64_t(sp) * nxi + xi) * kp * cpn;
#pragma unroll
  for (int r = 0; r < S::NACC; ++r) {
    const int k = kb * 64 + kq * 32 + S::acc_row(lane, r), c = cb * 64 + cq * 32 + i;
    pp[int64_t(k) * cpn + c] = acc[r];
  }
}

// M[xi][k][c] = sum over the splits, in split order; written over split 0's
// partial (each entry is read and written by its own thread only).  One
// thread per (xi, k, c), channels fastest, so the partial reads coalesce and
// the split loads of a thread are independent.
static __global__ void __launch_bounds__(256) k_wgrad_sum(float* __restrict__ part, WgArgs a, int32_t nxi) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int c = int(idx % a.C);
  const int64_t r = idx / a.C;
  const int k = int(r % a.K), xi = int(r / a.K);
  if (xi >= nxi) return;
  const int64_t kp = int64_t(a.nkb) * 64, cpn = int64_t(a.ncb) * 64, plane = int64_t(nxi) * kp * cpn;
  float* pp = part + (int64_t(xi) * kp + k) * cpn + c;
  float v = 0.0f;
#pragma unroll 8
  for (int sp = 0; sp < a.nsplit; ++sp) v += pp[sp * plane];
  pp[0] = v;
}

// dw[k][c][p] = sum_xi (prod over the axes of A'^T[p_ax][xi_ax]) M[xi][k][c],
// M summed over the splits by k_wgrad_sum: the N-mode product with A'^T
// written as one sum per output tap.  One thread per (k, p, c), channels
// fastest, so the M reads of a wave coalesce.
template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(256) k_wgrad_finish(const float* __restrict__ part, float* __restrict__ dw,
                                                      WgArgs a, FMats fw) {
  const MatRef<Which::AT, CONST, R, MM> ATp{&fw};  // A'^T of F(r, m): r x alpha
  constexpr int A = MM + R - 1, NXI = ipow(A, N), NOUT = ipow(R, N);
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int c = int(idx % a.C);
  const int64_t rest = idx / a.C;
  const int p = int(rest % NOUT), k = int(rest / NOUT);
  if (k >= a.K) return;
  int pa[3] = {0, 0, 0};                           // the tap's index per axis
  {
    int q = p;
#pragma unroll
    for (int ax = N - 1; ax >= 0; --ax) { pa[ax] = q % R; q /= R; }
  }
  const int64_t kp = int64_t(a.nkb) * 64, cpn = int64_t(a.ncb) * 64;
  const float* pp = part + int64_t(k) * cpn + c;
  float acc = 0.0f;
#pragma unroll
  for (int xi = 0; xi < NXI; ++xi) {
    float coef = 1.0f;
    int q = xi;
#pragma unroll
    for (int ax = N - 1; ax >= 0; --ax) {
      coef *= ATp(pa[ax], q % A);
      q /= A;
    }
    if (coef != 0.0f) acc = __builtin_fmaf(coef, pp[int64_t(xi) * kp * cpn], acc);
  }
  dw[(int64_t(k) * a.C + c) * NOUT + p] = acc;
}

}  // namespace wino
