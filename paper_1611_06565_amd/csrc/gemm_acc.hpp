// Batched GEMM with the inverse transform accumulated pass by pass, for
// output tiles of extent m = 2 (F(2^N, r^N)).
//
// The inverse transform of eq. (4) is linear: every output is a sum over the
// alpha^N elements xi of a coefficient (a product of A^T entries, one per
// axis) times M_xi.  So the products of one (tile, kernel) pair need not be
// live at once: a pass computes a few whole alpha-rows of elements (leading
// indices fixed, last index free), reduces each row by A^T along the last
// axis and adds it into the m^N outputs with the leading coefficients.  A
// work-group keeps one pass of accumulators and covers a 64-tile x 64-kernel
// block (twice the MFMA operand reuse of keeping all alpha^N elements
// resident), plus m^N output accumulators per pair.
//
// Operands (V tile rows and U kernel columns of one pass and one channel
// stage) are copied global -> LDS with 16-byte direct-to-LDS loads into a
// double buffer, so the next stage streams in while this one is multiplied,
// without holding registers.
//
// Layouts: V[T_pad/64][alpha^N][C_pad/4][64][4], U[alpha^N][C_pad/4][K_pad][4]
// (channel groups of 4 innermost: a lane's 16-byte LDS read holds 4 channels).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.hpp"
#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

struct AccArgs {
  int64_t vplane;     // floats per (tile block, element): C_pad * 64
  int64_t uplane;     // floats per element of U: C_pad * K_pad
  int64_t ystride_k;  // prod Y_i
  int32_t T, C_pad, K, K_pad;
  int32_t nkb;        // K_pad / 64
  int32_t nblocks;    // work-groups in the grid
  int32_t tiles[3], Y[3];
  int32_t relu;
};

template <int N, int MM, int R>
struct AccGeom {
  static constexpr int A = MM + R - 1;
  static constexpr int NXI = ipow(A, N);
  // elements per pass: whole rows of the last axis, at most 8 (128 accumulator
  // registers, leaving room for the m^N output accumulators)
  static constexpr int E = ipow(A, N - 1) > 8 ? 8 : ipow(A, N - 1);
  static constexpr int RP = E / A;                // alpha-rows per pass
  static constexpr int NROW = ipow(A, N - 1);     // alpha-rows in all
  static constexpr int NPASS = NXI / E;
  static constexpr int NOUT = ipow(MM, N);        // outputs per (tile, kernel)
  static constexpr int NLEAD = NOUT / MM;         // outputs of the leading axes
  static constexpr int TB = 64, KB = 64;          // tiles and kernels per work-group
  static constexpr int NW = 4, NT = 256;          // wave (tq, kq) owns a 32 x 32 quadrant
  static constexpr int SC = 128 / E;              // channels per stage: 64 KB of operands
  static constexpr int G4 = SC / 4;               // 4-channel groups per stage
  static constexpr int GPW = G4 / NW;             // groups per wave in the copies
  static constexpr int SA = E * G4 * TB * 4;      // floats of V per stage buffer
  static constexpr int SB = E * G4 * KB * 4;      // floats of U per stage buffer
  static constexpr int STAGE = SA + SB;
  static constexpr int PLANE = TB * KB;           // stitch plane of one output index
  static_assert(MM == 2, "m = 2 only: 2^N output accumulators per pair");
  static_assert(E % A == 0 && NXI % E == 0, "passes of whole alpha-rows");
  static_assert(SC % 8 == 0, "whole pairs of 4-channel groups per stage");
  static_assert(G4 % NW == 0, "copies split evenly over the waves");
  static_assert(NOUT % 2 == 0 && (NOUT / 2) * PLANE <= STAGE, "stitch fits the two buffers");
};

// One 16-byte direct-to-LDS copy per lane: lane l moves src[4l..4l+3] (its own
// global address) to dst[4l..4l+3] (dst is wave-uniform).  A plain function,
// not a template, so that the host pass never checks the builtin's gfx950-only
// operand size against the host target.
__device__ __forceinline__ void lds_copy16(const float* src, float* dst) {
  __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
}

// Coefficient of alpha-row `row` (leading element indices, last axis
// excluded) in the leading output index `oo`: the product over the leading
// axes of A^T[o_ax][xi_ax].  `row` is wave-uniform; the select chain keeps
// the compile-time matrices as immediates.
template <int N, int MM, int R, bool CONST>
__device__ __forceinline__ float lead_coef(const MatRef<Which::AT, CONST, MM, R>& AT, int row, int oo) {
  using G = AccGeom<N, MM, R>;
  float c = 0.0f;
#pragma unroll
  for (int q = 0; q < G::NROW; ++q) {
    float v = 1.0f;
    int rr = q, o2 = oo;
#pragma unroll
    for (int ax = 0; ax < N - 1; ++ax) {
      v *= AT(o2 % MM, rr % G::A);
      rr /= G::A;
      o2 /= MM;
    }
    c = (row == q) ? v : c;
  }
  return c;
}

template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(256) k_gemm_acc(const float* __restrict__ V,
                                                  const float* __restrict__ U,
                                                  float* __restrict__ y, AccArgs g, FMats fm) {
  using G = AccGeom<N, MM, R>;
  using S = MfmaShape<32>;
  constexpr int A = G::A, E = G::E, NOUT = G::NOUT, G4 = G::G4, RP = G::RP;
  constexpr int TB = G::TB, KB = G::KB, NW = G::NW;

  // Two operand buffers as distinct LDS objects: the compiler can then tell
  // that reads of one do not depend on the copies in flight into the other.
  __shared__ __attribute__((aligned(16))) float buf0[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf1[G::STAGE];

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tq = wave >> 1, kq = wave & 1;        // quadrant of the 64 x 64 block
  const int col = lane & 31, kr = lane >> 5;

  const int L = xcd_remap(int(blockIdx.x), g.nblocks);
  const int tb = L / g.nkb, kb = L % g.nkb;
  const int nstage = g.C_pad / G::SC;             // channel stages per pass

  // ---- direct-to-LDS copies of one (pass, stage) step.  Wave w copies the
  // 4-channel groups gi = w + NW*j of every element of the pass: 1 KB chunks
  // V[tb][xi][grp][0:64][0:4] and U[xi][grp][kb*64 : kb*64+64][0:4].
  const float* vsrc = V + int64_t(tb) * G::NXI * g.vplane + wave * (TB * 4) + lane * 4;
  const float* usrc = U + int64_t(kb) * (KB * 4) + int64_t(wave) * g.K_pad * 4 + lane * 4;
  const int64_t vstage = int64_t(G4) * TB * 4, ustage = int64_t(G4) * g.K_pad * 4;
  auto issue = [&](float* base, int pass, int st) {
    const float* vs = vsrc + int64_t(pass) * E * g.vplane + st * vstage;
    const float* us = usrc + int64_t(pass) * E * g.uplane + st * ustage;
#pragma unroll
    for (int e = 0; e < E; ++e)
#pragma unroll
      for (int j = 0; j < G::GPW; ++j) {
        const int gi = wave + NW * j;
        lds_copy16(vs + e * g.vplane + j * (NW * TB * 4), base + (e * G4 + gi) * 256);
        lds_copy16(us + e * g.uplane + int64_t(j) * NW * g.K_pad * 4,
                   base + G::SA + (e * G4 + gi) * 256);
      }
  };

  typename S::acc_t acc[E];
  float yacc[NOUT][S::NACC];
#pragma unroll
  for (int o = 0; o < NOUT; ++o)
#pragma unroll
    for (int r = 0; r < S::NACC; ++r) yacc[o][r] = 0.0f;

  const MatRef<Which::AT, CONST, MM, R> AT{&fm};
  const int aoff = (kr * TB + tq * 32 + col) * 4;
  const int boff = G::SA + (kr * KB + kq * 32 + col) * 4;

  // One step: wait for this step's operands, free the other buffer, start the
  // next step's copies into it, and multiply this one.
  auto step = [&](const float* cur, float* nxt, bool more, int npass, int nst) {
    __builtin_amdgcn_s_waitcnt(0x0f70);           // vmcnt(0), other counters untouched
    __syncthreads();                              // everyone's copies landed; nxt is free
    if (more) issue(nxt, npass, nst);
    const float* sa = cur + aoff;
    const float* sb = cur + boff;
    // pair p of 4-channel groups: lane half kr reads group 2p + kr, so k-step
    // j of the pair contracts channels 8p + j (kr = 0) and 8p + 4 + j (kr = 1).
    // Operands go in groups of 4 elements; the next group is read from LDS
    // while the MFMAs of this one run.
    constexpr int NG = (G4 / 2) * (E / 4);        // (pair, element group) steps
    float4 a4[2][4], b4[2][4];
    auto read_group = [&](int gidx, int slot) {
      const int p = gidx / (E / 4), e0 = (gidx % (E / 4)) * 4;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int off = ((e0 + e) * G4 + 2 * p) * 256;
        a4[slot][e] = *reinterpret_cast<const float4*>(sa + off);
        b4[slot][e] = *reinterpret_cast<const float4*>(sb + off);
      }
    };
    read_group(0, 0);
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      const int slot = gi & 1;
      if (gi + 1 < NG) read_group(gi + 1, slot ^ 1);
      const int e0 = (gi % (E / 4)) * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float4 av4 = a4[slot][e], bv4 = b4[slot][e];
          const float av = j == 0 ? av4.x : j == 1 ? av4.y : j == 2 ? av4.z : av4.w;
          const float bv = j == 0 ? bv4.x : j == 1 ? bv4.y : j == 2 ? bv4.z : bv4.w;
          acc[e0 + e] = S::mma(av, bv, acc[e0 + e]);
          if (gi + 1 < NG && j < 2) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // The stages of one pass alternate between the buffers; which buffer comes
  // first depends on the parity of the steps taken so far.  Both orders are
  // inlined with constant buffer addresses.
  auto run_pass = [&](float* b0, float* b1, int pass) __attribute__((always_inline)) {
    const bool last_pass = pass + 1 == G::NPASS;
    for (int st = 0; st < nstage; st += 2) {
      {
        const bool wrap = st + 1 == nstage;
        step(b0, b1, !(wrap && last_pass), wrap ? pass + 1 : pass, wrap ? 0 : st + 1);
      }
      if (st + 1 < nstage) {
        const bool wrap = st + 2 == nstage;
        step(b1, b0, !(wrap && last_pass), wrap ? pass + 1 : pass, wrap ? 0 : st + 2);
      }
    }
  };

  issue(buf0, 0, 0);
#pragma unroll 1
  for (int pass = 0; pass < G::NPASS; ++pass) {
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = typename S::acc_t{};
    if ((pass * nstage) & 1) run_pass(buf1, buf0, pass);
    else run_pass(buf0, buf1, pass);

    // pass complete: its elements are RP alpha-rows (leading indices fixed,
    // last index free).  Reduce each row along the last axis with A^T, then add
    // it to every output with the product of A^T over the leading indices.
    float c[G::NLEAD][RP];
#pragma unroll
    for (int oo = 0; oo < G::NLEAD; ++oo)
#pragma unroll
      for (int rp = 0; rp < RP; ++rp) c[oo][rp] = lead_coef<N, MM, R, CONST>(AT, pass * RP + rp, oo);
#pragma unroll
    for (int r = 0; r < S::NACC; ++r) {
      float rows[RP][MM];
#pragma unroll
      for (int rp = 0; rp < RP; ++rp) {
        float sv[A];
#pragma unroll
        for (int e = 0; e < A; ++e) sv[e] = acc[rp * A + e][r];
        apply_axis<1, A, MM, 1>(sv, rows[rp], AT);
      }
#pragma unroll
      for (int o = 0; o < NOUT; ++o)
#pragma unroll
        for (int rp = 0; rp < RP; ++rp)
          yacc[o][r] = __builtin_fmaf(c[o / MM][rp], rows[rp][o % MM], yacc[o][r]);
    }
  }

  // ---- stitch: outputs through LDS so that neighbouring lanes store
  // neighbouring outputs of a row.  Plane o ([k][t], t XOR-swizzled by k) lives
  // in buf0 for o < NOUT/2, else in buf1.
  __syncthreads();
  auto plane = [&](int o) { return (o < NOUT / 2 ? buf0 : buf1) + (o % (NOUT / 2)) * G::PLANE; };
#pragma unroll
  for (int o = 0; o < NOUT; ++o)
#pragma unroll
    for (int r = 0; r < S::NACC; ++r) {
      const int t = tq * 32 + S::acc_row(lane, r), k = kq * 32 + col;
      plane(o)[k * TB + (t ^ (k & 31))] = yacc[o][r];
    }
  __syncthreads();
  // item i: last-axis output fastest, then tile, then kernel, then the others
  const int ol = tid % MM;
  const int tl = (tid / MM) % TB;
  const int t = tb * TB + tl;
  if (t >= g.T) return;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<N>(t, g.tiles, ti);
  const int ylast = ti[N - 1] * MM + ol;
  if (ylast >= g.Y[N - 1]) return;
  constexpr int ITEMS = NOUT * TB * KB;
  constexpr int NT = G::NT;
  static_assert(NT % (MM * TB) == 0, "lanes tile the outputs");
  for (int i = tid; i < ITEMS; i += NT) {
    const int kl = (i / (MM * TB)) % KB;
    const int orest = i / (MM * TB * KB);          // outputs of the leading axes
    const int kg = kb * KB + kl;
    if (kg >= g.K) continue;
    int yc[3] = {0, 0, 0};
    bool in = true;
    int rem = orest;
#pragma unroll
    for (int ax = N - 2; ax >= 0; --ax) {
      const int oa = rem % MM;
      rem /= MM;
      yc[ax] = ti[ax] * MM + oa;
      in = in && yc[ax] < g.Y[ax];
    }
    if (!in) continue;
    yc[N - 1] = ylast;
    int64_t off = yc[0];
#pragma unroll
    for (int ax = 1; ax < N; ++ax) off = off * g.Y[ax] + yc[ax];
    float v = plane(orest * MM + ol)[kl * TB + (tl ^ (kl & 31))];
    if (g.relu) v = v > 0.0f ? v : 0.0f;
    y[(int64_t(n) * g.K + kg) * g.ystride_k + off] = v;
  }
}

}  // namespace wino
