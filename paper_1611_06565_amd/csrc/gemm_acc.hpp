// Batched GEMM with the inverse transform accumulated pass by pass, for
// output tiles of extent m = 2 (F(2^N, r^N)).
//
// The inverse transform of eq. (4) is linear: every output is a sum over the
// alpha^N elements xi of a coefficient (a product of A^T entries, one per
// axis) times M_xi.  So the products of one (tile, kernel) pair need not be
// live at once: a pass computes two elements (half a row of the last axis),
// reduces them by the matching columns of A^T along the last axis and adds
// the result into the m^N outputs with the product of A^T over the leading
// axes.  A work-group keeps one pass of accumulators and covers a 64-tile x
// 64-kernel block (twice the MFMA operand reuse of keeping all alpha^N
// elements resident); with two elements per pass a wave needs at most 256
// registers, so two work-groups share a CU and each one's barriers, copies
// and epilogues run under the other's MFMAs.
//
// Operands (V tile rows and U kernel columns of one pass and one channel
// stage) are copied global -> LDS with 16-byte direct-to-LDS loads into four
// stage buffers, three steps ahead, without holding registers.
//
// Layouts: V[T_pad/64][C_pad/4][alpha^N][64][4], U[alpha^N][C_pad/4][K_pad][4]
// (channel groups of 4 innermost: a lane's 16-byte LDS read holds 4 channels).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "kernels.hpp"
#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

struct AccArgs {
  int64_t vblock;     // floats per tile block of V: alpha^N * C_pad * 64
  int64_t uplane;     // floats per element of U: C_pad * K_pad
  int64_t ystride_k;  // prod Y_i
  int32_t T, C_pad, K, K_pad;
  int32_t nkb;        // K_pad / 64
  // Work per XCD (work-group b runs on XCD b % 8 as its unit b / 8): XCD x
  // owns blocks xb0[x] .. xb0[x] + xn[x] - 1, whole blocks first.  Its last
  // xs[x] blocks (those past its last full round of resident work-groups, or
  // all of them when it has fewer than a round) are tail blocks, split into
  // nparts parts of contiguous passes so the last round is shorter; the
  // parts' partial outputs go to part[(xt0[x] + s) * nparts + q][o][t][k]
  // (tail block s of XCD x, part q; TB x KB per output index o), and
  // k_part_reduce sums them in part order and applies bias and ReLU.
  int32_t xb0[8], xn[8], xs[8], xt0[8];
  int32_t tiles[3], Y[3];
  int32_t act;        // activation f of eq. (2): 0 none, 1 ReLU, 2 leaky ReLU
  float slope;        // leaky ReLU: f(v) = slope * v for v <= 0
  const float* bias;  // [K] or null: b_k of eq. (2), added before the activation
  float* part;
  int32_t nparts;
  // (2, 2, 2) max-pool in the epilogue (k_gemm_acc with POOL, k_part_reduce_pool):
  // pooled extents Y / 2 (floor) and the pooled stride per kernel
  int32_t Yp[3];
  int64_t ystride_p;
};

template <int N, int MM, int R>
struct AccGeom {
  static constexpr int A = MM + R - 1;
  static constexpr int NXI = ipow(A, N);
  static constexpr int E = 2;                     // elements per pass: half a row of the last axis
  static constexpr int HALVES = A / E;            // passes per row
  static constexpr int NROW = ipow(A, N - 1);     // rows of the last axis
  static constexpr int NPASS = NXI / E;
  static constexpr int NOUT = ipow(MM, N);        // outputs per (tile, kernel)
  static constexpr int NLEAD = NOUT / MM;         // outputs of the leading axes
  static constexpr int TB = 64, KB = 64;          // tiles and kernels per work-group
  static constexpr int NW = 4, NT = 256;          // wave (tq, kq) owns a 32 x 32 quadrant
  static constexpr int NBUF = 4;                  // stage buffers in LDS
  static constexpr int DEPTH = 3;                 // steps in flight ahead of the one multiplied
  static constexpr int SC = 16;                   // channels per stage
  static constexpr int G4 = SC / 4;               // 4-channel groups per stage
  static constexpr int NG = G4 / 2;               // operand groups (channel pairs) per step
  static constexpr int CH = E * G4;               // 1 KB chunks per operand per stage
  static constexpr int CPW = CH / NW;             // chunks per operand per wave
  static constexpr int CPS = 2 * CPW;             // copies per wave per step
  static constexpr int SA = CH * 256;             // floats of V (and of U) per stage
  static constexpr int STAGE = 2 * SA;            // 16 KB
  static constexpr int PLANE = TB * KB;           // stitch plane of one output index
  static constexpr int PPR = NBUF * (STAGE / PLANE);   // stitch planes per round
  static_assert(MM == 2, "m = 2 only: 2^N output accumulators per pair");
  static_assert(A % E == 0, "passes of half rows");
  static_assert(CH % NW == 0 && CPS == 4, "four copies per wave per step");
  static_assert(STAGE == PLANE && NOUT % PPR == 0, "stitch rounds of whole buffers");
  static_assert(DEPTH < NBUF, "a buffer is refilled only after it was multiplied");
};

// One 16-byte direct-to-LDS copy per lane: lane l moves the 16 bytes at
// sbase + lane_off (sbase wave-uniform, lane_off the lane's own byte offset)
// to dst[4l..4l+3] (dst is wave-uniform; M0 holds its LDS byte address).  Written as inline assembly so that the compiler does not
// track these copies: it would otherwise make LDS reads of other buffers wait
// for them.  Every wait for the copies is explicit (s_waitcnt vmcnt), and the
// stage barrier, which has a memory clobber, orders them against LDS reads.
// NT marks the load non-temporal.  V rows are copied that way although the
// other kernel blocks of a tile block read them too: temporal copies make the
// GEMM a little faster on its own but leave V in the caches (L2 and the
// memory-side cache) in place of the input x that the next input transform
// reads, which costs more than they gain.
// The source is a wave-uniform base (scalar registers) plus the lane's 32-bit
// byte offset, so the copies need no per-lane 64-bit address arithmetic (on
// the headline layer the product went from 615 to 575 us when the per-lane
// pointer adds and selects left the step loop).
template <bool NT>
__device__ __forceinline__ void lds_copy16(const float* sbase, uint32_t lane_off, float* dst) {
  // the low 32 bits of a generic pointer into LDS are its LDS byte address
  const uint32_t lds_addr =
      __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(dst)));
  if constexpr (NT) {
    asm volatile(
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1 nt"
        :
        : "v"(lane_off), "s"(sbase), "s"(lds_addr)
        : "m0");
  } else {
    asm volatile(
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1"
        :
        : "v"(lane_off), "s"(sbase), "s"(lds_addr)
        : "m0");
  }
}

// Work-group barrier for the copy pipeline.  __syncthreads() carries a release
// fence, which would wait for every copy still in flight (vmcnt(0)) and undo
// the pipelining; here the waits are explicit: the caller waits for its own
// copies of the step, and LDS reads are finished (lgkmcnt(0)) before any wave
// may overwrite a buffer.  The memory clobber keeps the compiler from moving
// memory accesses across it.
// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding (expcnt and lgkmcnt untouched).
constexpr int vmcnt_imm(int n) { return 0x0f70 | (n & 15) | (((n >> 4) & 3) << 14); }

__device__ __forceinline__ void stage_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);             // lgkmcnt(0), vmcnt and expcnt untouched
  asm volatile("s_barrier" ::: "memory");
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

// The same coefficients of the compiled-in matrices as a table in constant
// memory: the pass epilogue indexes it with wave-uniform row and half, so
// the coefficients arrive by scalar loads instead of select chains.
// lead[row][oo] = lead_coef(row, oo); at[h][ol][e] = A^T[ol][h * E + e].
template <int N, int MM, int R>
struct AccCoef {
  float lead[AccGeom<N, MM, R>::NROW][AccGeom<N, MM, R>::NLEAD];
  float at[AccGeom<N, MM, R>::HALVES][MM][AccGeom<N, MM, R>::E];
};
template <int N, int MM, int R>
constexpr AccCoef<N, MM, R> make_acc_coef() {
  using G = AccGeom<N, MM, R>;
  AccCoef<N, MM, R> t{};
  for (int q = 0; q < G::NROW; ++q)
    for (int oo = 0; oo < G::NLEAD; ++oo) {
      float v = 1.0f;
      int rr = q, o2 = oo;
      for (int ax = 0; ax < N - 1; ++ax) {
        v *= kDefaultF<MM, R>.AT[o2 % MM][rr % G::A];
        rr /= G::A;
        o2 /= MM;
      }
      t.lead[q][oo] = v;
    }
  for (int h = 0; h < G::HALVES; ++h)
    for (int ol = 0; ol < MM; ++ol)
      for (int e = 0; e < G::E; ++e) t.at[h][ol][e] = kDefaultF<MM, R>.AT[ol][h * G::E + e];
  return t;
}
template <int N, int MM, int R>
__constant__ AccCoef<N, MM, R> kAccCoef = make_acc_coef<N, MM, R>();

template <int N, int MM, int R, bool CONST, int POOL = 0>
__global__ void __launch_bounds__(256, 2) k_gemm_acc(const float* __restrict__ V,
                                                     const float* __restrict__ U,
                                                     float* __restrict__ y, AccArgs g, FMats fm) {
  using G = AccGeom<N, MM, R>;
  using S = MfmaShape<32>;
  constexpr int E = G::E, NOUT = G::NOUT, G4 = G::G4, NG = G::NG;
  constexpr int TB = G::TB, KB = G::KB, NW = G::NW, NBUF = G::NBUF, DEPTH = G::DEPTH;

  // The stage buffers are distinct LDS objects, always named with a
  // compile-time index.
  __shared__ __attribute__((aligned(16))) float buf0[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf1[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf2[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf3[G::STAGE];
  // copies past the last step land here, so every step issues the same copies
  // and no branch splits the MFMA sequence
  __shared__ __attribute__((aligned(16))) float dump[256];
  auto buf = [&](auto I) -> float* {
    constexpr int b = decltype(I)::value % NBUF;
    if constexpr (b == 0) return buf0;
    else if constexpr (b == 1) return buf1;
    else if constexpr (b == 2) return buf2;
    else return buf3;
  };
  auto bufi = [&](int b) -> float* { return b == 0 ? buf0 : b == 1 ? buf1 : b == 2 ? buf2 : buf3; };

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tq = wave >> 1, kq = wave & 1;        // quadrant of the 64 x 64 block
  const int col = lane & 31, kr = lane >> 5;

  // Work unit -> (block, passes).  Each XCD runs its own contiguous range of
  // blocks (consecutive blocks share V rows in its L2), whole blocks first,
  // then the nparts parts of each of its tail blocks, which would otherwise
  // run alone after the XCD's last full round of resident work-groups (or
  // leave most of the slots idle when there is less than a round).  Surplus
  // units exit at once.
  const int xcd = int(blockIdx.x) & 7, j = int(blockIdx.x) >> 3;
  const int xn = g.xn[xcd], xs = g.xs[xcd], np = g.nparts;
  const int nwhole = xn - xs;
  if (j >= nwhole + xs * np) return;
  const bool tail = j >= nwhole;
  const int tj = tail ? j - nwhole : 0;           // unit among the XCD's tail units
  const int blk = g.xb0[xcd] + (tail ? nwhole + tj / np : j);
  const int p0 = tail ? (tj % np) * (G::NPASS / np) : 0;
  const int npass = tail ? G::NPASS / np : G::NPASS;
  const int64_t pslot = tail ? int64_t(g.xt0[xcd]) * np + tj : 0;   // partial-output slot
  const int tb = blk / g.nkb, kb = blk % g.nkb;
  const int nstage = g.C_pad / G::SC;             // channel stages per pass
  const int nsteps = npass * nstage;

  // ---- direct-to-LDS copies of one (pass, stage) step.  Chunk c of an
  // operand is (element e, 4-channel group gi) = (c / G4, c % G4): 1 KB, either
  // V[tb][grp][xi][0:64][0:4] or U[xi][grp][kb*64 : kb*64+64][0:4], landing at
  // c * 256 floats of the V or U half of the buffer.  Wave w copies chunks
  // w, w + NW, ...
  constexpr int64_t VX = TB * 4, VG = int64_t(G::NXI) * TB * 4;    // V element / group strides
  // wave-uniform sources; lane l copies the 16 bytes at byte offset 16 l
  const float* vsrc = V + int64_t(tb) * g.vblock;
  const float* usrc = U + int64_t(kb) * (KB * 4);
  const uint32_t loff = uint32_t(lane) * 16u;
  int64_t voff[G::CPW], uoff[G::CPW];
#pragma unroll
  for (int i = 0; i < G::CPW; ++i) {
    const int c = wave + NW * i, e = c / G4, gi = c % G4;
    voff[i] = e * VX + gi * VG;
    uoff[i] = e * g.uplane + int64_t(gi) * g.K_pad * 4;
  }
  const int64_t vstage = G4 * VG, ustage = int64_t(G4) * g.K_pad * 4;
  // copy q of a step: chunk q / 2 of V (q even) or of U (q odd).  A step past
  // the last one (real == false) copies the block's first chunk again into
  // the dump area instead.
  auto copy_one = [&](const float* vs, const float* us, float* base, bool real, int q) {
    const int i = q >> 1, c = wave + NW * i;
    if ((q & 1) == 0) {
      lds_copy16<true>(real ? vs + voff[i] : vsrc, loff, real ? base + c * 256 : dump);
    } else {
      lds_copy16<false>(real ? us + uoff[i] : usrc, loff, real ? base + G::SA + c * 256 : dump);
    }
  };
  // copy cursor: the next step to copy, as (pass, stage)
  int cpass = p0, cst = 0;
  auto cursor_src = [&](const float*& vs, const float*& us) {
    vs = vsrc + int64_t(cpass) * E * VX + cst * vstage;
    us = usrc + int64_t(cpass) * E * g.uplane + cst * ustage;
  };
  auto advance = [&]() {
    const bool wrap = cst + 1 == nstage;
    cst = wrap ? 0 : cst + 1;
    cpass += wrap ? 1 : 0;
  };
  auto issue = [&](float* base, bool real) {
    const float* vs;
    const float* us;
    cursor_src(vs, us);
#pragma unroll
    for (int q = 0; q < G::CPS; ++q) copy_one(vs, us, base, real, q);
    advance();
  };

  typename S::acc_t acc[E];
  float yacc[NOUT][S::NACC];
#pragma unroll
  for (int o = 0; o < NOUT; ++o)
#pragma unroll
    for (int r = 0; r < S::NACC; ++r) yacc[o][r] = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = typename S::acc_t{};

  const MatRef<Which::AT, CONST, MM, R> AT{&fm};
  const int aoff = (kr * TB + tq * 32 + col) * 4;
  const int boff = G::SA + (kr * KB + kq * 32 + col) * 4;

  // Operand group p (a pair of 4-channel groups) of a step: lane half kr reads
  // group 2p + kr, so k-step j contracts channels 8p + j (kr = 0) and 8p + 4 + j
  // (kr = 1), for both elements of the pass.  Each group is read from LDS while
  // the MFMAs of the previous one run, across step boundaries too.
  float4 a4[2][E], b4[2][E];
  auto read_one = [&](const float* base, int p, int slot, int q) {   // q: A of e = q/2 (even), B (odd)
    const int e = q >> 1;
    const int off = (e * G4 + 2 * p) * 256;
    if ((q & 1) == 0) a4[slot][e] = *reinterpret_cast<const float4*>(base + aoff + off);
    else b4[slot][e] = *reinterpret_cast<const float4*>(base + boff + off);
  };
  // The 4 * E MFMAs of group p from `slot`, in a fixed order with the reads of
  // the next group (into the other slot) and, in a step's last group, the
  // copies of a later step.
  auto mma_group = [&](auto COPY, int slot, const float* nbase, int np, const float* vs,
                       const float* us, float* cbase, bool real) {
    constexpr bool copying = decltype(COPY)::value;
#pragma unroll
    for (int m = 0; m < 4 * E; ++m) {
      const int j = m / E, e = m % E;
      const float4 av4 = a4[slot][e], bv4 = b4[slot][e];
      const float av = j == 0 ? av4.x : j == 1 ? av4.y : j == 2 ? av4.z : av4.w;
      const float bv = j == 0 ? bv4.x : j == 1 ? bv4.y : j == 2 ? bv4.z : bv4.w;
      acc[e] = S::mma(av, bv, acc[e]);
      if (m < 2 * E) read_one(nbase, np, slot ^ 1, m);
      if constexpr (copying) {
        if (m & 1) copy_one(vs, us, cbase, real, m >> 1);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  static_assert(4 * E == 2 * G::CPS, "one copy after every other MFMA of a group");

  // Step s multiplies buffer s % NBUF, whose first group is already in slot
  // 0.  Before its last group it synchronises for step s + 1: wait for this
  // wave's copies of s + 1 (the CPS copies of s + 2 may stay in flight: every
  // step issues exactly CPS copies, real or dumped), barrier (all copies of
  // s + 1 landed; nobody reads buffer (s - 1) % NBUF any more); the last group
  // then refills that buffer with step s + DEPTH and reads the first group of
  // s + 1.  The last step does the same on buffers nobody reads again.
  using CopyOff = std::false_type;
  using CopyOn = std::true_type;
  static_assert(NG % 2 == 0, "a step's first group always uses slot 0");
  auto step = [&](auto I, int s) {
    constexpr int b = decltype(I)::value;
    const float* cur = buf(I);
#pragma unroll
    for (int p = 0; p + 1 < NG; ++p) mma_group(CopyOff{}, p & 1, cur, p + 1, nullptr, nullptr, nullptr, false);
    __builtin_amdgcn_s_waitcnt(0x0f74);           // vmcnt(4): the copies of s + 2 may be in flight
    static_assert(G::CPS == 4, "wait count matches the copies per step");
    stage_barrier();
    const bool real = s + DEPTH < nsteps;
    const float* vs;
    const float* us;
    cursor_src(vs, us);
    advance();
    mma_group(CopyOn{}, (NG - 1) & 1, buf(std::integral_constant<int, b + 1>{}), 0, vs, us,
              buf(std::integral_constant<int, b + DEPTH>{}), real);
  };

  auto epilogue_direct = [&](int pass) {
    const int row = pass / G::HALVES, h = pass % G::HALVES;
    float c[G::NLEAD], at[MM][E];
#pragma unroll
    for (int oo = 0; oo < G::NLEAD; ++oo) c[oo] = lead_coef<N, MM, R, CONST>(AT, row, oo);
#pragma unroll
    for (int ol = 0; ol < MM; ++ol)
#pragma unroll
      for (int e = 0; e < E; ++e) {
        float v = AT(ol, e);
#pragma unroll
        for (int hh = 1; hh < G::HALVES; ++hh) v = (h == hh) ? AT(ol, hh * E + e) : v;
        at[ol][e] = v;
      }
#pragma unroll
    for (int r = 0; r < S::NACC; ++r) {
      float rv[MM];
#pragma unroll
      for (int ol = 0; ol < MM; ++ol) {
        float v = at[ol][0] * acc[0][r];
#pragma unroll
        for (int e = 1; e < E; ++e) v = __builtin_fmaf(at[ol][e], acc[e][r], v);
        rv[ol] = v;
      }
#pragma unroll
      for (int o = 0; o < NOUT; ++o) yacc[o][r] = __builtin_fmaf(c[o / MM], rv[o % MM], yacc[o][r]);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = typename S::acc_t{};
  };
  // Pass epilogue for pass p = (row, half h): the two elements xi_last = 2h,
  // 2h + 1 of the row are reduced by the matching columns of A^T along the last
  // axis, then added to every output with the product of A^T over the leading
  // axes.  With the compiled-in matrices the reduced values are first summed
  // over the halves of the row (rsum), and added to the outputs once, after
  // the row's last half or the last pass of this work unit; with matrices
  // from the argument (their registers leave no room for rsum) every pass
  // adds its own.  The accumulators are cleared for the next pass.
  [[maybe_unused]] float rsum[MM][S::NACC];
  auto epilogue = [&](int pass) {
    if constexpr (!CONST) {
      epilogue_direct(pass);
      return;
    }
    const int row = pass / G::HALVES, h = pass % G::HALVES;
    const AccCoef<N, MM, R>& tab = kAccCoef<N, MM, R>;
    float at[MM][E];
#pragma unroll
    for (int ol = 0; ol < MM; ++ol)
#pragma unroll
      for (int e = 0; e < E; ++e) at[ol][e] = tab.at[h][ol][e];
    if (h == 0 || pass == p0) {                   // first half of a row seen by this unit
#pragma unroll
      for (int r = 0; r < S::NACC; ++r)
#pragma unroll
        for (int ol = 0; ol < MM; ++ol) {
          float v = at[ol][0] * acc[0][r];
#pragma unroll
          for (int e = 1; e < E; ++e) v = __builtin_fmaf(at[ol][e], acc[e][r], v);
          rsum[ol][r] = v;
        }
    } else {
#pragma unroll
      for (int r = 0; r < S::NACC; ++r)
#pragma unroll
        for (int ol = 0; ol < MM; ++ol) {
          float v = rsum[ol][r];
#pragma unroll
          for (int e = 0; e < E; ++e) v = __builtin_fmaf(at[ol][e], acc[e][r], v);
          rsum[ol][r] = v;
        }
    }
    if (h == G::HALVES - 1 || pass == p0 + npass - 1) {   // the row (or the unit) ends
      float c[G::NLEAD];
#pragma unroll
      for (int oo = 0; oo < G::NLEAD; ++oo) c[oo] = tab.lead[row][oo];
#pragma unroll
      for (int r = 0; r < S::NACC; ++r)
#pragma unroll
        for (int o = 0; o < NOUT; ++o) yacc[o][r] = __builtin_fmaf(c[o / MM], rsum[o % MM][r], yacc[o][r]);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = typename S::acc_t{};
  };

  // ---- prologue: copies of the first DEPTH steps, then the first group
  issue(buf0, true);
  issue(buf1, 1 < nsteps);
  issue(buf2, 2 < nsteps);
  static_assert(DEPTH == 3, "prologue fills three buffers");
  __builtin_amdgcn_s_waitcnt(0x0f78);             // vmcnt(8): step 0's copies landed
  static_assert(2 * G::CPS == 8, "prologue wait count");
  stage_barrier();
#pragma unroll
  for (int q = 0; q < 2 * E; ++q) read_one(buf0, 0, 0, q);

  // ---- steps, four per trip so that every buffer is named at compile time
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  static_assert(NBUF == 4, "the step loop unrolls four buffers");
  int s = 0, pass = p0, st = 0;
  auto finish = [&]() {                           // after a step: true when all are done
    ++s;
    if (++st == nstage) {
      epilogue(pass);
      st = 0;
      ++pass;
    }
    return s == nsteps;
  };
#pragma unroll 1
  for (;;) {
    step(I0{}, s);
    if (finish()) break;
    step(I1{}, s);
    if (finish()) break;
    step(I2{}, s);
    if (finish()) break;
    step(I3{}, s);
    if (finish()) break;
  }

  if (tail) {
    // partial outputs of this unit: part[pslot][o][t][k], lanes over k
    __builtin_amdgcn_s_waitcnt(0x0f70);           // vmcnt(0): no copy still writes LDS
    float* pp = g.part + pslot * NOUT * (TB * KB);
#pragma unroll
    for (int o = 0; o < NOUT; ++o)
#pragma unroll
      for (int r = 0; r < S::NACC; ++r) {
        const int tt = tq * 32 + S::acc_row(lane, r), k = kq * 32 + col;
        pp[(o * TB + tt) * KB + k] = yacc[o][r];
      }
    return;
  }

  if constexpr (POOL != 0) {
    // Window (2, 2, 2), stride 2: a tile of 2 is one window, whose 8 outputs
    // are this lane's yacc[0..7][r].  Bias, activation and the maximum in
    // registers, scanned in the stand-alone pool's order (first axis
    // slowest, strict comparison from -inf), so the result has the bits of
    // the forward followed by that pool; one store per complete window
    // (floor rounding drops the tiles cut by the output's end).
    static_assert(N == 3 && MM == 2, "the pooled epilogue takes 3-D tiles of 2");
    __builtin_amdgcn_s_waitcnt(0x0f70);           // vmcnt(0): no copy still writes LDS
    const int kg = kb * KB + kq * 32 + col;
    if (kg >= g.K) return;
    const float bk = g.bias != nullptr ? g.bias[kg] : 0.0f;
    float* const yk = y + int64_t(kg) * g.ystride_p;
#pragma unroll
    for (int r = 0; r < S::NACC; ++r) {
      const int t = tb * TB + tq * 32 + S::acc_row(lane, r);
      if (t >= g.T) continue;
      int ti[3] = {0, 0, 0};
      const int n = split_tile<N>(t, g.tiles, ti);
      if (ti[0] >= g.Yp[0] || ti[1] >= g.Yp[1] || ti[2] >= g.Yp[2]) continue;
      float best = -__builtin_inff();
#pragma unroll
      for (int o = 0; o < NOUT; ++o) {
        float v = yacc[o][r];
        if (g.bias != nullptr) v += bk;
        v = activate(v, g.act, g.slope);
        best = v > best ? v : best;
      }
      yk[int64_t(n) * g.K * g.ystride_p + (int64_t(ti[0]) * g.Yp[1] + ti[1]) * g.Yp[2] + ti[2]] = best;
    }
    return;
  }

  // ---- stitch: outputs through LDS so that neighbouring lanes store
  // neighbouring outputs of a row, PPR output planes per round.  Plane o
  // ([k][t], t XOR-swizzled by k) of a round lives in buffer o % PPR.
  __builtin_amdgcn_s_waitcnt(0x0f70);             // vmcnt(0): no copy still writes LDS
  const int ol = tid % MM;
  const int tl = (tid / MM) % TB;
  const int t = tb * TB + tl;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<N>(t < g.T ? t : 0, g.tiles, ti);
  const int ylast = ti[N - 1] * MM + ol;
  const bool mine = t < g.T && ylast < g.Y[N - 1];
  // thread (ol, tl) stores its tile's outputs for kernels k0, k0 + KS, ...
  constexpr int KS = G::NT / (MM * TB);
  static_assert(G::NT % (MM * TB) == 0, "lanes tile the outputs");
  const int k0 = tid / (MM * TB);
  float* const yn = y + int64_t(n) * g.K * g.ystride_k;
  constexpr int LPR = G::PPR / MM;                // leading output indices per round
#pragma unroll
  for (int o0 = 0; o0 < NOUT; o0 += G::PPR) {
    __syncthreads();                              // buffers free (last MFMA reads / previous round)
#pragma unroll
    for (int o = o0; o < o0 + G::PPR; ++o)
#pragma unroll
      for (int r = 0; r < S::NACC; ++r) {
        const int tt = tq * 32 + S::acc_row(lane, r), k = kq * 32 + col;
        bufi(o - o0)[k * TB + (tt ^ (k & 31))] = yacc[o][r];
      }
    __syncthreads();
    if (mine) {
#pragma unroll
      for (int orest = o0 / MM; orest < o0 / MM + LPR; ++orest) {   // leading output index
        int64_t off = 0;
        bool in = true;
#pragma unroll
        for (int ax = 0; ax < N - 1; ++ax) {
          const int oa = (orest / ipow(MM, N - 2 - ax)) % MM;
          const int yc = ti[ax] * MM + oa;
          in = in && yc < g.Y[ax];
          off = off * g.Y[ax] + yc;
        }
        if (!in) continue;
        off = off * g.Y[N - 1] + ylast;
        const float* pl = bufi(orest * MM + ol - o0);
        float* yo = yn + off;
#pragma unroll 8
        for (int kl = k0; kl < KB; kl += KS) {
          const int kg = kb * KB + kl;
          if (kg >= g.K) break;
          float v = pl[kl * TB + (tl ^ (kl & 31))];
          if (g.bias != nullptr) v += g.bias[kg];
          v = activate(v, g.act, g.slope);
          __builtin_nontemporal_store(v, yo + int64_t(kg) * g.ystride_k);
        }
      }
    }
  }
}

// Tail blocks of k_gemm_acc (TB x KB = 64 x 64) and k_gemm_acc4 (64 x 32):
// y = ReLU(sum over the parts, in part order, + bias) for every output of
// every tail block.  One thread per (tail block,
// output index, tile, kernel); lanes over kernels read the partials
// contiguously, and the part loads are independent (issued together), the
// adds in fixed order, so the results are bitwise reproducible.
template <int N, int MM, int TB, int KB>
__global__ void __launch_bounds__(256) k_part_reduce(float* __restrict__ y, AccArgs g, int32_t ntail) {
  constexpr int NOUT = ipow(MM, N);
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;   // ((tail block, o), tile, kernel)
  const int k_l = int(i % KB), tl = int((i / KB) % TB);
  const int64_t bo = i / (KB * TB);
  const int o = int(bo % NOUT), tix = int(bo / NOUT);
  if (tix >= ntail) return;
  int blk = -1;                                   // tail block tix -> its block
#pragma unroll
  for (int x = 0; x < 8; ++x)
    if (tix >= g.xt0[x] && tix < g.xt0[x] + g.xs[x]) blk = g.xb0[x] + g.xn[x] - g.xs[x] + (tix - g.xt0[x]);
  if (blk < 0) return;
  const int tb = blk / g.nkb, kb = blk % g.nkb;
  const int t = tb * TB + tl, kg = kb * KB + k_l;
  if (t >= g.T || kg >= g.K) return;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<N>(t, g.tiles, ti);
  int64_t off = 0;
#pragma unroll
  for (int ax = 0; ax < N; ++ax) {
    const int oa = (o / ipow(MM, N - 1 - ax)) % MM;
    const int yc = ti[ax] * MM + oa;
    if (yc >= g.Y[ax]) return;                  // cropped output of a partial tile
    off = off * g.Y[ax] + yc;
  }
  const float* pp = g.part + (int64_t(tix) * g.nparts * NOUT + o) * (TB * KB) + tl * KB + k_l;
  float v = 0.0f;
#pragma unroll 8
  for (int q = 0; q < g.nparts; ++q) v += __builtin_nontemporal_load(pp + int64_t(q) * NOUT * (TB * KB));
  if (g.bias != nullptr) v += g.bias[kg];
  v = activate(v, g.act, g.slope);
  y[(int64_t(n) * g.K + kg) * g.ystride_k + off] = v;
}

// k_part_reduce with the (2, 2, 2) max-pool of k_gemm_acc's pooled epilogue
// (3-D tiles of 2): one thread per (tail block, tile, kernel) forms the 8
// outputs of its tile as k_part_reduce does (parts summed in order, bias,
// activation) and stores their maximum, scanned in the stand-alone pool's
// order, for every complete window.
template <int N, int MM, int TB, int KB>
__global__ void __launch_bounds__(256) k_part_reduce_pool(float* __restrict__ y, AccArgs g, int32_t ntail) {
  static_assert(N == 3 && MM == 2, "windows of one tile of 2");
  constexpr int NOUT = ipow(MM, N);
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;   // (tail block, tile, kernel)
  const int k_l = int(i % KB), tl = int((i / KB) % TB);
  const int tix = int(i / (KB * TB));
  if (tix >= ntail) return;
  int blk = -1;                                   // tail block tix -> its block
#pragma unroll
  for (int x = 0; x < 8; ++x)
    if (tix >= g.xt0[x] && tix < g.xt0[x] + g.xs[x]) blk = g.xb0[x] + g.xn[x] - g.xs[x] + (tix - g.xt0[x]);
  if (blk < 0) return;
  const int tb = blk / g.nkb, kb = blk % g.nkb;
  const int t = tb * TB + tl, kg = kb * KB + k_l;
  if (t >= g.T || kg >= g.K) return;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<N>(t, g.tiles, ti);
  if (ti[0] >= g.Yp[0] || ti[1] >= g.Yp[1] || ti[2] >= g.Yp[2]) return;
  const float* pp = g.part + int64_t(tix) * g.nparts * NOUT * (TB * KB) + tl * KB + k_l;
  // each output's parts are added in part order, as k_part_reduce does; the
  // loads of four parts of all 8 outputs are issued together (a thread here
  // does 8 times the loads of a k_part_reduce thread)
  float v[NOUT];
#pragma unroll
  for (int o = 0; o < NOUT; ++o) v[o] = 0.0f;
  int q = 0;
  for (; q + 4 <= g.nparts; q += 4) {
    float ld[4][NOUT];
#pragma unroll
    for (int qq = 0; qq < 4; ++qq)
#pragma unroll
      for (int o = 0; o < NOUT; ++o)
        ld[qq][o] = __builtin_nontemporal_load(pp + (int64_t(q + qq) * NOUT + o) * (TB * KB));
#pragma unroll
    for (int qq = 0; qq < 4; ++qq)
#pragma unroll
      for (int o = 0; o < NOUT; ++o) v[o] += ld[qq][o];
  }
  for (; q < g.nparts; ++q)
#pragma unroll
    for (int o = 0; o < NOUT; ++o) v[o] += __builtin_nontemporal_load(pp + (int64_t(q) * NOUT + o) * (TB * KB));
  float best = -__builtin_inff();
#pragma unroll
  for (int o = 0; o < NOUT; ++o) {
    float u = v[o];
    if (g.bias != nullptr) u += g.bias[kg];
    u = activate(u, g.act, g.slope);
    best = u > best ? u : best;
  }
  y[(int64_t(n) * g.K + kg) * g.ystride_p + (int64_t(ti[0]) * g.Yp[1] + ti[1]) * g.Yp[2] + ti[2]] = best;
}

}  // namespace wino
