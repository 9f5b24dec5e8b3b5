// Batched GEMM with the inverse transform accumulated pass by pass, for 2-D
// output tiles of extent m = 4 (F(4^2, r^2)).
//
// The same scheme as k_gemm_acc (gemm_acc.hpp): a pass computes M_xi for two
// elements (a third of a row of the last axis), reduces them by the matching
// columns of A^T along the last axis and adds the result into the m^2 = 16
// outputs with A^T of the leading axis (eq. 4 is linear).  With 16 outputs
// per (tile, kernel) a wave owns 32 tiles x 16 kernels, as two 16 x 16 blocks
// of v_mfma_f32_16x16x4f32, so its output accumulators take 128 registers; a
// work-group of four waves covers 64 tiles x 32 kernels, twice the operand
// reuse of keeping all alpha^2 elements resident in registers, and two
// work-groups share a CU so that each one's barriers, copies and epilogues
// run under the other's MFMAs.
//
// Operands of one (pass, channel stage) step, V rows of 64 tiles and U columns
// of 32 kernels for 16 channels of two elements (12 KB), are copied global ->
// LDS with 16-byte direct-to-LDS loads into four stage buffers, three steps
// ahead.  A lane group kr (lanes 16 kr .. 16 kr + 15) of an MFMA operand reads
// 4-channel group kr of the stage as one float4 and k-step j uses its j-th
// channel, so the four k-steps of a step contract all 16 channels.
//
// Layouts: V[T_pad/64][C_pad/4][alpha^2][64][4], U[alpha^2][C_pad/4][K_pad][4].
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "gemm_acc.hpp"
#include "kernels.hpp"
#include "synth.hpp"
#include "transforms.hpp"

namespace wino {

template <int N, int MM, int R>
struct Acc4Geom {
  static constexpr int A = MM + R - 1;
  static constexpr int NXI = ipow(A, N);
  static constexpr int E = 2;                     // elements per pass
  static constexpr int HALVES = A / E;            // passes per row of the last axis
  static constexpr int NROW = ipow(A, N - 1);     // rows of the last axis
  static constexpr int NPASS = NXI / E;
  static constexpr int NOUT = ipow(MM, N);        // outputs per (tile, kernel)
  static constexpr int NLEAD = NOUT / MM;         // outputs of the leading axis
  static constexpr int TB = 64, KB = 32;          // tiles and kernels per work-group
  static constexpr int NW = 4, NT = 256;          // wave (tq, kq) owns 32 tiles x 16 kernels
  static constexpr int NH = 2;                    // 16 x 16 MFMA blocks per wave (tile halves)
  static constexpr int NACC = 4;                  // accumulator registers per block
  static constexpr int NBUF = 6;                  // stage buffers in LDS
  // steps copied ahead of the one multiplied: a step's buffer is refilled as
  // soon as its operands are in registers (all reads of it precede the step's
  // barrier), so all NBUF buffers are in flight
  static constexpr int DEPTH = NBUF;
  static constexpr int SC = 16;                   // channels per stage
  static constexpr int G4 = SC / 4;               // 4-channel groups per stage (= MFMA lane groups)
  static constexpr int SAV = E * G4 * TB * 4;     // floats of V per stage (1 KB chunks)
  static constexpr int SAU = E * G4 * KB * 4;     // floats of U per stage (512 B chunks)
  static constexpr int STAGE = SAV + SAU;         // 12 KB
  static constexpr int NCOPY = SAV / 256 + SAU / 256;   // 1 KB copies per step
  static constexpr int CPS = NCOPY / NW;          // copies per wave per step
  static constexpr int PLANE = TB * KB;           // stitch plane of one output index
  static constexpr int PPR = 4;                   // stitch planes per round (one per buffer)
  static_assert(N == 2 && MM == 4, "2-D, m = 4");
  static_assert(A % E == 0, "passes of whole thirds of a row");
  static_assert(NCOPY % NW == 0 && CPS == 3, "three copies per wave per step");
  static_assert(PLANE <= STAGE && NOUT % PPR == 0 && PPR % MM == 0 && PPR <= NBUF, "stitch rounds of whole output rows");
  static_assert(DEPTH <= NBUF && NBUF % 2 == 0, "a buffer is refilled once its operands are read; slots alternate");
  static_assert(KB * 4 * 2 == 256, "a U copy moves two 512 B chunks");
};

// The epilogue's coefficients of the compiled-in matrices as a table in
// constant memory, indexed by the wave-uniform row and third (scalar loads
// instead of select chains): lead[xr][o0] = A^T[o0][xr], at[h][ol][e] =
// A^T[ol][h * E + e].
template <int N, int MM, int R>
struct Acc4Coef {
  float lead[Acc4Geom<N, MM, R>::A][Acc4Geom<N, MM, R>::NLEAD];
  float at[Acc4Geom<N, MM, R>::HALVES][MM][Acc4Geom<N, MM, R>::E];
};
template <int N, int MM, int R>
constexpr Acc4Coef<N, MM, R> make_acc4_coef() {
  using G = Acc4Geom<N, MM, R>;
  Acc4Coef<N, MM, R> t{};
  for (int q = 0; q < G::A; ++q)
    for (int o0 = 0; o0 < G::NLEAD; ++o0) t.lead[q][o0] = kDefaultF<MM, R>.AT[o0][q];
  for (int h = 0; h < G::HALVES; ++h)
    for (int ol = 0; ol < MM; ++ol)
      for (int e = 0; e < G::E; ++e) t.at[h][ol][e] = kDefaultF<MM, R>.AT[ol][h * G::E + e];
  return t;
}
template <int N, int MM, int R>
__constant__ Acc4Coef<N, MM, R> kAcc4Coef = make_acc4_coef<N, MM, R>();

template <int N, int MM, int R, bool CONST>
__global__ void __launch_bounds__(256, 2) k_gemm_acc4(const float* __restrict__ V,
                                                      const float* __restrict__ U,
                                                      float* __restrict__ y, AccArgs g, FMats fm) {
  using G = Acc4Geom<N, MM, R>;
  using S = MfmaShape<16>;
  constexpr int A = G::A, E = G::E, NOUT = G::NOUT, G4 = G::G4, NH = G::NH, NACC = G::NACC;
  constexpr int TB = G::TB, KB = G::KB, NW = G::NW, NBUF = G::NBUF, DEPTH = G::DEPTH;
  static_assert(S::KSTEP == G4 && S::NACC == NACC, "lane groups = 4-channel groups");

  __shared__ __attribute__((aligned(16))) float buf0[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf1[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf2[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf3[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf4[G::STAGE];
  __shared__ __attribute__((aligned(16))) float buf5[G::STAGE];
  static_assert(NBUF == 6, "six stage buffers");
  // copies past the last step land here, so every step issues the same copies
  __shared__ __attribute__((aligned(16))) float dump[256];
  auto buf = [&](auto I) -> float* {
    constexpr int b = decltype(I)::value % NBUF;
    if constexpr (b == 0) return buf0;
    else if constexpr (b == 1) return buf1;
    else if constexpr (b == 2) return buf2;
    else if constexpr (b == 3) return buf3;
    else if constexpr (b == 4) return buf4;
    else return buf5;
  };
  auto bufi = [&](int b) -> float* { return b == 0 ? buf0 : b == 1 ? buf1 : b == 2 ? buf2 : buf3; };   // stitch

  const int tid = int(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tq = wave >> 1, kq = wave & 1;        // 32-tile half and 16-kernel half of the block
  const int row = lane & 15, kr = lane >> 4;      // MFMA operand row / column and lane group

  // Work unit -> (block, passes), as in k_gemm_acc; the 18 passes of a tail
  // block are split into nparts contiguous runs of 2 or 3.
  const int xcd = int(blockIdx.x) & 7, j = int(blockIdx.x) >> 3;
  const int xn = g.xn[xcd], xs = g.xs[xcd], np = g.nparts;
  const int nwhole = xn - xs;
  if (j >= nwhole + xs * np) return;
  const bool tail = j >= nwhole;
  const int tj = tail ? j - nwhole : 0;           // unit among the XCD's tail units
  const int blk = g.xb0[xcd] + (tail ? nwhole + tj / np : j);
  const int prt = tj % np;
  const int p0 = tail ? prt * G::NPASS / np : 0;
  const int npass = tail ? (prt + 1) * G::NPASS / np - p0 : G::NPASS;
  const int64_t pslot = tail ? int64_t(g.xt0[xcd]) * np + tj : 0;   // partial-output slot
  const int tb = blk / g.nkb, kb = blk % g.nkb;
  const int nstage = g.C_pad / G::SC;             // channel stages per pass
  const int nsteps = npass * nstage;

  // ---- direct-to-LDS copies of one (pass, stage) step.  Copy c < 8: V chunk
  // (e, gi) = (c / G4, c % G4), V[tb][grp][xi][0:64][0:4], to c * 256.  Copy
  // c >= 8: U chunks (e, gi) and (e, gi + 1), gi = 2 (u % 2), u = c - 8, e = u / 2:
  // lanes 0..31 move U[xi][grp][kb*32 + lane][0:4], lanes 32..63 the same of
  // group grp + 1, to SAV + (e * G4 + gi) * 128 (the two chunks are adjacent).
  // Wave w does copies w, w + 4 (V) and w + 8 (U), so whether a wave's copy
  // i is V or U is known at compile time.
  constexpr int64_t VX = TB * 4, VG = int64_t(G::NXI) * TB * 4;    // V element / group strides
  // wave-uniform sources plus the lane's byte offset (V: 16 l; U: lanes
  // 32..63 read the next channel group, K_pad * 16 bytes further)
  const float* vsrc = V + int64_t(tb) * g.vblock;
  const float* usrc = U + int64_t(kb) * (KB * 4);
  const uint32_t vloff = uint32_t(lane) * 16u;
  const uint32_t uloff = uint32_t(lane & 31) * 16u + uint32_t(lane >> 5) * uint32_t(g.K_pad) * 16u;
  int64_t off[G::CPS];
  int dsto[G::CPS];
  constexpr int NVC = G::SAV / 256 / NW;           // V copies per wave
  static_assert(NW == 4 && NVC == 2 && G::CPS == NVC + 1, "copies w, w + 4 of V and w + 8 of U");
#pragma unroll
  for (int i = 0; i < G::CPS; ++i) {
    const int c = wave + NW * i;
    if (i < NVC) {
      const int e = c / G4, gi = c % G4;
      off[i] = e * VX + gi * VG;
      dsto[i] = c * 256;
    } else {
      const int u = c - NW * NVC, e = u / 2, gi = 2 * (u % 2);
      off[i] = e * g.uplane + int64_t(gi) * g.K_pad * 4;
      dsto[i] = G::SAV + (e * G4 + gi) * 128;
    }
  }
  const int64_t vstage = G4 * VG, ustage = int64_t(G4) * g.K_pad * 4;
  // copy i of a step; a step past the last one (real == false) copies the
  // block's first V (or U) chunk again into the dump area instead
  auto copy_one = [&](auto I, const float* vs, const float* us, float* base, bool real) {
    constexpr int i = decltype(I)::value;
    // non-temporal V rows: see lds_copy16
    if constexpr (i < NVC) lds_copy16<true>(real ? vs + off[i] : vsrc, vloff, real ? base + dsto[i] : dump);
    else lds_copy16<false>(real ? us + off[i] : usrc, uloff, real ? base + dsto[i] : dump);
  };
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
    unroll<G::CPS>([&](auto I) { copy_one(I, vs, us, base, real); });
    advance();
  };

  typename S::acc_t acc[E][NH];
  float yacc[NOUT][NH][NACC];
#pragma unroll
  for (int o = 0; o < NOUT; ++o)
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
      for (int r = 0; r < NACC; ++r) yacc[o][h][r] = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e)
#pragma unroll
    for (int h = 0; h < NH; ++h) acc[e][h] = typename S::acc_t{};

  const MatRef<Which::AT, CONST, MM, R> AT{&fm};
  // lane group kr reads 4-channel group kr: V tile tq*32 + h*16 + row, U kernel kq*16 + row
  const int aoff = kr * TB * 4 + (tq * 32 + row) * 4;
  const int boff = G::SAV + kr * KB * 4 + (kq * 16 + row) * 4;

  // operands of one step in `slot`: A of element e, half h; B of element e
  float4 a4[2][E][NH], b4[2][E];
  constexpr int NREAD = E * (NH + 1);
  auto read_one = [&](const float* base, int slot, int q) {
    const int e = q / (NH + 1), w = q % (NH + 1);
    if (w < NH) a4[slot][e][w] = *reinterpret_cast<const float4*>(base + e * G4 * TB * 4 + aoff + w * 64);
    else b4[slot][e] = *reinterpret_cast<const float4*>(base + e * G4 * KB * 4 + boff);
  };
  // the 4 * E * NH MFMAs of a step from `slot`, with the reads of the next
  // step (other slot) and the copies of a later step in a fixed order
  constexpr int NMMA = G4 * E * NH;
  static_assert(NMMA == 16 && NREAD <= NMMA && G::CPS <= NMMA / 4, "placement of reads and copies");
  auto mma_step = [&](int slot, const float* nbase, const float* vs, const float* us, float* cbase, bool real) {
    unroll<NMMA>([&](auto M) {
      constexpr int m = decltype(M)::value;
      constexpr int jk = m / (E * NH), e = (m / NH) % E, h = m % NH;
      const float4 av4 = a4[slot][e][h], bv4 = b4[slot][e];
      const float av = jk == 0 ? av4.x : jk == 1 ? av4.y : jk == 2 ? av4.z : av4.w;
      const float bv = jk == 0 ? bv4.x : jk == 1 ? bv4.y : jk == 2 ? bv4.z : bv4.w;
      acc[e][h] = S::mma(av, bv, acc[e][h]);
      if constexpr (m < NREAD) read_one(nbase, slot ^ 1, m);
      if constexpr (m % 4 == 3 && m / 4 < G::CPS) copy_one(std::integral_constant<int, m / 4>{}, vs, us, cbase, real);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  // Step s multiplies buffer s % NBUF from slot s % 2 (read during step s - 1).
  // At its start it waits for this wave's copies of s + 1 (those of s + 2 ..
  // s + DEPTH - 1 may stay in flight: every step issues exactly CPS copies,
  // real or dumped) and synchronises: all copies of s + 1 landed, and every
  // wave has finished reading buffer s % NBUF into registers.  Its MFMAs then
  // run with the reads of step s + 1 and the copies of step s + DEPTH into
  // buffer (s + DEPTH) % NBUF = s % NBUF.
  auto step = [&](auto I, int s) {
    constexpr int b = decltype(I)::value;
    __builtin_amdgcn_s_waitcnt(vmcnt_imm((DEPTH - 2) * G::CPS));
    stage_barrier();
    const bool real = s + DEPTH < nsteps;
    const float* vs;
    const float* us;
    cursor_src(vs, us);
    advance();
    mma_step(b & 1, buf(std::integral_constant<int, b + 1>{}), vs, us, buf(std::integral_constant<int, b + DEPTH>{}),
             real);
  };

  // Pass epilogue, pass p = (row xi_0, third h): elements xi_1 = 2h, 2h + 1 of
  // the row are reduced by the matching columns of A^T, then added to every
  // output (o_0, o_1) with A^T[o_0][xi_0]; the accumulators are cleared.
  auto epilogue = [&](int pass) {
    const int xr = pass / G::HALVES, h3 = pass % G::HALVES;
    float c[G::NLEAD], at[MM][E];
    if constexpr (CONST) {
      const Acc4Coef<N, MM, R>& tab = kAcc4Coef<N, MM, R>;
#pragma unroll
      for (int o0 = 0; o0 < G::NLEAD; ++o0) c[o0] = tab.lead[xr][o0];
#pragma unroll
      for (int ol = 0; ol < MM; ++ol)
#pragma unroll
        for (int e = 0; e < E; ++e) at[ol][e] = tab.at[h3][ol][e];
    } else {
#pragma unroll
      for (int o0 = 0; o0 < G::NLEAD; ++o0) {
        float v = AT(o0, 0);
#pragma unroll
        for (int q = 1; q < A; ++q) v = (xr == q) ? AT(o0, q) : v;
        c[o0] = v;
      }
#pragma unroll
      for (int ol = 0; ol < MM; ++ol)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          float v = AT(ol, e);
#pragma unroll
          for (int hh = 1; hh < G::HALVES; ++hh) v = (h3 == hh) ? AT(ol, hh * E + e) : v;
          at[ol][e] = v;
        }
    }
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
      for (int r = 0; r < NACC; ++r) {
        float rv[MM];
#pragma unroll
        for (int ol = 0; ol < MM; ++ol) {
          float v = at[ol][0] * acc[0][h][r];
#pragma unroll
          for (int e = 1; e < E; ++e) v = __builtin_fmaf(at[ol][e], acc[e][h][r], v);
          rv[ol] = v;
        }
#pragma unroll
        for (int o = 0; o < NOUT; ++o) yacc[o][h][r] = __builtin_fmaf(c[o / MM], rv[o % MM], yacc[o][h][r]);
      }
#pragma unroll
    for (int e = 0; e < E; ++e)
#pragma unroll
      for (int h = 0; h < NH; ++h) acc[e][h] = typename S::acc_t{};
  };

  // ---- prologue: copies of the first DEPTH steps, then step 0's operands
  unroll<DEPTH>([&](auto I) { issue(buf(I), decltype(I)::value < nsteps); });
  __builtin_amdgcn_s_waitcnt(vmcnt_imm((DEPTH - 1) * G::CPS));   // step 0's copies landed
  stage_barrier();
#pragma unroll
  for (int q = 0; q < NREAD; ++q) read_one(buf0, 0, q);

  int s = 0, pass = p0, st = 0;
  auto finish = [&]() {
    ++s;
    if (++st == nstage) {
      epilogue(pass);
      st = 0;
      ++pass;
    }
    return s == nsteps;
  };
  // NBUF steps per trip so that every buffer is named at compile time
  bool done = false;
#pragma unroll 1
  while (!done) {
    unroll<NBUF>([&](auto I) {
      if (!done) {
        step(I, s);
        done = finish();
      }
    });
  }

  // ---- stitch: outputs through LDS, one output plane ([k][t], t XOR-swizzled
  // by k) per buffer, a whole leading output index (MM planes of the last
  // axis) per round; thread (ol, tl) stores its tile's output ol of the last
  // axis for every kernel, so neighbouring lanes store neighbouring outputs.
  __builtin_amdgcn_s_waitcnt(0x0f70);             // vmcnt(0): no copy still writes LDS
  if (tail) {
    // partial outputs of this unit: part[pslot][o][t][k], lanes over k
    float* pp = g.part + pslot * G::NOUT * (TB * KB);
#pragma unroll
    for (int o = 0; o < G::NOUT; ++o)
#pragma unroll
      for (int h = 0; h < NH; ++h)
#pragma unroll
        for (int r = 0; r < NACC; ++r) {
          const int tt = tq * 32 + h * 16 + S::acc_row(lane, r), k = kq * 16 + row;
          pp[(o * TB + tt) * KB + k] = yacc[o][h][r];
        }
    return;
  }
  // the block's bias values go through LDS: a global load inside the store
  // loop would make its stores wait for each other (vmcnt counts both)
  __shared__ float bsm[KB];
  if (g.bias != nullptr && tid < KB) {
    const int kg = kb * KB + tid;
    bsm[tid] = kg < g.K ? g.bias[kg] : 0.0f;
  }
  const int ol = tid % MM;
  const int tl = (tid / MM) % TB;
  static_assert(G::NT == MM * TB, "one thread per (output of the last axis, tile)");
  const int t = tb * TB + tl;
  int ti[3] = {0, 0, 0};
  const int n = split_tile<N>(t < g.T ? t : 0, g.tiles, ti);
  const int ylast = ti[N - 1] * MM + ol;
  const bool mine = t < g.T && ylast < g.Y[N - 1];
  float* const yn = y + int64_t(n) * g.K * g.ystride_k;
#pragma unroll
  for (int o0 = 0; o0 < NOUT; o0 += G::PPR) {
    __syncthreads();                              // buffers free (last MFMA reads / previous round)
#pragma unroll
    for (int o = o0; o < o0 + G::PPR; ++o)
#pragma unroll
      for (int h = 0; h < NH; ++h)
#pragma unroll
        for (int r = 0; r < NACC; ++r) {
          const int tt = tq * 32 + h * 16 + S::acc_row(lane, r), k = kq * 16 + row;
          bufi(o - o0)[k * TB + (tt ^ (k & 31))] = yacc[o][h][r];
        }
    __syncthreads();
    if (mine) {
#pragma unroll
      for (int orest = o0 / MM; orest < (o0 + G::PPR) / MM; ++orest) {   // leading output index
        const int yc = ti[0] * MM + orest;
        if (yc >= g.Y[0]) continue;
        const int64_t off2 = int64_t(yc) * g.Y[N - 1] + ylast;
        const float* pl = bufi(orest * MM + ol - o0);
        float* yo = yn + off2;
#pragma unroll 8
        for (int kl = 0; kl < KB; ++kl) {
          const int kg = kb * KB + kl;
          if (kg >= g.K) break;
          float v = pl[kl * TB + (tl ^ (kl & 31))];
          if (g.bias != nullptr) v += bsm[kl];
          v = activate(v, g.act, g.slope);
          __builtin_nontemporal_store(v, yo + int64_t(kg) * g.ystride_k);
        }
      }
    }
  }
}

}  // namespace wino
