// Operand layouts and work-group blocking of every compiled size, as
// compile-time constants shared by the kernels and the host-side planner
// (plain C++: the planner builds without the HIP compiler).
#pragma once

#include "synth.hpp"

namespace wino {

// The (N, m, r) compiled on the layouts below (KIND 0-2): F(2,3) and F(4,3)
// in 2-D and 3-D, F(3,2) in 2-D and 3-D, and in 2-D the alpha = 8 sizes of
// Table 1, F(5,4), F(4,5), F(3,6).  The 3-D alpha = 8 sizes (KIND 4) and the
// per-axis tiles (KIND 3) have their own traits below.
#define WINO_SIZES(X) \
  X(2, 2, 3) X(3, 2, 3) X(2, 4, 3) X(3, 4, 3) X(2, 5, 4) X(2, 4, 5) X(2, 3, 6) X(2, 3, 2) X(3, 3, 2)

// GEMM kind, block (tiles and kernels per work-group), operand load width
// and channel group per (N, m, r).
//   KIND 0 (m = 2) and 1 (F(4^2)): pass-accumulating GEMMs (gemm_acc.hpp,
//     gemm_acc4.hpp) on 64-tile blocks of V with channel groups of 4.
//   KIND 2 (F(4^3) and the other 2-D sizes): k_gemm_inv, all alpha^N
//     elements resident, 16-tile blocks.  A GEMM
//     "stage" covers KSTEP * VEC channels: lane group kr of an MFMA operand
//     loads channels VEC*kr .. VEC*kr+VEC-1 of the stage, and k-step j uses
//     the j-th of them; the stage is KSTEP groups of VEC channels (CG = VEC),
//     so that one input-transform work-group (16 tiles x one group) writes
//     256 contiguous bytes per element.
template <int N, int MM, int R>
struct Blocking {
  static constexpr int A = MM + R - 1;
  static constexpr int NXI = ipow(A, N);
  static constexpr int KIND = MM == 2 ? 0 : ((N == 2 && MM == 4 && R == 3) ? 1 : 2);
  static constexpr bool ACC = KIND == 0;                         // k_gemm_acc
  static constexpr bool PASS = KIND != 2;                        // k_gemm_acc or k_gemm_acc4
  static constexpr int BLK = PASS ? 64 : 16;                     // tiles per V block
  static constexpr int KBLK = KIND == 0 ? 64 : (KIND == 1 ? 32 : 16);   // kernels padded to this
  static constexpr int KSTEP = 4;                                // channels per MFMA (k_gemm_inv)
  static constexpr int VEC = 4;                                  // floats per operand load (k_gemm_inv)
  static constexpr int STAGE = KSTEP * VEC;                      // channels per GEMM stage (k_gemm_inv)
  static constexpr int CG = 4;                                   // channels per V group
  static constexpr int CGU = CG;                                 // channels per U group
  // channels are padded to whole operand stages of the GEMM (16 channels)
  static constexpr int CPAD = 16;
};

// The same constants as run-time values, for the planner.
struct SizeTraits {
  int A, NXI, KIND, BLK, KBLK, CG, CGU, CPAD;
  int TB, KB;   // tiles and kernels per product work-group
};

template <int N, int MM, int R>
constexpr SizeTraits size_traits() {
  using B = Blocking<N, MM, R>;
  SizeTraits t{};
  t.A = B::A; t.NXI = B::NXI; t.KIND = B::KIND; t.BLK = B::BLK; t.KBLK = B::KBLK;
  t.CG = B::CG; t.CGU = B::CGU; t.CPAD = B::CPAD;
  t.TB = B::PASS ? 64 : B::BLK;
  t.KB = B::KBLK;
  return t;
}

// Anisotropic 3-D tiles (F(M0, R) on axis 0, F(M1, R) on axes 1 and 2):
// k_input_ax and k_gemm_ax on the F(4^3) layouts (16-tile V blocks of
// 4-channel groups, 16-kernel blocks).
template <int M0, int M1, int R>
constexpr SizeTraits size_traits_ax() {
  SizeTraits t{};
  t.A = 0;
  t.NXI = (M0 + R - 1) * (M1 + R - 1) * (M1 + R - 1);
  t.KIND = 3;
  t.BLK = 16; t.KBLK = 16; t.CG = 4; t.CGU = 4; t.CPAD = 16;
  t.TB = 16; t.KB = 16;
  return t;
}

// 3-D sizes with alpha = 8 (F(5^3, 4^3), F(4^3, 5^3), F(3^3, 6^3)): k_input_a8
// and k_gemm_a8 on the F(4^3) layouts (16-tile V blocks of 4-channel groups,
// 16-kernel blocks, channels padded to 16).
template <int MM, int R>
constexpr SizeTraits size_traits_a8() {
  SizeTraits t{};
  t.A = MM + R - 1;
  t.NXI = t.A * t.A * t.A;
  t.KIND = 4;
  t.BLK = 16; t.KBLK = 16; t.CG = 4; t.CGU = 4; t.CPAD = 16;
  t.TB = 16; t.KB = 16;
  return t;
}

}  // namespace wino
