// libwino: plan construction, argument checking and kernel dispatch behind the
// C ABI declared in include/wino.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>

#include "gemm_acc.hpp"
#include "gemm_acc4.hpp"
#include "kernels.hpp"
#include "synth.hpp"
#include "wgrad.hpp"
#include "wino.h"

using namespace wino;

struct wino_plan_s {
  int N, m, r, alpha, nxi, C, K;
  int C_pad, K_pad;
  int64_t batch;
  int64_t X[3], Y[3], tiles[3];
  int32_t pad[3];
  int64_t T, T_pad;
  int blk, kblk, cg, cgu;
  int32_t n_user_pts;     // the caller's points (0: default set), kept for wino_plan_adjoint
  double user_pts[kMaxAlpha];
  // weight gradient: F(r, m) on the same points (its B^T is the forward's)
  bool wgrad_ok;
  FMats fmw;
  int32_t wg_nsplit, wg_kpad4;
  int64_t wg_d_floats, wg_part_floats;
  // k_gemm_acc tail split, fixed at plan time from the device's compute
  // units: the last xtail[x] blocks of XCD x are done in nparts parts each
  int nparts;             // 1: no split
  int32_t xtail[8];
  int64_t ntail;          // sum of xtail
  int64_t v_floats;       // V in the workspace (rounded up to 256 bytes)
  int64_t part_floats;    // partial outputs after V when nparts > 1
  uint32_t flags;
  bool const_mats;
  double AT[kMaxAlpha][kMaxAlpha], BT[kMaxAlpha][kMaxAlpha], G[kMaxAlpha][kMaxAlpha];
  FMats fm;
};

namespace {

// Compute units of the current device (cached per device).
int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cached[dev] = n;
  }
  return cached[dev];
}


constexpr int64_t kMaxI32 = 0x7fffffff;

int64_t round_up(int64_t v, int64_t b) { return (v + b - 1) / b * b; }

// Nearest small rational to a double point, accepted only if it rounds back
// to exactly the same double.
bool rationalize(double v, Rat* out) {
  if (!std::isfinite(v) || std::fabs(v) > 1048576.0) return false;
  // continued-fraction convergents h/k
  int64_t h0 = 0, h1 = 1, k0 = 1, k1 = 0;
  double x = v;
  for (int it = 0; it < 40; ++it) {
    const double a = std::floor(x);
    if (std::fabs(a) > 4.0e6) return false;
    const int64_t ai = int64_t(a);
    const int64_t h2 = ai * h1 + h0, k2 = ai * k1 + k0;
    if (k2 > (int64_t(1) << 20) || k2 <= 0) break;
    h0 = h1; h1 = h2; k0 = k1; k1 = k2;
    if (double(h1) / double(k1) == v) {
      *out = rat(h1, k1);
      return true;
    }
    const double f = x - a;
    if (f == 0.0) break;
    x = 1.0 / f;
  }
  return false;
}

// The (N, m, r) with compiled kernels: F(2,3) and F(4,3) in 2-D and 3-D;
// in 2-D also the other sizes of Table 1, F(3,2) (alpha = 4) and F(5,4),
// F(4,5), F(3,6) (alpha = 8).
#define WINO_SIZES(X) \
  X(2, 2, 3) X(3, 2, 3) X(2, 4, 3) X(3, 4, 3) X(2, 5, 4) X(2, 4, 5) X(2, 3, 6) X(2, 3, 2)

bool supported(int N, int m, int r) {
#define WINO_SUPPORTED(N_, M_, R_) \
  if (N == N_ && m == M_ && r == R_) return true;
  WINO_SIZES(WINO_SUPPORTED)
#undef WINO_SUPPORTED
  return false;
}

wino_status launch_status() {
  return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EDEVICE;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---------------------------------------------------------------- dispatch
template <int N, int MM, int R, bool CONST>
struct Launch {
  static constexpr int A = MM + R - 1;
  static constexpr int NXI = ipow(A, N);
  static constexpr int BLK = Blocking<N, MM, R>::BLK;
  static constexpr int CG = Blocking<N, MM, R>::CG;
  static constexpr int CGU = Blocking<N, MM, R>::CGU;
  // k_gemm_inv work-group shape: F(4^3): 12 waves x three alpha-rows (18
  // elements); 2-D sizes: alpha waves x one alpha-row (alpha elements).  The last
  // axis is reduced in registers, 16-byte operand loads, no register ring
  // (the other waves of the SIMD hide the load latency).
  static constexpr int NW = (N == 3 && A == 6) ? 12 : ipow(A, N - 1);
  static constexpr int LOC = 1;
  static constexpr int VEC = Blocking<N, MM, R>::VEC;
  static constexpr int DEPTH = 1;

  static wino_status filter(const wino_plan_s& p, const float* w, float* U, bool adjoint, hipStream_t s) {
    FilterArgs a{};
    a.uplane = int64_t(p.C_pad) * p.K_pad;
    a.C = p.C; a.K = p.K; a.C_pad = p.C_pad; a.K_pad = p.K_pad;
    a.adjoint = adjoint ? 1 : 0;
    const int64_t n = int64_t(p.C_pad) * p.K_pad;   // C_pad is a multiple of CGU
    // one thread per (channel, kernel): small work-groups spread the few
    // threads of a layer (8192 for C = 64, K = 128) over more CUs
    const unsigned grid = unsigned((n + 63) / 64);
    hipLaunchKernelGGL((k_filter<N, MM, R, CONST>), dim3(grid), dim3(64), 0, s, w, U, a, p.fm);
    return launch_status();
  }

  static wino_status input(const wino_plan_s& p, const float* x, float* V, hipStream_t s) {
    InputArgs a{};
    a.xstride_c = 1;
    for (int i = 0; i < N; ++i) a.xstride_c *= p.X[i];
    a.C = p.C; a.C_pad = p.C_pad;
    a.T = int32_t(p.T); a.T_pad = int32_t(p.T_pad);
    for (int i = 0; i < 3; ++i) {
      a.X[i] = int32_t(p.X[i]); a.tiles[i] = int32_t(p.tiles[i]); a.pad[i] = p.pad[i];
    }
    const int64_t groups = p.C_pad / CG;
    a.ntb = int32_t(p.T_pad / BLK);
    if constexpr (Blocking<N, MM, R>::NXI > 64) {
      // large windows: A threads per (tile, channel), one V block (BLK tiles
      // x one channel group) per work-group.  Row-aligned loads when every
      // block is BLK tiles of one input row, rows are whole 16-byte units and
      // a window starts at most 2 values left of its tile.
      constexpr int A = Blocking<N, MM, R>::A;
      static_assert(BLK * CG == 64, "one pair per lane");
      const int64_t nb = (p.T_pad / BLK) * groups;
      a.nblocks = int32_t(nb);
      // (x is 16-byte aligned: the entry points check it)
      a.rowfast = (p.tiles[N - 1] % BLK == 0 && p.X[N - 1] % 4 == 0 && p.pad[N - 1] <= 2) ? 1 : 0;
      hipLaunchKernelGGL((k_input_split<N, MM, R, CONST>), dim3(unsigned(nb)), dim3(A * 64), 0, s, x, V,
                         a, p.fm);
    } else {
      constexpr int GPW = 256 / (BLK * CG);
      const int64_t nb = (p.T_pad / BLK) * ((groups + GPW - 1) / GPW);
      a.nblocks = int32_t(nb);
      // m = 2: aligned pairs plus neighbouring lanes when the last axis has
      // pad 1 and an even length (x is 16-byte aligned: the entry points check it)
      a.rowfast = (MM == 2 && p.pad[N - 1] == 1 && p.X[N - 1] % 2 == 0) ? 1 : 0;
      hipLaunchKernelGGL((k_input<N, MM, R, CONST>), dim3(unsigned(nb)), dim3(256), 0, s, x, V, a, p.fm);
    }
    return launch_status();
  }

  // Weight gradient (wgrad.hpp): V by the forward's input transform, D by
  // k_dy, partial products over tile-block ranges, then their sum and A'^T.
  static wino_status wgrad(const wino_plan_s& p, const float* x, const float* dy, float* dw, float* ws,
                           hipStream_t s) {
    if constexpr ((BLK != 64 && BLK != 16) || CG != 4) {
      return WINO_EUNSUPPORTED;
    } else {
      float* V = ws;
      float* D = ws + p.v_floats;
      float* part = D + p.wg_d_floats;
      wino_status st = input(p, x, V, s);
      if (st != WINO_OK) return st;
      WgArgs a{};
      a.ystride_k = 1;
      for (int i = 0; i < N; ++i) a.ystride_k *= p.Y[i];
      a.T = int32_t(p.T); a.ntb = int32_t((p.T_pad + 63) / 64); a.nvb = int32_t(p.T_pad / BLK);
      a.K = p.K; a.K_pad4 = p.wg_kpad4; a.C = p.C; a.C_pad = p.C_pad;
      a.nkb = (p.wg_kpad4 + 63) / 64; a.ncb = (p.C_pad + 63) / 64;
      a.nsplit = p.wg_nsplit;
      for (int i = 0; i < 3; ++i) { a.tiles[i] = int32_t(p.tiles[i]); a.Y[i] = int32_t(p.Y[i]); }
      const int64_t nb = int64_t(a.nsplit) * NXI * a.nkb * a.ncb;
      a.nblocks = int32_t(nb);
      const int64_t dy_grid = int64_t(a.ntb) * (a.K_pad4 / 4) * (NXI > 64 ? A : 1);   // k_dy: planes for alpha^N > 64
      hipLaunchKernelGGL((k_dy<N, MM, R, CONST>), dim3(unsigned(dy_grid)), dim3(256), 0, s, dy, D, a, p.fmw);
      hipLaunchKernelGGL((k_wgrad_gemm<BLK>), dim3(unsigned(nb)), dim3(256), 0, s, V, D, part, a, int32_t(NXI));
      const int64_t nkc = int64_t(p.K) * p.C;
      hipLaunchKernelGGL(k_wgrad_sum, dim3(unsigned((nkc * NXI + 255) / 256)), dim3(256), 0, s, part, a,
                         int32_t(NXI));
      const int64_t ntap = nkc * ipow(R, N);
      hipLaunchKernelGGL((k_wgrad_finish<N, MM, R, CONST>), dim3(unsigned((ntap + 255) / 256)), dim3(256), 0, s, part,
                         dw, a, p.fmw);
      return launch_status();
    }
  }

  // Per-XCD work ranges of a pass-accumulating GEMM (k_gemm_acc, k_gemm_acc4):
  // work-groups go to the 8 XCDs round-robin; each XCD takes a contiguous
  // range of blocks, and the plan's tail blocks of each XCD are split into
  // p.nparts parts.  Returns the grid size.
  template <int TB, int KB>
  static int64_t acc_setup(const wino_plan_s& p, AccArgs& a, const float* bias) {
    a.vblock = int64_t(p.nxi) * p.C_pad * TB;
    a.uplane = int64_t(p.C_pad) * p.K_pad;
    a.ystride_k = 1;
    for (int i = 0; i < N; ++i) a.ystride_k *= p.Y[i];
    a.T = int32_t(p.T); a.C_pad = p.C_pad; a.K = p.K; a.K_pad = p.K_pad;
    a.nkb = p.K_pad / KB;
    const int64_t nb = (p.T_pad / TB) * int64_t(a.nkb);
    for (int i = 0; i < 3; ++i) { a.tiles[i] = int32_t(p.tiles[i]); a.Y[i] = int32_t(p.Y[i]); }
    a.relu = (p.flags & WINO_RELU) ? 1 : 0;
    a.bias = bias;
    a.nparts = p.nparts;
    constexpr int NX = 8;
    int64_t maxu = 0, t0 = 0;
    for (int x = 0; x < NX; ++x) {
      const int64_t n = nb / NX + (x < nb % NX ? 1 : 0);
      const int64_t b0 = x * (nb / NX) + (x < nb % NX ? x : nb % NX);
      const int64_t sx = p.nparts > 1 ? p.xtail[x] : 0;
      const int64_t units = n - sx + sx * p.nparts;
      a.xb0[x] = int32_t(b0); a.xn[x] = int32_t(n); a.xs[x] = int32_t(sx); a.xt0[x] = int32_t(t0);
      t0 += sx;
      maxu = maxu > units ? maxu : units;
    }
    return NX * maxu;
  }

  static wino_status gemm(const wino_plan_s& p, const float* V, float* part, const float* U, const float* bias,
                          float* y, hipStream_t s) {
    constexpr int KIND = Blocking<N, MM, R>::KIND;
    if constexpr (KIND == 0) {
      using G = AccGeom<N, MM, R>;
      AccArgs a{};
      // tail blocks: passes split over p.nparts units, whose partial outputs
      // (after V in the workspace) are summed in order
      a.part = part;
      const int64_t grid = acc_setup<G::TB, G::KB>(p, a, bias);
      hipLaunchKernelGGL((k_gemm_acc<N, MM, R, CONST>), dim3(unsigned(grid)), dim3(G::NT), 0, s, V, U, y, a,
                         p.fm);
      if (p.nparts > 1) {
        const int64_t items = p.ntail * ipow(MM, N) * G::TB * G::KB;
        hipLaunchKernelGGL((k_part_reduce<N, MM, G::TB, G::KB>), dim3(unsigned((items + 255) / 256)), dim3(256),
                           0, s, y, a, int32_t(p.ntail));
      }
      return launch_status();
    } else if constexpr (KIND == 1) {
      using G = Acc4Geom<N, MM, R>;
      AccArgs a{};
      a.part = part;
      const int64_t grid = acc_setup<G::TB, G::KB>(p, a, bias);
      hipLaunchKernelGGL((k_gemm_acc4<N, MM, R, CONST>), dim3(unsigned(grid)), dim3(G::NT), 0, s, V, U, y, a,
                         p.fm);
      if (p.nparts > 1) {
        const int64_t items = p.ntail * ipow(MM, N) * G::TB * G::KB;
        hipLaunchKernelGGL((k_part_reduce<N, MM, G::TB, G::KB>), dim3(unsigned((items + 255) / 256)), dim3(256),
                           0, s, y, a, int32_t(p.ntail));
      }
      return launch_status();
    } else {
      using Geo = GemmGeom<N, MM, R, BLK, NW, LOC>;
      GemmArgs g{};
      g.uplane = int64_t(p.C_pad) * p.K_pad;
      g.ystride_k = 1;
      for (int i = 0; i < N; ++i) g.ystride_k *= p.Y[i];
      g.T = int32_t(p.T); g.T_pad = int32_t(p.T_pad);
      g.C_pad = p.C_pad; g.K = p.K; g.K_pad = p.K_pad;
      g.nkb = p.K_pad / BLK;
      const int64_t nb = (p.T_pad / BLK) * int64_t(g.nkb);
      g.nblocks = int32_t(nb);
      for (int i = 0; i < 3; ++i) { g.tiles[i] = int32_t(p.tiles[i]); g.Y[i] = int32_t(p.Y[i]); }
      g.relu = (p.flags & WINO_RELU) ? 1 : 0;
      g.bias = bias;
      hipLaunchKernelGGL((k_gemm_inv<N, MM, R, CONST, BLK, NW, LOC, VEC, DEPTH>), dim3(unsigned(nb)),
                         dim3(Geo::NT), 0, s, V, U, y, g, p.fm);
      return launch_status();
    }
  }
};

template <template <int, int, int, bool> class L, typename F>
wino_status dispatch(const wino_plan_s& p, F&& f) {
#define WINO_CASE(N_, M_, R_)                                            \
  if (p.N == N_ && p.m == M_ && p.r == R_)                               \
    return p.const_mats ? f(L<N_, M_, R_, true>{}) : f(L<N_, M_, R_, false>{});
  WINO_SIZES(WINO_CASE)
#undef WINO_CASE
  return WINO_EUNSUPPORTED;
}

template <int N, int M, int R> void groups_of(int* cg, int* cgu, int* cpad, int* kblk) {
  *cg = Blocking<N, M, R>::CG;
  *cgu = Blocking<N, M, R>::CGU;
  *cpad = Blocking<N, M, R>::CPAD;
  *kblk = Blocking<N, M, R>::KBLK;
}
// Channel groups of the V (cg) and U (cgu) layouts, channel padding multiple
// and kernel padding multiple of an instantiation.
void channel_groups(int N, int m, int r, int* cg, int* cgu, int* cpad, int* kblk) {
  *cg = *cgu = *cpad = *kblk = 1;
#define WINO_GROUPS(N_, M_, R_) \
  if (N == N_ && m == M_ && r == R_) groups_of<N_, M_, R_>(cg, cgu, cpad, kblk);
  WINO_SIZES(WINO_GROUPS)
#undef WINO_GROUPS
}

int block_for(int N, int m, int r) {
#define WINO_BLOCK(N_, M_, R_) \
  if (N == N_ && m == M_ && r == R_) return Blocking<N_, M_, R_>::BLK;
  WINO_SIZES(WINO_BLOCK)
#undef WINO_BLOCK
  return 32;
}

}  // namespace

extern "C" {

wino_status wino_plan(int N, int m, int r, int C, int K, const int64_t* dims, const wino_opts* opts,
                      wino_plan_t** out) {
  if (out == nullptr || dims == nullptr) return WINO_EINVAL;
  if (N < 1 || N > 3 || m < 1 || r < 1 || C < 1 || K < 1) return WINO_EINVAL;
  if (m + r - 1 > kMaxAlpha) return WINO_EUNSUPPORTED;
  if (!supported(N, m, r)) return WINO_EUNSUPPORTED;
  wino_opts o{};
  if (opts) o = *opts;
  if (o.flags & ~(WINO_RELU | WINO_NO_SPLIT)) return WINO_EINVAL;
  const int alpha = m + r - 1;

  wino_plan_s p{};
  p.N = N; p.m = m; p.r = r; p.alpha = alpha; p.C = C; p.K = K;
  p.flags = o.flags;
  p.batch = dims[0];
  if (p.batch < 1 || p.batch > kMaxI32) return WINO_EINVAL;
  int64_t T = p.batch;
  for (int i = 0; i < 3; ++i) { p.X[i] = 1; p.Y[i] = 1; p.tiles[i] = 1; p.pad[i] = 0; }
  for (int i = 0; i < N; ++i) {
    const int64_t X = dims[1 + i];
    const int32_t pad = o.pad[i];
    if (X < 1 || X > kMaxI32 || pad < 0 || pad > 1 << 20) return WINO_EINVAL;
    const int64_t Y = X + 2 * int64_t(pad) - r + 1;
    if (Y < 1) return WINO_EINVAL;
    p.X[i] = X; p.pad[i] = pad; p.Y[i] = Y;
    p.tiles[i] = (Y + m - 1) / m;
    T *= p.tiles[i];
    if (T > kMaxI32) return WINO_EINVAL;
  }
  p.T = T;
  p.blk = block_for(N, m, r);
  p.T_pad = round_up(T, p.blk);
  int cpad = 1, kblk = 1;
  channel_groups(N, m, r, &p.cg, &p.cgu, &cpad, &kblk);
  p.C_pad = int(round_up(C, cpad));   // whole operand stages / channel groups
  {
    int cg_, cgu_, cpad_, kblk_;
    channel_groups(N, m, r, &cg_, &cgu_, &cpad_, &kblk_);
    p.kblk = kblk_;
    p.K_pad = int(round_up(K, kblk_));
  }
  if (p.T_pad > kMaxI32) return WINO_EINVAL;
  if (p.C_pad > (1 << 18)) return WINO_EINVAL;  // bounds the input-transform grid
  p.nxi = 1;
  for (int i = 0; i < N; ++i) p.nxi *= alpha;
  if ((p.T_pad / p.blk) * (p.K_pad / p.blk) > kMaxI32) return WINO_EINVAL;   // GEMM grid
  // workspace: V, then the partial outputs of k_gemm_acc's tail blocks.  The
  // GEMM's 64 x 64 blocks go to the 8 XCDs in contiguous ranges, two
  // resident work-groups per CU; an XCD's blocks past its last full round
  // (all of them when it has less than a round) are its tail.  Each tail
  // block is split into nparts parts by passes (a power of two; at most 8
  // when full rounds precede, since every part writes a whole partial output)
  // so that the tail units still have a CU each: one work-group alone on a CU
  // already runs the MFMA pipes nearly full, so filling the second slot of a
  // CU gains little against the partial outputs' traffic.
  p.v_floats = round_up(int64_t(p.nxi) * p.C_pad * p.T_pad, 64);
  p.nparts = 1;
  p.ntail = 0;
  p.part_floats = 0;
  for (int x = 0; x < 8; ++x) p.xtail[x] = 0;
  const int cus = cu_count();
  const bool acc4 = N == 2 && m == 4 && r == 3;   // k_gemm_acc4: 64 x 32 blocks
  if ((m == 2 || acc4) && !(o.flags & WINO_NO_SPLIT) && cus >= 8) {
    const int kbw = acc4 ? 32 : 64;                 // kernels per block
    const int64_t nb = (p.T_pad / 64) * (p.K_pad / kbw);
    const int64_t sx = 2 * int64_t(cus / 8);        // resident work-groups per XCD
    const int64_t cx = cus / 8;                     // CUs per XCD
    const int npass = p.nxi / 2;
    int64_t rmax = 0;
    bool rounds = false;
    for (int x = 0; x < 8; ++x) {
      const int64_t n = nb / 8 + (x < nb % 8 ? 1 : 0);
      rmax = n % sx > rmax ? n % sx : rmax;
      rounds = rounds || n >= sx;
    }
    const int cap = rounds ? 8 : 32;
    int np = 1;
    if (rmax > 0)
      while (np * 2 <= npass && np * 2 <= cap && rmax * np * 2 <= cx) np *= 2;
    if (np > 1) {
      int nout = 1;
      for (int i = 0; i < N; ++i) nout *= m;
      for (int x = 0; x < 8; ++x) {
        const int64_t n = nb / 8 + (x < nb % 8 ? 1 : 0);
        p.xtail[x] = int32_t(n % sx);
        p.ntail += n % sx;
      }
      p.nparts = np;
      p.part_floats = p.ntail * np * nout * 64 * kbw;
    }
  }
  if ((p.T_pad / p.blk) * (p.C_pad / p.cg) > kMaxI32) return WINO_EINVAL;     // input grid

  // Transform synthesis (a1): exact rationals, one rounding per entry.
  Rat pts[kMaxAlpha];
  int np = alpha - 1;
  bool defaults = false;
  if (o.points == nullptr) {
    if (o.n_points != 0) return WINO_EINVAL;
    int cnt = 0;
    const Rat* d = default_points(m, r, &cnt);
    if (d == nullptr || cnt != np) return WINO_EUNSUPPORTED;
    for (int i = 0; i < np; ++i) pts[i] = d[i];
    defaults = true;
  } else {
    if (o.n_points != np) return WINO_EINVAL;
    for (int i = 0; i < np; ++i)
      if (!rationalize(o.points[i], &pts[i])) return WINO_EINVAL;
    p.n_user_pts = np;
    for (int i = 0; i < np; ++i) p.user_pts[i] = o.points[i];
    int cnt = 0;
    const Rat* d = default_points(m, r, &cnt);
    defaults = d != nullptr && cnt == np;
    for (int i = 0; defaults && i < np; ++i) defaults = eq(d[i], pts[i]);
  }
  const RatMats R = synthesize(m, r, pts);
  if (!R.ok) return WINO_EINVAL;
  for (int i = 0; i < kMaxAlpha; ++i)
    for (int j = 0; j < kMaxAlpha; ++j) {
      p.AT[i][j] = to_f64(R.AT[i][j]);
      p.BT[i][j] = to_f64(R.BT[i][j]);
      p.G[i][j] = to_f64(R.G[i][j]);
    }
  p.fm = to_fmats(R);
  p.const_mats = defaults;
  // weight gradient: F(r, m) on the same points (V in 64- or 16-tile blocks
  // of 4-channel groups: every size)
  {
    p.wgrad_ok = false;
    int cg_, cgu_, cpad_, kblk_;
    channel_groups(N, m, r, &cg_, &cgu_, &cpad_, &kblk_);
    if ((p.blk == 64 || p.blk == 16) && cg_ == 4) {
      const RatMats Rw = synthesize(r, m, pts);
      bool same = Rw.ok;
      for (int i = 0; same && i < alpha; ++i)
        for (int j = 0; same && j < alpha; ++j) same = eq(Rw.BT[i][j], R.BT[i][j]);
      if (same) {
        p.wgrad_ok = true;
        p.fmw = to_fmats(Rw);
        p.wg_kpad4 = int(round_up(K, 4));
        const int64_t nkb = (p.wg_kpad4 + 63) / 64, ncb = (p.C_pad + 63) / 64, ntb = (p.T_pad + 63) / 64;
        const int64_t units = int64_t(p.nxi) * nkb * ncb;
        int64_t ns = (2048 + units - 1) / units;
        ns = ns < ntb ? ns : ntb;
        p.wg_nsplit = int32_t(ns < 1 ? 1 : ns);
        p.wg_d_floats = round_up(int64_t(p.nxi) * p.wg_kpad4 * ntb * 64, 64);
        p.wg_part_floats = int64_t(p.wg_nsplit) * p.nxi * nkb * 64 * ncb * 64;
        if (units * p.wg_nsplit > kMaxI32) p.wgrad_ok = false;                      // product grid
        if (int64_t(K) * C * (p.nxi > r * r * r ? p.nxi : r * r * r) > kMaxI32 * int64_t(256))
          p.wgrad_ok = false;                                                        // sum and tap grids
      }
    }
  }

  wino_plan_s* h = new (std::nothrow) wino_plan_s(p);
  if (h == nullptr) return WINO_EINVAL;
  *out = h;
  return WINO_OK;
}

void wino_destroy(wino_plan_t* plan) { delete plan; }

wino_status wino_plan_describe(const wino_plan_t* p, wino_plan_desc* d) {
  if (p == nullptr || d == nullptr) return WINO_EINVAL;
  std::memset(d, 0, sizeof(*d));
  d->N = p->N; d->m = p->m; d->r = p->r; d->alpha = p->alpha; d->n_xi = p->nxi;
  d->C = p->C; d->K = p->K; d->C_pad = p->C_pad; d->K_pad = p->K_pad;
  d->batch = p->batch;
  for (int i = 0; i < 3; ++i) { d->X[i] = p->X[i]; d->Y[i] = p->Y[i]; d->tiles[i] = p->tiles[i]; }
  d->T = p->T; d->T_pad = p->T_pad;
  d->block_tiles = p->blk;
  d->block_kernels = p->K_pad > 0 ? p->kblk : 0;
  d->channel_group = p->cg;
  d->filter_channel_group = p->cgu;
  d->gemm_parts = p->nparts;
  d->gemm_tail_blocks = p->ntail;
  d->default_points = p->const_mats ? 1 : 0;
  return WINO_OK;
}

size_t wino_filter_bytes(const wino_plan_t* p) {
  return p ? size_t(p->nxi) * size_t(p->C_pad) * size_t(p->K_pad) * sizeof(float) : 0;
}

size_t wino_workspace_bytes(const wino_plan_t* p) {
  return p ? size_t(p->v_floats + p->part_floats) * sizeof(float) : 0;
}

size_t wino_forward_workspace_bytes(const wino_plan_t* p) { return wino_workspace_bytes(p); }

wino_status wino_output_dims(const wino_plan_t* p, int64_t* out) {
  if (p == nullptr || out == nullptr) return WINO_EINVAL;
  out[0] = p->batch;
  out[1] = p->K;
  for (int i = 0; i < p->N; ++i) out[2 + i] = p->Y[i];
  return WINO_OK;
}

wino_status wino_get_matrices(const wino_plan_t* p, double* AT, double* BT, double* G) {
  if (p == nullptr) return WINO_EINVAL;
  const int a = p->alpha;
  if (AT) for (int i = 0; i < p->m; ++i) for (int j = 0; j < a; ++j) AT[i * a + j] = p->AT[i][j];
  if (BT) for (int i = 0; i < a; ++i) for (int j = 0; j < a; ++j) BT[i * a + j] = p->BT[i][j];
  if (G) for (int i = 0; i < a; ++i) for (int j = 0; j < p->r; ++j) G[i * p->r + j] = p->G[i][j];
  return WINO_OK;
}

wino_status wino_transform_filter(const wino_plan_t* p, const float* w, float* U, void* stream) {
  if (p == nullptr || w == nullptr || U == nullptr) return WINO_EINVAL;
  if (!aligned16(w) || !aligned16(U)) return WINO_EINVAL;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  return dispatch<Launch>(*p, [&](auto L) { return decltype(L)::filter(*p, w, U, false, s); });
}

size_t wino_weight_gradient_workspace_bytes(const wino_plan_t* p) {
  if (p == nullptr || !p->wgrad_ok) return 0;
  return size_t(p->v_floats + p->wg_d_floats + p->wg_part_floats) * sizeof(float);
}

wino_status wino_weight_gradient(const wino_plan_t* p, const float* x, const float* dy, float* dw, void* ws,
                                 size_t ws_bytes, void* stream) {
  if (p == nullptr || x == nullptr || dy == nullptr || dw == nullptr || ws == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(dy) || !aligned16(dw) || !aligned16(ws)) return WINO_EINVAL;
  if (!p->wgrad_ok) return WINO_EUNSUPPORTED;
  if (ws_bytes < wino_weight_gradient_workspace_bytes(p)) return WINO_EWORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  float* w = static_cast<float*>(ws);
  return dispatch<Launch>(*p, [&](auto L) { return decltype(L)::wgrad(*p, x, dy, dw, w, s); });
}

wino_status wino_transform_filter_adjoint(const wino_plan_t* p, const float* w, float* U, void* stream) {
  if (p == nullptr || w == nullptr || U == nullptr) return WINO_EINVAL;
  if (!aligned16(w) || !aligned16(U)) return WINO_EINVAL;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  return dispatch<Launch>(*p, [&](auto L) { return decltype(L)::filter(*p, w, U, true, s); });
}

// The adjoint of a layer's correlation (the data gradient, §3.1's eq. (2)
// read backwards): dx[n][c][q] = sum_k sum_p w[k][c][p] dy~[n][k][q - p + pad],
// with dy~ zero outside [0, Y).  Substituting p' = r - 1 - p makes it the
// correlation of dy with the kernel w'[c][k][p'] = w[k][c][r - 1 - p'] and
// padding r - 1 - pad, whose output extent is X again.
wino_status wino_plan_adjoint(const wino_plan_t* f, wino_plan_t** out) {
  if (f == nullptr || out == nullptr) return WINO_EINVAL;
  wino_opts o{};
  for (int i = 0; i < f->N; ++i) {
    if (f->pad[i] > f->r - 1) return WINO_EINVAL;
    o.pad[i] = f->r - 1 - f->pad[i];
  }
  o.points = f->n_user_pts > 0 ? f->user_pts : nullptr;
  o.n_points = f->n_user_pts;
  o.flags = f->flags & WINO_NO_SPLIT;
  int64_t dims[4] = {f->batch, 1, 1, 1};
  for (int i = 0; i < f->N; ++i) dims[1 + i] = f->Y[i];
  return wino_plan(f->N, f->m, f->r, f->K, f->C, dims, &o, out);
}

wino_status wino_transform_input(const wino_plan_t* p, const float* x, void* ws, size_t ws_bytes,
                                 void* stream) {
  if (p == nullptr || x == nullptr || ws == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(ws)) return WINO_EINVAL;
  if (ws_bytes < wino_workspace_bytes(p)) return WINO_EWORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  float* V = static_cast<float*>(ws);
  return dispatch<Launch>(*p, [&](auto L) { return decltype(L)::input(*p, x, V, s); });
}

wino_status wino_gemm_inverse_ex(const wino_plan_t* p, void* ws, size_t ws_bytes, const float* U,
                                 const float* bias, float* y, void* stream) {
  if (p == nullptr || ws == nullptr || U == nullptr || y == nullptr) return WINO_EINVAL;
  if (!aligned16(ws) || !aligned16(U) || !aligned16(y)) return WINO_EINVAL;
  if (bias != nullptr && (reinterpret_cast<uintptr_t>(bias) & 3u) != 0) return WINO_EINVAL;
  if (ws_bytes < wino_workspace_bytes(p)) return WINO_EWORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const float* V = static_cast<const float*>(ws);
  float* part = p->nparts > 1 ? static_cast<float*>(ws) + p->v_floats : nullptr;
  return dispatch<Launch>(*p, [&](auto L) { return decltype(L)::gemm(*p, V, part, U, bias, y, s); });
}

wino_status wino_gemm_inverse(const wino_plan_t* p, void* ws, size_t ws_bytes, const float* U,
                              float* y, void* stream) {
  return wino_gemm_inverse_ex(p, ws, ws_bytes, U, nullptr, y, stream);
}

wino_status wino_forward_ex(const wino_plan_t* p, const float* x, const float* U, const float* bias,
                            float* y, void* ws, size_t ws_bytes, void* stream) {
  if (p == nullptr || x == nullptr || U == nullptr || y == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(U) || !aligned16(y)) return WINO_EINVAL;
  if (bias != nullptr && (reinterpret_cast<uintptr_t>(bias) & 3u) != 0) return WINO_EINVAL;
  if (ws == nullptr) return WINO_EINVAL;
  if (!aligned16(ws)) return WINO_EINVAL;
  if (ws_bytes < wino_workspace_bytes(p)) return WINO_EWORKSPACE;
  wino_status st = wino_transform_input(p, x, ws, ws_bytes, stream);
  if (st != WINO_OK) return st;
  return wino_gemm_inverse_ex(p, ws, ws_bytes, U, bias, y, stream);
}

wino_status wino_forward(const wino_plan_t* p, const float* x, const float* U, float* y, void* ws,
                         size_t ws_bytes, void* stream) {
  return wino_forward_ex(p, x, U, nullptr, y, ws, ws_bytes, stream);
}

wino_status wino_maxpool3d(const int64_t* dims, const int32_t* window, const float* x, float* y,
                           void* stream) {
  if (dims == nullptr || window == nullptr || x == nullptr || y == nullptr) return WINO_EINVAL;
  if (!aligned16(x) || !aligned16(y)) return WINO_EINVAL;
  PoolArgs a{};
  a.lead = dims[0];
  if (a.lead < 1) return WINO_EINVAL;
  int64_t total = a.lead;
  for (int i = 0; i < 3; ++i) {
    if (dims[1 + i] < 1 || dims[1 + i] > kMaxI32 || window[i] < 1) return WINO_EINVAL;
    a.X[i] = int32_t(dims[1 + i]);
    a.p[i] = window[i];
    a.Y[i] = a.X[i] / a.p[i];
    if (a.Y[i] < 1) return WINO_EINVAL;
    total *= a.Y[i];
  }
  a.total = total;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (a.p[2] == 2 && a.X[2] % 4 == 0) {
    // Y_3 = X_3 / 2 is even: whole output pairs, 16-byte aligned input rows
    hipLaunchKernelGGL(k_maxpool3d_pair, dim3(unsigned((total / 2 + 255) / 256)), dim3(256), 0, s, x, y, a);
  } else {
    hipLaunchKernelGGL(k_maxpool3d, dim3(unsigned((total + 255) / 256)), dim3(256), 0, s, x, y, a);
  }
  return launch_status();
}

// Growth of fp32 rounding error through the transforms of a point set
// (§2.2 and §3.3 note that the choice of points trades accuracy): for
// |g|, |d| <= 1 the first-order error of output i of the 1-D algorithm
// A^T [(G g) . (B^T d)] is at most u sum_xi |A^T[i][xi]| |G[xi]|_1 |B^T[xi]|_1,
// against at most r for the direct sum; kappa_1 = max_i of that sum / r, and
// the N-D transforms, products over the axes, give kappa_1^N.
static bool growth_of(int N, int m, int r, const Rat* pts, double* out) {
  const RatMats R = synthesize(m, r, pts);
  if (!R.ok) return false;
  const int a = m + r - 1;
  double k1 = 0.0;
  for (int i = 0; i < m; ++i) {
    double sum = 0.0;
    for (int x = 0; x < a; ++x) {
      double gn = 0.0, bn = 0.0;
      for (int k = 0; k < r; ++k) gn += std::fabs(to_f64(R.G[x][k]));
      for (int j = 0; j < a; ++j) bn += std::fabs(to_f64(R.BT[x][j]));
      sum += std::fabs(to_f64(R.AT[i][x])) * gn * bn;
    }
    k1 = std::fmax(k1, sum / r);
  }
  *out = std::pow(k1, N);
  return true;
}

wino_status wino_points_error_growth(int N, int m, int r, const double* points, int n_points,
                                     double* growth) {
  if (growth == nullptr || N < 1 || N > 3 || m < 1 || r < 1 || m + r - 1 > kMaxAlpha) return WINO_EINVAL;
  const int np = m + r - 2;
  Rat pts[kMaxAlpha];
  if (points == nullptr) {
    int cnt = 0;
    const Rat* d = default_points(m, r, &cnt);
    if (d == nullptr || cnt != np) return WINO_EINVAL;
    for (int i = 0; i < np; ++i) pts[i] = d[i];
  } else {
    if (n_points != np) return WINO_EINVAL;
    for (int i = 0; i < np; ++i)
      if (!rationalize(points[i], &pts[i])) return WINO_EINVAL;
  }
  return growth_of(N, m, r, pts, growth) ? WINO_OK : WINO_EINVAL;
}

wino_status wino_search_points(int N, int m, int r, double* points, double* growth) {
  if (points == nullptr || growth == nullptr || N < 1 || N > 3 || m < 1 || r < 1 ||
      m + r - 1 > kMaxAlpha)
    return WINO_EINVAL;
  const int np = m + r - 2;
  // candidates: 0 (when the count is odd) and pairs +-p, p from a pool of
  // small rationals; every subset of pairs of the right size is tried
  static const Rat pool[] = {{1, 1}, {2, 1}, {1, 2}, {3, 1}, {1, 3}, {3, 2}, {2, 3}, {4, 1}, {1, 4}};
  constexpr int NP = int(sizeof(pool) / sizeof(pool[0]));
  const int pairs = np / 2;
  const bool zero = (np % 2) == 1;
  if (pairs > NP) return WINO_EUNSUPPORTED;
  double best = 0.0;
  bool found = false;
  Rat best_pts[kMaxAlpha];
  for (uint32_t mask = 0; mask < (1u << NP); ++mask) {
    if (__builtin_popcount(mask) != pairs) continue;
    Rat pts[kMaxAlpha];
    int n = 0;
    if (zero) pts[n++] = rat(0);
    for (int i = 0; i < NP; ++i)
      if (mask & (1u << i)) {
        pts[n++] = pool[i];
        pts[n++] = neg(pool[i]);
      }
    double g = 0.0;
    if (!growth_of(N, m, r, pts, &g)) continue;
    // ties go to the earlier subset: pool order prefers small integers
    if (!found || g < best * (1.0 - 1e-12)) {
      best = g;
      found = true;
      for (int i = 0; i < np; ++i) best_pts[i] = pts[i];
    }
  }
  if (!found) return WINO_EUNSUPPORTED;
  for (int i = 0; i < np; ++i) points[i] = to_f64(best_pts[i]);
  *growth = best;
  return WINO_OK;
}

const char* wino_status_string(wino_status s) {
  switch (s) {
    case WINO_OK: return "ok";
    case WINO_EINVAL: return "invalid argument";
    case WINO_EUNSUPPORTED: return "unsupported (N, m, r)";
    case WINO_EWORKSPACE: return "workspace too small";
    case WINO_EDEVICE: return "device launch failed";
  }
  return "unknown status";
}

}  // extern "C"
