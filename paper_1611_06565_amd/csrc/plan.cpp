// libwino host side: plan construction, size queries, transform synthesis,
// accuracy queries and argument checks behind the C ABI of include/wino.h.
// No device code and no HIP headers: every size, byte count and launch grid
// is computed here in 64-bit integers with overflow checks before anything
// is narrowed, and a plan whose numbers do not fit is refused.
#include "plan.hpp"

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>

#include "layout.hpp"
#include "synth.hpp"

using namespace wino;

namespace {

constexpr int64_t kMaxI32 = 0x7fffffff;
constexpr int64_t kMaxChannels = int64_t(1) << 20;   // C and K
constexpr int64_t kMaxPad = int64_t(1) << 20;
constexpr int64_t kMaxFloats = int64_t(1) << 60;     // any tensor or workspace, in floats
constexpr int64_t kMaxLaunch = (int64_t(1) << 32) - 1;   // work-items per grid axis

// a * b, false on signed overflow or a negative operand.
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  return !__builtin_mul_overflow(a, b, out);
}
bool mul3_ok(int64_t a, int64_t b, int64_t c, int64_t* out) {
  int64_t t = 0;
  return mul_ok(a, b, &t) && mul_ok(t, c, out);
}
// ceil(a / b) for a >= 0, b > 0 (no overflow: a < 2^63).
int64_t cdiv(int64_t a, int64_t b) { return a / b + (a % b != 0 ? 1 : 0); }
// a rounded up to a multiple of b, false on overflow.
bool round_up(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b <= 0) return false;
  return mul_ok(cdiv(a, b), b, out);
}
// A grid of `groups` work-groups of `threads` work-items fits one launch.
bool grid_ok(int64_t groups, int threads, uint32_t* out) {
  int64_t items = 0;
  if (groups < 0 || groups > kMaxI32 || !mul_ok(groups, threads, &items) || items > kMaxLaunch) return false;
  *out = uint32_t(groups);
  return true;
}

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


bool traits_of(int N, int m, int r, SizeTraits* t) {
#define WINO_TRAITS(N_, M_, R_)                    \
  if (N == N_ && m == M_ && r == R_) {             \
    *t = size_traits<N_, M_, R_>();                \
    return true;                                   \
  }
  WINO_SIZES(WINO_TRAITS)
#undef WINO_TRAITS
  if (N == 3 && m == 5 && r == 4) { *t = size_traits_a8<5, 4>(); return true; }
  if (N == 3 && m == 4 && r == 5) { *t = size_traits_a8<4, 5>(); return true; }
  if (N == 3 && m == 3 && r == 6) { *t = size_traits_a8<3, 6>(); return true; }
  return false;
}

// Tail split and per-XCD ranges of a pass-accumulating product (k_gemm_acc,
// k_gemm_acc4) over nb blocks.  Work-groups reach the 8 XCDs round-robin and
// each XCD takes a contiguous range of blocks; two work-groups are resident
// per CU.  An XCD's blocks past its last full round (all of them when it has
// less than a round) are its tail.  Each tail block is split into nparts
// parts by passes (a power of two; at most 8 when full rounds precede, since
// every part writes a whole partial output) so that the tail units still
// have a CU each: one work-group alone on a CU already runs the MFMA pipes
// nearly full, so filling the second slot of a CU gains little against the
// partial outputs' traffic.
bool acc_geometry(wino_plan_s& p, const SizeTraits& t, bool split, int cus) {
  const int64_t nb = (p.T_pad / t.TB) * (p.K_pad / t.KB);
  p.nparts = 1;
  p.ntail = 0;
  p.part_floats = 0;
  for (int x = 0; x < 8; ++x) p.xtail[x] = 0;
  if (split && cus >= 8) {
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
      const int nout = ipow(p.m, p.N);
      for (int x = 0; x < 8; ++x) {
        const int64_t n = nb / 8 + (x < nb % 8 ? 1 : 0);
        p.xtail[x] = int32_t(n % sx);
        p.ntail += n % sx;
      }
      p.nparts = np;
      if (!mul3_ok(p.ntail * np, int64_t(nout), int64_t(t.TB) * t.KB, &p.part_floats)) return false;
    }
  }
  int64_t maxu = 0, t0 = 0;
  for (int x = 0; x < 8; ++x) {
    const int64_t n = nb / 8 + (x < nb % 8 ? 1 : 0);
    const int64_t b0 = x * (nb / 8) + (x < nb % 8 ? x : nb % 8);
    const int64_t sx = p.nparts > 1 ? p.xtail[x] : 0;
    const int64_t units = n - sx + sx * p.nparts;
    if (b0 > kMaxI32 || n > kMaxI32 || t0 > kMaxI32) return false;
    p.acc_xb0[x] = int32_t(b0); p.acc_xn[x] = int32_t(n); p.acc_xs[x] = int32_t(sx); p.acc_xt0[x] = int32_t(t0);
    t0 += sx;
    maxu = maxu > units ? maxu : units;
  }
  if (!grid_ok(8 * maxu, 256, &p.grid_gemm)) return false;
  p.grid_reduce = 0;
  if (p.nparts > 1) {
    int64_t items = 0;
    if (!mul3_ok(p.ntail, int64_t(ipow(p.m, p.N)), int64_t(t.TB) * t.KB, &items)) return false;
    if (!grid_ok(cdiv(items, 256), 256, &p.grid_reduce)) return false;
  }
  return true;
}

// Weight-gradient geometry (F(r, m) on the forward's points, V reused): the
// transformed output gradients D, the partial products of the tile ranges
// and the grids of its four kernels.  Leaves wgrad_ok false when F(r, m)'s
// data transform differs from the forward's or a grid does not fit.
void wgrad_geometry(wino_plan_s& p, const SizeTraits& t, const Rat* pts, const RatMats& R) {
  p.wgrad_ok = false;
  if (!((t.BLK == 64 || t.BLK == 16) && t.CG == 4)) return;
  if (t.KIND == 4) return;   // the 3-D alpha = 8 sizes have no weight gradient
  const RatMats Rw = synthesize(p.r, p.m, pts);
  bool same = Rw.ok;
  for (int i = 0; same && i < p.alpha; ++i)
    for (int j = 0; same && j < p.alpha; ++j) same = eq(Rw.BT[i][j], R.BT[i][j]);
  if (!same) return;
  int64_t kpad4 = 0;
  if (!round_up(p.K, 4, &kpad4)) return;
  p.fmw = to_fmats(Rw);
  p.wg_kpad4 = int32_t(kpad4);
  const int64_t nkb = cdiv(kpad4, 64), ncb = cdiv(p.C_pad, 64), ntb = cdiv(p.T_pad, 64);
  const int64_t units = int64_t(p.nxi) * nkb * ncb;
  int64_t ns = cdiv(2048, units);
  ns = ns < ntb ? ns : ntb;
  p.wg_nsplit = int32_t(ns < 1 ? 1 : ns);
  int64_t dfl = 0, pfl = 0, t1 = 0;
  if (!mul3_ok(int64_t(p.nxi), kpad4, ntb, &t1) || !mul_ok(t1, 64, &t1) || !round_up(t1, 64, &dfl)) return;
  if (!mul3_ok(int64_t(p.wg_nsplit), int64_t(p.nxi), nkb * 64, &t1) || !mul_ok(t1, ncb * 64, &pfl)) return;
  if (dfl > kMaxFloats || pfl > kMaxFloats) return;
  p.wg_d_floats = dfl;
  p.wg_part_floats = pfl;
  int64_t g = 0;
  if (!mul3_ok(ntb, kpad4 / 4, int64_t(p.nxi > 64 ? p.alpha : 1), &g) || !grid_ok(g, 256, &p.grid_dy)) return;
  if (!mul_ok(units, p.wg_nsplit, &g) || !grid_ok(g, 256, &p.grid_wgemm)) return;
  if (!mul3_ok(int64_t(p.K), int64_t(p.C), int64_t(p.nxi), &g) || !grid_ok(cdiv(g, 256), 256, &p.grid_wsum)) return;
  if (!mul3_ok(int64_t(p.K), int64_t(p.C), int64_t(ipow(p.r, p.N)), &g) ||
      !grid_ok(cdiv(g, 256), 256, &p.grid_wfin))
    return;
  p.wgrad_ok = true;
}

// Growth of fp32 rounding error through the transforms of a point set
// (§2.2 and §3.3 note that the choice of points trades accuracy): for
// |g|, |d| <= 1 the first-order error of output i of the 1-D algorithm
// A^T [(G g) . (B^T d)] is at most u sum_xi |A^T[i][xi]| |G[xi]|_1 |B^T[xi]|_1,
// against at most r for the direct sum; kappa_1 = max_i of that sum / r, and
// the N-D transforms, products over the axes, give kappa_1^N.
bool growth_of(int N, int m, int r, const Rat* pts, double* out) {
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

}  // namespace

namespace wino {

wino_status pool_geometry(const int64_t* dims, const int32_t* window, PoolGeom* g) {
  if (dims == nullptr || window == nullptr || g == nullptr) return WINO_EINVAL;
  PoolGeom q{};
  q.lead = dims[0];
  if (q.lead < 1) return WINO_EINVAL;
  int64_t total = q.lead, in = q.lead;
  for (int i = 0; i < 3; ++i) {
    if (dims[1 + i] < 1 || dims[1 + i] > kMaxI32 || window[i] < 1) return WINO_EINVAL;
    q.X[i] = int32_t(dims[1 + i]);
    q.p[i] = window[i];
    q.Y[i] = q.X[i] / q.p[i];
    if (q.Y[i] < 1) return WINO_EINVAL;
    if (!mul_ok(total, q.Y[i], &total) || !mul_ok(in, q.X[i], &in)) return WINO_EINVAL;
  }
  if (in > kMaxFloats) return WINO_EINVAL;   // input offsets stay far inside int64
  q.total = total;
  q.pair = q.p[2] == 2 && q.X[2] % 4 == 0;   // Y_3 even: whole output pairs, 16-byte aligned rows
  if (!grid_ok(cdiv(q.pair ? total / 2 : total, 256), 256, &q.grid)) return WINO_EINVAL;
  *g = q;
  return WINO_OK;
}

}  // namespace wino

extern "C" {

wino_status wino_plan(int N, int m, int r, int C, int K, const int64_t* dims, const wino_opts* opts,
                      wino_plan_t** out) {
  if (out == nullptr || dims == nullptr) return WINO_EINVAL;
  if (N < 1 || N > 3 || m < 1 || r < 1 || C < 1 || K < 1) return WINO_EINVAL;
  if (C > kMaxChannels || K > kMaxChannels) return WINO_EINVAL;
  if (m + r - 1 > kMaxAlpha) return WINO_EUNSUPPORTED;
  wino_opts o{};
  if (opts) o = *opts;
  if (o.flags & ~(WINO_RELU | WINO_NO_SPLIT | WINO_LEAKY_RELU | WINO_NO_FUSE)) return WINO_EINVAL;
  if ((o.flags & WINO_RELU) && (o.flags & WINO_LEAKY_RELU)) return WINO_EINVAL;
  if ((o.flags & WINO_LEAKY_RELU) && !std::isfinite(o.slope)) return WINO_EINVAL;
  // per-axis output tiles (eq. 4): tile[i] = 0 keeps m
  int ms[3] = {1, 1, 1};
  bool aniso = false;
  for (int i = 0; i < 3; ++i) {
    if (o.tile[i] < 0 || o.tile[i] > kMaxAlpha || (i >= N && o.tile[i] != 0)) return WINO_EINVAL;
    if (i < N) ms[i] = o.tile[i] != 0 ? o.tile[i] : m;
    aniso = aniso || (i < N && ms[i] != ms[0]);
  }
  if (!aniso) m = ms[0];   // the same tile on every axis: an isotropic plan of that m
  if (m + r - 1 > kMaxAlpha) return WINO_EUNSUPPORTED;
  SizeTraits t{};
  if (aniso) {
    // compiled: 3-D, r = 3, F(m0, 3) on axis 0 and F(m1, 3) on axes 1 and 2,
    // {m0, m1} = {2, 4}; each axis takes its F(m, r)'s default points
    if (N != 3 || r != 3 || ms[1] != ms[2] || ms[0] == ms[1]) return WINO_EUNSUPPORTED;
    if (ms[0] == 2 && ms[1] == 4) t = size_traits_ax<2, 4, 3>();
    else if (ms[0] == 4 && ms[1] == 2) t = size_traits_ax<4, 2, 3>();
    else return WINO_EUNSUPPORTED;
    if (o.points != nullptr || o.n_points != 0) return WINO_EINVAL;
  } else if (!traits_of(N, m, r, &t)) {
    return WINO_EUNSUPPORTED;
  }
  const int alpha = aniso ? 0 : m + r - 1;

  wino_plan_s p{};
  p.N = N; p.m = m; p.r = r; p.alpha = alpha; p.C = C; p.K = K;
  p.aniso = aniso;
  for (int i = 0; i < 3; ++i) {
    p.mv[i] = ms[i];
    p.av[i] = i < N ? ms[i] + r - 1 : 1;
  }
  p.flags = o.flags;
  p.slope = (o.flags & WINO_LEAKY_RELU) ? o.slope : 0.0f;
  p.kind = t.KIND;
  p.batch = dims[0];
  if (p.batch < 1 || p.batch > kMaxI32) return WINO_EINVAL;
  int64_t T = p.batch;
  int64_t xin = int64_t(C) * p.batch, yout = int64_t(K) * p.batch;
  for (int i = 0; i < 3; ++i) { p.X[i] = 1; p.Y[i] = 1; p.tiles[i] = 1; p.pad[i] = 0; }
  for (int i = 0; i < N; ++i) {
    const int64_t X = dims[1 + i];
    const int32_t pad = o.pad[i];
    if (X < 1 || X > kMaxI32 || pad < 0 || pad > kMaxPad) return WINO_EINVAL;
    const int64_t Y = X + 2 * int64_t(pad) - r + 1;
    if (Y < 1 || Y > kMaxI32) return WINO_EINVAL;
    p.X[i] = X; p.pad[i] = pad; p.Y[i] = Y;
    p.tiles[i] = (Y + ms[i] - 1) / ms[i];
    T *= p.tiles[i];                          // < 2^31 * 2^31: no overflow before the check
    if (T > kMaxI32) return WINO_EINVAL;
    if (!mul_ok(xin, X, &xin) || !mul_ok(yout, Y, &yout)) return WINO_EINVAL;
  }
  if (xin > kMaxFloats || yout > kMaxFloats) return WINO_EINVAL;
  p.T = T;
  p.blk = t.BLK;
  p.kblk = t.KBLK;
  p.cg = t.CG;
  p.cgu = t.CGU;
  p.nxi = t.NXI;
  int64_t tpad = 0, cpad = 0, kpad = 0;
  if (!round_up(T, p.blk, &tpad) || tpad > kMaxI32) return WINO_EINVAL;
  if (!round_up(C, t.CPAD, &cpad) || !round_up(K, t.KBLK, &kpad)) return WINO_EINVAL;
  p.T_pad = tpad;
  p.C_pad = int(cpad);   // <= 2^20 + 15: whole operand stages / channel groups
  p.K_pad = int(kpad);

  // byte counts: U and V, then the workspace (V rounded up to 256 bytes,
  // then the partial outputs of the product's tail blocks)
  int64_t uf = 0, vf = 0;
  if (!mul3_ok(int64_t(p.nxi), cpad, kpad, &uf) || uf > kMaxFloats) return WINO_EINVAL;
  if (!mul3_ok(int64_t(p.nxi), cpad, tpad, &vf) || !round_up(vf, 64, &p.v_floats) || p.v_floats > kMaxFloats)
    return WINO_EINVAL;

  // launch grids (k_filter_a8: one thread per (channel, kernel, first-axis plane))
  if (!grid_ok(cdiv(cpad * kpad * (t.KIND == 4 ? t.A : 1), 64), 64, &p.grid_filter)) return WINO_EINVAL;
  const int64_t groups = cpad / p.cg;
  int64_t ig = 0;
  if (aniso) {
    // k_input_ax: one V block per work-group, alpha0 waves
    if (!mul_ok(tpad / p.blk, groups, &ig) || !grid_ok(ig, p.av[0] * 64, &p.grid_input)) return WINO_EINVAL;
  } else if (t.KIND == 4) {
    // k_input_a8: half a V block (8 tiles x one channel group) per work-group
    if (!mul_ok(tpad / p.blk, 2 * groups, &ig) || !grid_ok(ig, 256, &p.grid_input)) return WINO_EINVAL;
  } else if (p.nxi > 64) {
    // k_input_split: one V block (BLK tiles x one channel group) per work-group
    if (!mul_ok(tpad / p.blk, groups, &ig) || !grid_ok(ig, alpha * 64, &p.grid_input)) return WINO_EINVAL;
  } else {
    // k_input: 256 threads over BLK tiles x 256 / (BLK * CG) channel groups
    const int64_t gpw = 256 / (int64_t(p.blk) * p.cg);
    if (!mul_ok(tpad / p.blk, cdiv(groups, gpw), &ig) || !grid_ok(ig, 256, &p.grid_input)) return WINO_EINVAL;
  }
  p.gemm_nkb = int32_t(kpad / t.KB);
  if (t.KIND == 0 || t.KIND == 1) {
    if (!acc_geometry(p, t, !(o.flags & WINO_NO_SPLIT), device_cu_count())) return WINO_EINVAL;
  } else {
    // k_gemm_inv, k_gemm_ax, k_gemm_a8: one (tile block, kernel block) per
    // work-group, up to 12 waves (16 for k_gemm_a8)
    p.nparts = 1;
    p.grid_reduce = 0;
    int64_t gg = 0;
    if (!mul_ok(tpad / p.blk, kpad / t.KB, &gg) || !grid_ok(gg, t.KIND == 4 ? 1024 : 768, &p.grid_gemm))
      return WINO_EINVAL;
    // k_gemm_inv (3-D), k_gemm_ax and k_gemm_a8 read a wave's U operands of a
    // stage through one buffer resource: the byte offsets of its element
    // planes of C_pad x K_pad floats (at most 18; 4 for k_gemm_a8), plus the
    // lane's, stay below 2^32
    const bool buffered = (t.KIND == 2 && N == 3) || t.KIND == 3;
    if (buffered && (int64_t(18) * cpad * kpad + 4 * kpad + 64) * 4 >= (int64_t(1) << 32)) return WINO_EINVAL;
    if (t.KIND == 4 && (int64_t(4) * cpad * kpad + 4 * kpad + 64) * 4 >= (int64_t(1) << 32)) return WINO_EINVAL;
  }
  if (p.v_floats + p.part_floats > kMaxFloats) return WINO_EINVAL;
  // F(4^3) with few kernels: the input transform runs inside the product
  // (recomputed for each block of 16 kernels, so only while there are at
  // most 4 such blocks); same grid as k_gemm_inv
  // (its offsets inside one channel's input volume and into U are 32-bit)
  // (k_fused43 reads U from one buffer base per chunk: element offsets of up
  // to 182 planes of C_pad x K_pad floats stay below 2^32 bytes)
  p.fused = !aniso && N == 3 && m == 4 && r == 3 && p.K_pad <= 64 && !(o.flags & WINO_NO_FUSE) &&
            p.X[0] * p.X[1] * p.X[2] <= kMaxI32 && uf <= kMaxI32 &&
            (int64_t(182) * cpad * kpad + 4 * kpad + 64) * 4 < (int64_t(1) << 32);
  if (p.fused && !grid_ok(int64_t(p.T_pad / p.blk) * (p.K_pad / 16), 768, &p.grid_fused)) return WINO_EINVAL;

  if (aniso) {
    // every axis uses its F(m, r)'s default points, compiled into the kernels
    p.const_mats = true;
    p.wgrad_ok = false;
    wino_plan_s* h = new (std::nothrow) wino_plan_s(p);
    if (h == nullptr) return WINO_EINVAL;
    *out = h;
    return WINO_OK;
  }

  // Transform synthesis (a1): exact rationals, one rounding per entry.
  Rat pts[kMaxAlpha];
  const int np = alpha - 1;
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
  wgrad_geometry(p, t, pts, R);

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
  d->block_kernels = p->kblk;
  d->channel_group = p->cg;
  d->filter_channel_group = p->cgu;
  d->gemm_parts = p->nparts;
  d->gemm_tail_blocks = p->ntail;
  d->default_points = p->const_mats ? 1 : 0;
  d->fused = p->fused ? 1 : 0;
  for (int i = 0; i < 3; ++i) { d->tile[i] = p->mv[i]; d->alpha_axis[i] = p->av[i]; }
  return WINO_OK;
}

size_t wino_filter_bytes(const wino_plan_t* p) {
  return p ? size_t(p->nxi) * size_t(p->C_pad) * size_t(p->K_pad) * sizeof(float) : 0;
}

size_t wino_workspace_bytes(const wino_plan_t* p) {
  return p ? size_t(p->v_floats + p->part_floats) * sizeof(float) : 0;
}

size_t wino_forward_workspace_bytes(const wino_plan_t* p) {
  if (p == nullptr) return 0;
  return p->fused ? 0 : wino_workspace_bytes(p);
}

size_t wino_weight_gradient_workspace_bytes(const wino_plan_t* p) {
  if (p == nullptr || !p->wgrad_ok) return 0;
  return size_t(p->v_floats + p->wg_d_floats + p->wg_part_floats) * sizeof(float);
}

wino_status wino_output_dims(const wino_plan_t* p, int64_t* out) {
  if (p == nullptr || out == nullptr) return WINO_EINVAL;
  out[0] = p->batch;
  out[1] = p->K;
  for (int i = 0; i < p->N; ++i) out[2 + i] = p->Y[i];
  return WINO_OK;
}

wino_status wino_get_matrices(const wino_plan_t* p, double* AT, double* BT, double* G) {
  if (p == nullptr) return WINO_EINVAL;
  if (p->aniso) return WINO_EUNSUPPORTED;   // one triple per axis
  const int a = p->alpha;
  if (AT) for (int i = 0; i < p->m; ++i) for (int j = 0; j < a; ++j) AT[i * a + j] = p->AT[i][j];
  if (BT) for (int i = 0; i < a; ++i) for (int j = 0; j < a; ++j) BT[i * a + j] = p->BT[i][j];
  if (G) for (int i = 0; i < a; ++i) for (int j = 0; j < p->r; ++j) G[i * p->r + j] = p->G[i][j];
  return WINO_OK;
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
  if (f->aniso)
    for (int i = 0; i < f->N; ++i) o.tile[i] = f->mv[i];
  int64_t dims[4] = {f->batch, 1, 1, 1};
  for (int i = 0; i < f->N; ++i) dims[1 + i] = f->Y[i];
  return wino_plan(f->N, f->m, f->r, f->K, f->C, dims, &o, out);
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
