// Transform synthesis for F(m, r) in exact rational arithmetic.
//
// §2.1-§2.2: the only input of synthesis is the modulus polynomial
// m(x) = prod_j (x - p_j) over alpha-1 distinct finite points plus the point
// at infinity (alpha = m + r - 1).  Theorem 1 (CRT) turns polynomial
// multiplication modulo m(x) into one product per point; for the valid
// correlation of eq. (2) that yields, in closed form,
//
//   A^T[i][j] = p_j^i                     (j < alpha-1),  A^T[i][alpha-1] = [i == m-1]
//   B^T row j = coefficients of m(x) / (x - p_j), ascending, then 0
//   B^T row alpha-1 = coefficients of m(x), ascending
//   G[j][k]   = p_j^k / prod_{i != j} (p_j - p_i),          G[alpha-1] = e_{r-1}
//
// so that y_i = sum_j A^T[i][j] (G g)_j (B^T d)_j = sum_k g_k d_{i+k}.
// The CRT constant of each reconstruction polynomial sits in G (the cached
// side).  When the x^1 coefficient of m(x) is negative, B^T rows 0 and
// alpha-1, G row 0 and A^T column alpha-1 are negated: a diagonal rescaling
// that leaves the result unchanged and matches the F(2,3) matrices printed in
// §2.2 entry for entry (§3.3's F(4,3) matrices need no flip).
//
// Everything here is constexpr so the default point sets become compile-time
// float constants in the kernels (zero and unit entries fold away), while the
// same code runs on the host for caller-chosen points.
#pragma once

#include <cstdint>
#include <utility>

namespace wino {

constexpr int kMaxAlpha = 8;

// b^e for small non-negative e; iterative (not recursive) so that device
// code can always inline it (constexpr functions serve host and device).
constexpr int ipow(int b, int e) {
  int r = 1;
  for (int i = 0; i < e; ++i) r *= b;
  return r;
}

struct Rat {
  int64_t n = 0, d = 1;  // d > 0, gcd(|n|, d) == 1
};

// Bound on numerators and denominators: keeps every intermediate product of
// the synthesis and the float rounding below inside 128-bit integers.
constexpr int64_t kRatLimit = int64_t(1) << 32;

constexpr Rat rat_norm(__int128 n, __int128 d, bool& ok) {
  if (d == 0) { ok = false; return {}; }
  if (d < 0) { n = -n; d = -d; }
  __int128 a = n < 0 ? -n : n, b = d;
  while (b != 0) { __int128 t = a % b; a = b; b = t; }
  if (a > 1) { n /= a; d /= a; }
  if (n >= kRatLimit || n <= -kRatLimit || d >= kRatLimit) { ok = false; return {}; }
  return {int64_t(n), int64_t(d)};
}
constexpr Rat rat(int64_t n, int64_t d = 1) { bool ok = true; return rat_norm(n, d, ok); }
constexpr Rat add(Rat a, Rat b, bool& ok) {
  return rat_norm(__int128(a.n) * b.d + __int128(b.n) * a.d, __int128(a.d) * b.d, ok);
}
constexpr Rat sub(Rat a, Rat b, bool& ok) {
  return rat_norm(__int128(a.n) * b.d - __int128(b.n) * a.d, __int128(a.d) * b.d, ok);
}
constexpr Rat mul(Rat a, Rat b, bool& ok) {
  return rat_norm(__int128(a.n) * b.n, __int128(a.d) * b.d, ok);
}
constexpr Rat dvd(Rat a, Rat b, bool& ok) {
  return rat_norm(__int128(a.n) * b.d, __int128(a.d) * b.n, ok);
}
constexpr Rat neg(Rat a) { return {-a.n, a.d}; }
constexpr bool eq(Rat a, Rat b) { return a.n == b.n && a.d == b.d; }

constexpr int bitlen(unsigned __int128 v) {
  int b = 0;
  while (v != 0) { ++b; v >>= 1; }
  return b;
}

// Round n/d to the nearest binary floating-point value with MANT significand
// bits, ties to even (exact integer arithmetic; no double rounding).
template <typename F, int MANT>
constexpr F rat_to_fp(Rat q) {
  if (q.n == 0) return F(0);
  const bool negative = q.n < 0;
  const unsigned __int128 n = negative ? (unsigned __int128)(-(__int128)q.n) : (unsigned __int128)q.n;
  const unsigned __int128 d = (unsigned __int128)q.d;
  int s = (MANT - 1) - (bitlen(n) - bitlen(d));  // n*2^s/d in [2^(MANT-2), 2^MANT)
  unsigned __int128 num = 0, den = 0, quo = 0;
  for (int iter = 0; iter < 3; ++iter) {
    num = s >= 0 ? (n << s) : n;
    den = s >= 0 ? d : (d << (-s));
    quo = num / den;
    if (quo < ((unsigned __int128)1 << (MANT - 1))) { ++s; continue; }
    if (quo >= ((unsigned __int128)1 << MANT)) { --s; continue; }
    break;
  }
  const unsigned __int128 rem = num - quo * den;
  if (2 * rem > den || (2 * rem == den && (quo & 1))) ++quo;
  F v = F(uint64_t(quo));
  for (int i = 0; i < s; ++i) v = v * F(0.5);
  for (int i = 0; i < -s; ++i) v = v * F(2);
  return negative ? -v : v;
}
constexpr float to_f32(Rat q) { return rat_to_fp<float, 24>(q); }
constexpr double to_f64(Rat q) { return rat_to_fp<double, 53>(q); }

struct RatMats {
  int m = 0, r = 0, alpha = 0;
  bool ok = false;
  Rat AT[kMaxAlpha][kMaxAlpha] = {};  // m x alpha
  Rat BT[kMaxAlpha][kMaxAlpha] = {};  // alpha x alpha
  Rat G[kMaxAlpha][kMaxAlpha] = {};   // alpha x r
};

// Float copies in the layout the kernels read (row-major, padded to 8x8).
struct FMats {
  float AT[kMaxAlpha][kMaxAlpha];
  float BT[kMaxAlpha][kMaxAlpha];
  float G[kMaxAlpha][kMaxAlpha];
};

constexpr RatMats synthesize(int m, int r, const Rat* pts) {
  RatMats M{};
  M.m = m;
  M.r = r;
  M.alpha = m + r - 1;
  const int alpha = M.alpha, np = alpha - 1;
  if (m < 1 || r < 1 || alpha > kMaxAlpha) return M;
  bool ok = true;
  for (int i = 0; i < np; ++i)
    for (int j = 0; j < i; ++j)
      if (eq(pts[i], pts[j])) return M;  // points must be distinct

  // A^T: powers of the points; the infinity column picks the top output.
  for (int i = 0; i < m; ++i) {
    for (int j = 0; j < np; ++j) {
      Rat p = rat(1);
      for (int e = 0; e < i; ++e) p = mul(p, pts[j], ok);
      M.AT[i][j] = p;
    }
    M.AT[i][np] = rat(i == m - 1 ? 1 : 0);
  }
  // m(x) = prod_j (x - p_j), ascending coefficients c[0..np].
  Rat c[kMaxAlpha + 1] = {};
  c[0] = rat(1);
  for (int j = 0; j < np; ++j) {
    for (int e = j + 1; e >= 1; --e) c[e] = sub(c[e - 1], mul(pts[j], c[e], ok), ok);
    c[0] = neg(mul(pts[j], c[0], ok));
  }
  // B^T rows: m(x)/(x - p_j) by synthetic division; infinity row = m(x).
  for (int j = 0; j < np; ++j) {
    Rat q[kMaxAlpha] = {};
    q[np - 1] = c[np];
    for (int e = np - 1; e >= 1; --e) q[e - 1] = add(c[e], mul(pts[j], q[e], ok), ok);
    for (int e = 0; e < alpha; ++e) M.BT[j][e] = e < np ? q[e] : rat(0);
  }
  for (int e = 0; e < alpha; ++e) M.BT[np][e] = c[e];
  // G rows: powers over the CRT denominator; infinity row picks g_{r-1}.
  for (int j = 0; j < np; ++j) {
    Rat Nj = rat(1);
    for (int i = 0; i < np; ++i)
      if (i != j) Nj = mul(Nj, sub(pts[j], pts[i], ok), ok);
    Rat p = rat(1);
    for (int k = 0; k < r; ++k) {
      M.G[j][k] = dvd(p, Nj, ok);
      p = mul(p, pts[j], ok);
    }
  }
  for (int k = 0; k < r; ++k) M.G[np][k] = rat(k == r - 1 ? 1 : 0);
  // Sign convention of the printed F(2,3) matrices.
  if (np >= 1 && c[1].n < 0) {
    for (int e = 0; e < alpha; ++e) {
      M.BT[0][e] = neg(M.BT[0][e]);
      M.BT[np][e] = neg(M.BT[np][e]);
    }
    for (int k = 0; k < r; ++k) M.G[0][k] = neg(M.G[0][k]);
    for (int i = 0; i < m; ++i) M.AT[i][np] = neg(M.AT[i][np]);
  }
  M.ok = ok;
  return M;
}

constexpr FMats to_fmats(const RatMats& R) {
  FMats F{};
  for (int i = 0; i < kMaxAlpha; ++i)
    for (int j = 0; j < kMaxAlpha; ++j) {
      F.AT[i][j] = to_f32(R.AT[i][j]);
      F.BT[i][j] = to_f32(R.BT[i][j]);
      F.G[i][j] = to_f32(R.G[i][j]);
    }
  return F;
}

// Default interpolation points per (m, r): the first m + r - 2 entries of
// the ladder {0, 1, -1, 2, -2, 1/2, -1/2} (infinity implied).  F(2,3) gets
// the §2.2 set {0, 1, -1}; F(4,3) gets {0, 1, -1, 2, -2} (the §3.3 set
// {0, 1, -1, 1/3, -1/3} is accepted as an explicit choice but loses about an
// order of magnitude of fp32 accuracy in 3-D); F(5,4) and the other alpha = 8
// sizes of Table 1 get all seven.
constexpr int kLadderLen = kMaxAlpha - 1;
constexpr Rat kLadder[kLadderLen] = {{0, 1}, {1, 1}, {-1, 1}, {2, 1}, {-2, 1}, {1, 2}, {-1, 2}};
template <int K, class Seq = std::make_integer_sequence<int, K>> struct LadderPrefix;
template <int K, int... I> struct LadderPrefix<K, std::integer_sequence<int, I...>> {
  static_assert(K >= 1 && K <= kLadderLen, "alpha in 2..8");
  static constexpr Rat pts[K] = {kLadder[I]...};
};
template <int M, int R> struct DefaultPoints : LadderPrefix<M + R - 2> {};

template <int M, int R>
inline constexpr RatMats kDefaultRat = synthesize(M, R, DefaultPoints<M, R>::pts);

template <int M, int R>
inline constexpr FMats kDefaultF = to_fmats(kDefaultRat<M, R>);

// Host helper: the default points for (m, r), or nullptr.
inline const Rat* default_points(int m, int r, int* count) {
  const int k = m + r - 2;
  if (m < 1 || r < 1 || k < 1 || k > kLadderLen) {
    *count = 0;
    return nullptr;
  }
  *count = k;
  return kLadder;
}

}  // namespace wino
