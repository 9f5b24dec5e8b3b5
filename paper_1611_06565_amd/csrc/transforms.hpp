// Separable per-axis transforms on register tiles (eq. 3: the n-mode product).
//
// A tile of extents [E_0]..[E_{N-1}] lives in a flat float array, last axis
// fastest.  Transforming along axis `ax` with an (OUT x IN) matrix replaces
// extent IN by OUT on that axis: eq. (4) applies B^T (data), G (kernel) or
// A^T (inverse) this way along every axis in turn.
//
// Matrices come either as compile-time constants (default interpolation
// points) or from a kernel argument (caller-chosen points).  Zero terms are
// skipped and +-1 terms become plain adds, the GPU counterpart of the paper's
// sparse traversal of the transform matrices (§3.2).  Constant matrices are
// further applied with shared sub-expressions found at compile time (see
// ConstPlan), so the two forms may round differently in the last bits.
#pragma once

#include <type_traits>
#include <utility>

#include "synth.hpp"

namespace wino {

// Which matrix of the triple a transform reads.
enum class Which { AT, BT, G };

template <Which W, bool CONST, int M_, int R_>
struct MatRef {
  static constexpr bool kConst = CONST;
  static constexpr Which kWhich = W;
  static constexpr int kM = M_, kR = R_;
  const FMats* rt;
  __device__ __forceinline__ float operator()(int i, int j) const {
    if constexpr (CONST) {
      if constexpr (W == Which::AT) return kDefaultF<M_, R_>.AT[i][j];
      else if constexpr (W == Which::BT) return kDefaultF<M_, R_>.BT[i][j];
      else return kDefaultF<M_, R_>.G[i][j];
    } else {
      if constexpr (W == Which::AT) return rt->AT[i][j];
      else if constexpr (W == Which::BT) return rt->BT[i][j];
      else return rt->G[i][j];
    }
  }
};

// out = sum_i M(j, i) * in_i, skipping zero coefficients and turning +-1 into
// adds; the first non-zero term initialises the sum.
template <int IN, class Mat>
__device__ __forceinline__ float dot_row(const Mat& M, int j, const float* v, int stride) {
  float acc = 0.0f;
  bool first = true;
#pragma unroll
  for (int i = 0; i < IN; ++i) {
    const float c = M(j, i);
    if (c == 0.0f) continue;
    const float x = v[i * stride];
    if (first) {
      acc = (c == 1.0f) ? x : (c == -1.0f ? -x : c * x);
      first = false;
    } else if (c == 1.0f) {
      acc += x;
    } else if (c == -1.0f) {
      acc -= x;
    } else {
      acc = __builtin_fmaf(c, x, acc);
    }
  }
  return acc;
}

template <Which W, int M_, int R_>
__host__ __device__ constexpr float const_entry(int i, int j) {
  if constexpr (W == Which::AT) return kDefaultF<M_, R_>.AT[i][j];
  else if constexpr (W == Which::BT) return kDefaultF<M_, R_>.BT[i][j];
  else return kDefaultF<M_, R_>.G[i][j];
}

// Compile-time application plan of a constant OUT x IN matrix.
//
// Row pairs: rows o < o2 that agree on the even columns and are opposite on
// the odd ones (the rows of points a and -a in B^T and G) share the even part
// E and the odd part O of row o: out_o = E + O, out_o2 = E - O.
// Column pairs: columns i < i2 whose entries agree up to sign in every row
// (the columns of points a and -a in A^T) are read through s = v_i + v_i2 and
// d = v_i - v_i2, each row taking s or d with the coefficient of column i.
// Every sum starts from a +1 term when there is one (no multiply).
template <Which W, int M_, int R_, int OUT, int IN>
struct ConstPlan {
  static constexpr float c(int o, int i) { return const_entry<W, M_, R_>(o, i); }
  // operands: 0..IN-1 = v_i, IN + i = s of pair (i, i2), 2 IN + i = d
  struct Terms {
    int n = 0;
    float coef[kMaxAlpha] = {};
    int op[kMaxAlpha] = {};
  };
  struct Info {
    int rowp[kMaxAlpha] = {};    // partner row (> o), -1 if none
    bool row2[kMaxAlpha] = {};   // o is the second row of a pair
    int colp[kMaxAlpha] = {};    // partner column (> i), -1 if none
    bool col2[kMaxAlpha] = {};   // i is the second column of a pair
  };
  static constexpr bool rows_pair(int o, int o2) {
    bool odd_nz = false, even_nz = false;
    for (int i = 0; i < IN; ++i) {
      const float a = c(o, i), b = c(o2, i);
      if (i % 2 == 0) {
        if (a != b) return false;
        even_nz = even_nz || a != 0.0f;
      } else {
        if (a != -b) return false;
        odd_nz = odd_nz || a != 0.0f;
      }
    }
    return odd_nz && even_nz;
  }
  static constexpr bool cols_pair(int i, int i2) {
    int plus = 0, minus = 0;
    for (int o = 0; o < OUT; ++o) {
      const float a = c(o, i), b = c(o, i2);
      if (a == 0.0f && b == 0.0f) continue;
      if (a == b) ++plus;
      else if (a == -b) ++minus;
      else return false;
    }
    return plus + minus >= 3;  // at least one add saved
  }
  static constexpr Info make_info() {
    Info f{};
    for (int o = 0; o < kMaxAlpha; ++o) f.rowp[o] = f.colp[o] = -1;
    for (int o = 0; o < OUT; ++o) {
      if (f.row2[o] || f.rowp[o] >= 0) continue;
      for (int o2 = o + 1; o2 < OUT; ++o2)
        if (!f.row2[o2] && f.rowp[o2] < 0 && rows_pair(o, o2)) {
          f.rowp[o] = o2; f.row2[o2] = true;
          break;
        }
    }
    bool any_row = false;
    for (int o = 0; o < OUT; ++o) any_row = any_row || f.rowp[o] >= 0;
    if (!any_row) {
      for (int i = 0; i < IN; ++i) {
        if (f.col2[i] || f.colp[i] >= 0) continue;
        for (int i2 = i + 1; i2 < IN; ++i2)
          if (!f.col2[i2] && f.colp[i2] < 0 && cols_pair(i, i2)) {
            f.colp[i] = i2; f.col2[i2] = true;
            break;
          }
      }
    }
    return f;
  }
  // terms of row o; part 0 = all columns, 1 = even only, 2 = odd only
  static constexpr Terms terms(int o, int part) {
    const Info info = make_info();
    Terms t{};
    for (int i = 0; i < IN; ++i) {
      if (part == 1 && i % 2 != 0) continue;
      if (part == 2 && i % 2 == 0) continue;
      if (info.col2[i]) continue;
      const float a = c(o, i);
      if (a == 0.0f) continue;
      int op = i;
      if (info.colp[i] >= 0) op = (c(o, info.colp[i]) == a ? IN : 2 * IN) + i;
      t.coef[t.n] = a; t.op[t.n] = op; ++t.n;
    }
    // a +1 term first
    for (int k = 1; k < t.n; ++k)
      if (t.coef[k] == 1.0f && t.coef[0] != 1.0f) {
        const float cc = t.coef[0]; const int oo = t.op[0];
        t.coef[0] = t.coef[k]; t.op[0] = t.op[k];
        t.coef[k] = cc; t.op[k] = oo;
        break;
      }
    return t;
  }
};

template <int... I, class F>
__device__ __forceinline__ void unroll_seq(std::integer_sequence<int, I...>, F&& f) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void unroll(F&& f) {
  unroll_seq(std::make_integer_sequence<int, N>{}, f);
}

// One row of a matrix: for a constant matrix the terms of row O (no shared
// sub-expressions), a +1 term first; otherwise dot_row.
template <int IN, int O, class Mat>
__device__ __forceinline__ float row_dot(const Mat& M, const float* v, int vs) {
  if constexpr (Mat::kConst) {
    constexpr auto t = [] {
      typename ConstPlan<Mat::kWhich, Mat::kM, Mat::kR, kMaxAlpha, IN>::Terms r{};
      for (int i = 0; i < IN; ++i) {
        const float a = const_entry<Mat::kWhich, Mat::kM, Mat::kR>(O, i);
        if (a != 0.0f) { r.coef[r.n] = a; r.op[r.n] = i; ++r.n; }
      }
      for (int k = 1; k < r.n; ++k)
        if (r.coef[k] == 1.0f && r.coef[0] != 1.0f) {
          const float cc = r.coef[0]; const int oo = r.op[0];
          r.coef[0] = r.coef[k]; r.op[0] = r.op[k]; r.coef[k] = cc; r.op[k] = oo;
          break;
        }
      return r;
    }();
    float acc = 0.0f;
    unroll<t.n>([&](auto K) {
      constexpr int k = decltype(K)::value;
      constexpr float cf = t.coef[k];
      constexpr int opi = t.op[k];
      const float x = v[opi * vs];
      if constexpr (k == 0) {
        if constexpr (cf == 1.0f) acc = x;
        else if constexpr (cf == -1.0f) acc = -x;
        else acc = cf * x;
      } else if constexpr (cf == 1.0f) {
        acc += x;
      } else if constexpr (cf == -1.0f) {
        acc -= x;
      } else {
        acc = __builtin_fmaf(cf, x, acc);
      }
    });
    return acc;
  } else {
    return dot_row<IN>(M, O, v, vs);
  }
}

// Sum of a compile-time term list over the operand array.
template <class P, int O, int PART>
__device__ __forceinline__ float const_sum(const float* ops) {
  constexpr auto t = P::terms(O, PART);
  float acc = 0.0f;
  unroll<t.n>([&](auto K) {
    constexpr int k = decltype(K)::value;
    constexpr float cf = t.coef[k];
    constexpr int opi = t.op[k];
    const float x = ops[opi];
    if constexpr (k == 0) {
      if constexpr (cf == 1.0f) acc = x;
      else if constexpr (cf == -1.0f) acc = -x;
      else acc = cf * x;
    } else if constexpr (cf == 1.0f) {
      acc += x;
    } else if constexpr (cf == -1.0f) {
      acc -= x;
    } else {
      acc = __builtin_fmaf(cf, x, acc);
    }
  });
  return acc;
}

// out[o * os] = sum_i M(o, i) * v[i * vs] for all o < OUT.
template <int IN, int OUT, class Mat>
__device__ __forceinline__ void apply_vec(const Mat& M, const float* v, int vs, float* out, int os) {
  if constexpr (Mat::kConst) {
    using P = ConstPlan<Mat::kWhich, Mat::kM, Mat::kR, OUT, IN>;
    constexpr auto info = P::make_info();
    float ops[3 * IN];
#pragma unroll
    for (int i = 0; i < IN; ++i) ops[i] = v[i * vs];
    unroll<IN>([&](auto I) {
      constexpr int i = decltype(I)::value;
      if constexpr (info.colp[i] >= 0) {
        constexpr int i2 = info.colp[i];
        ops[IN + i] = ops[i] + ops[i2];
        ops[2 * IN + i] = ops[i] - ops[i2];
      }
    });
    unroll<OUT>([&](auto O) {
      constexpr int o = decltype(O)::value;
      if constexpr (info.rowp[o] >= 0) {
        constexpr int o2 = info.rowp[o];
        const float e = const_sum<P, o, 1>(ops);
        const float d = const_sum<P, o, 2>(ops);
        out[o * os] = e + d;
        out[o2 * os] = e - d;
      } else if constexpr (!info.row2[o]) {
        out[o * os] = const_sum<P, o, 0>(ops);
      }
    });
  } else {
#pragma unroll
    for (int o = 0; o < OUT; ++o) out[o * os] = dot_row<IN>(M, o, v, vs);
  }
}

// src [PRE][IN][POST] -> dst [PRE][OUT][POST], matrix OUT x IN.
template <int PRE, int IN, int OUT, int POST, class Mat>
__device__ __forceinline__ void apply_axis(const float* src, float* dst, const Mat& M) {
#pragma unroll
  for (int p = 0; p < PRE; ++p)
#pragma unroll
    for (int q = 0; q < POST; ++q)
      apply_vec<IN, OUT>(M, src + p * IN * POST + q, POST, dst + p * OUT * POST + q, POST);
}

// Full N-D transform of an [IN]^N tile into [OUT]^N, axis 0 first.
template <int N, int IN, int OUT, class Mat>
__device__ __forceinline__ void transform_nd(const float* src, float* dst, const Mat& M) {
  static_assert(N >= 1 && N <= 3, "N in 1..3");
  if constexpr (N == 1) {
    apply_axis<1, IN, OUT, 1>(src, dst, M);
  } else if constexpr (N == 2) {
    float t[OUT * IN];
    apply_axis<1, IN, OUT, IN>(src, t, M);
    apply_axis<OUT, IN, OUT, 1>(t, dst, M);
  } else {
    float t1[OUT * IN * IN];
    float t2[OUT * OUT * IN];
    apply_axis<1, IN, OUT, IN * IN>(src, t1, M);
    apply_axis<OUT, IN, OUT, IN>(t1, t2, M);
    apply_axis<OUT * OUT, IN, OUT, 1>(t2, dst, M);
  }
}

// 3-D transform with its own matrix per axis (eq. 4's C_n, B_n, A_n):
// [I0][I1][I2] -> [O0][O1][O2], axis 0 first.
template <int I0, int O0, int I1, int O1, int I2, int O2, class M0, class M1, class M2>
__device__ __forceinline__ void transform3_axes(const float* src, float* dst, const M0& a, const M1& b,
                                                const M2& c) {
  float t1[O0 * I1 * I2];
  float t2[O0 * O1 * I2];
  apply_axis<1, I0, O0, I1 * I2>(src, t1, a);
  apply_axis<O0, I1, O1, I2>(t1, t2, b);
  apply_axis<O0 * O1, I2, O2, 1>(t2, dst, c);
}

}  // namespace wino
