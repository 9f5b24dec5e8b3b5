// Separable per-axis transforms on register tiles (eq. 3: the n-mode product).
//
// A tile of extents [E_0]..[E_{N-1}] lives in a flat float array, last axis
// fastest.  Transforming along axis `ax` with an (OUT x IN) matrix replaces
// extent IN by OUT on that axis: eq. (4) applies B^T (data), G (kernel) or
// A^T (inverse) this way along every axis in turn.
//
// Matrices come either as compile-time constants (default interpolation
// points: zero terms vanish and +-1 terms become plain adds at compile time,
// the GPU counterpart of the paper's sparse traversal of the transform
// matrices, §3.2) or from a kernel argument for caller-chosen points.  Both
// forms run the same sequence of operations, so they round identically.
#pragma once

#include "synth.hpp"

namespace wino {

// Iterative (not recursive) so that device code can always inline it.
__host__ __device__ constexpr int ipow(int b, int e) {
  int r = 1;
  for (int i = 0; i < e; ++i) r *= b;
  return r;
}

// Which matrix of the triple a transform reads.
enum class Which { AT, BT, G };

template <Which W, bool CONST, int M_, int R_>
struct MatRef {
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

// src [PRE][IN][POST] -> dst [PRE][OUT][POST], matrix OUT x IN.
template <int PRE, int IN, int OUT, int POST, class Mat>
__device__ __forceinline__ void apply_axis(const float* src, float* dst, const Mat& M) {
#pragma unroll
  for (int p = 0; p < PRE; ++p)
#pragma unroll
    for (int q = 0; q < POST; ++q)
#pragma unroll
      for (int j = 0; j < OUT; ++j)
        dst[(p * OUT + j) * POST + q] = dot_row<IN>(M, j, src + p * IN * POST + q, POST);
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

}  // namespace wino
