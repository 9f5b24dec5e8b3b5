"""Reference N-D Winograd correlation (oracle; test infrastructure only).

Written from §3.2-§4.1, step by step:

1. tile the input: overlapping alpha^N windows stepping by m along each axis
   (§3.3), alpha = m + r - 1; T_i = ceil(Y_i / m) tiles per axis, reads outside
   the zero-padded input are zero;
2. kernel transform  U = g x_1 G x_2 G ... x_N G          (eq. 3 and 4)
3. data transform    V = d x_1 B^T ... x_N B^T            (eq. 4)
4. for every transformed element xi, one matrix product over channels
   M_xi = V_xi [T x C] . U_xi [C x K]                     (eq. 5)
5. inverse transform Y = M x_1 A^T ... x_N A^T            (eq. 4)
6. stitch the m^N output tiles and crop to Y.

The n-mode product is eq. (3): (X x_n U)_{..j..} = sum_{i_n} x_{..i_n..} u_{j,i_n}.

Eq. (4) lets every axis n carry its own transform triple (C_n, B_n, A_n):
``m`` may be one output-tile extent for all axes or a tuple with one per axis,
each axis then using F(m_n, r)'s matrices (default points of F(m_n, r)), its
own tile extent alpha_n = m_n + r - 1 and stride m_n.

Arithmetic is fp64 by default; with ``exact=True`` every array is an object
array of ``fractions.Fraction`` and the result is exact.

Pins (tests/test_oracle_winograd.py): exact agreement with the direct
correlation on small integer inputs for N = 1, 2, 3, every supported (m, r),
ragged tiles and padding; the §2.2 hand example; separability (the N-D
transform equals a Kronecker-product matrix and any axis order gives the same
result); the 2-D case equals A[(C g C^T) . (B d B^T)]A^T of §3.2.
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction

import numpy as np

from .toomcook import default_points, winograd_matrices


def mode_n_product(X, U, n):
    """Eq. (3): contract axis n of X with the columns of U (J x I_n)."""
    U = np.asarray(U)
    out = np.tensordot(X, U, axes=([n], [1]))          # moves the new axis last
    return np.moveaxis(out, -1, n)


def mode_products(X, mats, axes):
    """X x_{axes[0]} mats[0] x_{axes[1]} mats[1] ... (applied in that order)."""
    for U, n in zip(mats, axes):
        X = mode_n_product(X, U, n)
    return X


def matrices(m, r, points=None, exact=False):
    pts = default_points(m, r) if points is None else points
    AT, BT, G = winograd_matrices(m, r, pts)
    if exact:
        cv = lambda M: np.array(M, dtype=object)
    else:
        cv = lambda M: np.array([[float(c) for c in row] for row in M], dtype=np.float64)
    return cv(AT), cv(BT), cv(G)


def _as(x, exact):
    if exact:
        a = np.asarray(x)
        out = np.empty(a.shape, dtype=object)
        flat = out.reshape(-1)
        for i, v in enumerate(a.reshape(-1)):
            flat[i] = Fraction(v) if not isinstance(v, Fraction) else v
        return out
    return np.asarray(x, dtype=np.float64)


def per_axis(m, N):
    """The output-tile extent of every axis: m repeated, or m itself if a tuple."""
    if isinstance(m, (tuple, list)):
        if len(m) != N:
            raise ValueError("one tile extent per axis")
        return tuple(int(v) for v in m)
    return (int(m),) * N


def tile_counts(X, pad, m, r):
    ms = per_axis(m, len(X))
    Y = tuple(xi + 2 * pad - r + 1 for xi in X)
    return Y, tuple(math.ceil(yi / mi) for yi, mi in zip(Y, ms))


def _axis_matrices(m, r, N, points, exact):
    """(A^T, B^T, G) of every axis; a point set applies only to isotropic tiles."""
    ms = per_axis(m, N)
    if points is not None and len(set(ms)) > 1:
        raise ValueError("caller points need the same tile extent on every axis")
    return [matrices(mi, r, points, exact) for mi in ms]


def _extend(x, pad, m, r, exact):
    """Step 1: zero-extended input large enough for every tile window."""
    ms = per_axis(m, x.ndim - 2)
    Y, T = tile_counts(x.shape[2:], pad, m, r)
    if any(yi < 1 for yi in Y):
        raise ValueError("output extent must be positive")
    ext = tuple(ti * mi + r - 1 for ti, mi in zip(T, ms))
    zero = Fraction(0) if exact else 0.0
    xe = np.full(x.shape[:2] + ext, zero, dtype=object if exact else np.float64)
    sl_dst, sl_src = [], []
    for xi, ei in zip(x.shape[2:], ext):
        hi = min(xi, ei - pad)
        sl_dst.append(slice(pad, pad + hi))
        sl_src.append(slice(0, hi))
    xe[(slice(None), slice(None)) + tuple(sl_dst)] = x[(slice(None), slice(None)) + tuple(sl_src)]
    return xe, Y, T


def transform_filter(w, m, r, points=None, exact=False):
    """Step 2: U[k][c] = g x_1 G_1 ... x_N G_N  ->  [K][C][alpha_1..alpha_N]."""
    N = np.ndim(w) - 2
    mats = _axis_matrices(m, r, N, points, exact)
    w = _as(w, exact)
    return mode_products(w, [G for _, _, G in mats], [2 + a for a in range(N)])


def transform_input(x, m, r, pad=0, points=None, exact=False):
    """Steps 1 and 3: V[t][c] = d_t x_1 B_1^T ... x_N B_N^T for every tile t
    (t linear over sample and tile grid, last axis fastest) -> [T][C][alpha_1..]."""
    N = np.ndim(x) - 2
    ms = per_axis(m, N)
    alphas = tuple(mi + r - 1 for mi in ms)
    mats = _axis_matrices(m, r, N, points, exact)
    x = _as(x, exact)
    xe, Y, T = _extend(x, pad, m, r, exact)
    n, C = x.shape[:2]
    tiles = list(itertools.product(range(n), *[range(ti) for ti in T]))
    V = np.empty((len(tiles), C) + alphas, dtype=xe.dtype)
    for ti, t in enumerate(tiles):
        sl = (t[0], slice(None)) + tuple(slice(tj * mi, tj * mi + ai) for tj, mi, ai in zip(t[1:], ms, alphas))
        V[ti] = mode_products(xe[sl], [BT for _, BT, _ in mats], [1 + a for a in range(N)])
    return V


def winograd_forward(x, w, m, r, pad=0, points=None, relu=False, exact=False):
    """Steps 1-6 above.  x: [n][C][X..], w: [K][C][r..] -> y [n][K][Y..]; m is
    one tile extent or one per axis."""
    N = np.ndim(x) - 2
    ms = per_axis(m, N)
    alphas = tuple(mi + r - 1 for mi in ms)
    mats = _axis_matrices(m, r, N, points, exact)
    x = _as(x, exact)
    n = x.shape[0]
    Y, T = tile_counts(x.shape[2:], pad, m, r)
    if any(yi < 1 for yi in Y):
        raise ValueError("output extent must be positive")
    U = transform_filter(w, m, r, points, exact)               # step 2: [K][C][alpha..]
    V = transform_input(x, m, r, pad, points, exact)           # steps 1, 3: [T][C][alpha..]
    K = U.shape[0]
    Tn = V.shape[0]
    tiles = list(itertools.product(range(n), *[range(ti) for ti in T]))

    # Step 4: eq. (5), one [T x C] . [C x K] product per element xi.
    Mt = np.empty((Tn, K) + alphas, dtype=V.dtype)
    for xi in itertools.product(*[range(a) for a in alphas]):
        sel = (slice(None), slice(None)) + xi
        Mt[sel] = np.dot(V[sel], U[sel].T)                   # [T][C] . [C][K]

    # Step 5: inverse transform of every (tile, kernel), A_n^T along axis n.
    S = mode_products(Mt, [AT for AT, _, _ in mats], [2 + a for a in range(N)])   # [T][K][m..]

    # Step 6: stitch and crop.
    full = tuple(ti * mi for ti, mi in zip(T, ms))
    y = np.empty((n, K) + full, dtype=S.dtype)
    for ti, t in enumerate(tiles):
        sl = (t[0], slice(None)) + tuple(slice(tj * mi, tj * mi + mi) for tj, mi in zip(t[1:], ms))
        y[sl] = S[ti]
    y = y[(slice(None), slice(None)) + tuple(slice(0, yi) for yi in Y)]
    if relu:
        zero = Fraction(0) if exact else 0.0
        y = np.where(y > 0, y, zero)
    return y
