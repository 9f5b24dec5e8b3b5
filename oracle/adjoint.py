"""Data gradient of a layer: the adjoint of the correlation of eq. (2)
(oracle; test infrastructure only).

For y = corr(x, w) of §3.1's eq. (2) without bias and activation, the gradient
of a loss with respect to x is the adjoint map applied to dy = dL/dy: every
input position collects, from each output whose receptive field holds it, the
weight that joined them times that output's gradient,

    dx[n][c][q] = sum_k sum_p w[k][c][p] * dy[n][k][q - p + pad],

over the offsets p with 0 <= q - p + pad < Y.  Written here as it reads from
the forward sum: output o met padded input position o + p through w[k][c][p],
so dy[n][k][o] * w[k][c][p] is scattered back to o + p, one kernel offset at a
time, and the padding border is cut off at the end.  fp64 throughout.

Each function returns (dx, den) with den the same sum of |w| |dy|, the
denominator of the normalised error metric.

Pins (tests/test_oracle_adjoint.py): <corr(x), dy> = <x, adjoint(dy)> with the
forward oracle; the transpose of the forward map's explicit matrix (built
from unit inputs through the loop-nest oracle) on tiny inputs; torch's CPU
fp64 conv_transpose1d/2d/3d (a library routine for the same map); the
sampled form against the full one.
"""
from __future__ import annotations

import itertools

import numpy as np


def in_extent(Y, pad, r):
    """Input extent X of a layer with output extent Y (inverse of Y = X + 2 pad - r + 1)."""
    return tuple(int(y) - 2 * int(pad) + int(r) - 1 for y in Y)


def direct_adjoint(dy, w, pad=0, with_den=True):
    """dy [n][K][Y_1..Y_N], w [K][C][r..r] -> (dx [n][C][X..], den)."""
    dy = np.asarray(dy, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, K = dy.shape[:2]
    C, r = w.shape[1], w.shape[2]
    N = dy.ndim - 2
    Y = dy.shape[2:]
    X = in_extent(Y, pad, r)
    if min(X) < 1:
        raise ValueError("no input extent for these sizes")
    grid = (n, C) + tuple(x + 2 * pad for x in X)       # x zero-extended by pad
    buf = np.zeros(grid)
    mag = np.zeros(grid) if with_den else None
    ady, aw = (np.abs(dy), np.abs(w)) if with_den else (None, None)
    for p in itertools.product(range(r), repeat=N):
        sl = (slice(None), slice(None)) + tuple(slice(pi, pi + yi) for pi, yi in zip(p, Y))
        wp = w[(slice(None), slice(None)) + p]           # [K][C]
        buf[sl] += np.moveaxis(np.tensordot(dy, wp, axes=([1], [0])), -1, 1)
        if with_den:
            mag[sl] += np.moveaxis(np.tensordot(ady, aw[(slice(None), slice(None)) + p], axes=([1], [0])), -1, 1)
    crop = (slice(None), slice(None)) + tuple(slice(pad, pad + x) for x in X)
    return buf[crop], (mag[crop] if with_den else None)


def direct_adjoint_sampled(dy, w, pad, coords):
    """dx and den at coords [M][2 + N] = (n, c, q_1..q_N) only, by the gather
    form of the same sum."""
    dy = np.asarray(dy, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    coords = np.asarray(coords, dtype=np.int64)
    N = dy.ndim - 2
    r = w.shape[2]
    Y = dy.shape[2:]
    b, c, q = coords[:, 0], coords[:, 1], coords[:, 2:]
    out = np.zeros(len(coords))
    den = np.zeros(len(coords))
    for p in itertools.product(range(r), repeat=N):
        src = q - np.asarray(p) + pad                    # output position read
        ok = np.all((src >= 0) & (src < np.asarray(Y)), axis=1)
        s = np.where(ok[:, None], src, 0)
        g = dy[(b[:, None], np.arange(dy.shape[1])[None, :]) + tuple(s[:, i][:, None] for i in range(N))]
        wp = w[(slice(None), c) + p].T                   # [M][K]
        g = np.where(ok[:, None], g, 0.0)
        out += np.sum(g * wp, axis=1)
        den += np.sum(np.abs(g) * np.abs(wp), axis=1)
    return out, den
