"""Weight gradient of a layer (oracle; test infrastructure only).

For y = corr(x, w) of §3.1's eq. (2) without bias and activation, y is linear
in w, and the gradient of a loss with respect to w[k][c][p] collects, over
every sample and output position, the output gradient times the input value
that weight met:

    dw[k][c][p] = sum_n sum_o dy[n][k][o] * x~[n][c][o + p - pad],

with x~ the input zero-extended outside [0, X).  Written here one kernel
offset p at a time as a contraction over (n, o) of dy with the shifted input,
in fp64.  Returns (dw, den) with den = the same sum of |dy| |x~|, the
denominator of the normalised error metric.

Pins (tests/test_oracle_wgrad.py): <dy, corr(x, w)> = <w, dw> with the forward
oracle (y is linear in w); torch's CPU fp64 conv2d_weight / conv3d_weight
(library routines for the same map); and, on tiny inputs, the forward loop-nest
oracle applied to every unit kernel (dw[k][c][p] is the forward response to
the unit kernel at (k, c, p), dotted with dy).
"""
from __future__ import annotations

import itertools

import numpy as np


def direct_wgrad(x, dy, r, pad=0, with_den=True):
    """x [n][C][X..], dy [n][K][Y..] with Y = X + 2 pad - r + 1 ->
    (dw [K][C][r..r], den)."""
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    n, C = x.shape[:2]
    K = dy.shape[1]
    N = x.ndim - 2
    X, Y = x.shape[2:], dy.shape[2:]
    if tuple(Y) != tuple(xx + 2 * pad - r + 1 for xx in X) or dy.shape[0] != n:
        raise ValueError("dy does not have the layer's output shape")
    xp = np.pad(x, [(0, 0), (0, 0)] + [(pad, pad)] * N)
    dw = np.zeros((K, C) + (r,) * N)
    den = np.zeros_like(dw) if with_den else None
    axes = ([0] + list(range(2, 2 + N)),) * 2
    for p in itertools.product(range(r), repeat=N):
        win = xp[(slice(None), slice(None)) + tuple(slice(pi, pi + yi) for pi, yi in zip(p, Y))]
        dw[(slice(None), slice(None)) + p] = np.tensordot(dy, win, axes=axes)
        if with_den:
            den[(slice(None), slice(None)) + p] = np.tensordot(np.abs(dy), np.abs(win), axes=axes)
    return dw, den
