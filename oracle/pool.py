"""Max-pool for the C3D stack (oracle; test infrastructure only; not part of
the Winograd method).

Non-overlapping windows equal to the stride, floor rounding: an output of
extent floor(X_i / p_i) per axis, trailing remainders dropped.

Pins (tests/test_oracle_direct.py): equals torch CPU max_pool3d with
ceil_mode=False, and a hand-checked 1x2x2 example.
"""
from __future__ import annotations

import numpy as np


def maxpool(x, window):
    x = np.asarray(x)
    N = len(window)
    lead = x.shape[: x.ndim - N]
    X = x.shape[x.ndim - N:]
    Y = tuple(xi // pi for xi, pi in zip(X, window))
    x = x[(Ellipsis,) + tuple(slice(0, yi * pi) for yi, pi in zip(Y, window))]
    shp = lead
    for yi, pi in zip(Y, window):
        shp = shp + (yi, pi)
    v = x.reshape(shp)
    axes = tuple(len(lead) + 2 * a + 1 for a in range(N))
    return v.max(axis=axes)
