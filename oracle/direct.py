"""Direct N-D correlation, the plain definition of the layer (oracle; test
infrastructure only).

Eq. (2) of §3.1 defines each output as a sum over input channels and kernel
offsets of weight times shifted input, with no kernel flip; the bias b and
activation f are applied around it.  Reading of the index typo inside the
channel sum: the input is channel m of the previous layer.  Outputs cover the
valid extent Y = X + 2 pad - r + 1 (§2.2 gives S = D - G + 1 unpadded), with
x zero-extended outside [0, X).

The activation f of eq. (2) is the identity, ReLU (relu=True) or a leaky
ReLU (leaky=s: v for v > 0, s * v otherwise); the section allows a ReLU or
another non-linear activation for f.

Each function returns (y, den) where den = sum |w| |x| over the same
receptive field (plus |b_k| with a bias), the denominator of the normalised
error metric.  All
arithmetic is fp64 on the exact float32 input values.

Pins (tests/test_oracle_direct.py): the naive loop nest, the per-offset BLAS
form and the sampled form agree, and all equal torch's CPU fp64
conv1d/conv2d/conv3d (an independent library implementation of the same
correlation); the 1-D hand example of §2.2 gives [14, 20].
"""
from __future__ import annotations

import itertools

import numpy as np


def out_extent(X, pad, r):
    return tuple(int(x) + 2 * int(pad) - int(r) + 1 for x in X)


def activate(y, relu=False, leaky=None):
    """f of eq. (2) on an fp64 array (or scalar)."""
    if relu and leaky is not None:
        raise ValueError("one activation at most")
    if relu:
        return np.maximum(y, 0.0)
    if leaky is not None:
        return np.where(y > 0.0, y, float(leaky) * y)
    return y


def direct_naive(x, w, pad=0, relu=False, bias=None, leaky=None):
    """O1: the literal 2N+3 nested loops of eq. (2); tiny inputs only.

    x: [n][C][X_1..X_N], w: [K][C][r..r] -> (y [n][K][Y..], den)."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, C = x.shape[:2]
    K = w.shape[0]
    N = x.ndim - 2
    r = w.shape[2]
    X = x.shape[2:]
    Y = out_extent(X, pad, r)
    y = np.zeros((n, K) + Y)
    den = np.zeros((n, K) + Y)
    for b in range(n):
        for k in range(K):
            for o in itertools.product(*[range(v) for v in Y]):
                acc = 0.0 if bias is None else float(bias[k])
                mag = 0.0 if bias is None else abs(float(bias[k]))
                for c in range(C):
                    for p in itertools.product(range(r), repeat=N):
                        src = tuple(oi + pi - pad for oi, pi in zip(o, p))
                        if all(0 <= s < xs for s, xs in zip(src, X)):
                            v = x[(b, c) + src]
                            acc += w[(k, c) + p] * v
                            mag += abs(w[(k, c) + p]) * abs(v)
                if relu:
                    acc = max(acc, 0.0)
                elif leaky is not None and not acc > 0.0:
                    acc = float(leaky) * acc
                y[(b, k) + o] = acc
                den[(b, k) + o] = mag
    return y, den


def _padded(x, pad):
    N = x.ndim - 2
    return np.pad(x, [(0, 0), (0, 0)] + [(pad, pad)] * N)


def direct_blas(x, w, pad=0, relu=False, bias=None, with_den=True, leaky=None):
    """O2: one fp64 BLAS contraction per kernel offset p in [0, r)^N.

    y[n,k,o] = sum_p sum_c w[k,c,p] x~[n,c,o+p-pad]."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, C = x.shape[:2]
    K = w.shape[0]
    N = x.ndim - 2
    r = w.shape[2]
    Y = out_extent(x.shape[2:], pad, r)
    xp = _padded(x, pad)
    axp = np.abs(xp) if with_den else None
    aw = np.abs(w) if with_den else None
    y = np.zeros((K, n) + Y)
    den = np.zeros((K, n) + Y) if with_den else None
    for p in itertools.product(range(r), repeat=N):
        sl = (slice(None), slice(None)) + tuple(slice(pi, pi + yi) for pi, yi in zip(p, Y))
        win = xp[sl]                                        # [n][C][Y..]
        wk = w[(slice(None), slice(None)) + p]              # [K][C]
        y += np.tensordot(wk, win, axes=([1], [1]))         # [K][n][Y..]
        if with_den:
            den += np.tensordot(aw[(slice(None), slice(None)) + p], axp[sl], axes=([1], [1]))
    y = np.moveaxis(y, 0, 1)
    if with_den:
        den = np.moveaxis(den, 0, 1)
    if bias is not None:
        b = np.asarray(bias, dtype=np.float64).reshape((1, K) + (1,) * N)
        y = y + b
        if with_den:
            den = den + np.abs(b)
    return activate(y, relu, leaky), den


def direct_sampled(x, w, pad, coords, relu=False, chunk=2048, bias=None, leaky=None):
    """O3: outputs at selected positions only, one receptive field at a time.

    coords: int array [S][2+N] of (n, k, o_1..o_N).  Returns (y [S], den [S])."""
    x = np.asarray(x)
    w = np.asarray(w)
    coords = np.asarray(coords, dtype=np.int64)
    N = x.ndim - 2
    r = w.shape[2]
    X = x.shape[2:]
    offs = np.array(list(itertools.product(range(r), repeat=N)), dtype=np.int64)  # [P][N]
    ys, dens = [], []
    for s0 in range(0, len(coords), chunk):
        cc = coords[s0:s0 + chunk]
        src = cc[:, None, 2:] + offs[None, :, :] - pad                              # [S][P][N]
        inside = np.all((src >= 0) & (src < np.array(X)[None, None, :]), axis=2)     # [S][P]
        srcc = np.where(inside[..., None], src, 0)
        idx = (cc[:, 0][:, None, None], np.arange(x.shape[1])[None, :, None]) + tuple(
            srcc[:, None, :, a] for a in range(N))
        xv = x[idx].astype(np.float64) * inside[:, None, :]                          # [S][C][P]
        wv = w.reshape(w.shape[0], w.shape[1], -1)[cc[:, 1]].astype(np.float64)     # [S][C][P]
        yv = np.einsum("scp,scp->s", xv, wv)
        dv = np.einsum("scp,scp->s", np.abs(xv), np.abs(wv))
        if bias is not None:
            bv = np.asarray(bias, dtype=np.float64)[cc[:, 1]]
            yv = yv + bv
            dv = dv + np.abs(bv)
        ys.append(activate(yv, relu, leaky))
        dens.append(dv)
    return np.concatenate(ys), np.concatenate(dens)
