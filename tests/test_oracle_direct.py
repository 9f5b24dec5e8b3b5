"""Pins for the direct correlation (oracle/direct.py) and max-pool (oracle/pool.py).

The naive loop nest, the per-offset BLAS form and the sampled form must
agree with each other and with torch's CPU fp64 convNd (an independent
library implementation of the same cross-correlation); the 1-D hand example
of §2.2 gives [14, 20].
"""
import itertools

import numpy as np
import pytest
import torch

from golden_io import read_kv
from oracle.direct import direct_blas, direct_naive, direct_sampled
from oracle.pool import maxpool


def _rand(rng, shape, ints=False):
    if ints:
        return rng.integers(-3, 4, size=shape).astype(np.float32)
    return rng.standard_normal(shape).astype(np.float32)


SHAPES = [
    # N, n, C, K, X, r, pad
    (1, 2, 3, 2, (9,), 3, 0),
    (1, 1, 2, 3, (7,), 4, 1),
    (2, 2, 3, 2, (6, 7), 3, 1),
    (2, 1, 2, 2, (5, 5), 2, 0),
    (3, 1, 2, 3, (4, 5, 6), 3, 1),
    (3, 2, 1, 1, (3, 4, 3), 3, 0),
]


@pytest.mark.parametrize("N,n,C,K,X,r,pad", SHAPES)
def test_naive_equals_blas(N, n, C, K, X, r, pad):
    rng = np.random.default_rng(N * 100 + C)
    x = _rand(rng, (n, C) + X)
    w = _rand(rng, (K, C) + (r,) * N)
    for relu in (False, True):
        y1, d1 = direct_naive(x, w, pad, relu=relu)
        y2, d2 = direct_blas(x, w, pad, relu=relu)
        np.testing.assert_allclose(y1, y2, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(d1, d2, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("N,n,C,K,X,r,pad", SHAPES)
def test_blas_equals_torch_conv(N, n, C, K, X, r, pad):
    rng = np.random.default_rng(N * 10 + K)
    x = _rand(rng, (n, C) + X)
    w = _rand(rng, (K, C) + (r,) * N)
    y, den = direct_blas(x, w, pad)
    conv = {1: torch.nn.functional.conv1d, 2: torch.nn.functional.conv2d,
            3: torch.nn.functional.conv3d}[N]
    ref = conv(torch.from_numpy(x).double(), torch.from_numpy(w).double(), padding=pad).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
    dref = conv(torch.from_numpy(np.abs(x)).double(), torch.from_numpy(np.abs(w)).double(),
                padding=pad).numpy()
    np.testing.assert_allclose(den, dref, rtol=1e-12, atol=1e-12 * dref.max())


def test_sampled_equals_blas():
    rng = np.random.default_rng(3)
    x = _rand(rng, (2, 5, 6, 7, 5))
    w = _rand(rng, (4, 5, 3, 3, 3))
    y, den = direct_blas(x, w, 1)
    coords = np.array([(b, k, a, c, e) for b in range(2) for k in range(4)
                       for a in range(6) for c in range(7) for e in range(5)])
    ys, ds = direct_sampled(x, w, 1, coords, chunk=97)
    np.testing.assert_allclose(ys, y[tuple(coords.T)], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(ds, den[tuple(coords.T)], rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("N,n,C,K,X,r,pad", SHAPES[::2])
def test_bias_all_forms_and_torch(N, n, C, K, X, r, pad):
    """eq. (2)'s bias b_k: the three forms agree, torch's convNd with its bias
    argument agrees, the ReLU applies after the bias, and the denominator
    counts |b_k|."""
    rng = np.random.default_rng(N * 7 + K)
    x = _rand(rng, (n, C) + X)
    w = _rand(rng, (K, C) + (r,) * N)
    b = (3.0 * rng.standard_normal(K)).astype(np.float32)
    conv = {1: torch.nn.functional.conv1d, 2: torch.nn.functional.conv2d,
            3: torch.nn.functional.conv3d}[N]
    ref = conv(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
               bias=torch.from_numpy(b).double(), padding=pad).numpy()
    y0, d0 = direct_blas(x, w, pad)
    for relu in (False, True):
        want = np.maximum(ref, 0.0) if relu else ref
        y1, d1 = direct_naive(x, w, pad, relu=relu, bias=b)
        y2, d2 = direct_blas(x, w, pad, relu=relu, bias=b)
        np.testing.assert_allclose(y1, want, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
        np.testing.assert_allclose(y2, want, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
        dwant = d0 + np.abs(b).reshape((1, K) + (1,) * N)
        np.testing.assert_allclose(d1, dwant, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(d2, dwant, rtol=1e-13, atol=1e-13)
        coords = np.stack(np.meshgrid(*[np.arange(v) for v in y2.shape], indexing="ij"), -1).reshape(-1, 2 + N)
        ys, ds = direct_sampled(x, w, pad, coords, relu=relu, bias=b, chunk=13)
        np.testing.assert_allclose(ys, y2[tuple(coords.T)], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(ds, d2[tuple(coords.T)], rtol=1e-13, atol=1e-13)


def test_hand_example():
    ex = read_kv("f23_hand_example.txt")
    d = np.array([[[float(v) for v in ex["d"]]]], dtype=np.float32)
    g = np.array([[[float(v) for v in ex["g"]]]], dtype=np.float32)
    for fn in (direct_naive, direct_blas):
        y, den = fn(d, g, 0)
        assert y.reshape(-1).tolist() == [float(v) for v in ex["s"]]


def test_no_kernel_flip_one_hot():
    """A one-hot input returns the kernel mirrored about the centre: the layer
    is a correlation, not a convolution."""
    x = np.zeros((1, 1, 5, 5, 5), np.float32)
    x[0, 0, 2, 2, 2] = 1
    w = np.arange(27, dtype=np.float32).reshape(1, 1, 3, 3, 3)
    y, _ = direct_blas(x, w, 1)
    got = y[0, 0, 1:4, 1:4, 1:4]
    np.testing.assert_array_equal(got, w[0, 0, ::-1, ::-1, ::-1])


def test_maxpool_matches_torch():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 3, 5, 7, 9)).astype(np.float32)
    for win in [(1, 2, 2), (2, 2, 2)]:
        ref = torch.nn.functional.max_pool3d(torch.from_numpy(x), win, win, ceil_mode=False).numpy()
        np.testing.assert_array_equal(maxpool(x, win), ref)


def test_maxpool_hand_example():
    x = np.array([[1, 5, 2], [3, 4, 9]], dtype=np.float32).reshape(1, 1, 1, 2, 3)
    # floor rounding drops the last column: windows {1,5,3,4} -> 5
    assert maxpool(x, (1, 2, 2)).reshape(-1).tolist() == [5.0]


@pytest.mark.parametrize("N,n,C,K,X,r,pad", SHAPES[1::2])
@pytest.mark.parametrize("slope", [0.1, -0.5, 0.0, 2.0])
def test_leaky_relu_all_forms_and_torch(N, n, C, K, X, r, pad, slope):
    """A leaky ReLU as eq. (2)'s activation f, after the bias: the three forms
    agree with torch's CPU fp64 convNd followed by its leaky_relu; the
    denominator is the activation-free one (slope 0 equals the ReLU)."""
    rng = np.random.default_rng(N * 31 + C)
    x = _rand(rng, (n, C) + X)
    w = _rand(rng, (K, C) + (r,) * N)
    b = rng.standard_normal(K).astype(np.float32)
    conv = {1: torch.nn.functional.conv1d, 2: torch.nn.functional.conv2d,
            3: torch.nn.functional.conv3d}[N]
    ref = torch.nn.functional.leaky_relu(
        conv(torch.from_numpy(x).double(), torch.from_numpy(w).double(), bias=torch.from_numpy(b).double(),
             padding=pad), negative_slope=slope).numpy()
    tol = 1e-12 * np.abs(ref).max()
    y1, d1 = direct_naive(x, w, pad, bias=b, leaky=slope)
    y2, d2 = direct_blas(x, w, pad, bias=b, leaky=slope)
    np.testing.assert_allclose(y1, ref, rtol=1e-12, atol=tol)
    np.testing.assert_allclose(y2, ref, rtol=1e-12, atol=tol)
    _, d0 = direct_blas(x, w, pad, bias=b)
    np.testing.assert_array_equal(d2, d0)
    coords = np.stack(np.meshgrid(*[np.arange(v) for v in y2.shape], indexing="ij"), -1).reshape(-1, 2 + N)
    ys, _ = direct_sampled(x, w, pad, coords, bias=b, leaky=slope, chunk=11)
    np.testing.assert_allclose(ys, y2[tuple(coords.T)], rtol=1e-13, atol=1e-13)
    if slope == 0.0:
        yr, _ = direct_blas(x, w, pad, bias=b, relu=True)
        np.testing.assert_array_equal(np.abs(y2), yr)   # -0.0 from 0 * v compares equal
    pre, _ = direct_blas(x, w, pad, bias=b)
    assert np.any(pre < 0) and np.any(pre > 0)      # both sides of f are exercised
    with pytest.raises(ValueError):
        direct_blas(x, w, pad, relu=True, leaky=slope)
