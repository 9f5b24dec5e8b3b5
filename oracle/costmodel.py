"""Multiplication counts and ideal speed-ups (oracle; test infrastructure only).

Dense counts: a transform matrix of shape (a x b) applied to a vector costs
a*b multiplications; an n-mode product of an I^N tensor with a (J x I) matrix
costs J*I*I^(N-1).

* §2.2: F(S, G) needs S*G/D fewer multiplications than sliding windows, with
  D = S + G - 1; in N dimensions (S*G/D)^N (§3.2, Table 1).
* §3.3: explicit eq. (1) for F(2,3) costs 4 (product) + 16 (data transform)
  + 8 (inverse) = 28 multiplications with the kernel transform cached; a layer
  of M channels and M kernels costs 4M^2 + 16M + 8M.
* §3.3 / Fig. 1: per output tile of a C3D layer, direct correlation costs
  S^3 G^3 M K; fast tensor correlation costs D^3 M K (element-wise products)
  + 3 D^4 M (data transform, once per channel) + (S D^3 + S^2 D^2 + S^3 D) K
  (inverse transform, once per kernel, shrinking one axis at a time).

Pins (tests/test_oracle_costmodel.py): the counts quoted in §3.3 (28, 4M^2 +
24M), the >6-fold reduction at 100 channels and kernels and the roughly
three-times-smaller margin at 10, the 8-fold ceiling for the C3D matrices, and
Table 1's speed-up columns.
"""
from __future__ import annotations


def ideal_speedup(S, G, N):
    D = S + G - 1
    return (S * G / D) ** N


def explicit_1d_mults(S, G):
    D = S + G - 1
    return D + D * D + S * D


def layer_1d_mults(S, G, M):
    D = S + G - 1
    return D * M * M + D * D * M + S * D * M


def c3d_tile_mults(S, G, M, K):
    D = S + G - 1
    direct = S ** 3 * G ** 3 * M * K
    fast = D ** 3 * M * K + 3 * D ** 4 * M + (S * D ** 3 + S ** 2 * D ** 2 + S ** 3 * D) * K
    return direct, fast
