"""Plain, slow CPU oracle for the N-D Winograd forward.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the
HIP library (no headers, tables, constant generators or helpers); the two meet
only through seeded inputs from ``workloads``.

Modules
-------
``toomcook``  exact transform synthesis following §2.1 Algorithm 1 (CRT over
              linear moduli plus the point at infinity), turned into the
              correlation form the layer equation (2) needs.
``direct``    fp64 direct N-D correlation, eq. (2): a naive loop nest, a
              per-offset BLAS form, and a per-output sampled form, each also
              returning the magnitude denominator used by the error metric.
``winograd``  reference Winograd in fp64 or exact rationals via n-mode
              products, eq. (3)-(5), with the overlapping-tile decomposition
              of §3.3.
``metric``    normalised error |y - y_ref| / sum|w||x|.
``pool``      max-pool and ReLU for the C3D stack (not part of the method).
``costmodel`` multiplication counts and ideal speed-ups quoted in §3.2-§3.3
              and Table 1.

Every function in this package is pinned by a ``-m "not gpu"`` test against
something the paper or mathematics fixes (printed matrices, Table 1, a hand
worked example, brute-force exact agreement, a library convolution); see the
module docstrings for the pins.
"""
