"""Pins of the normalised error metric (oracle/metric.py), CPU only.

The metric decides every GPU parity verdict, so it is pinned by hand-computed
cases whose values follow from its definition (|y - y_ref| / den, den clamped
below at 1e-3 of its mean, the largest value and its position), and planted
slips in a copy of the function (a dropped absolute value, min in place of
max, a floor tied to the largest denominator, a constant result) must each
fail one of them.
"""
import inspect
import math

import numpy as np
import pytest

import oracle.metric as om


def _hand_cases(fn):
    """Run every hand case through fn; returns a list of failures (empty: pinned)."""
    bad = []

    # 1. known max and argmax.  errors: |1-1.5|/2 = 0.25, |2-2|/4 = 0,
    #    |0-3|/0.5 = 6 (y below y_ref), |7-6|/1 = 1; den mean 1.875, no clamp
    y = np.array([[1.0, 2.0], [0.0, 7.0]])
    y_ref = np.array([[1.5, 2.0], [3.0, 6.0]])
    den = np.array([[2.0, 4.0], [0.5, 1.0]])
    e = fn(y, y_ref, den)
    if e["max"] != 6.0:
        bad.append(("max", e["max"]))
    if e["argmax"] != (1, 0):
        bad.append(("argmax", e["argmax"]))
    if e["clamped"] != 0 or e["nonfinite"] != 0:
        bad.append(("counts", e["clamped"], e["nonfinite"]))

    # 2. a zero denominator is clamped at 1e-3 * mean(den): den = [0, 10, 10, 10],
    #    mean 7.5, floor 7.5e-3; the only nonzero difference sits there
    y = np.array([1e-6, 5.0, -2.0, 0.25])
    y_ref = np.array([0.0, 5.0, -2.0, 0.25])
    den = np.array([0.0, 10.0, 10.0, 10.0])
    e = fn(y, y_ref, den)
    want = 1e-6 / 7.5e-3
    if not math.isclose(e["max"], want, rel_tol=1e-12):
        bad.append(("clamp max", e["max"], want))
    if e["clamped"] != 1:
        bad.append(("clamped", e["clamped"]))
    if e["argmax"] != (0,):
        bad.append(("clamp argmax", e["argmax"]))

    # 3. a NaN output is counted and makes the error infinite
    y = np.array([1.0, np.nan, 3.0])
    y_ref = np.array([1.0, 2.0, 3.0])
    den = np.array([1.0, 1.0, 1.0])
    e = fn(y, y_ref, den)
    if e["nonfinite"] != 1 or e["max"] != math.inf or e["argmax"] != (1,):
        bad.append(("nan", e))

    # 4. an infinite output likewise; a non-finite reference gives inf too
    e = fn(np.array([np.inf, 0.0]), np.array([1.0, 0.0]), np.array([1.0, 1.0]))
    if e["nonfinite"] != 1 or e["max"] != math.inf:
        bad.append(("inf", e))
    e = fn(np.array([1.0, 0.0]), np.array([np.nan, 0.0]), np.array([1.0, 1.0]))
    if e["max"] != math.inf:
        bad.append(("nan ref", e))

    # 5. every output equal: zero error
    y = np.arange(6.0).reshape(2, 3)
    e = fn(y, y.copy(), np.ones((2, 3)))
    if e["max"] != 0.0 or e["p9999"] != 0.0:
        bad.append(("equal", e))

    # 6. the 99.99th percentile of 10^4 + 1 errors 0, 1e-4, ..., 1 (den 1)
    #    is 0.9999 (linear interpolation between order statistics)
    errs = np.arange(10001) / 10000.0
    e = fn(errs, np.zeros_like(errs), np.ones_like(errs))
    if not math.isclose(e["p9999"], 0.9999, rel_tol=1e-12) or e["max"] != 1.0:
        bad.append(("p9999", e["p9999"], e["max"]))

    # 7. an empty comparison has no error and no position
    e = fn(np.zeros(0), np.zeros(0), np.zeros(0))
    if e["max"] != 0.0 or e["argmax"] is not None:
        bad.append(("empty", e))
    return bad


def test_metric_hand_cases():
    assert _hand_cases(om.normalised_error) == []


def test_metric_shape_mismatch_raises():
    with pytest.raises(ValueError):
        om.normalised_error(np.zeros(3), np.zeros(3), np.zeros(4))


def _planted(old, new):
    """A copy of normalised_error with one source fragment replaced."""
    src = inspect.getsource(om.normalised_error)
    assert old in src, old          # the slip must really be planted
    ns = {"np": np}
    exec(src.replace(old, new, 1), ns)
    return ns["normalised_error"]


SLIPS = {
    "dropped_abs": ("np.abs(y - y_ref)", "(y - y_ref)"),
    "min_for_max": ("np.argmax(err)", "np.argmin(err)"),
    "floor_from_max_den": ("den.mean()", "den.max()"),
    "constant_zero": ('"max": float(err.reshape(-1)[i])', '"max": 0.0'),
    "no_clamp_count": ("np.count_nonzero(den < floor)", "0"),
    "nan_not_counted": ("np.count_nonzero(~np.isfinite(y))", "0"),
    "nonfinite_dropped": ("np.where(np.isfinite(err), err, np.inf)", "np.where(np.isfinite(err), err, 0.0)"),
}


@pytest.mark.parametrize("slip", sorted(SLIPS))
def test_metric_slips_caught(slip):
    old, new = SLIPS[slip]
    assert _hand_cases(_planted(old, new)) != []
