"""Normalised error metric (oracle; test infrastructure only).

err = |y - y_ref| / den, den = sum |w| |x| over the receptive field (the bound
any summation order of eq. (2) can reach with unit roundoff).  Where den is
tiny compared with its mean (an all-zero receptive field), a transform method
may still leave rounding residue from the other elements of its tile, so den
is clamped below at 1e-3 of its mean and the clamped count is reported.
"""
from __future__ import annotations

import numpy as np


def normalised_error(y, y_ref, den, floor_frac=1e-3):
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    den = np.asarray(den, dtype=np.float64)
    if y.shape != y_ref.shape or y.shape != den.shape:
        raise ValueError(f"shape mismatch {y.shape} {y_ref.shape} {den.shape}")
    if y.size == 0:
        return {"max": 0.0, "p9999": 0.0, "argmax": None, "clamped": 0, "nonfinite": 0}
    mean = float(den.mean()) if den.size else 0.0
    floor = max(floor_frac * mean, np.finfo(np.float64).tiny)
    dc = np.maximum(den, floor)
    err = np.abs(y - y_ref) / dc
    nonfinite = int(np.count_nonzero(~np.isfinite(y)))
    err = np.where(np.isfinite(err), err, np.inf)
    i = int(np.argmax(err))
    return {
        "max": float(err.reshape(-1)[i]),
        "p9999": float(np.quantile(err, 0.9999)),
        "argmax": tuple(int(v) for v in np.unravel_index(i, err.shape)),
        "clamped": int(np.count_nonzero(den < floor)),
        "nonfinite": nonfinite,
    }
