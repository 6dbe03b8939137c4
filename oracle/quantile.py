"""p99 outlier threshold (oracle; test infrastructure only).

Section 3.4 combines Root's shape-dependent coefficients with p99 outlier
clipping of the momentum; Table 8 gives the Root quantile ratio 0.99; Section 2
("Root optimizer") describes the removal of momentum outliers by
soft-thresholding.  Readings: one threshold per matrix, on the absolute values
of the momentum as given; the "linear" quantile definition (the one NumPy and
PyTorch use by default) computed from exact order statistics:

    v = sorted |M| (binary32 values), N = number of elements,
    h = q * (N - 1) in binary64 (q is the binary32 ratio widened),
    lo = floor(h), f = h - lo,
    tau = fl32(v[lo] + f * (v[lo + 1] - v[lo]))   (binary64 steps, one product
                                                    then one sum, then rounded)

and the clipped momentum is clamp(M, -tau, tau), which is exactly M minus the
soft-threshold S_tau(M).
"""
from __future__ import annotations

import numpy as np


def clip_threshold(m: np.ndarray, q: float = 0.99) -> np.float32:
    a = np.abs(np.asarray(m, dtype=np.float32)).reshape(-1)
    if not np.all(np.isfinite(a)):
        raise ValueError("non-finite input")
    n = a.size
    if n == 0:
        raise ValueError("empty matrix")
    h = np.float64(np.float32(q)) * np.float64(n - 1)
    lo = int(np.floor(h))
    f = h - np.float64(lo)
    if lo >= n - 1:
        return np.float32(np.max(a))
    # np.partition returns the same two order statistics a full sort would.
    part = np.partition(a, [lo, lo + 1])
    va = np.float64(part[lo])
    vb = np.float64(part[lo + 1])
    return np.float32(va + f * (vb - va))


def clip(m: np.ndarray, tau: np.float32) -> np.ndarray:
    return np.clip(np.asarray(m, dtype=np.float32), -tau, tau).astype(np.float32)
