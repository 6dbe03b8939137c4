"""Seeded synthetic momentum matrices for the Newton-Schulz orthogonalisation path.

This module holds no arithmetic of the method: it only draws random matrices.
Both the CPU oracle (tests, CPU baseline) and the GPU harness (bench, GPU tests)
read their inputs from here, so both sides always see the same bytes.

The paper measures on momentum taken from real pretraining runs (Section 4.3,
Table 6 "Root" rows: four decoder blocks, five NS iterations).  That data is
not available, so heavy-tailed synthetic matrices stand in for it: Gaussian or
Student-t entries, lognormal per-row scales and sparse large outliers mimic
the outlier structure that motivates the p99 clipping of Section 3.4.

Recipe (every case): values are drawn in float64 from
``numpy.random.Generator(PCG64(seed))``, cast to float32, then the modifiers
are applied in float32 in the order listed for the case.
"""
from __future__ import annotations

import numpy as np

__all__ = ["CASES", "case_matrices", "case_shapes", "matrix", "small_case"]


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _normal_outliers(rng, rows, cols, factor):
    x = rng.standard_normal((rows, cols)).astype(np.float32)
    n = rows * cols
    k = int(round(0.001 * n))
    pos = rng.choice(n, size=k, replace=False)
    flat = x.reshape(-1)
    flat[pos] *= np.float32(factor)
    return x


def _student_t_unit_rms(rng, rows, cols, df=4.0):
    x = rng.standard_t(df, size=(rows, cols)).astype(np.float32)
    rms = np.float32(np.sqrt(np.mean(np.square(x, dtype=np.float64))))
    return (x / rms).astype(np.float32)


def _row_lognormal(rng, x):
    f = rng.lognormal(0.0, 1.0, size=(x.shape[0], 1)).astype(np.float32)
    return (x * f).astype(np.float32)


def _normal_rows(rng, rows, cols):
    x = rng.standard_normal((rows, cols)).astype(np.float32)
    return _row_lognormal(rng, x)


def _t_rows(rng, rows, cols):
    x = rng.standard_t(4.0, size=(rows, cols)).astype(np.float32)
    return _row_lognormal(rng, x)


# name -> (description, list of (label, rows, cols)) ; the generator order is the list order.
_BLOCK = [("q", 3072, 3072), ("k", 1024, 3072), ("v", 1024, 3072), ("o", 3072, 3072),
          ("gate", 8192, 3072), ("up", 8192, 3072), ("down", 3072, 8192)]

CASES = {
    "single_256x512": "one 256x512 N(0,1) matrix, 0.1% of positions x20, seed 0",
    "square_4096": "one 4096x4096 Student-t(4) matrix scaled to unit RMS, seed 1",
    "rect_3072x8192_pair": "3072x8192 and 8192x3072, N(0,1) x per-row lognormal(0,1), seed 2",
    "block3b_x4": "four 3B-shaped decoder blocks (q,k,v,o,gate,up,down), Student-t(4) x per-row "
                  "lognormal(0,1), seed 3, 28 matrices",
    "stress_8192x28672_plus_256x512sq": "one 8192x28672 plus 256 of 512x512, N(0,1), 0.1% x50, seed 4",
    # the shapes of the paper's isolated Root measurement (Section 4, native-hardware
    # efficiency: four decoder blocks, d = 4096, d_ff = 11008, 8 KV heads of 128)
    "paper_d4096_x4": "four d=4096 decoder blocks (q,o 4096x4096; k,v 1024x4096; gate,up 11008x4096; "
                      "down 4096x11008), Student-t(4) x per-row lognormal(0,1), seed 5, 28 matrices",
}
_BLOCK_D4096 = [("q", 4096, 4096), ("k", 1024, 4096), ("v", 1024, 4096), ("o", 4096, 4096),
                ("gate", 11008, 4096), ("up", 11008, 4096), ("down", 4096, 11008)]


def case_shapes(name: str):
    """List of (label, rows, cols) for a case, in generation order."""
    if name == "single_256x512":
        return [("m0", 256, 512)]
    if name == "square_4096":
        return [("m0", 4096, 4096)]
    if name == "rect_3072x8192_pair":
        return [("wide", 3072, 8192), ("tall", 8192, 3072)]
    if name == "block3b_x4":
        return [(f"b{b}.{lab}", r, c) for b in range(4) for (lab, r, c) in _BLOCK]
    if name == "stress_8192x28672_plus_256x512sq":
        return [("big", 8192, 28672)] + [(f"s{i}", 512, 512) for i in range(256)]
    if name == "paper_d4096_x4":
        return [(f"b{b}.{lab}", r, c) for b in range(4) for (lab, r, c) in _BLOCK_D4096]
    raise KeyError(name)


def case_matrices(name: str, limit: int | None = None):
    """Generate the matrices of a case (a list of float32 C-contiguous arrays).

    ``limit`` stops after that many matrices; the ones produced are identical to
    the first ``limit`` matrices of the full case (one generator, fixed order).
    """
    shapes = case_shapes(name)
    if limit is not None:
        shapes = shapes[:limit]
    out = []
    if name == "single_256x512":
        rng = _rng(0)
        out = [_normal_outliers(rng, 256, 512, 20.0)]
    elif name == "square_4096":
        rng = _rng(1)
        out = [_student_t_unit_rms(rng, 4096, 4096)]
    elif name == "rect_3072x8192_pair":
        rng = _rng(2)
        out = [_normal_rows(rng, r, c) for (_, r, c) in shapes]
    elif name == "block3b_x4":
        rng = _rng(3)
        out = [_t_rows(rng, r, c) for (_, r, c) in shapes]
    elif name == "stress_8192x28672_plus_256x512sq":
        rng = _rng(4)
        out = [_normal_outliers(rng, r, c, 50.0) for (_, r, c) in shapes]
    elif name == "paper_d4096_x4":
        rng = _rng(5)
        out = [_t_rows(rng, r, c) for (_, r, c) in shapes]
    return [np.ascontiguousarray(m) for m in out]


def matrix(rows: int, cols: int, seed: int, kind: str = "t_rows") -> np.ndarray:
    """One extra seeded matrix of any shape, for tests at sizes between the cases."""
    rng = _rng(seed)
    if kind == "t_rows":
        return np.ascontiguousarray(_t_rows(rng, rows, cols))
    if kind == "normal_outliers":
        return np.ascontiguousarray(_normal_outliers(rng, rows, cols, 20.0))
    if kind == "normal":
        return np.ascontiguousarray(rng.standard_normal((rows, cols)).astype(np.float32))
    raise KeyError(kind)


def small_case():
    """The small case the oracle finishes in seconds (one 256x512 matrix)."""
    return case_matrices("single_256x512")
