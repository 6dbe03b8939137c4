"""NVFP4 number formats, written from their definitions (oracle; test infrastructure only).

Section 2 ("NVFP4 format"): an element is E2M1 (1 sign, 2 exponent, 1 mantissa
bit), each 16-element block shares an FP8 E4M3 scale s, and the tensor has an
FP32 global scale s_g; the decoded value is x_E2M1 * s * s_g.

E2M1 magnitudes, indexed by the 3-bit code (OCP 4-bit float): 0, 0.5, 1, 1.5,
2, 3, 4, 6.  E4M3 here is the OCP "E4M3FN" variant: exponent bias 7, no
infinities, code 0x7F is NaN, largest finite 448, subnormals m/8 * 2^-6.

Rounding is round-to-nearest with ties to the even code (RTN, Section 2
"Others"; Section 3.4 "All quantizations use RTN").  This module implements it
as an explicit nearest-grid-point search, deliberately unlike the bit
manipulation a GPU would use.
"""
from __future__ import annotations

import numpy as np

E2M1_GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)
E2M1_MAX = 6.0
E4M3_MAX = 448.0


def e4m3_table() -> np.ndarray:
    """Magnitude of every non-negative finite E4M3FN code 0..126, by the format definition."""
    vals = np.empty(127, dtype=np.float64)
    for code in range(127):
        e, m = code >> 3, code & 7
        if e == 0:
            vals[code] = (m / 8.0) * 2.0 ** -6
        else:
            vals[code] = (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return vals


E4M3_GRID = e4m3_table()


def round_to_grid(v: np.ndarray, grid: np.ndarray) -> np.ndarray:
    """Index of the grid point nearest to each v (v >= 0, v <= grid[-1]); ties -> even index.

    Distances are taken in float64.  Away from a tie the comparison cannot be
    flipped by rounding; at a tie both operands lie in neighbouring binades and
    the float64 differences of float32 inputs and grid points are exact.
    """
    v = np.asarray(v, dtype=np.float64)
    if np.any(v < 0) or np.any(v > grid[-1]) or np.any(np.isnan(v)):
        raise ValueError("round_to_grid: value outside [0, grid max]")
    hi = np.searchsorted(grid, v, side="left")
    hi = np.clip(hi, 0, len(grid) - 1)
    lo = np.clip(hi - 1, 0, len(grid) - 1)
    d_lo = v - grid[lo]
    d_hi = grid[hi] - v
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    return np.where(take_hi, hi, lo).astype(np.int64)


def e4m3_encode(v: np.ndarray) -> np.ndarray:
    """E4M3FN code (uint8) of each non-negative float32 v <= 448, round-to-nearest-even."""
    return round_to_grid(np.asarray(v, dtype=np.float32), E4M3_GRID).astype(np.uint8)


def e4m3_decode(code: np.ndarray) -> np.ndarray:
    """float64 value of each E4M3FN code (sign bit honoured; 0x7F/0xFF rejected)."""
    code = np.asarray(code, dtype=np.uint8)
    mag = code & 0x7F
    if np.any(mag == 0x7F):
        raise ValueError("E4M3 NaN code")
    val = E4M3_GRID[mag]
    return np.where(code & 0x80, -val, val)


def e2m1_index(y: np.ndarray) -> np.ndarray:
    """3-bit E2M1 magnitude index of each y in [0, 6], round-to-nearest-even."""
    return round_to_grid(y, E2M1_GRID).astype(np.uint8)


def e2m1_decode(code: np.ndarray) -> np.ndarray:
    """float64 value of 4-bit E2M1 codes (bit 3 = sign, bits 0-2 = magnitude index)."""
    code = np.asarray(code, dtype=np.uint8)
    val = E2M1_GRID[code & 7]
    return np.where(code & 8, -val, val)


def pack_nibbles(codes: np.ndarray) -> np.ndarray:
    """Pack 4-bit codes along the last axis, two per byte, element 2j in the low nibble."""
    codes = np.asarray(codes, dtype=np.uint8)
    lo = codes[..., 0::2]
    hi = codes[..., 1::2]
    return (lo | (hi << 4)).astype(np.uint8)


def unpack_nibbles(packed: np.ndarray) -> np.ndarray:
    """Inverse of ``pack_nibbles``."""
    packed = np.asarray(packed, dtype=np.uint8)
    out = np.empty(packed.shape[:-1] + (packed.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = packed & 0xF
    out[..., 1::2] = packed >> 4
    return out
