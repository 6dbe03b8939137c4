"""NVFP4 quantiser Q_1x16 / Q_16x1 (oracle; test infrastructure only).

Follows Section 2 ("NVFP4 format": E2M1 elements, one E4M3 scale per 1x16 or
16x1 block, one FP32 global scale, decode x_E2M1 * s * s_g) and Section 3.4
(every NS quantisation uses RTN and adaptive 4/6 block scaling, after the fresh
16x16 random Hadamard rotation).  The paper fixes the decode but not the encode;
the readings taken here are:

* global scale   s_g = fl32(amax / (6 * 448)), amax over the rotated matrix;
                 amax = 0 gives s_g = 0 and all-zero scales and magnitudes;
* block scale    for a candidate M in {6} (or {6, 4} with adaptive 4/6):
                 v = fl32(bmax / fl32(M * s_g)), s = E4M3_RNE(min(v, 448)),
                 r = fl32(s * s_g);
* elements       y = fl32(|u| / r), q = E2M1_RNE(min(y, 6)); r = 0 gives q = 0;
                 the code keeps the IEEE sign bit of u even when q = 0;
* adaptive 4/6   E_M = sum_i (u_i - q_i * s * s_g)^2 in float64, summed in
                 element order; M = 4 is kept iff E_4 < E_6 (ties keep M = 6).
                 Only the chosen scale byte is stored: decoding is always
                 q * s * s_g.

axis = 1 quantises 16 consecutive elements of a row (Q_1x16).  axis = 0
quantises 16 consecutive elements of a column (Q_16x1); its result is laid out
as the transposed matrix quantised along rows, which is the K-contiguous form a
product over that axis consumes.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .formats import E2M1_GRID, E4M3_GRID, e2m1_index, e4m3_encode, pack_nibbles
from .rht import rotate_blocks_f32

SG_DIVISOR = np.float32(6.0 * 448.0)


@dataclass
class NVFP4:
    codes: np.ndarray    # (rows, cols) uint8, 4-bit codes: bit 3 sign, bits 0-2 E2M1 index
    scales: np.ndarray   # (rows, cols // 16) uint8, E4M3FN bits
    sg: np.float32       # global scale
    m4: np.ndarray       # (rows, cols // 16) bool, True where M = 4 was chosen (diagnostic)

    @property
    def packed(self) -> np.ndarray:
        return pack_nibbles(self.codes)

    def block_values(self) -> np.ndarray:
        """float64 q * s for every element (exact), without the global scale."""
        q = E2M1_GRID[self.codes & 7]
        q = np.where(self.codes & 8, -q, q)
        s = E4M3_GRID[self.scales & 0x7F]
        rows, cols = self.codes.shape
        return (q.reshape(rows, cols // 16, 16) * s[..., None]).reshape(rows, cols)

    def dequantize(self) -> np.ndarray:
        """float64 q * s * s_g for every element (exact)."""
        return self.block_values() * np.float64(self.sg)


def quantize(x: np.ndarray, axis: int = 1, signs: np.ndarray | None = None,
             adaptive46: bool = True, rows: np.ndarray | None = None) -> NVFP4:
    """Quantise a float32 matrix to NVFP4 along ``axis`` (see module docstring).

    ``rows`` (optional) selects rows of the blocked layout (rows of x for axis 1,
    columns of x for axis 0) to encode; the tensor scale still comes from the
    whole matrix, so each selected row equals the same row of the full result.
    """
    x = np.asarray(x, dtype=np.float32)
    if x.ndim != 2:
        raise ValueError("quantize expects a matrix")
    if not np.all(np.isfinite(x)):
        raise ValueError("non-finite input")
    if axis == 0:
        x = x.T
    elif axis != 1:
        raise ValueError("axis must be 0 or 1")
    nrows, cols = x.shape
    if cols % 16:
        raise ValueError("blocked axis must be a multiple of 16")
    blocks = np.ascontiguousarray(x).reshape(nrows, cols // 16, 16)
    u = rotate_blocks_f32(blocks, signs) if signs is not None else blocks.astype(np.float32)
    neg = np.signbit(u)
    mag = np.abs(u)
    amax = np.float32(mag.max()) if mag.size else np.float32(0.0)
    sg = np.float32(amax / SG_DIVISOR)
    if rows is not None:
        rows_idx = np.asarray(rows, dtype=np.int64)
        u, neg, mag = u[rows_idx], neg[rows_idx], mag[rows_idx]
        rows = len(rows_idx)
    else:
        rows = u.shape[0]
    nblk = rows * (cols // 16)
    if sg == 0:
        codes = (neg.astype(np.uint8) << 3).reshape(rows, cols)
        return NVFP4(codes, np.zeros((rows, cols // 16), np.uint8), np.float32(0.0),
                     np.zeros((rows, cols // 16), bool))
    bmax = mag.max(axis=-1)
    best = None
    for M in ((6, 4) if adaptive46 else (6,)):
        den = np.float32(np.float32(M) * sg)
        v = np.minimum((bmax / den).astype(np.float32), np.float32(448.0))
        scode = e4m3_encode(v)
        s = E4M3_GRID[scode].astype(np.float32)
        r = (s * sg).astype(np.float32)
        with np.errstate(divide="ignore", invalid="ignore"):
            y = (mag / r[..., None]).astype(np.float32)
        y = np.where(r[..., None] > 0, np.minimum(y, np.float32(6.0)), np.float32(0.0))
        idx = e2m1_index(y.reshape(-1)).reshape(y.shape)
        dec = (E2M1_GRID[idx] * s.astype(np.float64)[..., None]) * np.float64(sg)
        dec = np.where(neg, -dec, dec)
        diff = u.astype(np.float64) - dec
        err = np.zeros(bmax.shape, dtype=np.float64)
        for i in range(16):
            err = err + diff[..., i] * diff[..., i]
        cand = (scode, idx, err)
        if best is None:
            best = cand
            m4 = np.zeros(bmax.shape, bool)
        else:
            take = cand[2] < best[2]
            m4 = take
            best = (np.where(take, cand[0], best[0]),
                    np.where(take[..., None], cand[1], best[1]),
                    np.where(take, cand[2], best[2]))
    scode, idx, _ = best
    codes = ((neg.astype(np.uint8) << 3) | idx.astype(np.uint8)).reshape(rows, cols)
    assert scode.size == nblk
    return NVFP4(codes, scode.astype(np.uint8), sg, m4)
