"""Fresh 16x16 random Hadamard transform (oracle; test infrastructure only).

Sections 2 ("Others": Hadamard transforms with butterfly implementations),
3.2 and 3.4 (H_16^r, "a fresh 16x16 random Hadamard transform").  Reading:
H_16^r = diag(d) * H_16 / 4 with H_16 the Sylvester Hadamard matrix and d a
vector of 16 random signs.  A 1x16 row block x maps to x * H_16^r, which equals
the fast Walsh-Hadamard transform of (d * x) divided by 4; the 16x1 column
view (H_16^r)^T applies the same map to a column block.  H_16^r is orthogonal,
so the rotation cancels inside each product of the NS iteration.

Signs: one 16-sign vector per NS step k, from output k+1 of the SplitMix64
generator (Steele, Lea and Flood, OOPSLA 2014) started at state ``seed``: bit i
set means d_i = -1.  The GPU library implements the same published generator
on its own; nothing is shared.
"""
from __future__ import annotations

import numpy as np

_MASK = (1 << 64) - 1
_GAMMA = 0x9E3779B97F4A7C15


def splitmix64(state: int, index: int) -> int:
    """Output number ``index`` (1-based) of SplitMix64 started at ``state``."""
    z = (state + _GAMMA * index) & _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def step_signs(seed: int, step: int) -> np.ndarray:
    """The 16 signs d of NS step ``step`` (0-based) as float32 +-1."""
    bits = splitmix64(seed, step + 1)
    return np.array([-1.0 if (bits >> i) & 1 else 1.0 for i in range(16)], dtype=np.float32)


def sylvester16() -> np.ndarray:
    """H_16 by the Sylvester construction H_{2n} = [[H, H], [H, -H]] (float64)."""
    h = np.array([[1.0]])
    while h.shape[0] < 16:
        h = np.block([[h, h], [h, -h]])
    return h


def rotate_blocks_f32(blocks: np.ndarray, signs: np.ndarray) -> np.ndarray:
    """Apply H_16^r to every 16-vector in the last axis, emulating binary32 exactly.

    u = x * d (exact), then the in-place butterfly with strides 1, 2, 4, 8, each
    (u_i, u_{i+h}) <- (fl32(u_i + u_{i+h}), fl32(u_i - u_{i+h})), then * 0.25.
    """
    u = (np.asarray(blocks, dtype=np.float32) * signs.astype(np.float32)).astype(np.float32)
    lead = u.shape[:-1]
    h = 1
    while h < 16:
        v = u.reshape(lead + (16 // (2 * h), 2, h))
        a = v[..., 0, :]
        b = v[..., 1, :]
        u = np.stack([a + b, a - b], axis=-2).reshape(lead + (16,)).astype(np.float32)
        h *= 2
    return (u * np.float32(0.25)).astype(np.float32)


def unrotate_blocks_f32(blocks: np.ndarray, signs: np.ndarray) -> np.ndarray:
    """Apply (H_16^r)^-1 to every 16-vector in the last axis, in binary32.

    (diag(d) H_16 / 4)^-1 = (H_16 / 4) diag(d), because H_16 H_16 = 16 I: the
    unsigned butterfly (strides 1, 2, 4, 8, each pair rounded to binary32), then
    * 0.25, then the signs d.
    """
    u = np.asarray(blocks, dtype=np.float32)
    lead = u.shape[:-1]
    h = 1
    while h < 16:
        v = u.reshape(lead + (16 // (2 * h), 2, h))
        a = v[..., 0, :]
        b = v[..., 1, :]
        u = np.stack([a + b, a - b], axis=-2).reshape(lead + (16,)).astype(np.float32)
        h *= 2
    return ((u * np.float32(0.25)).astype(np.float32) * signs.astype(np.float32)).astype(np.float32)
