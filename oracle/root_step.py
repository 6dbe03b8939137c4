"""The Root parameter update around the NS orthogonalisation (oracle; test infrastructure only).

Section 2 ("Root optimizer") orthogonalises the clipped first moment with the NS
iteration; Section 3.4 runs it in NVFP4; the training setup (Section 4, Table 8)
uses Root with weight decay 0.1 and BF16 master weights (Section 3.3: no FP32
master copy).  The paper does not print the update rule around the
orthogonalised momentum O; the readings taken here:

* decoupled weight decay and a per-matrix update scale s (the caller's; the
  library's helper uses Muon's sqrt(max(1, rows / cols))):
      W <- W - lr (s O + wd W)
  evaluated in binary32 in this order: c1 = fl32(1 - fl32(lr wd)),
  c2 = fl32(lr s), W' = bf16(fl32(fl32(W c1) - fl32(c2 O)));
* bf16() rounds a binary32 value to the nearest BF16 (ties to even): the top 16
  bits of the binary32 pattern after adding 0x7FFF plus the lowest kept bit.
"""
from __future__ import annotations

import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Binary32 -> BF16 bit patterns (uint16), round to nearest, ties to even (finite inputs)."""
    b = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    r = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def bf16_value(h: np.ndarray) -> np.ndarray:
    """BF16 bit patterns -> binary32 values (exact)."""
    return (np.asarray(h, np.uint16).astype(np.uint32) << 16).view(np.float32)


def apply_update(w_bf16: np.ndarray, o: np.ndarray, lr: float, wd: float, scale: float) -> np.ndarray:
    """New BF16 weights (uint16 patterns) from BF16 weights and the orthogonalised momentum."""
    lr, wd, scale = np.float32(lr), np.float32(wd), np.float32(scale)
    c1 = np.float32(np.float32(1.0) - np.float32(lr * wd))
    c2 = np.float32(lr * scale)
    w = bf16_value(w_bf16)
    t = (w * c1).astype(np.float32) - (c2 * np.asarray(o, np.float32)).astype(np.float32)
    return bf16_round(t.astype(np.float32))


def muon_scale(rows: int, cols: int) -> float:
    """Muon's shape factor sqrt(max(1, rows / cols)) (binary32)."""
    return float(np.float32(np.sqrt(max(1.0, rows / cols))))
