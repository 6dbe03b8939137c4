"""NVFP4 storage of the first moment feeding the NS orthogonalisation (oracle; test infrastructure only).

Section 3.3 stores the optimizer's first moment in NVFP4 after a 16-element
Hadamard mixing, with stochastic rounding (SR) and adaptive 4/6 block scaling,
and Section 3.4 feeds that momentum to the NVFP4 Root iteration; Section 2
("AdamW optimizer") gives the first-moment update m_t = b1 m_{t-1} + (1 - b1) g_t.
The paper fixes none of the arithmetic; the readings taken here:

* state S_t of an R x C momentum: the NVFP4 record of the NS quantiser along
  rows (codes, E4M3 scales, FP32 tensor scale), encoded at optimizer step t after
  the rotation H_16^r with the signs of SplitMix64 output t + 1 of ``seed``
  (the same sign rule as the NS steps, with the optimizer step as counter);
* decode of S_{t-1}: u = fl32(q * s * s_g) per element (one rounding: q s is
  exact), then the inverse rotation in binary32 (``rht.unrotate_blocks_f32``)
  with the signs of step t - 1; at t = 0 the previous momentum is 0;
* update: m_t = fl32(b1 m_hat + b2 g) with b2 = fl32(1 - b1), the two products
  exact and their sum rounded once in binary64, then to binary32;
* m_t (binary32) is the input of the orthogonalisation;
* encode of m_t: rotation, tensor scale and the 4/6 choice exactly as the NS
  quantiser (the choice by the round-to-nearest errors, so that it does not
  depend on the random draws); with SR the element codes are then drawn: with
  x = |u| / r the exact quotient (r = fl32(s s_g)), lo and hi the E2M1 grid
  points with lo <= x < hi, the magnitude rounds up to hi iff
  rho 2^-24 < (x - lo) / (hi - lo), rho a 24-bit uniform integer; x >= 6 gives
  6; the sign bit is kept; r = 0 gives magnitude 0.  The comparison is exact:
  rho (hi - lo) r < (|u| - lo r) 2^24 holds every term exactly in binary64;
* draws: the element at flat index e (matrix b, row i, column j:
  e = (b R + i) C + j) takes 24 bits of SplitMix64 output floor(e / 2) + 1 of the
  state SplitMix64(seed XOR 0x5352, t + 1): bits 40..63 for even e, bits 16..39
  for odd e (one 64-bit output serves two elements).
"""
from __future__ import annotations

import numpy as np

from .formats import E2M1_GRID, E4M3_GRID
from .quantize import NVFP4, quantize
from .rht import _GAMMA, _MASK, rotate_blocks_f32, splitmix64, step_signs, unrotate_blocks_f32

SR_TAG = 0x5352


def sr_key(seed: int, step: int) -> int:
    """State of the draw stream of optimizer step ``step``."""
    return splitmix64(seed ^ SR_TAG, step + 1)


def sr_draws(key: int, count: int, offset: int = 0) -> np.ndarray:
    """24-bit draws for e = offset .. offset + count - 1: z = SplitMix64(key, e // 2 + 1),
    rho_e = z >> 40 for even e and (z >> 16) & 0xFFFFFF for odd e.

    The same three-line SplitMix64 mix as ``rht.splitmix64``, on uint64 arrays
    (NumPy's uint64 arithmetic wraps modulo 2^64).
    """
    e = np.arange(offset, offset + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(key) + np.uint64(_GAMMA) * (e // np.uint64(2) + np.uint64(1))
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    assert _MASK == (1 << 64) - 1
    odd = (e & np.uint64(1)) == np.uint64(1)
    return np.where(odd, (z >> np.uint64(16)) & np.uint64(0xFFFFFF), z >> np.uint64(40)).astype(np.uint32)


def sr_magnitudes(u: np.ndarray, r: np.ndarray, rho: np.ndarray) -> np.ndarray:
    """E2M1 indices of |u| / r rounded stochastically with draws rho (all arrays broadcast).

    u: binary32 values; r: binary32 scales (> 0 or 0); rho: 24-bit integers.
    """
    a = np.abs(np.asarray(u, np.float32)).astype(np.float64)
    r = np.asarray(r, np.float32).astype(np.float64)
    rho = np.asarray(rho, np.uint32).astype(np.float64)
    lo_idx = np.zeros(np.broadcast(a, r).shape, dtype=np.int64)
    for k in range(1, 8):   # largest grid point g with g r <= |u| (exact products)
        lo_idx = np.where(E2M1_GRID[k] * r <= a, k, lo_idx)
    lo = E2M1_GRID[lo_idx]
    hi = E2M1_GRID[np.minimum(lo_idx + 1, 7)]
    up = (lo_idx < 7) & (rho * (hi - lo) * r < (a - lo * r) * 2.0 ** 24)
    idx = np.where(up, lo_idx + 1, lo_idx)
    return np.where(r > 0, idx, 0)


def decode_state(state: NVFP4, signs: np.ndarray | None) -> np.ndarray:
    """The binary32 momentum a state encodes (inverse rotation with ``signs``)."""
    q = E2M1_GRID[state.codes & 7]
    q = np.where(state.codes & 8, -q, q)
    rows, cols = state.codes.shape
    s = E4M3_GRID[state.scales & 0x7F]
    qs = (q.reshape(rows, cols // 16, 16) * s[..., None])        # exact
    u = (qs * np.float64(state.sg)).astype(np.float32)           # one rounding
    if signs is not None:
        u = unrotate_blocks_f32(u, signs)
    return u.reshape(rows, cols)


def encode_state(m: np.ndarray, signs: np.ndarray | None, adaptive46: bool,
                 draws: np.ndarray | None, rows: np.ndarray | None = None) -> NVFP4:
    """NVFP4 record of a binary32 momentum; ``draws`` (24-bit, one per element of the
    encoded rows) selects SR.  ``rows`` (optional) encodes only those rows, with the
    tensor scale of the whole matrix (as ``quantize``)."""
    m = np.asarray(m, np.float32)
    rec = quantize(m, axis=1, signs=signs, adaptive46=adaptive46, rows=rows)
    if draws is None:
        return rec
    if rows is not None:
        m = m[np.asarray(rows, dtype=np.int64)]
    rows, cols = m.shape
    blocks = m.reshape(rows, cols // 16, 16)
    u = rotate_blocks_f32(blocks, signs) if signs is not None else blocks
    s = E4M3_GRID[rec.scales & 0x7F].astype(np.float32)
    r = (s * rec.sg).astype(np.float32)
    idx = sr_magnitudes(u, r[..., None], np.asarray(draws).reshape(rows, cols // 16, 16))
    neg = np.signbit(u).astype(np.uint8)
    codes = ((neg << 3) | idx.astype(np.uint8)).reshape(rows, cols)
    return NVFP4(codes, rec.scales, rec.sg, rec.m4)


def momentum_step(g: np.ndarray, prev: NVFP4 | None, beta: float, seed: int, step: int,
                  hadamard: bool = True, adaptive46: bool = True, sr: bool = True,
                  batch_index: int = 0):
    """One optimizer step of the first moment: returns (m_t binary32, state S_t).

    ``prev`` is S_{step-1} (ignored at step 0); ``batch_index`` is the matrix's
    position b in a batch of equal shapes (it offsets the draw indices).
    """
    g = np.asarray(g, np.float32)
    rows, cols = g.shape
    b1 = np.float32(beta)
    b2 = np.float32(np.float32(1.0) - b1)
    if step > 0:
        m_hat = decode_state(prev, step_signs(seed, step - 1) if hadamard else None)
    else:
        m_hat = np.zeros_like(g)
    m = (np.float64(b1) * m_hat.astype(np.float64) + np.float64(b2) * g.astype(np.float64)).astype(np.float32)
    draws = None
    if sr:
        draws = sr_draws(sr_key(seed, step), rows * cols, batch_index * rows * cols).reshape(rows, cols)
    state = encode_state(m, step_signs(seed, step) if hadamard else None, adaptive46, draws)
    return m, state
