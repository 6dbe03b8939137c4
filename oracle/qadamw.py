"""Quantized-state AdamW (oracle; test infrastructure only).

Section 3.3: the first moment is stored with the first-moment recipe (Hadamard
mixing, SR, adaptive 4/6: ``oracle.momentum``); the second moment v_t goes through
an ordered pipeline before NVFP4 storage: (1) square root, (2) subtraction of a
BF16 mean per 256-element tile, (3) the 16-element Hadamard transform; it is
stored as 4-bit E2M1 codes with one BF16 scale per 16 elements and one BF16 mean
per 256 (5.0625 bits per element); reconstruction inverts the transform and the
mean separation and squares.  Section 2 ("AdamW optimizer") gives the moment
updates; master weights are BF16 (Section 3.3).  Readings where the paper is silent:

* a parameter is a flat vector of N elements, N a multiple of 256; tile k holds
  elements 256k .. 256k + 255, block j of a tile its elements 16j .. 16j + 15;
* v_t = fl32(b2 v_hat + c2 fl32(g g)), b2 = beta2, c2 = fl32(1 - beta2), the two
  products exact and their sum rounded once in binary64 (v_hat = 0 at step 0);
* encode: y = fl32(sqrt(v_t)); the tile sum S is binary64: each block summed in
  element order, then the 16 block sums pairwise ((0+1)+(2+3)) + ..., a binary
  tree; mean mu = bf16(fl32(S / 256)); residual r = fl32(y - mu); rotation
  H_16^r with the signs of SplitMix64 output t + 1 of ``seed`` (binary32, as the
  NS quantiser); block scale for M in {6} or {6, 4}: s = bf16(fl32(bmax / M));
  codes E2M1_RNE(min(fl32(|u| / s), 6)) (s = 0: magnitude 0), sign bit kept; 4/6
  keeps M = 4 iff its binary64 squared error sum (element order) is smaller;
  round to nearest (the paper attaches SR to the first moment only);
* decode: u = fl32(q s) (exact), the inverse rotation (binary32) with the signs of
  step t - 1, y_hat = fl32(r + mu), v_hat = fl32(y_hat y_hat);
* update (binary32, IEEE division and square root): bc1 = fl32(1 - beta1^(t+1)),
  bc2 = fl32(1 - beta2^(t+1)) with the powers formed by repeated binary64
  multiplication of the binary32 betas; upd = fl32(fl32(m_t / bc1) /
  fl32(fl32(sqrt(fl32(v_t / bc2))) + eps)); W' = bf16(fl32(fl32(W c1) - fl32(lr upd))),
  c1 = fl32(1 - fl32(lr wd)); m_t and v_t are the binary32 moments of this step
  (before their storage rounding).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import momentum
from .formats import E2M1_GRID, e2m1_index
from .rht import rotate_blocks_f32, step_signs, unrotate_blocks_f32
from .root_step import bf16_round, bf16_value

TILE = 256


@dataclass
class VState:
    codes: np.ndarray    # (N,) uint8 4-bit codes
    scales: np.ndarray   # (N/16,) uint16 BF16 block scales
    means: np.ndarray    # (N/256,) uint16 BF16 tile means


def tile_means(y: np.ndarray) -> np.ndarray:
    """BF16 bit patterns of the tile means of binary32 y (N,), summed as defined above."""
    blocks = np.asarray(y, np.float32).astype(np.float64).reshape(-1, 16, 16)
    b = np.zeros(blocks.shape[:2])
    for i in range(16):                       # element order within a block
        b = b + blocks[:, :, i]
    while b.shape[1] > 1:                     # pairwise tree over the 16 block sums
        b = b[:, 0::2] + b[:, 1::2]
    return bf16_round((b[:, 0] / TILE).astype(np.float32))


def encode_v(v: np.ndarray, signs: np.ndarray | None, adaptive46: bool = True) -> VState:
    """Second-moment state (square root, tile-mean separation, rotation, NVFP4 with BF16 scales)."""
    v = np.asarray(v, np.float32)
    y = np.sqrt(v).astype(np.float32)
    means = tile_means(y)
    mu = np.repeat(bf16_value(means), TILE)
    r = (y - mu).astype(np.float32).reshape(-1, 16)
    u = rotate_blocks_f32(r, signs) if signs is not None else r
    neg = np.signbit(u)
    mag = np.abs(u)
    bmax = mag.max(axis=1)
    best = None
    for M in ((6, 4) if adaptive46 else (6,)):
        s = bf16_value(bf16_round((bmax / np.float32(M)).astype(np.float32)))
        with np.errstate(divide="ignore", invalid="ignore"):
            y_el = (mag / s[:, None]).astype(np.float32)
        y_el = np.where(s[:, None] > 0, np.minimum(y_el, np.float32(6.0)), np.float32(0.0))
        idx = e2m1_index(y_el.reshape(-1)).reshape(y_el.shape)
        dec = E2M1_GRID[idx] * s.astype(np.float64)[:, None]
        diff = u.astype(np.float64) - np.where(neg, -dec, dec)
        err = np.zeros(len(bmax))
        for i in range(16):
            err = err + diff[:, i] * diff[:, i]
        cand = (bf16_round(s), idx, err)
        if best is None:
            best = cand
        else:
            take = cand[2] < best[2]
            best = (np.where(take, cand[0], best[0]), np.where(take[:, None], cand[1], best[1]),
                    np.where(take, cand[2], best[2]))
    codes = ((neg.astype(np.uint8) << 3) | best[1].astype(np.uint8)).reshape(-1)
    return VState(codes, best[0].astype(np.uint16), means)


def decode_v(st: VState, signs: np.ndarray | None) -> np.ndarray:
    q = E2M1_GRID[st.codes & 7]
    q = np.where(st.codes & 8, -q, q).reshape(-1, 16)
    u = (q * bf16_value(st.scales).astype(np.float64)[:, None]).astype(np.float32)   # exact
    r = unrotate_blocks_f32(u, signs) if signs is not None else u
    y = (r.reshape(-1) + np.repeat(bf16_value(st.means), TILE)).astype(np.float32)
    return (y * y).astype(np.float32)


def bias_correction(beta: float, t: int) -> np.float32:
    p = 1.0
    b = float(np.float32(beta))
    for _ in range(t + 1):
        p = p * b
    return np.float32(1.0 - p)


def adamw_step(g, w_bf16, m_prev, v_prev: VState | None, step: int, lr: float, wd: float, beta1: float,
               beta2: float, eps: float, seed: int, hadamard: bool = True, adaptive46: bool = True,
               sr: bool = True):
    """One Q-AdamW step of a flat parameter: returns (new BF16 weights, m state, v state, m_t, v_t)."""
    g = np.asarray(g, np.float32)
    n = g.size
    m_t, m_state = momentum.momentum_step(g.reshape(n // TILE, TILE), m_prev, beta1, seed, step,
                                          hadamard=hadamard, adaptive46=adaptive46, sr=sr)
    m_t = m_t.reshape(-1)
    sg_prev = step_signs(seed, step - 1) if (hadamard and step > 0) else None
    v_hat = decode_v(v_prev, sg_prev) if step > 0 else np.zeros(n, np.float32)
    b2 = np.float32(beta2)
    c2 = np.float32(np.float32(1.0) - b2)
    gg = (g * g).astype(np.float32)
    v_t = (np.float64(b2) * v_hat.astype(np.float64) + np.float64(c2) * gg.astype(np.float64)).astype(np.float32)
    v_state = encode_v(v_t, step_signs(seed, step) if hadamard else None, adaptive46)
    bc1, bc2 = bias_correction(beta1, step), bias_correction(beta2, step)
    mh = (m_t / bc1).astype(np.float32)
    vh = (v_t / bc2).astype(np.float32)
    den = (np.sqrt(vh).astype(np.float32) + np.float32(eps)).astype(np.float32)
    upd = (mh / den).astype(np.float32)
    lr32, wd32 = np.float32(lr), np.float32(wd)
    c1 = np.float32(np.float32(1.0) - np.float32(lr32 * wd32))
    w = bf16_value(w_bf16)
    w_new = bf16_round(((w * c1).astype(np.float32) - (lr32 * upd).astype(np.float32)).astype(np.float32))
    return w_new, m_state, v_state, m_t, v_t
