"""Pins of the quantized-state AdamW oracle (oracle/qadamw.py).

* tile means: equal to the correctly rounded mean (math.fsum) on random tiles, and
  to the constant itself on constant tiles;
* the second-moment storage round-trips exactly where every stage is exact
  (square roots of binary32 squares, zero-sum residuals on the E2M1 grid times a
  BF16 scale), and its reconstruction error stays below direct NVFP4 storage of
  v on heavy-tailed synthetic second moments (the ordering of Section 3.3's
  component analysis; the paper's values come from real training states);
* bias corrections and the update in closed form (beta = 0, eps = 0: the update
  is the sign of g; beta = 1/2 corrections 1/2, 3/4, 7/8).
"""
import math

import numpy as np

from oracle import qadamw as Q
from oracle.formats import E2M1_GRID
from oracle.quantize import quantize
from oracle.root_step import bf16_round, bf16_value


def test_tile_means_match_exact_mean():
    rng = np.random.default_rng(0)
    y = np.abs(rng.standard_t(3, 256 * 400)).astype(np.float32) * np.float32(1e-3)
    got = Q.tile_means(y)
    want = [bf16_round(np.float32(math.fsum(map(float, y[k * 256:(k + 1) * 256])) / 256))
            for k in range(400)]
    assert np.array_equal(got, np.array(want, np.uint16))
    c = np.full(512, np.float32(0.3359375), np.float32)
    assert np.array_equal(Q.tile_means(c), bf16_round(np.float32([0.3359375, 0.3359375])))


def test_v_storage_exact_round_trip():
    rng = np.random.default_rng(1)
    s = np.float32(2.0 ** -4)
    half = rng.choice(E2M1_GRID, size=(4, 8, 16)) * rng.choice([-1, 1], size=(4, 8, 16))
    half[..., 0] = 6.0                                    # block maximum 6 s: the scale is s itself
    r = np.concatenate([half, -half], axis=1).astype(np.float32) * s   # zero-sum tiles
    y = (np.float32(1.0) + r).reshape(-1).astype(np.float32)
    v = (y * y).astype(np.float32)
    st = Q.encode_v(v, None, adaptive46=True)
    assert np.array_equal(bf16_value(st.means), np.ones(4, np.float32))
    assert np.array_equal(Q.decode_v(st, None), v)


def test_v_pipeline_beats_direct_nvfp4():
    rng = np.random.default_rng(2)
    n = 256 * 256
    scale = np.repeat(rng.lognormal(0, 1, n // 256), 256)
    v = np.zeros(n)
    for _ in range(20):                                   # EMA of squared heavy-tailed gradients
        g = rng.standard_t(3, n) * scale * 1e-3
        v = 0.95 * v + 0.05 * g * g
    v = v.astype(np.float32)
    signs = Q.step_signs(4, 0)
    full = Q.decode_v(Q.encode_v(v, signs), signs)
    direct = quantize(v.reshape(-1, 256), axis=1, adaptive46=True).dequantize().reshape(-1)
    e_full = np.linalg.norm(full - v) / np.linalg.norm(v)
    e_direct = np.linalg.norm(direct - v) / np.linalg.norm(v)
    assert e_full < e_direct


def test_bias_correction_and_sign_update():
    assert [Q.bias_correction(0.5, t) for t in range(3)] == [np.float32(0.5), np.float32(0.75), np.float32(0.875)]
    rng = np.random.default_rng(3)
    g = rng.standard_normal(512).astype(np.float32)
    w0 = bf16_round(np.zeros(512, np.float32))
    w1, _, vst, m_t, v_t = Q.adamw_step(g, w0, None, None, 0, 2.0 ** -10, 0.0, 0.0, 0.0, 0.0, 1)
    assert np.array_equal(m_t, g) and np.array_equal(v_t, g * g)
    assert np.array_equal(bf16_value(w1), np.where(g > 0, np.float32(-2.0 ** -10), np.float32(2.0 ** -10)))
    z = Q.encode_v(np.zeros(512, np.float32), Q.step_signs(1, 0))
    assert not np.any(z.scales) and not np.any(z.means) and not np.any(Q.decode_v(z, Q.step_signs(1, 0)))
