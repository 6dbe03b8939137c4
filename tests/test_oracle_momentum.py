"""Pins of the first-moment state oracle (oracle/momentum.py).

* the draws equal the scalar SplitMix64 of ``oracle.rht`` (itself pinned to the
  published reference outputs in tests/golden/splitmix64.txt);
* the inverse rotation undoes the rotation exactly where binary32 is exact
  (small integers) and equals (H/4) diag(d) computed as a binary64 matrix product;
* stochastic rounding against exact rational arithmetic (Python fractions) on
  random and crafted quotients, and its mean over a uniform grid of draws equals
  the quotient to within 2^-16 of the grid gap (unbiasedness);
* the state's codes stay within one grid step of round-to-nearest, the decode is
  the quantiser's dequantisation, and the update's special cases beta = 0, 1/2, 1;
* averaged over seeds the decoded stochastic states approach the momentum far
  closer than round-to-nearest does (the bias SR removes).
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import momentum as M
from oracle import rht
from oracle.formats import E2M1_GRID, E4M3_GRID
from oracle.quantize import quantize
from paper_2607_04422_amd import workloads


def test_sr_draws_match_scalar_generator():
    for key, off in [(0, 0), (0x123456789ABCDEF, 5), (M.sr_key(7, 3), (1 << 33) - 10)]:
        d = M.sr_draws(key, 40, off)
        want = [(rht.splitmix64(key, e // 2 + 1) >> (16 if e % 2 else 40)) & 0xFFFFFF for e in range(off, off + 40)]
        assert d.tolist() == want
        assert d.max() < (1 << 24)


def test_unrotate_inverts_rotate_on_small_integers():
    rng = np.random.default_rng(0)
    x = rng.integers(-8, 9, size=(50, 16)).astype(np.float32)
    for seed in range(4):
        d = rht.step_signs(seed, 2)
        u = rht.rotate_blocks_f32(x, d)
        assert np.array_equal(rht.unrotate_blocks_f32(u, d), x)


def test_unrotate_is_the_inverse_matrix():
    rng = np.random.default_rng(1)
    u = rng.standard_normal((200, 16)).astype(np.float32)
    d = rht.step_signs(9, 0)
    want = (u.astype(np.float64) @ (rht.sylvester16() / 4.0)) * d.astype(np.float64)
    got = rht.unrotate_blocks_f32(u, d)
    assert np.max(np.abs(got - want)) <= 8 * np.finfo(np.float32).eps * np.max(np.abs(want))


def _sr_fraction(u, r, rho):
    if r == 0:
        return 0
    x = Fraction(abs(float(u))) / Fraction(float(r))
    lo = max(k for k in range(8) if Fraction(E2M1_GRID[k]) <= x)
    if lo == 7:
        return 7
    frac = (x - Fraction(E2M1_GRID[lo])) / Fraction(E2M1_GRID[lo + 1] - E2M1_GRID[lo])
    return lo + 1 if Fraction(int(rho), 1 << 24) < frac else lo


def test_sr_against_fractions():
    rng = np.random.default_rng(2)
    r = np.float32(E4M3_GRID[rng.integers(1, 127, 400)] * np.float32(0.37))
    y = rng.uniform(0, 7, 400)
    u = (y * r * rng.choice([-1, 1], 400)).astype(np.float32)
    # crafted: on the grid, one ulp either side of grid points and midpoints, saturation
    r0 = np.float32(0.75)
    pts = []
    for gp in list(E2M1_GRID) + [0.25, 0.75, 1.25, 2.5, 3.5, 5.0, 6.5, 9.0]:
        v = np.float32(gp * r0)
        pts += [v, np.nextafter(v, np.float32(0)), np.nextafter(v, np.float32(np.inf))]
    u = np.concatenate([u, np.array(pts, np.float32)])
    r = np.concatenate([r, np.full(len(pts), r0, np.float32)])
    u = np.concatenate([u, np.float32([1.0, -2.0])])
    r = np.concatenate([r, np.float32([0.0, 0.0])])
    for rho in [0, 1, 1 << 23, (1 << 24) - 1] + list(rng.integers(0, 1 << 24, 6)):
        got = M.sr_magnitudes(u, r, np.full(u.shape, rho, np.uint32))
        want = [_sr_fraction(a, b, rho) for a, b in zip(u, r)]
        assert got.tolist() == want, rho


def test_sr_unbiased_over_uniform_draws():
    rng = np.random.default_rng(3)
    r = np.float32(0.5)
    rho = np.arange(0, 1 << 24, 256, dtype=np.uint32)
    for y in list(rng.uniform(0, 6, 20)) + [0.1, 1.999, 4.5, 5.99]:
        u = np.float32(y * r)
        x = float(u) / float(r)
        idx = M.sr_magnitudes(np.full(rho.shape, u), r, rho)
        mean = E2M1_GRID[idx].mean()
        lo = E2M1_GRID[E2M1_GRID <= x].max()
        gap = E2M1_GRID[E2M1_GRID > x].min() - lo
        assert abs(mean - x) <= gap * 2.0 ** -16 + 1e-15


def test_state_codes_neighbour_rtn_and_decode():
    g = workloads.matrix(64, 256, seed=4, kind="normal_outliers")
    d = rht.step_signs(5, 1)
    draws = M.sr_draws(M.sr_key(5, 1), g.size).reshape(g.shape)
    sr = M.encode_state(g, d, True, draws)
    rtn = M.encode_state(g, d, True, None)
    ref = quantize(g, axis=1, signs=d, adaptive46=True)
    assert np.array_equal(rtn.codes, ref.codes) and np.array_equal(rtn.scales, ref.scales)
    assert np.array_equal(sr.scales, rtn.scales) and sr.sg == rtn.sg
    assert np.array_equal(sr.codes & 8, rtn.codes & 8)
    assert np.max(np.abs((sr.codes & 7).astype(int) - (rtn.codes & 7))) <= 1
    assert np.count_nonzero(sr.codes != rtn.codes) > 0
    plain = M.decode_state(rtn, None)
    assert np.array_equal(plain, rtn.dequantize().astype(np.float32))
    rot = M.decode_state(rtn, d)
    assert np.array_equal(rot, rht.unrotate_blocks_f32(plain.reshape(64, 16, 16), d).reshape(64, 256))


def test_update_special_cases():
    g = workloads.matrix(32, 64, seed=6)
    m0, s0 = M.momentum_step(g, None, 0.5, 1, 0)
    assert np.array_equal(m0, g * np.float32(0.5))
    m1, _ = M.momentum_step(g, s0, 1.0, 1, 1)
    assert np.array_equal(m1, M.decode_state(s0, rht.step_signs(1, 0)))
    m2, _ = M.momentum_step(g, s0, 0.0, 1, 1)
    assert np.array_equal(m2, g)
    z, sz = M.momentum_step(np.zeros_like(g), None, 0.9, 1, 0)
    # zero magnitudes (rotated zeros may carry the sign bit: -0 keeps it)
    assert sz.sg == 0 and not np.any(sz.codes & 7) and not np.any(sz.scales) and not np.any(z)


def test_sr_states_unbiased_over_seeds():
    m = workloads.matrix(32, 128, seed=7)
    rtn = M.decode_state(M.encode_state(m, rht.step_signs(0, 0), True, None), rht.step_signs(0, 0))
    acc = np.zeros(m.shape)
    n = 64
    for seed in range(n):
        d = rht.step_signs(seed, 0)
        st = M.encode_state(m, d, True, M.sr_draws(M.sr_key(seed, 0), m.size).reshape(m.shape))
        acc += M.decode_state(st, d)
    mean_err = np.linalg.norm(acc / n - m)
    assert mean_err < 0.5 * np.linalg.norm(rtn - m)
