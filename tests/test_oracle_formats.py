"""Pins for the oracle's number formats and Hadamard rotation (CPU only)."""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import formats, rht

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLD, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def test_e4m3_table_matches_torch_float8():
    codes = torch.arange(127, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(formats.E4M3_GRID, ref)


def test_e4m3_golden_points():
    for code, val in _rows("e4m3_points.txt"):
        assert formats.E4M3_GRID[int(code, 16)] == float(val)


def _fp32_neighbourhood(centres, k=64):
    bits = np.asarray(centres, dtype=np.float32).view(np.uint32).astype(np.int64)
    offs = np.arange(-k, k + 1)
    b = (bits[:, None] + offs[None, :]).reshape(-1)
    b = b[(b >= 0) & (b < 0x7F800000)]
    return np.unique(b.astype(np.uint32)).view(np.float32)


def test_e4m3_encode_matches_torch_cast_near_every_boundary():
    g = formats.E4M3_GRID
    mids = (g[:-1] + g[1:]) / 2
    x = _fp32_neighbourhood(np.concatenate([g, mids]), k=256)
    rng = np.random.default_rng(0)
    x = np.concatenate([x, (rng.random(2_000_000) * 448).astype(np.float32),
                        np.exp2(rng.uniform(-30, 8.8, 1_000_000)).astype(np.float32)])
    x = x[(x >= 0) & (x <= 448)]
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(formats.e4m3_encode(x), ref)


def test_e4m3_saturating_points():
    # the quantiser clamps to 448 before rounding; RNE itself also sends 449 and 464 to 448
    ref = torch.tensor([449.0, 464.0]).to(torch.float8_e4m3fn).view(torch.uint8).tolist()
    assert ref == [0x7E, 0x7E]
    assert formats.e4m3_encode(np.minimum(np.float32([449, 464, 448]), 448)).tolist() == [0x7E] * 3
    with pytest.raises(ValueError):
        formats.e4m3_encode(np.float32([449]))
    assert formats.E4M3_GRID[formats.e4m3_encode(np.float32([2.0 ** -10]))[0]] == 0.0
    assert formats.E4M3_GRID[formats.e4m3_encode(np.float32([1.5 * 2.0 ** -10]))[0]] == 2.0 ** -9


def _e2m1_bruteforce(y):
    """Nearest grid point by exact rational distance, ties to the even index."""
    fy = Fraction(float(y))
    grid = [Fraction(v).limit_denominator() for v in formats.E2M1_GRID]
    d = [abs(fy - g) for g in grid]
    best = min(d)
    cands = [i for i, di in enumerate(d) if di == best]
    return min(cands, key=lambda i: (i % 2, i))


def test_e2m1_tie_table():
    for y, idx, val in _rows("e2m1_ties.txt"):
        got = int(formats.e2m1_index(np.float32([float(y)]))[0])
        assert got == int(idx)
        assert formats.E2M1_GRID[got] == float(val)


def test_e2m1_bruteforce_neighbourhoods():
    g = formats.E2M1_GRID
    mids = (g[:-1] + g[1:]) / 2
    x = _fp32_neighbourhood(np.concatenate([g, mids]), k=40)
    x = x[(x >= 0) & (x <= 6)]
    rng = np.random.default_rng(1)
    x = np.concatenate([x, (rng.random(3000) * 6).astype(np.float32)])
    got = formats.e2m1_index(x)
    ref = np.array([_e2m1_bruteforce(v) for v in x])
    assert np.array_equal(got, ref)


def test_nibble_packing_order():
    codes = np.arange(16, dtype=np.uint8).reshape(1, 16)
    packed = formats.pack_nibbles(codes)
    assert packed[0, 0] == 0x10 and packed[0, 7] == 0xFE
    assert np.array_equal(formats.unpack_nibbles(packed), codes)


def test_splitmix64_published_outputs():
    for idx, hx in _rows("splitmix64.txt"):
        assert rht.splitmix64(0, int(idx)) == int(hx, 16)


def test_hadamard_orthogonal_exactly():
    for step in range(4):
        d = rht.step_signs(1234, step).astype(np.float64)
        h = np.diag(d) @ rht.sylvester16() / 4.0
        assert np.array_equal(h @ h.T, np.eye(16))
    from scipy.linalg import hadamard
    assert np.array_equal(rht.sylvester16(), hadamard(16))


def test_butterfly_equals_matrix_product():
    rng = np.random.default_rng(2)
    d = rht.step_signs(7, 3)
    h = np.diag(d.astype(np.float64)) @ rht.sylvester16() / 4.0
    # small integers: every butterfly is exact, so the product must match bit for bit
    xi = rng.integers(-1000, 1000, size=(300, 16)).astype(np.float32)
    assert np.array_equal(rht.rotate_blocks_f32(xi, d).astype(np.float64), xi.astype(np.float64) @ h)
    # general floats: equal to binary32 rounding (4 rounded additions)
    xf = rng.standard_normal((2000, 16)).astype(np.float32)
    ref = xf.astype(np.float64) @ h
    got = rht.rotate_blocks_f32(xf, d).astype(np.float64)
    scale = np.abs(xf).astype(np.float64) @ np.abs(h)
    assert np.all(np.abs(got - ref) <= 4 * 2.0 ** -24 * scale * 4 + 1e-30)
