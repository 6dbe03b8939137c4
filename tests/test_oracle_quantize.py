"""Pins for the oracle's NVFP4 quantiser (CPU only): enumeration, invariances, brute-force 4/6."""
import numpy as np
import pytest

from oracle import formats, rht
from oracle.quantize import quantize

E2 = formats.E2M1_GRID
E4 = formats.E4M3_GRID


def _enumeration_matrix(sg_exp):
    """Rows of 16-blocks built as q * s * s_g for every sign, magnitude and finite positive scale.

    s_g is a power of two so that every product below is exact; one block at scale
    448 with element 6 fixes amax = 2688 * s_g.  Each block holds element 6 (its
    block maximum) so that the M=6 scale is exactly s.
    """
    sg = np.float32(2.0 ** sg_exp)
    blocks, exp_codes, exp_scales = [], [], []
    for sc in range(1, 127):
        s = E4[sc]
        for start in range(0, 16, 15):
            idx = np.array([(start + j) % 16 for j in range(16)]) % 8   # magnitudes 0..7 twice
            sign = (np.arange(16) + sc + start) % 2
            idx[0] = 7
            vals = np.where(sign, -1.0, 1.0) * E2[idx] * s * float(sg)
            blocks.append(vals)
            exp_codes.append((sign << 3) | idx)
            exp_scales.append(sc)
    x = np.array(blocks, dtype=np.float64)
    assert np.array_equal(x.astype(np.float32).astype(np.float64), x)
    return x.astype(np.float32), np.array(exp_codes, np.uint8), np.array(exp_scales, np.uint8), sg


@pytest.mark.parametrize("sg_exp", [-20, -3, 0, 5])
@pytest.mark.parametrize("adaptive", [False, True])
def test_enumeration_round_trip(sg_exp, adaptive):
    x, codes, scales, sg = _enumeration_matrix(sg_exp)
    q = quantize(x, 1, None, adaptive)
    assert q.sg == sg
    assert np.array_equal(q.scales[:, 0], scales)
    assert np.array_equal(q.codes, codes)
    assert np.array_equal(q.dequantize(), x.astype(np.float64))


def test_zero_and_signed_zero():
    x = np.zeros((2, 32), np.float32)
    x[1, 3] = -0.0
    q = quantize(x, 1)
    assert q.sg == 0 and not q.scales.any()
    assert q.codes[1, 3] == 8 and q.codes[0, 3] == 0


def test_zero_block_beside_nonzero_block():
    x = np.zeros((1, 32), np.float32)
    x[0, 20] = 2688.0                     # s_g = 1, s = 448: decodes exactly
    q = quantize(x, 1)
    assert q.scales[0, 0] == 0 and not q.codes[0, :16].any()
    assert q.dequantize()[0, 20] == 2688.0


def test_saturation_and_midpoint_ties():
    # block max 6*s*sg with s=1, sg=1/448: elements at E2M1 midpoints round to even
    sg = np.float32(1.0)
    big = np.zeros(16, np.float32); big[0] = 2688.0           # fixes amax -> sg = 1
    blk = np.float32([6, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 0.5, 1, 1.5, 2, 3, 4, 5.9, 6])
    x = np.stack([big, blk])
    q = quantize(x, 1, None, adaptive46=False)
    assert q.sg == sg and q.scales[1, 0] == 0x38               # s = 1
    assert list(E2[q.codes[1] & 7]) == [6, 0, 1, 1, 2, 2, 4, 4, 0.5, 1, 1.5, 2, 3, 4, 6, 6]


def test_scale_underflow_to_zero_keeps_signs():
    # a block far below the matrix maximum gets scale 0 and zero magnitudes
    x = np.zeros((2, 16), np.float32)
    x[0, 0] = 1.0
    x[1, :] = -1e-9
    q = quantize(x, 1, None, adaptive46=False)
    assert q.scales[1, 0] == 0
    assert np.all(q.codes[1] == 8)


def test_subnormal_scales():
    sg = np.float32(2.0 ** -4)
    x = np.zeros((2, 16), np.float32)
    x[0, 0] = 2688 * sg
    for m in range(1, 8):
        s = m * 2.0 ** -9
        x[1, :] = 0
        x[1, 0] = 6 * s * sg
        x[1, 1] = -1.5 * s * sg
        q = quantize(x, 1, None, adaptive46=False)
        assert q.scales[1, 0] == m
        assert q.codes[1, 0] == 7 and q.codes[1, 1] == 8 | 3


@pytest.mark.parametrize("signs", [None, rht.step_signs(3, 1)])
def test_power_of_two_and_negation_invariance(signs):
    rng = np.random.default_rng(4)
    x = (rng.standard_normal((48, 64)) * np.exp(rng.standard_normal((48, 1)))).astype(np.float32)
    q = quantize(x, 1, signs)
    for k in (-7, 3):
        qs = quantize((x * np.float32(2.0 ** k)).astype(np.float32), 1, signs)
        assert qs.sg == np.float32(q.sg * np.float32(2.0 ** k))
        assert np.array_equal(qs.codes, q.codes) and np.array_equal(qs.scales, q.scales)
    qn = quantize(-x, 1, signs)
    assert np.array_equal(qn.codes, q.codes ^ 8)
    assert np.array_equal(qn.scales, q.scales) and qn.sg == q.sg


def test_axis0_is_transposed_axis1():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((64, 48)).astype(np.float32)
    d = rht.step_signs(9, 0)
    a = quantize(x, 0, d)
    b = quantize(np.ascontiguousarray(x.T), 1, d)
    assert np.array_equal(a.codes, b.codes) and np.array_equal(a.scales, b.scales) and a.sg == b.sg


def _brute_block(u, sg, M):
    """Quantise one rotated block by the definition, one element at a time in Python floats."""
    bmax = max(abs(float(t)) for t in u)
    den = np.float32(np.float32(M) * sg)
    v = min(np.float32(np.float32(bmax) / den), np.float32(448.0))
    sc = int(formats.e4m3_encode(np.float32([v]))[0])
    s = np.float32(E4[sc])
    r = np.float32(s * sg)
    codes, err = [], 0.0
    for t in u:
        t = np.float32(t)
        if r == 0:
            idx = 0
        else:
            y = min(np.float32(abs(t) / r), np.float32(6.0))
            idx = int(formats.e2m1_index(np.float32([y]))[0])
        neg = bool(np.signbit(t))
        codes.append((8 if neg else 0) | idx)
        dec = (-1 if neg else 1) * E2[idx] * float(s) * float(sg)
        err = err + (float(t) - dec) * (float(t) - dec)
    return sc, codes, err


def test_adaptive46_choice_bruteforce():
    rng = np.random.default_rng(6)
    x = (rng.standard_t(3, size=(40, 64))).astype(np.float32)
    d = rht.step_signs(11, 2)
    q = quantize(x, 1, d, adaptive46=True)
    u = rht.rotate_blocks_f32(x.reshape(40, 4, 16), d)
    n4 = 0
    for i in range(40):
        for b in range(4):
            s6, c6, e6 = _brute_block(u[i, b], q.sg, 6)
            s4, c4, e4 = _brute_block(u[i, b], q.sg, 4)
            use4 = e4 < e6
            n4 += use4
            assert q.scales[i, b] == (s4 if use4 else s6)
            assert list(q.codes[i, b * 16:(b + 1) * 16]) == (c4 if use4 else c6)
    assert 0 < n4 < 160


def test_block_on_m4_grid_chooses_m4():
    sg = np.float32(1.0)
    x = np.zeros((2, 16), np.float32)
    x[0, 0] = 2688
    x[1, :] = np.float32([4, 3, 2, 1.5, 1, 0.5, 0, 3, 4, 2, 1, 0.5, 3, 1.5, 2, 4]) * np.float32(8.0)
    q = quantize(x, 1, None, adaptive46=True)
    assert q.m4[1, 0]
    assert E4[q.scales[1, 0]] == 8.0
    assert np.array_equal(q.dequantize()[1], x[1].astype(np.float64))
    q6 = quantize(x, 1, None, adaptive46=False)
    assert not np.array_equal(q6.dequantize()[1], x[1].astype(np.float64))


def test_rejects_non_finite():
    x = np.zeros((1, 16), np.float32)
    x[0, 4] = np.nan
    with pytest.raises(ValueError):
        quantize(x, 1)


@pytest.mark.parametrize("axis", [0, 1])
def test_row_subset_equals_full(axis):
    rng = np.random.default_rng(8)
    x = rng.standard_normal((64, 96)).astype(np.float32)
    d = rht.step_signs(2, 4)
    full = quantize(x, axis, d)
    sel = np.array([0, 5, 17, 40])
    part = quantize(x, axis, d, rows=sel)
    assert part.sg == full.sg
    assert np.array_equal(part.codes, full.codes[sel]) and np.array_equal(part.scales, full.scales[sel])
