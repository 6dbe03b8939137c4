"""Brute-force pins of one NVFP4 Newton-Schulz step and of the normalisation (CPU only).

The NVFP4 step of Section 3.4 (display equation) is re-derived here in scalar
exact-rational arithmetic, written separately from the oracle: every binary32
operation is the exact result rounded once (to nearest, ties to even, with
binary32's subnormals) by integer arithmetic, the E4M3 and E2M1 roundings are
nearest-point searches over the format definitions, the 4/6 block errors are
summed in Python floats (IEEE binary64) in element order, and every product's
sum is an exact integer before its single rounding to binary64.  The oracle
must agree with it bit for bit on A, qA, B, qB and X_{k+1}, with the rotation
on and off and with adaptive 4/6 on and off.  Slips such as pairing qB's tensor
scale with qX's instead of qXt's, rounding P to binary32 before it is combined
with A, or a transposed operand change these bits.

The normalisation X_0 = fl32(X * fl32(1 / (||X||_F + eps))) is pinned by what
the definition fixes: the Frobenius norm of X_0 (math.fsum) equals
nu / (nu + eps) to a few binary32 ulps, eps decides the result where nu is
comparable to it, a zero matrix stays zero, and a matrix of +-1 entries maps to
+-fl32(1 / (n + eps)).
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import ns, rht
from oracle.quantize import NVFP4, quantize

# ---------------------------------------------------------------------------
# exact binary32 rounding of a rational


def fl32(v: Fraction) -> Fraction:
    """Round a rational to the nearest binary32 value (ties to even, subnormals kept)."""
    if v == 0:
        return Fraction(0)
    neg = v < 0
    a = -v if neg else v
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    quantum = max(e - 23, -149)
    scaled = a / Fraction(2) ** quantum
    n = scaled.numerator // scaled.denominator
    rem = scaled - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = n * Fraction(2) ** quantum
    assert r < Fraction(2) ** 128
    return -r if neg else r


def as_f32(v: Fraction) -> float:
    return float(v)   # a binary32 value is exact in binary64


# the format definitions: E4M3FN (bias 7, three mantissa bits, subnormals m/8 2^-6,
# largest finite 448) and the E2M1 magnitudes of the 3-bit codes
E4M3 = [(Fraction(c & 7, 8) * Fraction(2) ** -6) if (c >> 3) == 0 else
        (1 + Fraction(c & 7, 8)) * Fraction(2) ** ((c >> 3) - 7) for c in range(127)]
E2M1 = [Fraction(0), Fraction(1, 2), Fraction(1), Fraction(3, 2), Fraction(2), Fraction(3), Fraction(4), Fraction(6)]


def nearest_even(v: Fraction, grid) -> int:
    best = None
    for i, g in enumerate(grid):
        d = abs(v - g)
        if best is None or d < best[0] or (d == best[0] and i % 2 == 0):
            best = (d, i)
    return best[1]


# ---------------------------------------------------------------------------
# scalar quantiser (Section 2 NVFP4 decode; readings of the encode as the oracle's header)


def rotate16(block, signs):
    """diag(d) H_16 / 4 applied to one 16-element block, every butterfly rounded to binary32."""
    u = [x * (float(signs[i]) if signs is not None else 1.0) for i, x in enumerate(block)]
    if signs is None:
        return u
    h = 1
    while h < 16:
        for i0 in range(0, 16, 2 * h):
            for j in range(i0, i0 + h):
                a, b = u[j], u[j + h]
                s, d = a + b, a - b
                u[j] = s if s == 0 else as_f32(fl32(Fraction(a) + Fraction(b)))
                u[j + h] = d if d == 0 else as_f32(fl32(Fraction(a) - Fraction(b)))
        h *= 2
    return [v if v == 0 else as_f32(fl32(Fraction(v) / 4)) for v in u]


def quantize_bf(x, axis, signs, adaptive46):
    """(codes, scale codes, s_g) of Q_1x16 (axis 1) or Q_16x1 (axis 0, laid out transposed)."""
    rows = [list(map(float, r)) for r in (np.asarray(x, np.float32).T if axis == 0 else np.asarray(x, np.float32))]
    nb = len(rows[0]) // 16
    blocks = [[rotate16(r[16 * b:16 * b + 16], signs) for b in range(nb)] for r in rows]
    amax = max((abs(v) for r in blocks for blk in r for v in blk), default=0.0)
    sg = fl32(Fraction(amax) / 2688)
    codes, scodes = [], []
    for r in blocks:
        crow, srow = [], []
        for u in r:
            signbits = [8 if math.copysign(1.0, v) < 0 else 0 for v in u]
            if sg == 0:
                crow += signbits
                srow.append(0)
                continue
            bmax = Fraction(max(abs(v) for v in u))
            best = None
            for M in ((6, 4) if adaptive46 else (6,)):
                den = fl32(M * sg)
                v = min(fl32(bmax / den), Fraction(448))
                sc = nearest_even(v, E4M3)
                s = E4M3[sc]
                rr = fl32(s * sg)
                idx = [0 if rr == 0 else nearest_even(min(fl32(abs(Fraction(uu)) / rr), Fraction(6)), E2M1)
                       for uu in u]
                err = 0.0
                for uu, ii in zip(u, idx):
                    dec = float(E2M1[ii] * s) * float(sg)
                    dec = -dec if math.copysign(1.0, uu) < 0 else dec
                    diff = uu - dec
                    err = err + diff * diff
                if best is None or err < best[0]:
                    best = (err, sc, idx)
            _, sc, idx = best
            crow += [sb | i for sb, i in zip(signbits, idx)]
            srow.append(sc)
        codes.append(crow)
        scodes.append(srow)
    return codes, scodes, sg


def decoded_ints(codes, scodes):
    """Every element as the integer q * s * 2^10 (exact: q in halves, s a multiple of 2^-9)."""
    out = []
    for crow, srow in zip(codes, scodes):
        r = []
        for k, c in enumerate(crow):
            v = E2M1[c & 7] * E4M3[srow[k // 16]] * 1024
            assert v.denominator == 1
            r.append(-int(v) if c & 8 else int(v))
        out.append(r)
    return out


def dot64(a, b) -> float:
    """binary64 rounding of the exact sum of products of two rows of decoded_ints (scaled back)."""
    return float(Fraction(sum(p * q for p, q in zip(a, b)), 1 << 20))


def f32_of(v: float) -> float:
    return float(np.float32(v))   # binary64 -> binary32 is one correctly rounded step


def step_bf(x, a, b, c, signs, adaptive46):
    """One NVFP4 NS step from the definitions; returns every intermediate."""
    x = np.asarray(x, np.float32)
    m, n = x.shape
    a64, b64, c64 = (float(np.float32(t)) for t in (a, b, c))
    qx = quantize_bf(x, 1, signs, adaptive46)
    qxt = quantize_bf(x, 0, signs, adaptive46)
    dx = decoded_ints(qx[0], qx[1])
    sgx2 = float(qx[2]) * float(qx[2])
    A = np.array([[f32_of(sgx2 * dot64(dx[i], dx[j])) for j in range(m)] for i in range(m)], np.float32)
    qa = quantize_bf(A, 1, signs, adaptive46)
    da = decoded_ints(qa[0], qa[1])
    sga2 = float(qa[2]) * float(qa[2])
    B = np.array([[f32_of(b64 * float(A[i, j]) + c64 * (sga2 * dot64(da[i], da[j]))) for j in range(m)]
                  for i in range(m)], np.float32)
    qb = quantize_bf(B, 1, signs, adaptive46)
    db = decoded_ints(qb[0], qb[1])
    dxt = decoded_ints(qxt[0], qxt[1])
    alpha = float(qb[2]) * float(qxt[2])
    X1 = np.array([[f32_of(a64 * float(x[i, j]) + alpha * dot64(db[i], dxt[j])) for j in range(n)]
                   for i in range(m)], np.float32)
    return dict(qx=qx, qxt=qxt, A=A, qa=qa, B=B, qb=qb, X1=X1)


def _same_q(q: NVFP4, ref):
    codes, scodes, sg = ref
    assert np.array_equal(q.codes, np.array(codes, np.uint8))
    assert np.array_equal(q.scales, np.array(scodes, np.uint8))
    assert np.float32(q.sg).view(np.uint32) == np.float32(float(sg)).view(np.uint32)


def _bits(v):
    return np.asarray(v, np.float32).view(np.uint32)


def _input(shape, seed):
    """Clipped, normalised, oriented X_0 of a heavy-tailed matrix with a zero block and a -0.0."""
    rng = np.random.default_rng(seed)
    m = (rng.standard_t(3, size=shape) * rng.lognormal(0, 1, size=(shape[0], 1))).astype(np.float32)
    m[0, :16] = 0.0
    m[1, 3] = -0.0
    x, _, _ = ns.prepare(m)
    return x


@pytest.mark.parametrize("shape", [(16, 32), (48, 32)])
@pytest.mark.parametrize("hadamard", [True, False])
@pytest.mark.parametrize("adaptive46", [True, False])
def test_ns_step_matches_exact_rational_brute_force(shape, hadamard, adaptive46):
    x = _input(shape, 7 + shape[0])
    coeffs = (3.4445, -4.7750, 2.0315)
    signs = rht.step_signs(11, 2) if hadamard else None
    tr = {}
    x1 = ns.ns_step_nvfp4(x, *coeffs, signs, adaptive46, trace=tr)
    bf = step_bf(x, *coeffs, signs, adaptive46)
    _same_q(tr["qx"], bf["qx"])
    _same_q(tr["qxt"], bf["qxt"])
    assert np.array_equal(_bits(tr["A"]), _bits(bf["A"]))
    _same_q(tr["qa"], bf["qa"])
    assert np.array_equal(_bits(tr["B"]), _bits(bf["B"]))
    _same_q(tr["qb"], bf["qb"])
    assert np.array_equal(_bits(x1), _bits(bf["X1"]))


def test_brute_force_detects_a_swapped_tensor_scale():
    # the pin is sharp: the same step with qB's tensor scale paired with qX's changes X_{k+1}
    x = _input((16, 32), 3)
    coeffs = (3.4445, -4.7750, 2.0315)
    signs = rht.step_signs(1, 0)
    tr = {}
    x1 = ns.ns_step_nvfp4(x, *coeffs, signs, True, trace=tr)
    assert tr["qx"].sg != tr["qxt"].sg
    wrong = ns.f32(np.float64(np.float32(coeffs[0])) * x.astype(np.float64) +
                   (np.float64(tr["qb"].sg) * np.float64(tr["qx"].sg)) * ns.block_dot64(tr["qb"], tr["qxt"]))
    assert not np.array_equal(_bits(wrong), _bits(x1))


# ---------------------------------------------------------------------------
# exact products


def _nvfp4(rng, rows, cols, spread):
    """Random NVFP4 operand whose block exponents span `spread` binades within each row."""
    codes = rng.integers(0, 16, size=(rows, cols)).astype(np.uint8)
    top = rng.integers(8, 15, size=(rows, 1))
    ef = np.clip(top - rng.integers(0, spread + 1, size=(rows, cols // 16)), 0, 15)
    scales = ((ef << 3) | rng.integers(0, 8, size=(rows, cols // 16))).astype(np.uint8)
    scales[scales == 0x7F] = 0x7E
    return NVFP4(codes, scales, np.float32(1.0), np.zeros((rows, cols // 16), bool))


@pytest.mark.parametrize("spread", [2, 15])
def test_block_dot64_is_the_correctly_rounded_exact_sum(spread):
    # spread 15 forces the math.fsum path on most entries, spread 2 the BLAS path
    rng = np.random.default_rng(spread)
    qa, qb = _nvfp4(rng, 24, 4096, spread), _nvfp4(rng, 20, 4096, spread)
    got = ns.block_dot64(qa, qb)
    da, db = qa.block_values(), qb.block_values()
    for i in range(0, 24, 5):
        for j in range(0, 20, 3):
            assert got[i, j] == math.fsum(da[i] * db[j])
    g = ns.block_dot64(qa)
    assert np.array_equal(g, g.T)
    for i in range(0, 24, 7):
        for j in range(0, 24, 5):
            assert g[i, j] == math.fsum(da[i] * da[j])


# ---------------------------------------------------------------------------
# normalisation (Muon convention read for Section 2; eps = 1e-7)


@pytest.mark.parametrize("shape,scale", [((16, 32), 1.0), ((64, 48), 1e-3), ((8, 160), 3e4)])
def test_normalise_has_unit_frobenius_norm(shape, scale):
    rng = np.random.default_rng(shape[0])
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    nu = math.sqrt(math.fsum(float(v) * float(v) for v in x.ravel()))
    x0 = ns.normalise(x)
    got = math.sqrt(math.fsum(float(v) * float(v) for v in x0.ravel()))
    want = nu / (nu + float(np.float32(1e-7)))
    assert abs(got - want) <= 4 * 2.0 ** -24 * want


def test_normalise_eps_decides_near_zero():
    # nu = eps: X_0 = X / (2 eps), whose norm is 1/2
    x = np.zeros((16, 16), np.float32)
    eps = float(np.float32(1e-7))
    x[3, 5] = np.float32(eps)
    x0 = ns.normalise(x)
    assert abs(float(x0[3, 5]) - 0.5) <= 2.0 ** -24
    assert np.count_nonzero(x0) == 1


def test_normalise_zero_matrix_stays_zero():
    x0 = ns.normalise(np.zeros((16, 48), np.float32))
    assert np.all(x0 == 0) and np.all(np.isfinite(x0))


def test_normalise_unit_entries():
    # 256 entries of +-1: nu = 16 exactly, every |X_0| = fl32(1 / (16 + eps)) (eps binary32)
    rng = np.random.default_rng(5)
    x = np.where(rng.random((16, 16)) < 0.5, -1.0, 1.0).astype(np.float32)
    x0 = ns.normalise(x)
    inv = fl32(1 / (16 + Fraction(float(np.float32(1e-7)))))
    assert np.all(np.abs(x0) == np.float32(float(inv)))
    assert np.array_equal(np.signbit(x0), np.signbit(x))
