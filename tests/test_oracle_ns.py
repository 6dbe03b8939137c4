"""Pins for the oracle's Newton-Schulz recurrence (CPU only)."""
import numpy as np
import pytest
import torch

from oracle import ns, rht
from oracle.quantize import quantize
from paper_2607_04422_amd import workloads

CONV = [(15 / 8, -10 / 8, 3 / 8)] * 5


def _rel(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


@pytest.mark.parametrize("shape", [(64, 64), (48, 160), (96, 32)])
@pytest.mark.parametrize("coeffs", [[ns.MUON_COEFFS] * 5, CONV, [(3.0, -3.2, 1.2), (2.0, -1.5, 0.5)]])
def test_exact_ns_equals_svd_closed_form(shape, coeffs):
    rng = np.random.default_rng(0)
    m = rng.standard_normal(shape).astype(np.float32)
    out = ns.orthogonalize(m, coeffs, clip_on=False, mode="exact")
    x0, tall, _ = ns.prepare(m, clip_on=False)
    ref = ns.closed_form(x0.astype(np.float64), coeffs)
    ref = ref.T if tall else ref
    assert _rel(out, ref) < 1e-12


def test_muon_singular_value_band():
    # the band p^5 maps [0.01, 1] into, from a dense evaluation of the scalar polynomial
    s = np.linspace(0.01, 1.0, 200001)
    t = s.copy()
    for _ in range(5):
        t = ns.poly(t, *ns.MUON_COEFFS)
    lo, hi = t.min(), t.max()
    assert 0.68 < lo < 0.69 and 1.13 < hi < 1.14
    grid = np.linspace(0, 1, 100001)
    pmax = ns.poly(grid, *ns.MUON_COEFFS).max()
    assert abs(pmax - 1.2024) < 1e-3
    # a matrix whose singular values all lie in [0.01, 1] lands in that band after exact NS
    rng = np.random.default_rng(1)
    u, _ = np.linalg.qr(rng.standard_normal((40, 40)))
    v, _ = np.linalg.qr(rng.standard_normal((80, 40)))
    sig = np.linspace(0.01, 1.0, 40)
    x = (u * sig) @ v.T
    for _ in range(5):
        x = ns.ns_step_exact(x, *ns.MUON_COEFFS)
    out_s = np.linalg.svd(x, compute_uv=False)
    assert out_s.min() >= lo - 1e-9 and out_s.max() <= hi + 1e-9


def test_rotations_cancel_when_quantisation_is_identity():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((32, 64)) / 40
    for k in range(3):
        d = rht.step_signs(5, k)
        assert _rel(ns.ns_step_exact(x, *CONV[0], signs=d), ns.ns_step_exact(x, *CONV[0])) < 1e-13


def test_rotation_placement_sensitivity():
    # a rotation on only one side of a product must not cancel: guards the H placement
    rng = np.random.default_rng(3)
    x = rng.standard_normal((32, 64)) / 40
    d = rht.step_signs(5, 0)
    xh = ns.rotate64(x, d, 1)
    assert _rel(xh @ x.T, x @ x.T) > 0.1


def test_quantised_step_structure():
    m = workloads.matrix(64, 128, 7)
    x, _, _ = ns.prepare(m)
    d = rht.step_signs(0, 0)
    tr = {}
    ns.ns_step_nvfp4(x, *CONV[0], signs=d, trace=tr)
    A, B = tr["A"], tr["B"]
    assert np.array_equal(A, A.T) and np.array_equal(B, B.T)
    qa0 = quantize(A, 0, d)
    assert np.array_equal(qa0.codes, tr["qa"].codes) and np.array_equal(qa0.scales, tr["qa"].scales)
    # operands decode close to the rotated matrices they stand for (NVFP4 error level)
    assert _rel(tr["qx"].dequantize(), ns.rotate64(x, d, 1)) < 0.12
    assert _rel(tr["qxt"].dequantize(), ns.rotate64(x.T, d, 1)) < 0.12


def test_quantiser_identity_reduces_to_exact_step():
    # with amax fixing s_g and values exactly on the NVFP4 grid, A = X X^T exactly
    x = np.zeros((16, 32), np.float32)
    x[:, :16] = np.float32(1.0)
    tr = {}
    ns.ns_step_nvfp4(x, 1.0, 0.0, 0.0, None, trace=tr)
    assert np.array_equal(tr["A"].astype(np.float64), x.astype(np.float64) @ x.T.astype(np.float64))


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(4)
    x = (rng.standard_normal(200000) * np.exp2(rng.integers(-20, 20, 200000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ns.to_bf16(x.astype(np.float64)), ref)


def test_bf16_path_close_to_exact():
    m = workloads.matrix(64, 192, 8)
    e = ns.orthogonalize(m, CONV, mode="exact")
    b = ns.orthogonalize(m, CONV, mode="bf16")
    assert _rel(b, e) < 2e-2


def test_quantised_route_sanity_band():
    # Section 3.4 reports a few-percent NS error for the proposed route vs about 10% for
    # the plain route on unknown inputs; here: the proposed route stays within a sanity band
    m = workloads.small_case()[0]
    e = ns.orthogonalize(m, CONV, mode="exact")
    q = ns.orthogonalize(m, CONV, mode="nvfp4", seed=1)
    err = _rel(q, e)
    assert 0.005 < err < 0.2
