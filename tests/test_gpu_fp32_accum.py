"""NVFP4 iteration with binary32 product accumulation (FP4ROOT_F_FP32_ACCUM).

In this mode each product adds its exact 16-element block products into one binary32
MFMA accumulator over the whole contraction (tensor-core style) instead of forming the
exact value.  What stays exact is checked exactly, the rest against bounds:
* every quantisation of a traced step equals the oracle's quantisation of the GPU's
  own stage input, bit for bit (the quantisers do not change);
* every product lies within the binary32 accumulation bound of the exact product of
  the same NVFP4 operands: |C - C_exact| <= (K + 2) 2^-24 s_a s_b sum_k |a_k b_k| plus
  the final rounding (K the contraction length; each of the K additions rounds once);
* over five steps the iteration's distance to the unquantised binary64 iteration is
  that of the exact path within a small margin (the accumulation changes which codes
  round where, not the method's accuracy).
"""
import math

import numpy as np
import pytest
import torch

from oracle import ns, rht
from oracle.quantize import quantize
from paper_2607_04422_amd import workloads
from tests.error_study import run_case
from tests.gpu_util import assert_same_nvfp4, gpu_nvfp4, need_gpu, np_, rel_fro

pytestmark = pytest.mark.gpu

F = None
U = 2.0 ** -24
MIXED = [(3.0, -3.2, 1.2)] * 3 + [(1.875, -1.25, 0.375)] * 2


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _decoded(q):
    """D(q) = q * s per element (no tensor scale), binary64, exact."""
    I, E, _ = ns._integer_rows(q)
    return I * np.ldexp(1.0, E - 11)


def _abs_dot(qa, qb=None):
    da = np.abs(_decoded(qa))
    db = da if qb is None else np.abs(_decoded(qb))
    return da @ db.T


def _within(got, ref, bound, what):
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    bad = err > bound
    assert not bad.any(), (what, int(bad.sum()), float((err / np.maximum(bound, 1e-300)).max()))


def _check_step_fp32(x0, a, b, c, flags, seed, step, tr, x1):
    signs = rht.step_signs(seed, step) if flags & F.F_HADAMARD else None
    ad = bool(flags & F.F_ADAPTIVE46)
    m, n = x0.shape
    qx = gpu_nvfp4(tr["qx_codes"][0], tr["qx_scales"][0], tr["qx_sg"])
    qxt = gpu_nvfp4(tr["qxt_codes"][0], tr["qxt_scales"][0], tr["qxt_sg"])
    assert_same_nvfp4(qx, quantize(x0, 1, signs, ad), "qX")
    assert_same_nvfp4(qxt, quantize(x0, 0, signs, ad), "qXt")
    # A = s^2 D(qX) D(qX)^T, binary32 accumulation over K = n
    A = np_(tr["A"][0])
    sx2 = np.float64(qx.sg) ** 2
    A_ex = sx2 * ns.block_dot64(qx)
    _within(A, A_ex, (n + 2) * U * sx2 * _abs_dot(qx) + U * np.abs(A_ex), "A")
    assert np.array_equal(A, A.T)
    qa = gpu_nvfp4(tr["qa_codes"][0], tr["qa_scales"][0], tr["qa_sg"])
    assert_same_nvfp4(qa, quantize(A, 1, signs, ad), "qA")
    # B = fl32(b A + c P), P accumulated in binary32 over K = m
    B = np_(tr["B"][0])
    sa2 = np.float64(qa.sg) ** 2
    bb, cc = np.float64(np.float32(b)), np.float64(np.float32(c))
    B_ex = bb * A.astype(np.float64) + cc * sa2 * ns.block_dot64(qa)
    _within(B, B_ex, abs(cc) * (m + 2) * U * sa2 * _abs_dot(qa) + 2 * U * np.abs(B_ex), "B")
    assert np.array_equal(B, B.T)
    qb = gpu_nvfp4(tr["qb_codes"][0], tr["qb_scales"][0], tr["qb_sg"])
    assert_same_nvfp4(qb, quantize(B, 1, signs, ad), "qB")
    # X_{k+1} = fl32(a X_k + s_B s_Xt D(qB) D(qXt)^T), binary32 accumulation over K = m
    sbx = np.float64(qb.sg) * np.float64(qxt.sg)
    X_ex = np.float64(np.float32(a)) * x0.astype(np.float64) + sbx * ns.block_dot64(qb, qxt)
    _within(x1, X_ex, (m + 2) * U * sbx * _abs_dot(qb, qxt) + 2 * U * np.abs(X_ex), "X")


@pytest.mark.parametrize("shape", [(64, 128), (256, 512), (272, 400), (144, 144), (272, 144), (512, 1536)])
@pytest.mark.parametrize("flags", [6, 0])
def test_ns_step_stages_fp32_accum(shape, flags):
    m, n = shape
    x0, _, _ = ns.prepare(workloads.matrix(m, n, seed=m + n, kind="t_rows"))
    if x0.shape != (m, n):
        x0 = np.ascontiguousarray(x0.T)
    a, b, c = MIXED[0]
    f = flags | F.F_FP32_ACCUM
    x = torch.from_numpy(x0).cuda()
    tr = F.fp4root_ns_step(x, a, b, c, flags=f, seed=77, step=2, trace=True)
    _check_step_fp32(x0, a, b, c, flags, 77, 2, tr, np_(x))
    # the untraced call produces the same bits (the accumulation order is fixed)
    y = torch.from_numpy(x0).cuda()
    F.fp4root_ns_step(y, a, b, c, flags=f, seed=77, step=2)
    assert torch.equal(x, y)


def test_fp32_accum_rejected_with_bf16_path():
    x = torch.from_numpy(workloads.matrix(64, 128, seed=1)).cuda()
    # the workspace query rejects the configuration (the binding raises before any launch)
    with pytest.raises(ValueError):
        F.fp4root_orthogonalize([x], steps=2, flags=F.F_CLIP | F.F_BF16_PATH | F.F_FP32_ACCUM)
    with pytest.raises(F.Fp4RootError):
        F.fp4root_ns_step(x, 1.5, -0.5, 0.0, flags=F.F_BF16_PATH | F.F_FP32_ACCUM)


@pytest.mark.parametrize("which", ["small", "kv"])
def test_fp32_accum_keeps_the_iterations_accuracy(which):
    """Five steps: distance to the unquantised binary64 iteration within a small margin of
    the exact path's, and the output close to the exact path's (the oracle's)."""
    if which == "small":
        mats = workloads.small_case()
    else:
        mats = [workloads.matrix(1024, 3072, seed=33, kind="t_rows")]
    routes = {"exact": (F.F_DEFAULT, "shape"), "fp32": (F.F_DEFAULT | F.F_FP32_ACCUM, "shape")}
    res = run_case(F, mats, routes=routes)
    e_ex, e32 = res["exact"]["err"], res["fp32"]["err"]
    assert res["fp32"]["finite"] and res["exact"]["finite"]
    assert e32 <= 1.25 * e_ex + 0.01, (e32, e_ex)
    ins = [torch.from_numpy(m).cuda() for m in mats]
    ex = F.fp4root_orthogonalize(ins, steps=5)
    f32 = F.fp4root_orthogonalize(ins, steps=5, flags=F.F_DEFAULT | F.F_FP32_ACCUM)
    f32b = F.fp4root_orthogonalize(ins, steps=5, flags=F.F_DEFAULT | F.F_FP32_ACCUM)
    for a, b, c in zip(ex, f32, f32b):
        assert torch.equal(b, c)                      # deterministic
        d = rel_fro(np_(b), np_(a))
        assert math.isfinite(d) and d <= 0.25, d      # same iteration, other rounding of the products


def test_fp32_accum_grouped_call_equals_single_calls_and_replays():
    """Each output is one binary32 chain in contraction order whatever the launch: a call over
    six shape groups (grouped Gram launches, per-launch tile forms) gives every matrix the
    bits of a call on that matrix alone, and a HIP-graph replay gives the eager call's bits."""
    shapes = [(128, 256), (256, 128), (144, 144), (96, 400), (32, 1024), (272, 400), (128, 256)]
    mats = [workloads.matrix(r, c, seed=70 + i, kind="normal_outliers") for i, (r, c) in enumerate(shapes)]
    flags = F.F_DEFAULT | F.F_FP32_ACCUM
    ins = [torch.from_numpy(m).cuda() for m in mats]
    orth = F.Orthogonalizer(ins, steps=5, flags=flags, seed=4)
    eager = [o.clone() for o in orth()]
    assert orth.status() == 0
    for i, m in enumerate(mats):
        alone = F.fp4root_orthogonalize([torch.from_numpy(m).cuda()], steps=5, flags=flags, seed=4)[0]
        assert torch.equal(alone, eager[i]), i
    graph = orth.capture()
    for r in range(3):
        for o in orth.outputs:
            o.zero_()
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(eager, orth.outputs)):
            assert torch.equal(a, b), (r, i)
