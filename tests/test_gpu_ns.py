"""GPU parity of the Newton-Schulz path against the oracle.

Each stage of a step is checked against the oracle fed with the GPU's own
previous stage (quantisations bit for bit, products to the binary32 value),
then whole orthogonalisations end to end within the 1e-3 relative Frobenius
tolerance (the products are exact, so the observed error is expected to be 0).
"""
import numpy as np
import pytest
import torch

from oracle import ns, rht
from oracle.quantize import quantize
from paper_2607_04422_amd import workloads
from tests.gpu_util import assert_same_nvfp4, gpu_nvfp4, need_gpu, np_, rel_fro

pytestmark = pytest.mark.gpu

F = None
TOL = 1e-3
# BF16 comparison path: products accumulate in binary32 before their bf16 rounding,
# so about one element in 2^14 rounds to the neighbouring bf16 value (a 2^-8
# relative change of that element); through five steps these flips move the output
# by up to about 2^-8 relative.  Tolerance: 2^-7.
TOL_BF16 = 2.0 ** -7
CONV = [(1.875, -1.25, 0.375)] * 5
MIXED = [(3.0, -3.2, 1.2)] * 3 + [(1.875, -1.25, 0.375)] * 2


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _check_step(x0, a, b, c, flags, seed, step, tr, x1):
    """Stage-by-stage comparison of one traced GPU step with the oracle."""
    signs = rht.step_signs(seed, step) if flags & F.F_HADAMARD else None
    ad = bool(flags & F.F_ADAPTIVE46)
    qx = gpu_nvfp4(tr["qx_codes"][0], tr["qx_scales"][0], tr["qx_sg"])
    qxt = gpu_nvfp4(tr["qxt_codes"][0], tr["qxt_scales"][0], tr["qxt_sg"])
    assert_same_nvfp4(qx, quantize(x0, 1, signs, ad), "qX")
    assert_same_nvfp4(qxt, quantize(x0, 0, signs, ad), "qXt")
    # every product is the binary32 rounding of its exact value (the oracle's products
    # are correctly rounded binary64 sums), so the stages agree bit for bit
    A = np_(tr["A"][0])
    A_ref = ns.f32((np.float64(qx.sg) ** 2) * ns.block_dot64(qx))
    assert np.array_equal(A, A.T)
    assert np.array_equal(A, A_ref), f"A: {np.count_nonzero(A != A_ref)} of {A.size} differ"
    qa = gpu_nvfp4(tr["qa_codes"][0], tr["qa_scales"][0], tr["qa_sg"])
    assert_same_nvfp4(qa, quantize(A, 1, signs, ad), "qA")
    B = np_(tr["B"][0])
    P = (np.float64(qa.sg) ** 2) * ns.block_dot64(qa)
    B_ref = ns.f32(np.float64(np.float32(b)) * A.astype(np.float64) + np.float64(np.float32(c)) * P)
    assert np.array_equal(B, B.T)
    assert np.array_equal(B, B_ref), f"B: {np.count_nonzero(B != B_ref)} of {B.size} differ"
    qb = gpu_nvfp4(tr["qb_codes"][0], tr["qb_scales"][0], tr["qb_sg"])
    assert_same_nvfp4(qb, quantize(B, 1, signs, ad), "qB")
    X_ref = ns.f32(np.float64(np.float32(a)) * x0.astype(np.float64)
                   + np.float64(qb.sg) * np.float64(qxt.sg) * ns.block_dot64(qb, qxt))
    assert np.array_equal(x1, X_ref), f"X: {np.count_nonzero(x1 != X_ref)} of {x1.size} differ"


@pytest.mark.parametrize("shape", [(64, 128), (256, 512), (272, 400), (144, 144), (272, 144)])
@pytest.mark.parametrize("flags", [6, 0])
def test_ns_step_stages(shape, flags):
    m, n = shape
    x0, _, _ = ns.prepare(workloads.matrix(m, n, seed=m + n, kind="t_rows"))
    if x0.shape != (m, n):
        x0 = np.ascontiguousarray(x0.T)
    a, b, c = MIXED[0]
    x = torch.from_numpy(x0).cuda()
    tr = F.fp4root_ns_step(x, a, b, c, flags=flags, seed=77, step=2, trace=True)
    _check_step(x0, a, b, c, flags, 77, 2, tr, np_(x))
    # the untraced call produces the same bits
    y = torch.from_numpy(x0).cuda()
    F.fp4root_ns_step(y, a, b, c, flags=flags, seed=77, step=2)
    assert torch.equal(x, y)


def test_ns_step_matches_oracle_step():
    x0, _, _ = ns.prepare(workloads.matrix(256, 768, seed=4))
    x = torch.from_numpy(x0).cuda()
    for k, (a, b, c) in enumerate(MIXED):
        ref = ns.ns_step_nvfp4(np_(x), a, b, c, rht.step_signs(5, k), True)
        F.fp4root_ns_step(x, a, b, c, flags=6, seed=5, step=k)
        assert np.array_equal(np_(x), ref), k


def _orth_case(mats, coeffs, flags, seed=0, mode="nvfp4"):
    ins = [torch.from_numpy(m).cuda() for m in mats]
    orth = F.Orthogonalizer(ins, steps=len(coeffs), coeffs=coeffs, flags=flags, seed=seed)
    outs = orth()
    assert orth.status() == 0
    errs = []
    for m, o in zip(mats, outs):
        ref = ns.orthogonalize(m, coeffs, clip_on=bool(flags & F.F_CLIP), hadamard=bool(flags & F.F_HADAMARD),
                               adaptive46=bool(flags & F.F_ADAPTIVE46), seed=seed, mode=mode)
        errs.append(rel_fro(np_(o), ref))
    return errs


def test_orthogonalize_small_case():
    mats = workloads.small_case()
    errs = _orth_case(mats, MIXED, F.F_DEFAULT, seed=3)
    assert max(errs) <= TOL, errs


@pytest.mark.parametrize("flags", [7, 6, 1, 0])
def test_orthogonalize_mixed_shapes(flags):
    # wide, tall, square and ragged shapes in one call; equal canonical shapes are batched
    shapes = [(128, 256), (256, 128), (144, 144), (96, 400), (400, 96), (128, 256)]
    mats = [workloads.matrix(r, c, seed=10 + i, kind="normal_outliers") for i, (r, c) in enumerate(shapes)]
    errs = _orth_case(mats, MIXED, flags, seed=11)
    assert max(errs) <= TOL, errs


def test_orthogonalize_many_shape_groups():
    # seven canonical shapes: the symmetric products of one step run in two grouped
    # launches (four products, then three); contractions that are not multiples of 64,
    # matrices smaller than one tile, tall inputs; products exact, so outputs equal
    shapes = [(32, 1024), (272, 400), (208, 80), (144, 144), (48, 48), (112, 336), (64, 64), (400, 272)]
    mats = [workloads.matrix(r, c, seed=40 + i, kind="normal_outliers") for i, (r, c) in enumerate(shapes)]
    errs = _orth_case(mats, MIXED, F.F_DEFAULT, seed=12)
    assert max(errs) == 0.0, errs


def test_orthogonalize_bf16_path():
    mats = [workloads.matrix(256, 512, seed=1), workloads.matrix(384, 128, seed=2)]
    errs = _orth_case(mats, MIXED, F.F_CLIP | F.F_BF16_PATH, mode="bf16")
    assert max(errs) <= TOL_BF16, errs


def test_orthogonalize_default_coeffs_and_zero_steps():
    m = workloads.matrix(128, 384, seed=21)
    x = torch.from_numpy(m).cuda()
    out0 = F.fp4root_orthogonalize([x], steps=0)[0]
    x_ref, _, _ = ns.prepare(m)
    assert np.array_equal(np_(out0), x_ref)
    co = F.fp4root_default_coeffs(128, 384, 5)
    out = F.fp4root_orthogonalize([x], steps=5)[0]
    ref = ns.orthogonalize(m, co, seed=0)
    assert rel_fro(np_(out), ref) <= TOL


def test_orthogonalize_large_group_copy_out():
    """More than 32 matrices of one shape are written back by the copy-out kernel
    (tall ones transposed back): exact at zero steps, the oracle's NS after five."""
    mats = [workloads.matrix(96, 32, seed=50 + i) for i in range(40)]
    mats += [workloads.matrix(32, 64, seed=90 + i) for i in range(36)]
    ins = [torch.from_numpy(m).cuda() for m in mats]
    out0 = F.fp4root_orthogonalize(ins, steps=0)
    for i in (0, 17, 39, 40, 75):
        x_ref, tall, _ = ns.prepare(mats[i])
        assert np.array_equal(np_(out0[i]), x_ref.T if tall else x_ref), i
    outs = F.fp4root_orthogonalize(ins, steps=5, coeffs=MIXED)
    for i in (0, 39, 40, 75):
        assert rel_fro(np_(outs[i]), ns.orthogonalize(mats[i], MIXED, seed=0)) <= TOL, i


def test_in_place_and_determinism():
    m = workloads.matrix(256, 512, seed=31)
    x1 = torch.from_numpy(m).cuda()
    out1 = F.fp4root_orthogonalize([x1], steps=5, coeffs=MIXED)[0]
    x2 = torch.from_numpy(m).cuda()
    F.fp4root_orthogonalize([x2], outputs=[x2], steps=5, coeffs=MIXED)
    assert torch.equal(out1, x2)


@pytest.mark.parametrize("flags", ["default", "no_clip", "bf16_no_clip"])
@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -float("inf")])
def test_nonfinite_input_reported(flags, bad):
    fl = {"default": F.F_DEFAULT, "no_clip": F.F_HADAMARD | F.F_ADAPTIVE46, "bf16_no_clip": F.F_BF16_PATH}[flags]
    m = workloads.matrix(64, 128, seed=1)
    m[3, 3] = bad
    orth = F.Orthogonalizer([torch.from_numpy(m).cuda()], steps=1, coeffs=MIXED[:1], flags=fl)
    orth()
    assert orth.status() == -4
    # a finite input afterwards clears the report
    m[3, 3] = 0.5
    orth2 = F.Orthogonalizer([torch.from_numpy(m).cuda()], steps=1, coeffs=MIXED[:1], flags=fl)
    orth2()
    assert orth2.status() == 0


def test_graph_replay_equals_eager_call():
    # the whole orthogonalisation recorded in a HIP graph: every replay, with eager
    # work of the program between the replays, gives the eager call's bits
    mats = [workloads.matrix(256, 512, seed=3), workloads.matrix(512, 256, seed=4), workloads.matrix(256, 512, seed=5)]
    ins = [torch.from_numpy(m).cuda() for m in mats]
    orth = F.Orthogonalizer(ins, steps=5, flags=F.F_DEFAULT, seed=2)
    eager = [o.clone() for o in orth()]
    assert orth.status() == 0
    graph = orth.capture()
    other = F.Orthogonalizer([torch.from_numpy(workloads.matrix(128, 256, seed=9)).cuda()], steps=2,
                             coeffs=MIXED[:2], flags=F.F_DEFAULT)
    for r in range(4):
        for o in orth.outputs:
            o.zero_()
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(eager, orth.outputs)):
            assert torch.equal(a, b), (r, i)
        assert orth.status() == 0
        other()                         # eager work between the replays
        torch.cuda.synchronize()


def _degenerate_inputs():
    """The method's degenerate inputs, each (name, matrix): zero, constant (rank 1, every
    block tied), one non-zero entry (clipped away at p99), rank 1, zero rows and columns,
    rows or columns spread over 2^+-40 (blocks far below the tensor maximum: E4M3 scales
    that underflow or are subnormal), +-1 entries (ties of the 4/6 choice), the smallest
    side (16, one block per row; tall), and inputs of extreme magnitude."""
    rng = np.random.default_rng(2024)
    cases = [("zero", np.zeros((64, 128), np.float32)),
             ("constant", np.full((128, 256), 0.5, np.float32))]
    m = np.zeros((64, 64), np.float32)
    m[3, 17] = -2.5
    cases.append(("single_entry", m))
    u, v = rng.standard_normal(128), rng.standard_normal(384)
    cases.append(("rank1", np.outer(u, v).astype(np.float32)))
    m = rng.standard_normal((128, 256)).astype(np.float32)
    m[::2] = 0.0
    m[:, 64:80] = 0.0
    cases.append(("zero_rows_cols", m))
    cases.append(("range_rows", (rng.standard_normal((96, 192))
                                 * np.exp2(rng.integers(-40, 41, size=(96, 1)))).astype(np.float32)))
    cases.append(("range_cols", (rng.standard_normal((64, 256))
                                 * np.exp2(rng.integers(-30, 31, size=(1, 256)))).astype(np.float32)))
    cases.append(("signs", np.where(rng.random((112, 224)) < 0.5, -1.0, 1.0).astype(np.float32)))
    cases.append(("side16", rng.standard_normal((16, 16)).astype(np.float32)))
    cases.append(("tall_side16", rng.standard_normal((48, 16)).astype(np.float32)))
    cases.append(("huge", (rng.standard_normal((64, 128)) * 1e30).astype(np.float32)))
    cases.append(("tiny", (rng.standard_normal((80, 160)) * 1e-27).astype(np.float32)))
    return cases


@pytest.mark.parametrize("flags", ["default", "no_clip", "plain"])
def test_orthogonalize_degenerate_inputs(flags):
    # all in one call (eleven shape groups), the library's coefficients per shape; the
    # products are exact, so every output equals the oracle's bit for bit
    fl = {"default": F.F_DEFAULT, "no_clip": F.F_HADAMARD | F.F_ADAPTIVE46, "plain": 0}[flags]
    cases = _degenerate_inputs()
    ins = [torch.from_numpy(m).cuda() for _, m in cases]
    orth = F.Orthogonalizer(ins, steps=5, flags=fl, seed=9)
    outs = orth()
    assert orth.status() == 0
    for (name, m), o in zip(cases, outs):
        co = F.fp4root_default_coeffs(m.shape[0], m.shape[1], 5)
        ref = ns.orthogonalize(m, co, clip_on=bool(fl & F.F_CLIP), hadamard=bool(fl & F.F_HADAMARD),
                               adaptive46=bool(fl & F.F_ADAPTIVE46), seed=9)
        got = np_(o)
        assert np.array_equal(got, ref), (name, int(np.count_nonzero(got != ref)))


@pytest.mark.parametrize("scale", [1e-25, 1e-27, 1e-30])
def test_ns_step_stages_extreme_scales(scale):
    # normalised inputs of 1e-18 .. 1e-23 (the norm is far below eps): A and B hold
    # binary32 subnormals, their tensor scales are subnormal (1e-27) or underflow to
    # zero with a non-zero amax (1e-30); every stage still matches bit for bit
    m = (np.random.default_rng(11).standard_normal((80, 160)) * scale).astype(np.float32)
    x0, _, _ = ns.prepare(m)
    a, b, c = F.fp4root_default_coeffs(80, 160, 5)[0]
    x = torch.from_numpy(x0).cuda()
    tr = F.fp4root_ns_step(x, a, b, c, flags=6, seed=31, step=0, trace=True)
    _check_step(x0, a, b, c, 6, 31, 0, tr, np_(x))
