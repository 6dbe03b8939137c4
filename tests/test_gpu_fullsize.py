"""GPU parity at the full workload sizes, in the launch configuration bench.py times.

* Clipping and normalisation at full size: a zero-step fp4root_orthogonalize call
  returns the clipped, normalised input (p99 threshold from the exact radix
  select, Frobenius norm fused into its last pass); it must equal the oracle's
  prepare() bit for bit on every matrix of the 3B-shaped set, the 4096^2 case,
  the 3072x8192 pair and the 8192x28672 stress matrix.
* Five NS steps at full size, fed forward: each step runs traced on the whole
  shape group (the kernels and grids of the orthogonalisation), and every stage
  of one batch member is checked against the oracle applied to the GPU's own
  inputs of that stage: the quantisations of X, X^T, A and B bit for bit on
  24 sampled rows, and A, B and X_{k+1} on those whole rows, equal to the
  binary32 value (both sides form each product's sum exactly).  Groups: the
  12 x 3072x8192 and 8 x 3072^2 groups of the 3B set, the 4096^2 case, the tall
  member of the 3072x8192 pair; the 8192x28672 matrix for two steps.
* End to end: the 28-matrix set through one call as bench.py makes it (its
  1024 x 3072 outputs against the oracle) and a sample of the 256 512 x 512
  stress companions.
"""
import time

import numpy as np
import pytest
import torch

from oracle import ns, rht
from oracle.quantize import NVFP4, quantize
from paper_2607_04422_amd import workloads
from tests.gpu_util import assert_same_nvfp4, gpu_nvfp4, need_gpu, np_, rel_fro

pytestmark = pytest.mark.gpu

F = None
TOL = 1e-3


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


# ---------------------------------------------------------------------------
# clipping and normalisation


def _prep_parity(mats, label):
    ins = [torch.from_numpy(m).cuda() for m in mats]
    orth = F.Orthogonalizer(ins, steps=0, flags=F.F_DEFAULT, clip_quantile=0.99, eps=1e-7, seed=0)
    outs = orth()
    assert orth.status() == 0
    _log(f"{label}: gpu done")
    for i, (m, o) in enumerate(zip(mats, outs)):
        ref, tall, _ = ns.prepare(m)
        ref = ref.T if tall else ref
        got = np_(o)
        assert np.array_equal(got, ref), f"{label} #{i}: {np.count_nonzero(got != ref)} of {got.size} differ"
    _log(f"{label}: {len(mats)} matrices equal")


def test_prepare_full_size_block3b_set():
    _prep_parity(workloads.case_matrices("block3b_x4"), "3B set")


def test_prepare_full_size_square_and_pair():
    _prep_parity(workloads.case_matrices("square_4096"), "4096^2")
    _prep_parity(workloads.case_matrices("rect_3072x8192_pair"), "3072x8192 pair")


def test_prepare_full_size_stress_matrix():
    big = workloads.case_matrices("stress_8192x28672_plus_256x512sq", limit=1)
    _prep_parity(big, "8192x28672")


# ---------------------------------------------------------------------------
# five NS steps, fed forward


def _rows(q: NVFP4, r) -> NVFP4:
    return NVFP4(q.codes[r], q.scales[r], q.sg, q.m4[r] if q.m4.ndim else q.m4)


def _traced_steps(x0_all, member, coeffs, seed, label, first=0, check_qxt=True):
    """Traced GPU steps first .. len(coeffs) - 1 on the whole batch; every stage of
    batch member `member` against the oracle applied to the GPU's inputs of that stage."""
    B, m, n = x0_all.shape
    x = torch.from_numpy(x0_all).cuda()
    rng = np.random.default_rng(1000 + member)
    f64, f32c = np.float64, lambda v: np.float64(np.float32(v))
    for k in range(first, len(coeffs)):
        a, b, c = coeffs[k]
        xk = np_(x[member])                       # this step's input: the GPU's X_k
        tr = F.fp4root_ns_step(x, a, b, c, flags=F.F_HADAMARD | F.F_ADAPTIVE46, seed=seed, step=k, trace=True)
        torch.cuda.synchronize()
        d = rht.step_signs(seed, k)
        rows = np.sort(rng.choice(m, 24, replace=False))
        cols = np.sort(rng.choice(n, 24, replace=False))
        tag = f"{label} step {k}"
        qx = gpu_nvfp4(tr["qx_codes"][member], tr["qx_scales"][member], tr["qx_sg"][member:member + 1])
        qxt = gpu_nvfp4(tr["qxt_codes"][member], tr["qxt_scales"][member], tr["qxt_sg"][member:member + 1])
        assert_same_nvfp4(_rows(qx, rows), quantize(xk, 1, d, True, rows=rows), f"{tag} qX")
        if check_qxt:
            assert_same_nvfp4(_rows(qxt, cols), quantize(xk, 0, d, True, rows=cols), f"{tag} qXt")
        A = np_(tr["A"][member])
        assert np.array_equal(A, A.T), f"{tag}: A not symmetric"
        ref = ns.f32((f64(qx.sg) * f64(qx.sg)) * ns.block_dot64(_rows(qx, rows), qx))
        assert np.array_equal(A[rows], ref), f"{tag} A: {np.count_nonzero(A[rows] != ref)} differ"
        qa = gpu_nvfp4(tr["qa_codes"][member], tr["qa_scales"][member], tr["qa_sg"][member:member + 1])
        assert_same_nvfp4(_rows(qa, rows), quantize(A, 1, d, True, rows=rows), f"{tag} qA")
        Bm = np_(tr["B"][member])
        P = (f64(qa.sg) * f64(qa.sg)) * ns.block_dot64(_rows(qa, rows), qa)
        ref = ns.f32(f32c(b) * A[rows].astype(np.float64) + f32c(c) * P)
        assert np.array_equal(Bm[rows], ref), f"{tag} B: {np.count_nonzero(Bm[rows] != ref)} differ"
        qb = gpu_nvfp4(tr["qb_codes"][member], tr["qb_scales"][member], tr["qb_sg"][member:member + 1])
        assert_same_nvfp4(_rows(qb, rows), quantize(Bm, 1, d, True, rows=rows), f"{tag} qB")
        x1 = np_(x[member])
        ref = ns.f32(f32c(a) * xk[rows].astype(np.float64)
                     + (f64(qb.sg) * f64(qxt.sg)) * ns.block_dot64(_rows(qb, rows), qxt))
        assert np.array_equal(x1[rows], ref), f"{tag} X: {np.count_nonzero(x1[rows] != ref)} differ"
        del tr
        _log(f"{tag}: every stage equal")


def _canonical_batch(mats):
    xs = [ns.prepare(mm)[0] for mm in mats]
    return np.ascontiguousarray(np.stack(xs))


def test_five_steps_3b_group_3072x8192():
    shapes = workloads.case_shapes("block3b_x4")
    mats = workloads.case_matrices("block3b_x4")
    group = [mm for (lab, r, c), mm in zip(shapes, mats) if min(r, c) == 3072 and max(r, c) == 8192]
    assert len(group) == 12
    x0 = _canonical_batch(group)
    del mats, group
    _traced_steps(x0, 7, F.fp4root_default_coeffs(3072, 8192, 5), seed=0, label="3072x8192 x12 #7")


def test_five_steps_3b_group_3072sq():
    shapes = workloads.case_shapes("block3b_x4")
    mats = workloads.case_matrices("block3b_x4")
    group = [mm for (lab, r, c), mm in zip(shapes, mats) if r == 3072 and c == 3072]
    assert len(group) == 8
    x0 = _canonical_batch(group)
    del mats, group
    _traced_steps(x0, 2, F.fp4root_default_coeffs(3072, 3072, 5), seed=0, label="3072^2 x8 #2")


def test_five_steps_square_4096():
    m = workloads.case_matrices("square_4096")[0]
    x0 = np.ascontiguousarray(ns.prepare(m)[0][None])
    del m
    _traced_steps(x0, 0, F.fp4root_default_coeffs(4096, 4096, 5), seed=1, label="4096^2")


def test_five_steps_rect_pair_tall_member():
    # 3072 x 8192 and 8192 x 3072: both run short side first as one batch of two
    # 3072 x 8192 matrices; member 1 is the tall one, transposed
    mats = workloads.case_matrices("rect_3072x8192_pair")
    assert mats[1].shape == (8192, 3072)
    x0 = _canonical_batch(mats)
    del mats
    _traced_steps(x0, 1, F.fp4root_default_coeffs(8192, 3072, 5), seed=2, label="8192x3072 (tall)")


def test_two_steps_stress_matrix():
    # 8192 x 28672 (235 M elements, K = 28672 for the Gram of qX), steps 0 and 1
    big = workloads.case_matrices("stress_8192x28672_plus_256x512sq", limit=1)[0]
    x0 = np.ascontiguousarray(ns.prepare(big)[0][None])
    del big
    _log("prepared")
    co = F.fp4root_default_coeffs(8192, 28672, 5)[:2]
    _traced_steps(x0, 0, co, seed=4, label="8192x28672")


# ---------------------------------------------------------------------------
# end to end


def test_bench_set_end_to_end_kv():
    mats = workloads.case_matrices("block3b_x4")
    shapes = workloads.case_shapes("block3b_x4")
    ins = [torch.from_numpy(m).cuda() for m in mats]
    orth = F.Orthogonalizer(ins, steps=5, flags=F.F_DEFAULT, clip_quantile=0.99, eps=1e-7, seed=0)
    outs = orth()
    assert orth.status() == 0
    _log("gpu done")
    picks = [i for i, (lab, r, c) in enumerate(shapes) if lab.endswith(".k") or lab.endswith(".v")][::3]
    for i in picks:
        m = mats[i]
        co = F.fp4root_default_coeffs(m.shape[0], m.shape[1], 5)
        ref = ns.orthogonalize(m, co, seed=0)
        got = np_(outs[i])
        _log(f"{shapes[i][0]} {m.shape}: rel err {rel_fro(got, ref):.3e}")
        assert np.array_equal(got, ref)


def test_stress_small_batch_end_to_end():
    mats = workloads.case_matrices("stress_8192x28672_plus_256x512sq")
    small = mats[1:]
    del mats
    ins = [torch.from_numpy(mm).cuda() for mm in small]
    outs = F.Orthogonalizer(ins, steps=5, flags=F.F_DEFAULT, seed=4)()
    co = F.fp4root_default_coeffs(512, 512, 5)
    for i in (0, 97, 255):
        ref = ns.orthogonalize(small[i], co, seed=4)
        got = np_(outs[i])
        _log(f"512x512 #{i}: rel err {rel_fro(got, ref):.3e}")
        assert np.array_equal(got, ref)
