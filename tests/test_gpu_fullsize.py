"""GPU parity at the full workload sizes, in the launch configuration bench.py times.

* The 28-matrix 3B-shaped set runs through one fp4root_orthogonalize call
  (three batched shape groups, default coefficients, clipping + Hadamard +
  adaptive 4/6, seed 0), exactly as bench.py does; its 1024 x 3072 outputs are
  compared with the oracle end to end (the oracle finishes those in seconds).
* For the big groups (12 x 3072x8192 and 8 x 3072x3072) one traced NS step runs
  on the whole batch (the same kernels and grids as the orthogonalisation); the
  oracle checks every stage of one batch member on sampled rows (quantisers,
  bit for bit) and sampled entries (products, to the binary32 value).
* The 4096 x 4096 square case and the 3072 x 8192 / 8192 x 3072 pair: one traced
  step each, checked the same way.
* The stress case: the 8192 x 28672 matrix (one traced step) and end-to-end
  parity for a sample of its 256 512 x 512 companions.
"""
import time

import numpy as np
import pytest
import torch

from oracle import ns, rht
from oracle.quantize import quantize
from paper_2607_04422_amd import workloads
from tests.gpu_util import assert_same_nvfp4, gpu_nvfp4, need_gpu, np_, rel_fro, ulp_diff

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
        err = rel_fro(np_(outs[i]), ref)
        _log(f"{shapes[i][0]} {m.shape}: rel err {err:.3e}")
        assert err <= TOL


def _sample_pairs(rng, m, n, k):
    return rng.integers(0, m, k), rng.integers(0, n, k)


def _check_traced_step(x0_all, member, a, b, c, seed, step, label, check_qxt=True):
    """One traced GPU step on the whole batch; stage checks on batch member `member`."""
    B, m, n = x0_all.shape
    x = torch.from_numpy(x0_all).cuda()
    tr = F.fp4root_ns_step(x, a, b, c, flags=F.F_HADAMARD | F.F_ADAPTIVE46, seed=seed, step=step,
                           trace=True)
    torch.cuda.synchronize()
    _log(f"{label}: gpu step done")
    x0 = x0_all[member]
    d = rht.step_signs(seed, step)
    rng = np.random.default_rng(member)
    rows_m = np.sort(rng.choice(m, 24, replace=False))
    rows_n = np.sort(rng.choice(n, 24, replace=False))
    qx = gpu_nvfp4(tr["qx_codes"][member], tr["qx_scales"][member], tr["qx_sg"][member:member + 1])
    qxt = gpu_nvfp4(tr["qxt_codes"][member], tr["qxt_scales"][member], tr["qxt_sg"][member:member + 1])
    sel = lambda q, r: type(q)(q.codes[r], q.scales[r], q.sg, q.m4[r] if q.m4.ndim else q.m4)
    assert_same_nvfp4(sel(qx, rows_m), quantize(x0, 1, d, True, rows=rows_m), f"{label} qX")
    if check_qxt:
        assert_same_nvfp4(sel(qxt, rows_n), quantize(x0, 0, d, True, rows=rows_n), f"{label} qXt")
    _log(f"{label}: quantisers of X ok")
    DX = qx.block_values()
    A = np_(tr["A"][member])
    ii, jj = _sample_pairs(rng, m, m, 400)
    ref = ns.f32((np.float64(qx.sg) ** 2) * np.einsum("ij,ij->i", DX[ii], DX[jj]))
    assert ulp_diff(A[ii, jj], ref).max() <= 1
    assert np.array_equal(A, A.T)
    qa = gpu_nvfp4(tr["qa_codes"][member], tr["qa_scales"][member], tr["qa_sg"][member:member + 1])
    assert_same_nvfp4(sel(qa, rows_m), quantize(A, 1, d, True, rows=rows_m), f"{label} qA")
    DA = qa.block_values()
    Bm = np_(tr["B"][member])
    P = (np.float64(qa.sg) ** 2) * np.einsum("ij,ij->i", DA[ii], DA[jj])
    refB = ns.f32(np.float64(np.float32(b)) * A[ii, jj].astype(np.float64) + np.float64(np.float32(c)) * P)
    assert ulp_diff(Bm[ii, jj], refB).max() <= 1
    qb = gpu_nvfp4(tr["qb_codes"][member], tr["qb_scales"][member], tr["qb_sg"][member:member + 1])
    assert_same_nvfp4(sel(qb, rows_m), quantize(Bm, 1, d, True, rows=rows_m), f"{label} qB")
    _log(f"{label}: A, qA, B, qB ok")
    x1 = np_(x[member])
    ii, jj = _sample_pairs(rng, m, n, 400)
    DB = qb.block_values()
    DXt = qxt.block_values()
    prod = np.einsum("ij,ij->i", DB[ii], DXt[jj])
    refX = ns.f32(np.float64(np.float32(a)) * x0[ii, jj].astype(np.float64)
                  + np.float64(qb.sg) * np.float64(qxt.sg) * prod)
    assert ulp_diff(x1[ii, jj], refX).max() <= 1
    _log(f"{label}: X update ok")


def _canonical_batch(mats):
    xs = [ns.prepare(mm)[0] for mm in mats]
    return np.ascontiguousarray(np.stack(xs))


def test_bench_group_3072x8192_step_stages():
    shapes = workloads.case_shapes("block3b_x4")
    mats = workloads.case_matrices("block3b_x4")
    group = [mm for (lab, r, c), mm in zip(shapes, mats) if min(r, c) == 3072 and max(r, c) == 8192]
    assert len(group) == 12
    x0 = _canonical_batch(group)
    del mats, group
    a, b, c = F.fp4root_default_coeffs(3072, 8192, 5)[0]
    _check_traced_step(x0, 7, a, b, c, seed=0, step=0, label="3072x8192 x12")


def test_bench_group_3072sq_step_stages():
    shapes = workloads.case_shapes("block3b_x4")
    mats = workloads.case_matrices("block3b_x4", limit=28)
    group = [mm for (lab, r, c), mm in zip(shapes, mats) if r == 3072 and c == 3072]
    assert len(group) == 8
    x0 = _canonical_batch(group)
    del mats, group
    a, b, c = F.fp4root_default_coeffs(3072, 3072, 5)[3]
    _check_traced_step(x0, 2, a, b, c, seed=5, step=3, label="3072x3072 x8")


def test_square_4096_step_stages():
    # one 4096 x 4096 Student-t matrix, square-shape coefficients (seed 1 inputs)
    m = workloads.case_matrices("square_4096")[0]
    x0 = ns.prepare(m)[0][None]
    del m
    a, b, c = F.fp4root_default_coeffs(4096, 4096, 5)[2]
    _check_traced_step(np.ascontiguousarray(x0), 0, a, b, c, seed=1, step=2, label="4096x4096")


def test_rect_pair_step_stages():
    # 3072 x 8192 and 8192 x 3072 with lognormal row scales: both run short side first
    # as one batch of two 3072 x 8192 matrices; member 1 is the tall one, transposed
    mats = workloads.case_matrices("rect_3072x8192_pair")
    assert mats[1].shape == (8192, 3072)
    x0 = _canonical_batch(mats)
    del mats
    a, b, c = F.fp4root_default_coeffs(8192, 3072, 5)[0]
    _check_traced_step(x0, 1, a, b, c, seed=2, step=0, label="8192x3072 (tall) in the pair")


def test_stress_big_matrix_step_stages():
    # 8192 x 28672 (235 M elements): the quantiser along m is checked bit for bit at
    # 3072 x 8192 above; here its codes enter the sampled update-product entries.
    big = workloads.case_matrices("stress_8192x28672_plus_256x512sq", limit=1)[0]
    _log("generated")
    x0 = ns.prepare(big)[0][None]
    del big
    _log("prepared")
    a, b, c = F.fp4root_default_coeffs(8192, 28672, 5)[1]
    _check_traced_step(np.ascontiguousarray(x0), 0, a, b, c, seed=9, step=1, label="8192x28672",
                       check_qxt=False)


def test_stress_small_batch_end_to_end():
    mats = workloads.case_matrices("stress_8192x28672_plus_256x512sq")
    small = mats[1:]
    del mats
    ins = [torch.from_numpy(mm).cuda() for mm in small]
    outs = F.Orthogonalizer(ins, steps=5, flags=F.F_DEFAULT, seed=4)()
    co = F.fp4root_default_coeffs(512, 512, 5)
    for i in (0, 97, 255):
        err = rel_fro(np_(outs[i]), ns.orthogonalize(small[i], co, seed=4))
        _log(f"512x512 #{i}: rel err {err:.3e}")
        assert err <= TOL
