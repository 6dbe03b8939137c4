"""The NVFP4 products' two tile forms give the same bits.

The products cover each 128 x 128 output tile either with four waves of 64 x 64
outputs or with eight waves of 32 x 64, chosen per launch by how many rounds of
resident workgroups the launch fills.  Every product is exact (the binary32
rounding of its exact value), so the two forms must agree bit for bit; the other
GPU tests hold the per-launch choice to the oracle, and since the small shapes
they use run the narrow form, these cases force each form on ragged shapes:
sides that are not multiples of 128 (tail tiles), of 64 (no chain records: every
block folds) or both, wide and tall inputs, and a partial last 64-element stage.
"""
import numpy as np
import pytest
import torch

from oracle import ns
from paper_2607_04422_amd import workloads
from tests.gpu_util import need_gpu, np_, rel_fro

pytestmark = pytest.mark.gpu

F = None
MIXED = [(3.0, -3.2, 1.2)] * 3 + [(1.875, -1.25, 0.375)] * 2
SHAPES = [(272, 400), (400, 272), (1088, 1216), (1216, 1088), (144, 1296), (1040, 1040)]


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _run(ins, mode):
    prev = F.fp4root_set_product_tiling(mode)
    try:
        outs = F.fp4root_orthogonalize(ins, steps=5, coeffs=MIXED)
        torch.cuda.synchronize()
    finally:
        F.fp4root_set_product_tiling(prev)
    return [np_(o) for o in outs]


def test_set_product_tiling_returns_previous_and_rejects_bad_modes():
    assert F.fp4root_set_product_tiling(2) == 0
    assert F.fp4root_set_product_tiling(1) == 2
    assert F.fp4root_set_product_tiling(0) == 1
    for bad in (-1, 3):
        with pytest.raises(F.Fp4RootError):
            F.fp4root_set_product_tiling(bad)
    assert F.fp4root_set_product_tiling(0) == 0


@pytest.mark.parametrize("shape", SHAPES)
def test_wide_and_narrow_tiles_agree(shape):
    r, c = shape
    mats = [workloads.matrix(r, c, seed=700 + i) for i in range(2)]
    ins = [torch.from_numpy(m).cuda() for m in mats]
    narrow = _run(ins, 1)
    wide = _run(ins, 2)
    auto = _run(ins, 0)
    for i in range(len(mats)):
        assert np.array_equal(narrow[i], wide[i]), (shape, i, np.count_nonzero(narrow[i] != wide[i]))
        assert np.array_equal(narrow[i], auto[i]), (shape, i)


def test_wide_tiles_match_the_oracle_on_a_ragged_shape():
    """One ragged case of the wide form against the oracle directly (272 x 400:
    tail tiles in both directions and a partial last stage)."""
    m = workloads.matrix(272, 400, seed=710)
    out = _run([torch.from_numpy(m).cuda()], 2)[0]
    assert rel_fro(out, ns.orthogonalize(m, MIXED, seed=0)) <= 1e-3


def test_mixed_groups_in_one_call_agree():
    """Several shape groups in one call (the Gram launches then hold several products)."""
    mats = [workloads.matrix(r, c, seed=720 + i) for i, (r, c) in enumerate(SHAPES)]
    ins = [torch.from_numpy(m).cuda() for m in mats]
    narrow = _run(ins, 1)
    wide = _run(ins, 2)
    for i in range(len(mats)):
        assert np.array_equal(narrow[i], wide[i]), (SHAPES[i], np.count_nonzero(narrow[i] != wide[i]))
