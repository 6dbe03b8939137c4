"""The error study on the GPU against the same study on the oracle.

For every route of the study (Section 3.4 routes, Fig. 3b coefficient sets,
and the BF16 products), the library's relative L2 error against the binary64
reference equals the oracle's (their outputs agree within the parity
tolerance), on the small 256 x 512 workload and a tall matrix with outliers;
and the proposed route's error is below the plain all-FP4 route's and below
the same route with the Muon coefficients.
"""
import math

import numpy as np
import pytest
import torch

from oracle import ns
from paper_2607_04422_amd import workloads
from tests.error_study import MUON, ROUTES, STEPS, ns_reference, run_case
from tests.gpu_util import need_gpu

pytestmark = pytest.mark.gpu

F = None


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _oracle_errors(mats):
    out = {}
    for name, (flags, kind) in ROUTES.items():
        num = den = 0.0
        for m in mats:
            co = [MUON] * STEPS if kind == "muon" else F.fp4root_default_coeffs(*m.shape, STEPS)
            clip_on = bool(flags & 1)
            q = ns.orthogonalize(m, co, clip_on=clip_on, hadamard=bool(flags & 2), adaptive46=bool(flags & 4),
                                 seed=0, mode="bf16" if flags & 8 else "nvfp4")
            x0, tall, _ = ns.prepare(m, clip_on)
            x0 = np.ascontiguousarray(x0.T) if tall else x0
            ref = ns_reference(torch.from_numpy(x0), co).numpy()
            num += float(np.sum((q.astype(np.float64) - ref) ** 2))
            den += float(np.sum(ref * ref))
        out[name] = math.sqrt(num / den)
    return out


def test_error_study_matches_oracle():
    mats = workloads.small_case() + [workloads.matrix(512, 256, seed=31, kind="normal_outliers")]
    got = run_case(F, mats, log=print)
    want = _oracle_errors(mats)
    for name in ROUTES:
        g, w = got[name], want[name]
        print(f"{name}: gpu {g['err']:.6g} oracle {w:.6g}")
        assert g["finite"], name
        assert abs(g["err"] - w) <= 1e-3 * max(1.0, w), name
    assert got["proposed"]["err"] < 0.5 * got["plain FP4 (Muon coefficients)"]["err"]
    assert got["proposed"]["err"] < 0.5 * got["proposed, Muon coefficients"]["err"]
