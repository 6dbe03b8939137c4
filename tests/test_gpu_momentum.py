"""GPU parity of the NVFP4 first-moment state (fp4root_momentum_update) with the oracle.

Over three optimizer steps with fresh seeded gradients, the library's m_t must
equal the oracle's bit for bit, and so must the new state (E2M1 codes, E4M3
scales, FP32 tensor scale), for stochastic and round-to-nearest rounding, with
and without the rotation and 4/6 selection, on ragged block counts and batches
(the draw index runs over the batch).  Also: a zero gradient, a K/V-shaped
1024 x 3072 matrix, in-place m = g, a non-finite gradient (device status) and
argument errors.
"""
import numpy as np
import pytest
import torch

from oracle import momentum as M
from oracle.formats import unpack_nibbles
from paper_2607_04422_amd import workloads
from tests.gpu_util import need_gpu, np_

pytestmark = pytest.mark.gpu

F = None


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _flags_to_oracle(flags):
    return dict(hadamard=bool(flags & F.F_HADAMARD), adaptive46=bool(flags & F.F_ADAPTIVE46),
                sr=bool(flags & F.F_STOCHASTIC))


def _run_steps(shape, batch, flags, steps=3, beta=0.9, seed=11, kind="normal_outliers", in_place=False):
    R, C = shape
    state = F.MomentumState(batch, R, C)
    prev = [None] * batch
    for t in range(steps):
        gs = [workloads.matrix(R, C, seed=1000 * t + 17 * b + 3, kind=kind) for b in range(batch)]
        g = torch.from_numpy(np.stack(gs)).cuda()
        m = F.fp4root_momentum_update(g, state, beta, t, flags=flags, seed=seed, m=g if in_place else None)
        assert F.fp4root_device_status(state.ws) == 0
        for b in range(batch):
            mo, so = M.momentum_step(gs[b], prev[b], beta, seed, t, batch_index=b, **_flags_to_oracle(flags))
            assert np.array_equal(np_(m[b]), mo), (shape, batch, flags, t, b, "m")
            assert np.float32(np_(state.tensor_scale)[b]) == so.sg, (shape, flags, t, b, "sg")
            assert np.array_equal(np_(state.scales[b]), so.scales), (shape, flags, t, b, "scales")
            got = unpack_nibbles(np_(state.codes[b]))
            bad = np.count_nonzero(got != so.codes)
            assert bad == 0, (shape, batch, flags, t, b, f"{bad} code mismatches")
            prev[b] = so


@pytest.mark.parametrize("flags", [22, 6, 16, 18, 20, 0])
@pytest.mark.parametrize("shape,batch", [((64, 128), 1), ((48, 400), 3), ((16, 16), 2)])
def test_momentum_parity(shape, batch, flags):
    _run_steps(shape, batch, flags)


def test_momentum_kv_shape_and_in_place():
    _run_steps((1024, 3072), 1, 22, steps=2, kind="t_rows")
    _run_steps((96, 256), 2, 22, steps=2, in_place=True)


def test_momentum_zero_gradient():
    R, C = 32, 64
    state = F.MomentumState(1, R, C)
    g = torch.zeros((R, C), device="cuda")
    m = F.fp4root_momentum_update(g, state, 0.9, 0, seed=2)
    assert not torch.any(m) and float(state.tensor_scale[0]) == 0.0
    assert not torch.any(state.scales) and not torch.any(state.codes & 0x77)
    m = F.fp4root_momentum_update(g, state, 0.9, 1, seed=2)
    assert not torch.any(m)


def test_momentum_nonfinite_and_errors():
    R, C = 32, 64
    state = F.MomentumState(1, R, C)
    g = torch.ones((R, C), device="cuda")
    g[3, 5] = float("nan")
    F.fp4root_momentum_update(g, state, 0.9, 0)
    assert F.fp4root_device_status(state.ws) == -4
    g = torch.ones((R, C), device="cuda")
    with pytest.raises(F.Fp4RootError):
        F.fp4root_momentum_update(g, state, 0.9, 0, flags=F.F_CLIP)
    with pytest.raises(F.Fp4RootError):
        F.fp4root_momentum_update(g, state, 1.5, 0)
    with pytest.raises(F.Fp4RootError):
        F.fp4root_momentum_update(g, state, 0.9, -1)
    bad = torch.ones((R, 40), device="cuda")   # 40 columns: not a multiple of 16
    with pytest.raises(F.Fp4RootError) as e:
        F.fp4root_momentum_update(bad, F.MomentumState(1, R, 40), 0.9, 0)
    assert e.value.code == -2
