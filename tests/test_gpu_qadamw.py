"""GPU parity of quantized-state AdamW (fp4root_qadamw_update) with the oracle.

Over three steps with fresh seeded heavy-tailed gradients: the BF16 weights, the
first-moment state (codes, E4M3 scales, tensor scale), this step's m_t, and the
second-moment state (codes, BF16 block scales, BF16 tile means) equal the
oracle's bit for bit, for several flag sets and for parameter lengths that leave
partial work groups; plus the non-finite and shape error paths.
"""
import numpy as np
import pytest
import torch

from oracle import qadamw as Q
from oracle.formats import unpack_nibbles
from tests.gpu_util import need_gpu, np_

pytestmark = pytest.mark.gpu

F = None


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _u16(t):
    return t.cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("flags", [22, 6, 16, 0])
@pytest.mark.parametrize("n", [256, 256 * 37, 65536])
def test_qadamw_parity(n, flags):
    rng = np.random.default_rng(n + flags)
    lr, wd, b1, b2, eps, seed = 1e-3, 0.1, 0.9, 0.95, 1e-8, 5
    w_np = Q.bf16_round((rng.standard_normal(n) * 0.02).astype(np.float32))
    w = torch.from_numpy(w_np.view(np.int16).copy()).cuda().view(torch.bfloat16)
    st = F.QAdamWState(n, keep_m=True)
    m_prev = v_prev = None
    for t in range(3):
        g_np = (rng.standard_t(3, n) * np.repeat(rng.lognormal(0, 1, n // 256), 256) * 1e-3).astype(np.float32)
        F.fp4root_qadamw_update(w, torch.from_numpy(g_np).cuda(), st, t, lr, wd, b1, b2, eps, flags=flags, seed=seed)
        assert F.fp4root_device_status(st.ws) == 0
        w_np, ms, vs, m_t, v_t = Q.adamw_step(g_np, w_np, m_prev, v_prev, t, lr, wd, b1, b2, eps, seed,
                                              hadamard=bool(flags & 2), adaptive46=bool(flags & 4),
                                              sr=bool(flags & 16))
        m_prev, v_prev = ms, vs
        assert np.array_equal(np_(st.m), m_t), (n, flags, t, "m_t")
        assert float(st.m_tensor_scale[0]) == ms.sg
        assert np.array_equal(np_(st.m_scales), ms.scales.reshape(-1)), (n, flags, t, "m scales")
        assert np.array_equal(unpack_nibbles(np_(st.m_codes)), ms.codes.reshape(-1)), (n, flags, t, "m codes")
        assert np.array_equal(_u16(st.v_means), vs.means), (n, flags, t, "v means")
        assert np.array_equal(_u16(st.v_scales), vs.scales), (n, flags, t, "v scales")
        bad = np.count_nonzero(unpack_nibbles(np_(st.v_codes)) != vs.codes)
        assert bad == 0, (n, flags, t, f"{bad} v code mismatches")
        assert np.array_equal(_u16(w.view(torch.int16)), w_np), (n, flags, t, "weights")


def test_qadamw_errors():
    n = 512
    st = F.QAdamWState(n)
    w = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    g = torch.ones(n, device="cuda")
    g[7] = float("nan")
    F.fp4root_qadamw_update(w, g, st, 0, 1e-3)
    assert F.fp4root_device_status(st.ws) == -4
    with pytest.raises(ValueError):
        F.QAdamWState(300)
    with pytest.raises(F.Fp4RootError):
        F.fp4root_qadamw_update(w, torch.ones(n, device="cuda"), st, 0, 1e-3, beta2=2.0)
    g1 = torch.ones(n, device="cuda")
    st.m = g1                                   # m may not alias g: rejected before any launch
    with pytest.raises(F.Fp4RootError):
        F.fp4root_qadamw_update(w, g1, st, 0, 1e-3)
