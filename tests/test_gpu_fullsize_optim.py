"""GPU parity of the optimizer-state paths at a workload size, in bench.py's launch shapes.

* First-moment state: one fp4root_momentum_update call on the batch of eight
  3072 x 3072 matrices (the q/o batch bench.py times), steps 0 and 1; the last
  matrix of the batch (its draws start at 7 * 3072^2) is checked in full against
  the oracle: m_t and the state, bit for bit.
* Quantized-state AdamW: one 3072 x 3072 parameter (9.4 M elements, one of the
  calls bench.py times), steps 0 and 1: weights, m_t and both states in full.
"""
import time

import numpy as np
import pytest
import torch

from oracle import momentum as M
from oracle import qadamw as Q
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


def _log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


def test_momentum_qo_batch_full_size():
    B, R, C, beta, seed = 8, 3072, 3072, 0.9, 21
    state = F.MomentumState(B, R, C)
    prev = None
    for t in range(2):
        gs = np.stack([workloads.matrix(R, C, seed=100 * t + b, kind="normal") for b in range(B)])
        m = F.fp4root_momentum_update(torch.from_numpy(gs).cuda(), state, beta, t, seed=seed)
        assert F.fp4root_device_status(state.ws) == 0
        _log(f"step {t}: gpu done")
        mo, so = M.momentum_step(gs[B - 1], prev, beta, seed, t, batch_index=B - 1)
        prev = so
        _log(f"step {t}: oracle done")
        assert np.array_equal(np_(m[B - 1]), mo)
        assert float(state.tensor_scale[B - 1]) == so.sg
        assert np.array_equal(np_(state.scales[B - 1]), so.scales)
        bad = np.count_nonzero(unpack_nibbles(np_(state.codes[B - 1])) != so.codes)
        assert bad == 0, f"step {t}: {bad} code mismatches"


def test_qadamw_qo_parameter_full_size():
    n, seed = 3072 * 3072, 8
    rng = np.random.default_rng(5)
    w_np = Q.bf16_round((rng.standard_normal(n) * 0.02).astype(np.float32))
    w = torch.from_numpy(w_np.view(np.int16).copy()).cuda().view(torch.bfloat16)
    st = F.QAdamWState(n, keep_m=True)
    m_prev = v_prev = None
    for t in range(2):
        g_np = workloads.matrix(3072, 3072, seed=40 + t).reshape(-1) * np.float32(1e-3)
        F.fp4root_qadamw_update(w, torch.from_numpy(g_np).cuda(), st, t, 1e-4, 0.1, 0.9, 0.95, 1e-8, seed=seed)
        assert F.fp4root_device_status(st.ws) == 0
        _log(f"step {t}: gpu done")
        w_np, ms, vs, m_t, _ = Q.adamw_step(g_np, w_np, m_prev, v_prev, t, 1e-4, 0.1, 0.9, 0.95, 1e-8, seed)
        m_prev, v_prev = ms, vs
        _log(f"step {t}: oracle done")
        assert np.array_equal(np_(st.m), m_t)
        assert float(st.m_tensor_scale[0]) == ms.sg
        assert np.array_equal(np_(st.m_scales), ms.scales.reshape(-1))
        assert np.array_equal(unpack_nibbles(np_(st.m_codes)), ms.codes.reshape(-1))
        assert np.array_equal(st.v_means.cpu().numpy().view(np.uint16), vs.means)
        assert np.array_equal(st.v_scales.cpu().numpy().view(np.uint16), vs.scales)
        assert np.array_equal(unpack_nibbles(np_(st.v_codes)), vs.codes)
        assert np.array_equal(w.view(torch.int16).cpu().numpy().view(np.uint16), w_np)
