"""GPU parity of the Root step around the orthogonalisation (fp4root_apply_update,
fp4root_root_step) with the oracle.

* apply: the BF16 weights after the update equal the oracle's bit for bit
  (random weights and directions, ragged element counts, zero count);
* the whole step, two optimizer steps over a wide, a tall and a square parameter:
  the first-moment states equal the oracle's bit for bit; the orthogonalised
  momentum (left in each parameter's scratch) is within the NS parity tolerance
  of the oracle chain (momentum, then clip + normalise + NVFP4 NS); and the new
  weights equal the oracle's update applied to the GPU's own orthogonalised
  momentum, bit for bit;
* a non-finite gradient is reported through the device status.
"""
import numpy as np
import pytest
import torch

from oracle import momentum as M
from oracle import ns
from oracle import root_step as R
from oracle.formats import unpack_nibbles
from tests.gpu_util import need_gpu, np_, rel_fro

pytestmark = pytest.mark.gpu

F = None


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _bf16_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("count", [0, 8, 2056, 600 * 1024 + 8])
def test_apply_update_parity(count):
    rng = np.random.default_rng(count)
    w32 = rng.standard_normal(count).astype(np.float32) * np.float32(0.05)
    o = rng.standard_normal(count).astype(np.float32) * np.float32(0.02)
    w = torch.from_numpy(w32).cuda().to(torch.bfloat16)
    w0 = _bf16_bits(w)
    F.fp4root_apply_update(w, torch.from_numpy(o).cuda(), 0.01, 0.1, 3.0 ** 0.5)
    want = R.apply_update(w0, o, 0.01, 0.1, np.float32(3.0 ** 0.5))
    assert np.array_equal(_bf16_bits(w), want)


def test_root_step_two_steps():
    shapes = [(64, 128), (192, 64), (96, 96)]
    rng = np.random.default_rng(7)
    ws = [torch.from_numpy(rng.standard_normal(s).astype(np.float32) * np.float32(0.05)).cuda().to(torch.bfloat16)
          for s in shapes]
    gs = [torch.empty(s, device="cuda") for s in shapes]
    lr, wd, beta = 0.02, 0.1, 0.9
    step = F.RootStep(ws, gs, lr=lr, wd=wd, beta=beta, seed=3, momentum_seed=9)
    prev = [None] * len(shapes)
    for t in range(2):
        g_np = [rng.standard_normal(s).astype(np.float32) for s in shapes]
        for g, a in zip(gs, g_np):
            g.copy_(torch.from_numpy(a))
        w_before = [_bf16_bits(w) for w in ws]
        step(t)
        assert step.status() == 0
        for p, (r, c) in enumerate(shapes):
            m_t, st = M.momentum_step(g_np[p], prev[p], beta, 9 + p, t)
            prev[p] = st
            gst = step.states[p]
            assert float(gst.tensor_scale[0]) == st.sg
            assert np.array_equal(np_(gst.scales[0]), st.scales)
            assert np.array_equal(unpack_nibbles(np_(gst.codes[0])), st.codes)
            co = F.fp4root_default_coeffs(r, c, 5)
            o_ref = ns.orthogonalize(m_t, co, seed=3)
            o_gpu = np_(step.scratch[p])
            assert rel_fro(o_gpu, o_ref) <= 1e-3, (p, t)
            want = R.apply_update(w_before[p], o_gpu, lr, wd, np.float32(R.muon_scale(r, c)))
            assert np.array_equal(_bf16_bits(ws[p]), want), (p, t)


@pytest.mark.parametrize("ns_flags", ["default", "no_clip"])
@pytest.mark.parametrize("bad", [float("inf"), float("nan")])
def test_root_step_nonfinite_gradient(ns_flags, bad):
    # the first of two parameters carries the bad value: neither the second
    # parameter's first-moment stage nor the orthogonalisation may clear the status
    flags = F.F_DEFAULT if ns_flags == "default" else F.F_HADAMARD | F.F_ADAPTIVE46
    ws = [torch.zeros((32, 64), device="cuda", dtype=torch.bfloat16) for _ in range(2)]
    gs = [torch.ones((32, 64), device="cuda") for _ in range(2)]
    gs[0][1, 2] = bad
    step = F.RootStep(ws, gs, lr=0.01, ns_flags=flags)
    step(0)
    assert step.status() == -4
    gs[0][1, 2] = 1.0
    step(1)
    assert step.status() == 0


def test_root_step_bad_parameter_leaves_states_unchanged():
    # a misaligned state pointer in the second parameter fails the call before the
    # first parameter's state is touched
    ws = [torch.zeros((32, 64), device="cuda", dtype=torch.bfloat16) for _ in range(2)]
    gs = [torch.ones((32, 64), device="cuda") for _ in range(2)]
    step = F.RootStep(ws, gs, lr=0.01)
    good_codes = step.params[1].m_codes
    step.params[1].m_codes = good_codes + 1
    with pytest.raises(F.Fp4RootError):
        step(0)
    torch.cuda.synchronize()
    assert float(step.states[0].tensor_scale[0]) == 0.0
    assert int(step.states[0].codes.count_nonzero()) == 0
    assert int(ws[0].view(torch.int16).count_nonzero()) == 0
    step.params[1].m_codes = good_codes
    step(0)
    assert step.status() == 0 and float(step.states[0].tensor_scale[0]) > 0.0
