"""fp4root_quantize_noalloc (no workspace, the library's fixed scratch) through the
C ABI against fp4root_quantize (caller workspace) on the same inputs: codes,
scales, tensor scales and clip thresholds equal bit for bit, over two calls in a
row (the second on a smaller input, so stale scratch contents would show), both
axes, with and without clipping; non-finite input reported through the status
output and cleared by the next call; batches beyond the scratch rejected before
any work."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_04422_amd import workloads
from tests.gpu_util import need_gpu

pytestmark = pytest.mark.gpu

F = None


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _outputs(B, R, C, axis):
    shape_c = (B, R, C // 2) if axis == 1 else (B, C, R // 2)
    shape_s = (B, R, C // 16) if axis == 1 else (B, C, R // 16)
    return (torch.full(shape_c, 0xAB, dtype=torch.uint8, device="cuda"),
            torch.full(shape_s, 0xCD, dtype=torch.uint8, device="cuda"),
            torch.full((B,), -1.0, device="cuda"), torch.full((B,), -1.0, device="cuda"),
            torch.full((1,), 7, dtype=torch.int32, device="cuda"))


def _noalloc(lib, x, axis, flags, seed, step):
    B, R, C = x.shape
    codes, scales, sg, tau, status = _outputs(B, R, C, axis)
    rc = lib.fp4root_quantize_noalloc(_p(x), B, R, C, C, R * C, axis, flags, 0.99, seed, step, _p(codes),
                                      _p(scales), _p(sg), _p(tau), _p(status), None)
    assert rc == 0
    torch.cuda.synchronize()
    return codes, scales, sg, tau, int(status[0])


def _with_workspace(lib, x, axis, flags, seed, step):
    B, R, C = x.shape
    codes, scales, sg, tau, _ = _outputs(B, R, C, axis)
    need = lib.fp4root_quantize_workspace(B, R, C, flags)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    rc = lib.fp4root_quantize(_p(x), B, R, C, C, R * C, axis, flags, 0.99, seed, step, _p(codes), _p(scales),
                              _p(sg), _p(tau), _p(ws), need, None)
    assert rc == 0
    torch.cuda.synchronize()
    return codes, scales, sg, tau, F.fp4root_device_status(ws)


def _batch(B, R, C, seed):
    return torch.from_numpy(np.stack([workloads.matrix(R, C, seed=seed + i, kind="t_rows") for i in range(B)])).cuda()


@pytest.mark.parametrize("axis", [1, 0])
@pytest.mark.parametrize("flags", [7, 6])
def test_noalloc_equals_workspace_call_twice(axis, flags):
    lib = F.load()
    for (B, R, C, seed) in ((40, 256, 512, 1), (3, 64, 128, 90)):   # the second call is smaller
        x = _batch(B, R, C, seed)
        got = _noalloc(lib, x, axis, flags, 5, 2)
        want = _with_workspace(lib, x, axis, flags, 5, 2)
        for g, w, what in zip(got[:3], want[:3], ("codes", "scales", "tensor scale")):
            assert torch.equal(g, w), (B, R, C, what)
        if flags & 1:
            assert torch.equal(got[3], want[3]), (B, R, C, "clip threshold")
        assert got[4] == 0 and want[4] == 0


def test_noalloc_status_and_limits():
    lib = F.load()
    x = _batch(2, 64, 128, 3)
    x[1, 5, 7] = float("nan")
    assert _noalloc(lib, x, 1, 7, 0, 0)[4] == -4
    x[1, 5, 7] = 0.25
    assert _noalloc(lib, x, 1, 7, 0, 0)[4] == 0
    # more matrices than the scratch holds: rejected synchronously, outputs untouched
    big = torch.zeros((257, 16, 16), device="cuda")
    codes, scales, sg, tau, status = _outputs(257, 16, 16, 1)
    rc = lib.fp4root_quantize_noalloc(_p(big), 257, 16, 16, 16, 256, 1, 7, 0.99, 0, 0, _p(codes), _p(scales),
                                      _p(sg), _p(tau), _p(status), None)
    assert rc == -3
    torch.cuda.synchronize()
    assert int(status[0]) == 7 and float(sg[0]) == -1.0
    # 256 matrices fit
    codes, scales, sg, tau, status = _outputs(256, 16, 16, 1)
    rc = lib.fp4root_quantize_noalloc(_p(big), 256, 16, 16, 16, 256, 1, 7, 0.99, 0, 0, _p(codes), _p(scales),
                                      _p(sg), _p(tau), _p(status), None)
    assert rc == 0
    torch.cuda.synchronize()
    assert int(status[0]) == 0 and float(sg.abs().max()) == 0.0
