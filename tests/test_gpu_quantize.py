"""GPU parity: the HIP quantiser against the oracle, bit for bit (codes, E4M3 scales, FP32 s_g)."""
import numpy as np
import pytest
import torch

from oracle import rht
from oracle.quantile import clip, clip_threshold
from oracle.quantize import quantize
from paper_2607_04422_amd import workloads
from tests.gpu_util import assert_same_nvfp4, gpu_nvfp4, need_gpu, np_

pytestmark = pytest.mark.gpu

F = None


def setup_module():
    global F
    need_gpu()
    from paper_2607_04422_amd import fp4root
    F = fp4root


SHAPES = [(16, 16), (48, 80), (256, 512), (272, 400), (1024, 3072)]
FLAGS = [0, 2, 4, 6, 7]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("flags", FLAGS)
@pytest.mark.parametrize("axis", [1, 0])
def test_quantize_parity(shape, flags, axis):
    r, c = shape
    m = workloads.matrix(r, c, seed=r * 7 + c, kind="t_rows")
    seed, step = 1234 + flags, 3
    x = torch.from_numpy(m).cuda()
    codes, scales, sg, tau, ws = F.fp4root_quantize(x, axis=axis, flags=flags, clip_quantile=0.99,
                                                    seed=seed, step=step)
    assert F.fp4root_device_status(ws) == 0
    src = m
    if flags & F.F_CLIP:
        t = clip_threshold(m, 0.99)
        assert np_(tau)[0] == t, f"clip threshold {np_(tau)[0]!r} != {t!r}"
        src = clip(m, t)
    signs = rht.step_signs(seed, step) if flags & F.F_HADAMARD else None
    ref = quantize(src, axis, signs, bool(flags & F.F_ADAPTIVE46))
    assert_same_nvfp4(gpu_nvfp4(codes, scales, sg), ref, f"{shape} axis={axis} flags={flags}")


def test_quantize_batch_and_strides():
    rng = np.random.default_rng(3)
    big = rng.standard_normal((3, 64, 160)).astype(np.float32)
    x = torch.from_numpy(big).cuda()[:, :, :128]       # row stride 160, batch stride 64*160
    codes, scales, sg, tau, _ = F.fp4root_quantize(x, axis=1, flags=7, seed=9)
    for b in range(3):
        src = clip(big[b, :, :128], clip_threshold(big[b, :, :128], 0.99))
        ref = quantize(src, 1, rht.step_signs(9, 0), True)
        assert_same_nvfp4(gpu_nvfp4(codes[b], scales[b], sg[b:b + 1]), ref, f"batch {b}")


def test_quantize_edge_cases():
    z = np.zeros((32, 64), np.float32)
    x = torch.from_numpy(z).cuda()
    for flags in (0, 6):
        codes, scales, sg, _, _ = F.fp4root_quantize(x, axis=1, flags=flags)
        assert np_(sg)[0] == 0 and not np_(scales).any()
        # a rotated zero block holds -0.0 where a sign was flipped: the sign bit is kept
        ref = quantize(z, 1, rht.step_signs(0, 0) if flags & 2 else None, bool(flags & 4))
        assert_same_nvfp4(gpu_nvfp4(codes, scales, sg), ref, f"zeros flags={flags}")
    m = np.zeros((32, 64), np.float32)
    m[3, 17] = -2.5e-30     # tiny single value: subnormal-range scale arithmetic
    m[20, 40] = 1e-38
    x = torch.from_numpy(m).cuda()
    for flags in (0, 6):
        codes, scales, sg, _, _ = F.fp4root_quantize(x, axis=1, flags=flags)
        ref = quantize(m, 1, rht.step_signs(0, 0) if flags & 2 else None, bool(flags & 4))
        assert_same_nvfp4(gpu_nvfp4(codes, scales, sg), ref, f"tiny flags={flags}")
    # a tensor scale just above 2^-40 with blocks in and below the subnormal range:
    # the rotated quarter of these underflows, the kernel's scaled copies do not
    rng = np.random.default_rng(4)
    m = np.zeros((32, 64), np.float32)
    m[0, 0] = 1e-7
    m[5, 3], m[5, 4], m[5, 9] = 1e-38, -3e-41, 1e-45
    m[9, 16:32] = (7e-39 * rng.standard_normal(16)).astype(np.float32)
    m[12, :16] = (2e-37 * rng.standard_normal(16)).astype(np.float32)
    m[17, 32:48] = (1e-12 * rng.standard_normal(16)).astype(np.float32)
    m[30, 48:] = (3e-9 * rng.standard_normal(16)).astype(np.float32)
    x = torch.from_numpy(m).cuda()
    for flags in (0, 6):
        codes, scales, sg, _, _ = F.fp4root_quantize(x, axis=1, flags=flags)
        if flags & 2:
            assert np_(sg)[0] >= 2.0 ** -40
        ref = quantize(m, 1, rht.step_signs(0, 0) if flags & 2 else None, bool(flags & 4))
        assert_same_nvfp4(gpu_nvfp4(codes, scales, sg), ref, f"small scale flags={flags}")


def test_quantize_nonfinite_reported():
    m = np.ones((32, 32), np.float32)
    m[5, 7] = np.inf
    x = torch.from_numpy(m).cuda()
    _, _, _, _, ws = F.fp4root_quantize(x, axis=1, flags=6)
    assert F.fp4root_device_status(ws) == -4
    m[5, 7] = np.nan
    x = torch.from_numpy(m).cuda()
    _, _, _, _, ws = F.fp4root_quantize(x, axis=0, flags=7)
    assert F.fp4root_device_status(ws) == -4


def test_quantize_full_size_sampled_rows():
    """3072 x 8192 (a 3B-shaped MLP matrix): full GPU quantisation, oracle on sampled rows."""
    m = workloads.matrix(3072, 8192, seed=11, kind="t_rows")
    x = torch.from_numpy(m).cuda()
    rng = np.random.default_rng(0)
    for axis in (1, 0):
        codes, scales, sg, _, _ = F.fp4root_quantize(x, axis=axis, flags=6, seed=5, step=1)
        nrows = m.shape[0] if axis == 1 else m.shape[1]
        sel = np.sort(rng.choice(nrows, 48, replace=False))
        ref = quantize(m, axis, rht.step_signs(5, 1), True, rows=sel)
        got = gpu_nvfp4(codes[sel], scales[sel], sg)
        assert_same_nvfp4(got, ref, f"full-size axis={axis}")


def test_quantize_adaptive_near_ties():
    """Blocks whose two 4/6 candidates have equal or nearly equal squared errors
    (a single spike representable under both scalings, spikes on the E4M3 grid,
    two-level blocks), where the binary32 error sums cannot decide and the
    binary64 recomputation must reproduce the reference choice (keep M = 4 only
    if strictly smaller)."""
    rng = np.random.default_rng(21)
    rows, cols = 64, 256
    m = np.zeros((rows, cols), np.float32)
    m[0, 0] = 2688.0                                  # amax: s_g = 1
    for r in range(rows):
        for b in range(cols // 16):
            blk = m[r, 16 * b:16 * b + 16]
            kind = (r + b) % 4
            e4 = 2.0 ** int(rng.integers(-6, 8))
            if kind == 0:      # one spike: 6 s and 4 (1.5 s) both exact
                blk[int(rng.integers(16))] = np.float32(6.0 * e4)
            elif kind == 1:    # two levels on both grids
                blk[:8] = np.float32(6.0 * e4)
                blk[8:] = np.float32(3.0 * e4)
            elif kind == 2:    # grid values plus a tiny perturbation
                blk[:] = np.float32(6.0 * e4) * (1 + np.float32(2.0 ** -20) * rng.standard_normal(16).astype(np.float32))
            else:              # random
                blk[:] = rng.standard_normal(16).astype(np.float32) * np.float32(e4)
    m[0, 0] = 2688.0
    x = torch.from_numpy(m).cuda()
    for axis in (1, 0):
        codes, scales, sg, _, _ = F.fp4root_quantize(x, axis=axis, flags=F.F_ADAPTIVE46, seed=0)
        ref = quantize(m, axis, None, True)
        assert_same_nvfp4(gpu_nvfp4(codes, scales, sg), ref, f"near ties axis={axis}")


def test_quantize_grid_midpoints():
    """Elements exactly on E2M1 grid midpoints of their block (ties to the even code)
    and a few ulps to either side: the hardware-rounded fast path must hand these
    blocks to the exact threshold comparisons and match the reference bit for bit."""
    rng = np.random.default_rng(5)
    rows, cols = 48, 256
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], np.float32)
    m = np.zeros((rows, cols), np.float32)
    for r in range(rows):
        for b in range(cols // 16):
            blk = m[r, 16 * b:16 * b + 16]
            s = np.float32(rng.choice([1.0, 1.125, 1.5, 1.875]) * 2.0 ** int(rng.integers(-8, 6)))
            blk[0] = np.float32(6.0) * s                    # block maximum: the M = 6 scale is s
            v = mids[rng.integers(0, 7, 15)] * s             # exact: at most 7 significant bits
            steps = rng.integers(-3, 4, 15)
            for i in range(15):
                x = v[i]
                for _ in range(abs(int(steps[i]))):
                    x = np.nextafter(x, np.float32(np.inf if steps[i] > 0 else -np.inf), dtype=np.float32)
                blk[1 + i] = x
            blk[:] *= rng.choice([-1.0, 1.0], 16).astype(np.float32)
    m[0, 0] = 2688.0                                        # s_g = 1
    x = torch.from_numpy(m).cuda()
    for flags in (0, F.F_ADAPTIVE46):
        for axis in (1, 0):
            codes, scales, sg, _, _ = F.fp4root_quantize(x, axis=axis, flags=flags, seed=0)
            ref = quantize(m, axis, None, bool(flags & F.F_ADAPTIVE46))
            assert_same_nvfp4(gpu_nvfp4(codes, scales, sg), ref, f"midpoints flags={flags} axis={axis}")
