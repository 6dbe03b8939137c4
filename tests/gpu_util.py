"""Shared helpers of the GPU parity tests: convert library outputs into oracle objects."""
import numpy as np
import torch

from oracle.formats import unpack_nibbles
from oracle.quantize import NVFP4


def np_(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def gpu_nvfp4(codes, scales, sg) -> NVFP4:
    """Wrap packed GPU codes / scales / tensor scale as the oracle's NVFP4 record."""
    c = unpack_nibbles(np_(codes))
    s = np_(scales)
    return NVFP4(c, s, np.float32(np_(sg).reshape(-1)[0]), np.zeros(s.shape, bool))


def assert_same_nvfp4(got: NVFP4, ref: NVFP4, what: str):
    assert got.sg == ref.sg, f"{what}: tensor scale {got.sg!r} != {ref.sg!r}"
    bad_s = np.count_nonzero(got.scales != ref.scales)
    bad_c = np.count_nonzero(got.codes != ref.codes)
    assert bad_s == 0 and bad_c == 0, f"{what}: {bad_s} scale and {bad_c} code mismatches"


def ulp_diff(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Distance in binary32 units in the last place (same-sign finite values)."""
    ia = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    ib = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    ia = np.where(ia < 0, -(ia & 0x7FFFFFFF), ia)
    ib = np.where(ib < 0, -(ib & 0x7FFFFFFF), ib)
    return np.abs(ia - ib)


def rel_fro(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def need_gpu():
    import pytest
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_04422_amd import fp4root
    fp4root.load()   # a missing library is a failure, not a skip
