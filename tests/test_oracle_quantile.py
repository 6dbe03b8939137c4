"""Pins for the oracle's p99 threshold (CPU only)."""
import numpy as np
import pytest

from oracle.quantile import clip, clip_threshold


def _sorted_def(a, q):
    v = np.sort(np.abs(a).ravel())
    h = np.float64(np.float32(q)) * (v.size - 1)
    lo = int(np.floor(h))
    if lo >= v.size - 1:
        return np.float32(v[-1])
    f = h - lo
    return np.float32(np.float64(v[lo]) + f * (np.float64(v[lo + 1]) - np.float64(v[lo])))


@pytest.mark.parametrize("n", [1, 2, 3, 17, 100, 101, 1000, 4096])
def test_matches_sort_definition(n):
    rng = np.random.default_rng(n)
    a = (rng.standard_normal(n) * 3).astype(np.float32)
    for q in (0.0, 0.5, 0.99, 1.0):
        assert clip_threshold(a, q) == _sorted_def(a, q)


def test_within_one_ulp_of_numpy_linear_quantile():
    rng = np.random.default_rng(1)
    for n in (1000, 77777, 262144):
        a = rng.standard_t(3, n).astype(np.float32)
        ref = np.quantile(np.abs(a).astype(np.float64), np.float64(np.float32(0.99)), method="linear")
        got = clip_threshold(a, 0.99)
        assert abs(np.float64(got) - ref) <= np.spacing(np.float32(ref))


def test_ties_and_clip():
    a = np.float32([1, 1, 1, 1, 5, -9])
    tau = clip_threshold(a, 0.5)
    assert tau == 1
    assert np.array_equal(clip(a, tau), np.float32([1, 1, 1, 1, 1, -1]))


def test_scale_invariance():
    rng = np.random.default_rng(2)
    a = rng.standard_normal(5000).astype(np.float32)
    assert clip_threshold(a * np.float32(8), 0.99) == clip_threshold(a, 0.99) * np.float32(8)
