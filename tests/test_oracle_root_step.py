"""Pins of the Root parameter update oracle (oracle/root_step.py).

* the BF16 rounding equals torch's float32 -> bfloat16 conversion (round to
  nearest even) on random, tie and boundary patterns;
* closed forms: lr = 0 keeps W; O = 0 and wd = 0 keep W; a one-ulp step
  (lr s = 2^-8 on W = 1, O = 1) gives 1 - 2^-8; pure decay on powers of two.
"""
import numpy as np
import torch

from oracle import root_step as R


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(5000).astype(np.float32) * np.float32(3.0),
                        # exact ties between neighbouring BF16 values, both parities
                        (np.arange(0, 64, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
                        ((np.arange(0x3F80, 0x3FC0, dtype=np.uint32) << 16) | 0x8000).view(np.float32),
                        ((np.arange(0xC080, 0xC0C0, dtype=np.uint32) << 16) | 0x8000).view(np.float32),
                        np.float32([0.0, -0.0, 1.0, -1.0, 3.0e38, 1e-40, -1e-40])])
    x = x[np.isfinite(x)]
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(R.bf16_round(x), want)
    assert np.array_equal(R.bf16_value(want), torch.from_numpy(want.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_update_closed_forms():
    rng = np.random.default_rng(1)
    w = R.bf16_round(rng.standard_normal((16, 32)).astype(np.float32))
    o = rng.standard_normal((16, 32)).astype(np.float32)
    assert np.array_equal(R.apply_update(w, o, 0.0, 0.1, 1.0), w)
    assert np.array_equal(R.apply_update(w, np.zeros_like(o), 0.5, 0.0, 1.0), w)
    one = R.bf16_round(np.float32([1.0]))
    got = R.bf16_value(R.apply_update(one, np.float32([1.0]), 2.0 ** -8, 0.0, 1.0))
    assert got[0] == np.float32(1.0 - 2.0 ** -8)
    p2 = R.bf16_round(np.float32([2.0, -4.0, 0.5]))
    got = R.bf16_value(R.apply_update(p2, np.zeros(3, np.float32), 0.5, 0.5, 0.0))
    assert np.array_equal(got, np.float32([1.5, -3.0, 0.375]))   # W (1 - 1/4), exact
    assert R.muon_scale(3072, 1024) == np.float32(np.sqrt(3.0)) and R.muon_scale(1024, 3072) == 1.0
