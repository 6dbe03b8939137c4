"""Component study of the optimizer-state pipelines on the oracle (Section 3.3).

Section 3.3 reports, on states from real training, that the full second-moment
pipeline (square root, BF16 tile mean, Hadamard) reconstructs far better than
direct NVFP4 storage, that removing the square root or the tile mean makes it
worse, and that without the tile mean it is worse than direct storage; and that
Hadamard mixing helps the first moment.  The paper's states are not available:
this study runs the same comparisons on seeded synthetic states (exponential
moving averages of Student-t(3) gradients with lognormal tile scales) and pins
the orderings that hold there.  The Hadamard comparisons do not reproduce on
such i.i.d. inputs (there is no localised energy to spread) and are reported,
not asserted.  ``python -m pytest tests/test_oracle_state_study.py -s`` prints
the table.
"""
import numpy as np

from oracle import momentum as M
from oracle import qadamw as Q
from oracle.quantize import quantize


def _states(n=256 * 1024, seed=2):
    rng = np.random.default_rng(seed)
    scale = np.repeat(rng.lognormal(0, 1, n // 256), 256)
    v = np.zeros(n)
    m = np.zeros(n)
    for _ in range(30):
        g = rng.standard_t(3, n) * scale * 1e-3
        v = 0.95 * v + 0.05 * g * g
        m = 0.9 * m + 0.1 * g
    return m.astype(np.float32), v.astype(np.float32)


def component_errors():
    m, v = _states()
    d = Q.step_signs(4, 0)

    def rel(a, b):
        return float(np.linalg.norm(np.asarray(a, np.float64) - b) / np.linalg.norm(b))

    out = {
        "v: full pipeline": rel(Q.decode_v(Q.encode_v(v, d), d), v),
        "v: no Hadamard": rel(Q.decode_v(Q.encode_v(v, None), None), v),
        "v: no square root": rel(Q.decode_v(Q.encode_v(v, d, sqrt=False), d, sqrt=False), v),
        "v: no tile mean": rel(Q.decode_v(Q.encode_v(v, d, mean=False), d), v),
        "v: direct NVFP4": rel(quantize(v.reshape(-1, 256), axis=1).dequantize().reshape(-1), v),
    }
    mm = m.reshape(-1, 256)
    out["m: Hadamard, RTN"] = rel(M.decode_state(M.encode_state(mm, d, True, None), d), mm)
    out["m: no Hadamard, RTN"] = rel(M.decode_state(M.encode_state(mm, None, True, None), None), mm)
    draws = M.sr_draws(M.sr_key(4, 0), mm.size).reshape(mm.shape)
    out["m: Hadamard, SR"] = rel(M.decode_state(M.encode_state(mm, d, True, draws), d), mm)
    return out


def test_component_orderings():
    e = component_errors()
    for k, x in e.items():
        print(f"{k:24s} relative L2 {x:.4f}   squared {x * x:.5f}")
    assert e["v: full pipeline"] < e["v: direct NVFP4"]
    assert e["v: no square root"] > e["v: full pipeline"]
    assert e["v: no tile mean"] > e["v: direct NVFP4"]
    assert e["m: Hadamard, SR"] > e["m: Hadamard, RTN"]   # SR trades variance for unbiasedness
