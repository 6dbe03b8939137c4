"""Error study of the NVFP4 Newton-Schulz iteration (Fig. 3b; Section 3.4 error numbers).

Section 3.4 compares routes by the relative L2 error of the NVFP4 iteration:
the plain all-FP4 route against the proposed one (shape-dependent
coefficients, p99 clipping, the random Hadamard rotation and adaptive 4/6
scaling in every quantisation), and Fig. 3b compares the shape-dependent
coefficients with the standard Muon ones.  This module measures that error
for the library's routes on the synthetic workloads:

    err = ||Y_q - Y_ref||_F / ||Y_ref||_F,

Y_q the library's output of the route (NVFP4 or BF16 products), Y_ref the same
five steps with the same coefficients in binary64 without quantisation, both
from the same X_0 (the library's own clipped and normalised input, taken with
zero NS steps).  Errors are aggregated over a workload's matrices as
sqrt(sum ||Y_q - Y_ref||^2 / sum ||Y_ref||^2).

The binary64 reference is plain torch float64 matrix products (on the GPU for
speed); `tests/test_error_study.py` pins it to the test oracle and to the
closed form U p(Sigma) V^T on the CPU.  This is measurement and test code:
the library does not use it.

    python tests/error_study.py [--cases a,b] [--json out.json]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2607_04422_amd import workloads  # noqa: E402

MUON = (3.4445, -4.7750, 2.0315)   # the standard Muon quintic
STEPS = 5

# name -> (flags, coefficient set); flags are the library's F_* bits
# (1 clip, 2 Hadamard, 4 adaptive 4/6, 8 BF16 products)
ROUTES = {
    "proposed": (7, "shape"),
    "proposed, Muon coefficients": (7, "muon"),
    "no clipping": (6, "shape"),
    "plain FP4, shape coefficients": (0, "shape"),
    "plain FP4 (Muon coefficients)": (0, "muon"),
    "BF16 products": (9, "shape"),
}


def ns_reference(x0: torch.Tensor, coeffs) -> torch.Tensor:
    """Unquantised NS in binary64 on the short side: A = X X^T, B = b A + c A A,
    X <- a X + B X per step; returns the input's orientation (float64)."""
    x = x0.to(torch.float64)
    tall = x.shape[0] > x.shape[1]
    if tall:
        x = x.T
    for a, b, c in coeffs:
        g = x @ x.T
        x = a * x + (b * g + c * (g @ g)) @ x
    return x.T if tall else x


def route_coeffs(F, kind: str, rows: int, cols: int):
    return [MUON] * STEPS if kind == "muon" else F.fp4root_default_coeffs(rows, cols, STEPS)


def run_case(F, mats, routes=ROUTES, seed: int = 0, log=None):
    """Errors of every route on one workload: {route: {"err", "max", "finite"}}."""
    dev = torch.device("cuda")
    ins = [torch.from_numpy(m).to(dev) for m in mats]
    out = {}
    for name, (flags, kind) in routes.items():
        t0 = time.time()
        x0s = F.Orthogonalizer(ins, steps=0, flags=flags, seed=seed)()
        if kind == "muon":
            orth = F.Orthogonalizer(ins, steps=STEPS, coeffs=[MUON] * STEPS, flags=flags, seed=seed)
        else:
            orth = F.Orthogonalizer(ins, steps=STEPS, flags=flags, seed=seed)
        ys = orth()
        st = orth.status()
        num = den = 0.0
        worst = 0.0
        for m, x0, y in zip(mats, x0s, ys):
            ref = ns_reference(x0, route_coeffs(F, kind, *m.shape))
            d2 = float(torch.sum((y.to(torch.float64) - ref) ** 2))
            r2 = float(torch.sum(ref * ref))
            num += d2
            den += r2
            worst = max(worst, math.sqrt(d2 / r2) if r2 > 0 else 0.0)
        err = math.sqrt(num / den) if den > 0 else 0.0
        finite = st == 0 and math.isfinite(err)
        out[name] = {"err": err, "max": worst, "finite": finite, "status": st}
        if log:
            log(f"{name}: err {err:.4g} (worst matrix {worst:.4g}, status {st}) {time.time() - t0:.1f}s")
        del x0s, ys, orth
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--cases", default=",".join(workloads.CASES))
    ap.add_argument("--json", default=None)
    args = ap.parse_args()
    from paper_2607_04422_amd import fp4root as F
    F.load()

    def log(msg):
        print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)

    results = {}
    for case in args.cases.split(","):
        log(f"case {case}: generating")
        mats = workloads.case_matrices(case)
        results[case] = run_case(F, mats, log=lambda s: log(f"  {case} | {s}"))
        del mats
        torch.cuda.empty_cache()
    names = list(ROUTES)
    print("| route | flags | coefficients | " + " | ".join(results) + " |")
    print("|---|---|---|" + "---|" * len(results))
    for n in names:
        flags, kind = ROUTES[n]
        cells = []
        for case in results:
            r = results[case][n]
            cells.append(f"{r['err']:.4f}" if r["finite"] else f"non-finite (status {r['status']})")
        print(f"| {n} | {flags} | {kind} | " + " | ".join(cells) + " |")
    if args.json:
        with open(args.json, "w") as f:
            json.dump(results, f, indent=1)


if __name__ == "__main__":
    main()
