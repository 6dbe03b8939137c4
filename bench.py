#!/usr/bin/env python3
"""Throughput of NVFP4 Newton-Schulz orthogonalisation on one MI355X.

One "step" is one fp4root_orthogonalize call over the whole matrix set: p99
clipping, Frobenius normalisation, five NVFP4 Newton-Schulz steps and the
write-back, for every matrix (paper Section 3.4; Table 6 "Root" rows: isolated
Root, five NS iterations, p99 clipping, aspect-ratio coefficients).  Inputs are
resident in HBM before the timed region starts.

Default workload: four 3B-shaped decoder blocks, 28 FP32 matrices
(q, o 3072x3072; k, v 1024x3072; gate, up 8192x3072; down 3072x8192), seeded
synthetic momentum (Student-t(4) entries, lognormal(0,1) row scales).

Prints ONE JSON line.  Also reports, on the same line: the in-library BF16 NS
path on the same inputs, a roofline figure for the dominant kernel measured
with HIP events on its launch stream, the CPU oracle timed on a bounded
sample of the same workload, and one step of the NVFP4 first-moment state
(fp4root_momentum_update, Section 3.3 storage recipe) over the same set,
against the HBM bandwidth (it moves 13.125 algorithmic bytes per element), and the
full Root optimizer step (fp4root_root_step: first moment, NVFP4 Root, BF16
parameter update) with its update kernel against the HBM bandwidth, and one
quantized-state AdamW step (fp4root_qadamw_update) with every matrix as a flat
parameter, against the HBM bandwidth.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

COPY_PROBE_BYTES = 256 << 20
METRIC = "NS-orthogonalised matrices/s + effective TFLOP/s (% MFMA peak), 3B-shaped set"
BF16_MFMA_PEAK_TFLOPS = 2516.6
# The exact NVFP4 products run on the f16 MFMA (32x32x16, decoded operands), whose dense
# peak is the bf16/fp16 one: 2.5 PFLOP/s.  With whole 4-block stages chained into one
# binary32 accumulator, the binary64 folds (2 VALU ops per output per 64-element stage)
# match that rate too: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz / 2 x 128 FLOP = 2516 TFLOP/s.
F16_MFMA_PEAK_TFLOPS = BF16_MFMA_PEAK_TFLOPS
HBM_PEAK_GBS = 8000.0   # MI355X HBM3E
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "k_gemm_fp4_update_block3b_x4_traffic.md")


def ns_flop(m: int, n: int, steps: int) -> float:
    """Algorithmic FLOP of `steps` NS steps on an m x n matrix (m <= n), Grams exploited."""
    return steps * (m * (m + 1) * n + m * (m + 1) * m + 2.0 * m * m * n)


def set_flop(shapes, steps):
    return sum(ns_flop(min(r, c), max(r, c), steps) for (r, c) in shapes)


def time_calls(fn, warmup, iters, torch, per_call=None):
    """Mean wall time of `iters` calls after `warmup` (synchronised on both sides).
    With a list `per_call`, also appends each call's duration in ms from HIP events
    recorded between the calls on the launch stream (torch's current stream)."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(iters + 1)] if per_call is not None else None
    t0 = time.perf_counter()
    for i in range(iters):
        if evs:
            evs[i].record()
        fn()
    if evs:
        evs[iters].record()
    torch.cuda.synchronize()
    t = (time.perf_counter() - t0) / iters
    if evs:
        per_call.extend(evs[i].elapsed_time(evs[i + 1]) for i in range(iters))
    return t


def spread(ms):
    """Median and 10th / 90th percentiles of per-call times (ms)."""
    v = sorted(ms)
    if not v:
        return None
    q = lambda f: v[min(len(v) - 1, max(0, int(round(f * (len(v) - 1)))))]
    return {"median": round(q(0.5), 3), "p10": round(q(0.1), 3), "p90": round(q(0.9), 3), "calls": len(v)}


def torch_bf16_reference(inputs, coeffs_for, steps, warmup, iters, torch):
    """The same five BF16 NS steps written with torch.bmm (hipBLASLt), as context for the
    in-library BF16 path: X bf16, A = X X^T, B = b A + c A A, X = a X + B X, batched per shape
    group, on inputs already clipped, normalised and oriented short side first."""
    groups = {}
    for t in inputs:
        r, c = t.shape
        x = t if r <= c else t.t()
        groups.setdefault((min(r, c), max(r, c)), []).append(x)
    xs = {k: torch.stack([(v / v.norm()).to(torch.bfloat16) for v in vs]).contiguous() for k, vs in groups.items()}

    def run():
        for (m, n), x0 in xs.items():
            co = coeffs_for(m, n)
            x = x0
            for (a, b, c) in co[:steps]:
                xt = x.transpose(1, 2).contiguous()
                A = torch.bmm(x, xt)
                B = b * A + c * torch.bmm(A, A)
                x = a * x + torch.bmm(B, x)
        return x

    t = time_calls(run, warmup, iters, torch)
    return t


SAMPLE_SHORT, SAMPLE_LONG = 1024, 3072   # about 5 s of oracle work per sample on a 16-core host


def _oracle_sample(m):
    """The part of a workload matrix the oracle is timed on: the matrix itself when it
    holds at most 1024 x 3072 elements, else its leading 1024 x 3072 block (3072 x 1024
    for a tall matrix), drawn from the same distribution."""
    r, c = m.shape
    if r * c <= SAMPLE_SHORT * SAMPLE_LONG:
        return m
    if r <= c:
        return np.ascontiguousarray(m[:min(r, SAMPLE_SHORT), :min(c, SAMPLE_LONG)])
    return np.ascontiguousarray(m[:min(r, SAMPLE_LONG), :min(c, SAMPLE_SHORT)])


def _quantised_elements(m, n, steps):
    """Elements the NS steps quantise: X along both axes, A and B (m <= n)."""
    return steps * (2.0 * m * n + 2.0 * m * m)


def cpu_baseline(case, coeffs_for, steps):
    """The oracle, as it stands, on a bounded sample of the workload: the first matrix of
    each distinct shape (at most three shapes), each whole or its leading 1024 x 3072
    block, about 5 s each on the host.  Its time is split into the clip and
    normalisation (scaled by elements), the quantisations (scaled by quantised elements)
    and the exact products (scaled by algorithmic FLOP); the rates over the samples are
    applied to every matrix of the set and summed."""
    from threadpoolctl import threadpool_info

    from oracle import ns
    from paper_2607_04422_amd import workloads

    shapes = workloads.case_shapes(case)
    picks, seen = [], set()
    for i, (_, r, c) in enumerate(shapes):
        key = (min(r, c), max(r, c))
        if key not in seen and len(picks) < 3:
            seen.add(key)
            picks.append(i)
    mats = workloads.case_matrices(case, limit=picks[-1] + 1)
    timing = {}
    units = {"prepare": 0.0, "quantize": 0.0, "products": 0.0}
    parts = []
    dt = 0.0
    for i in picks:
        sample = _oracle_sample(mats[i])
        r0, c0 = sample.shape
        ms, ns_ = min(r0, c0), max(r0, c0)
        t0 = time.perf_counter()
        ns.orthogonalize(sample, coeffs_for(r0, c0), seed=0, timing=timing)
        dt += time.perf_counter() - t0
        units["prepare"] += r0 * c0
        units["quantize"] += _quantised_elements(ms, ns_, steps)
        units["products"] += ns_flop(ms, ns_, steps)
        what = "whole" if sample is mats[i] else f"leading {r0}x{c0} block"
        parts.append(f"{shapes[i][0]} ({mats[i].shape[0]}x{mats[i].shape[1]}, {what})")
    del mats
    rate = {k: timing.get(k, 0.0) / units[k] for k in units}
    t_set = 0.0
    for (_, r, c) in shapes:
        m, n = min(r, c), max(r, c)
        t_set += (rate["prepare"] * r * c + rate["quantize"] * _quantised_elements(m, n, steps)
                  + rate["products"] * ns_flop(m, n, steps))
    threads = max((d.get("num_threads", 1) for d in threadpool_info()), default=1)
    return {
        "value": len(shapes) / t_set, "unit": "matrices/s", "cores": int(threads), "kind": "oracle",
        "sample": f"{', '.join(parts)}: clip + normalise + {steps} NVFP4 NS steps each, {dt:.1f} s on the host "
                  f"({timing.get('prepare', 0):.1f} s prepare, {timing.get('quantize', 0):.1f} s quantise, "
                  f"{timing.get('products', 0):.1f} s products); scaled to the {len(shapes)}-matrix set by "
                  f"elements, quantised elements and algorithmic FLOP; the products use {threads} BLAS "
                  f"threads, the quantiser one core",
        "sample_seconds": round(dt, 2),
        "estimated_set_seconds": round(t_set, 1),
        "host_cpu_count": os.cpu_count(),
    }


MOM_BYTES_PER_ELEMENT = 4 + 0.5 + 1 / 16 + 4 + 4 + 0.5 + 1 / 16   # update pass + encode pass


def momentum_bench(inputs, warmup, iters, torch, F):
    """One first-moment step (fp4root_momentum_update, stochastic rounding, rotation,
    4/6) over the whole set, one call per shape batch; inputs act as gradients."""
    groups = {}
    for t in inputs:
        groups.setdefault(tuple(t.shape), []).append(t)
    batches = []
    for (r, c), ts in groups.items():
        g = torch.stack(ts)
        batches.append((g, F.MomentumState(len(ts), r, c), torch.empty_like(g)))
    n = sum(g.numel() for g, _, _ in batches)
    step = [0]

    def run():
        for g, st, m in batches:
            F.fp4root_momentum_update(g, st, 0.9, step[0], seed=1, m=m)
        step[0] += 1

    run()
    torch.cuda.synchronize()
    if any(F.fp4root_device_status(st.ws) != 0 for _, st, _ in batches):
        return {"error": "device status"}
    calls = []
    t = time_calls(run, warmup, iters, torch, calls)
    gbs = n * MOM_BYTES_PER_ELEMENT / t / 1e9
    out = {"ms_per_step": round(t * 1e3, 4), "per_call_ms": spread(calls), "elements": n,
           "launches_per_step": 2 * len(batches), "bytes_per_element": MOM_BYTES_PER_ELEMENT,
           "achieved_GB_per_s": round(gbs, 1), "peak_GB_per_s": HBM_PEAK_GBS,
           "frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
           "flags": "hadamard+adaptive46+stochastic", "beta": 0.9}
    del batches
    return out


APPLY_BYTES_PER_ELEMENT = 2 + 4 + 2   # BF16 weights in and out, FP32 direction in


def root_step_bench(inputs, warmup, iters, torch, F):
    """The full Root optimizer step (first moment, NVFP4 Root, parameter update) over
    the set with BF16 weights, and the update kernel alone against HBM bandwidth."""
    weights = [torch.zeros(t.shape, dtype=torch.bfloat16, device=t.device) for t in inputs]
    step = F.RootStep(weights, inputs, lr=1.5e-4, wd=0.1, beta=0.9)
    k = [0]

    def run():
        step(k[0])
        k[0] += 1

    run()
    torch.cuda.synchronize()
    if step.status() != 0:
        return {"error": "device status"}
    calls = []
    t = time_calls(run, warmup, iters, torch, calls)
    n = sum(w.numel() for w in weights)

    def apply_all():
        for w, o in zip(weights, step.scratch):
            F.fp4root_apply_update(w, o, 1.5e-4, 0.1, 1.0)

    calls_a = []
    ta = time_calls(apply_all, warmup, iters, torch, calls_a)
    gbs = n * APPLY_BYTES_PER_ELEMENT / ta / 1e9
    out = {"ms_per_step": round(t * 1e3, 3), "per_call_ms": spread(calls), "parameters": len(weights),
           "lr": 1.5e-4, "wd": 0.1, "beta": 0.9, "weights": "bf16",
           "apply_update": {"ms": round(ta * 1e3, 4), "elements": n, "bytes_per_element": APPLY_BYTES_PER_ELEMENT,
                            "achieved_GB_per_s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
                            "launches": len(weights)}}
    del step, weights
    return out


# pass 1 (first moment read only, second moment, weights): g 4 + m state 0.5625 +
# v state 0.6328 + w 2 read, v state 0.6328 + w 2 written; pass 2 (first moment
# re-derived and encoded in place): g 4 + m state 0.5625 read, m state 0.5625 written
_M_STATE = 0.5 + 1 / 16
_V_STATE = 0.5 + 2 / 16 + 2 / 256
QADAMW_BYTES_PER_ELEMENT = (4 + _M_STATE + 2 * _V_STATE + 2 + 2) + (4 + 2 * _M_STATE)


def qadamw_bench(inputs, warmup, iters, torch, F):
    """One quantized-state AdamW step with every matrix of the set as a flat parameter."""
    params = []
    for t in inputs:
        n = t.numel()
        params.append((torch.zeros(n, dtype=torch.bfloat16, device=t.device), t.reshape(-1), F.QAdamWState(n)))
    k = [0]

    def run():
        for w, g, st in params:
            F.fp4root_qadamw_update(w, g, st, k[0], 1e-4, 0.1, 0.9, 0.95, 1e-8)
        k[0] += 1

    run()
    torch.cuda.synchronize()
    if any(F.fp4root_device_status(st.ws) != 0 for _, _, st in params):
        return {"error": "device status"}
    calls = []
    t = time_calls(run, warmup, iters, torch, calls)
    n = sum(w.numel() for w, _, _ in params)
    gbs = n * QADAMW_BYTES_PER_ELEMENT / t / 1e9
    out = {"ms_per_step": round(t * 1e3, 4), "per_call_ms": spread(calls), "parameters": len(params),
           "elements": n, "bytes_per_element": round(QADAMW_BYTES_PER_ELEMENT, 4),
           "achieved_GB_per_s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
           "state_bits_per_element": {"m": 4.5, "v": 5.0625}, "weights": "bf16",
           "flags": "hadamard+adaptive46+stochastic (m)"}
    del params
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20, help="timed orthogonalize calls")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--case", default="block3b_x4")
    ap.add_argument("--ns-steps", type=int, default=5)
    ap.add_argument("--no-bf16", action="store_true", help="skip the BF16 comparison path")
    ap.add_argument("--no-fp32-accum", action="store_true",
                    help="skip the NVFP4 path with binary32 product accumulation")
    ap.add_argument("--probe-fp32-accum", action="store_true",
                    help="with --probe: the calls use binary32 product accumulation (FP4ROOT_F_FP32_ACCUM)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-roofline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph replay of the call")
    ap.add_argument("--no-momentum", action="store_true",
                    help="skip the first-moment state update, the full Root step and Q-AdamW")
    ap.add_argument("--probe", action="store_true",
                    help="for hardware-counter runs: one warm and one profiled orthogonalize call, "
                         "then a plain 256 MiB device copy as the byte-count reference; no timing")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "fp4root runs on one GPU only: sharding across GPUs is not "
                          "implemented", "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_04422_amd import fp4root as F
    from paper_2607_04422_amd import workloads

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    F.load()
    dev = torch.device("cuda:0")
    shapes = workloads.case_shapes(args.case)
    mats = workloads.case_matrices(args.case)
    inputs = [torch.from_numpy(m).to(dev) for m in mats]
    del mats
    S = args.ns_steps
    flop = set_flop([(r, c) for (_, r, c) in shapes], S)

    probe_flags = F.F_DEFAULT | (F.F_FP32_ACCUM if args.probe and args.probe_fp32_accum else 0)
    orth = F.Orthogonalizer(inputs, steps=S, flags=probe_flags, clip_quantile=0.99, eps=1e-7, seed=0)
    orth()
    torch.cuda.synchronize()
    if orth.status() != 0:
        print(json.dumps({"error": f"device status {orth.status()}"}))
        sys.exit(1)
    if args.probe:
        orth()
        src = torch.empty(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"probe": args.case, "copy_bytes": COPY_PROBE_BYTES}), flush=True)
        return
    calls = []
    t_step = time_calls(orth, args.warmup, args.steps, torch, calls)
    value = len(shapes) / t_step
    tflops = flop / t_step / 1e12

    # the same call replayed from a HIP graph (one launch of the recorded kernels)
    graph_replay = None
    if not args.no_graph:
        eager = [o.clone() for o in orth.outputs]
        graph = orth.capture()
        graph.replay()
        torch.cuda.synchronize()
        same = all(torch.equal(a, b) for a, b in zip(eager, orth.outputs))
        del eager
        calls_g = []
        t_g = time_calls(graph.replay, args.warmup, args.steps, torch, calls_g)
        graph_replay = {"ms_per_step": round(t_g * 1e3, 4), "per_call_ms": spread(calls_g),
                        "matrices_per_s": round(len(shapes) / t_g, 2),
                        "tflops_effective": round(flop / t_g / 1e12, 2), "equals_eager": same}
        del graph

    roofline = None
    if not args.no_roofline:
        F.fp4root_timer_reset()
        F.fp4root_timer_enable(True)
        for _ in range(args.steps):
            orth()
        torch.cuda.synchronize()
        F.fp4root_timer_enable(False)
        per_kernel = {k: F.fp4root_timer_read(k) for k in (0, 1, 2)}
        F.fp4root_timer_reset()
        ms2, n2, fl2 = per_kernel[2]            # the update product X <- a X + qB qXt^T
        achieved = fl2 / (ms2 / 1e3) / 1e12 if ms2 > 0 else 0.0
        peak = F16_MFMA_PEAK_TFLOPS
        from paper_2607_04422_amd import prof
        traffic = prof.read_update_traffic(TRAFFIC_RECORD) if args.case == "block3b_x4" else None
        roofline = {
            "kernel": "k_gemm_fp4<update X> (exact NVFP4 product: f16 MFMA, chained block groups, "
                      "f64 accumulation)",
            "bound": "mfma", "achieved": round(achieved, 2), "peak": round(peak, 1), "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": round(traffic) if traffic is not None else None,
            "avg_launch_ms": round(ms2 / max(n2, 1), 4), "launches": n2,
            "all_products_tflops": round(sum(v[2] for v in per_kernel.values()) /
                                         (sum(v[0] for v in per_kernel.values()) / 1e3) / 1e12, 2),
            "products_share_of_step": round(sum(v[0] for v in per_kernel.values()) / args.steps /
                                            (t_step * 1e3), 4),
            "per_kernel_tflops": {str(k): round(v[2] / (v[0] / 1e3) / 1e12, 2) if v[0] else 0.0
                                  for k, v in per_kernel.items()},
        }

    bf16 = None
    if not args.no_bf16:
        orth16 = F.Orthogonalizer(inputs, steps=S, flags=F.F_CLIP | F.F_BF16_PATH, clip_quantile=0.99,
                                  eps=1e-7, seed=0)
        calls16 = []
        t16 = time_calls(orth16, args.warmup, args.steps, torch, calls16)
        bf16 = {"ms_per_step": round(t16 * 1e3, 3), "per_call_ms": spread(calls16),
                "matrices_per_s": round(len(shapes) / t16, 2),
                "tflops_effective": round(flop / t16 / 1e12, 2),
                "pct_bf16_peak": round(100 * flop / t16 / 1e12 / BF16_MFMA_PEAK_TFLOPS, 2),
                "nvfp4_speedup_vs_bf16": round(t16 / t_step, 3)}
        del orth16
        try:
            tt = torch_bf16_reference(inputs, lambda r, c: F.fp4root_default_coeffs(r, c, S), S,
                                      args.warmup, args.steps, torch)
            bf16["torch_bmm_reference"] = {
                "ms_per_step": round(tt * 1e3, 3), "tflops_effective": round(flop / tt / 1e12, 2),
                "note": "same BF16 NS with torch.bmm (hipBLASLt), NS steps only, context"}
        except Exception as exc:   # context only; never fails the bench line
            bf16["torch_bmm_reference"] = {"error": str(exc)[:200]}

    # The same NVFP4 iteration with binary32 product accumulation (FP4ROOT_F_FP32_ACCUM: one
    # MFMA accumulator per product, as tensor-core NVFP4 products accumulate): its time, its
    # update product's rate, and its distance to the exact path's output on these inputs.
    fp32acc = None
    if not args.no_fp32_accum:
        orth32 = F.Orthogonalizer(inputs, steps=S, flags=F.F_DEFAULT | F.F_FP32_ACCUM, clip_quantile=0.99,
                                  eps=1e-7, seed=0)
        orth32()
        torch.cuda.synchronize()
        num = sum(float(torch.sum((a.double() - b.double()) ** 2)) for a, b in zip(orth32.outputs, orth.outputs))
        den = sum(float(torch.sum(b.double() ** 2)) for b in orth.outputs)
        calls32 = []
        t32 = time_calls(orth32, args.warmup, args.steps, torch, calls32)
        F.fp4root_timer_reset()
        F.fp4root_timer_enable(True)
        for _ in range(args.steps):
            orth32()
        torch.cuda.synchronize()
        F.fp4root_timer_enable(False)
        ms3, n3, fl3 = F.fp4root_timer_read(2)
        F.fp4root_timer_reset()
        upd32 = fl3 / (ms3 / 1e3) / 1e12 if ms3 > 0 else 0.0
        fp32acc = {"ms_per_step": round(t32 * 1e3, 3), "per_call_ms": spread(calls32),
                   "matrices_per_s": round(len(shapes) / t32, 2),
                   "tflops_effective": round(flop / t32 / 1e12, 2),
                   "pct_bf16_mfma_peak": round(100 * flop / t32 / 1e12 / BF16_MFMA_PEAK_TFLOPS, 2),
                   "update_product_tflops": round(upd32, 2),
                   "update_product_frac": round(upd32 / F16_MFMA_PEAK_TFLOPS, 4),
                   "speedup_vs_exact": round(t_step / t32, 3),
                   "speedup_vs_bf16": round(bf16["ms_per_step"] / (t32 * 1e3), 3) if bf16 else None,
                   "rel_fro_distance_to_exact": float(np.sqrt(num / den)) if den > 0 else None,
                   "note": "products accumulate in binary32 in MFMA order (tensor-core style); the "
                           "quantisers are unchanged; not the oracle-exact path the line's value measures"}
        del orth32

    momentum = None
    root = None
    qadamw = None
    if not args.no_momentum and not args.probe:
        momentum = momentum_bench(inputs, args.warmup, args.steps, torch, F)
        root = root_step_bench(inputs, args.warmup, args.steps, torch, F)
        qadamw = qadamw_bench(inputs, args.warmup, args.steps, torch, F)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.case, lambda r, c: F.fp4root_default_coeffs(r, c, S), S)
        cpu["vs_gpu"] = round(value / cpu["value"], 1)

    line = {
        "metric": METRIC, "value": round(value, 3), "unit": "matrices/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(t_step * 1e3, 3),
        "per_call_ms": spread(calls),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "nvfp4 operands; f16 MFMA exact block products; f64 accumulation",
        "data": "synthetic",
        "config": {"workload": f"{args.case}: {workloads.CASES[args.case]}", "matrices": len(shapes),
                   "ns_steps": S, "clip_quantile": 0.99, "flags": "clip+hadamard+adaptive46",
                   "algorithmic_tflop_per_step": round(flop / 1e12, 3), "parallelism": "single GPU"},
        "tflops_effective": round(tflops, 2),
        "pct_bf16_mfma_peak": round(100 * tflops / BF16_MFMA_PEAK_TFLOPS, 2),
        "graph_replay": graph_replay,
        "roofline": roofline,
        "bf16_path": bf16,
        "fp32_accumulation": fp32acc,
        "momentum_state_update": momentum,
        "root_optimizer_step": root,
        "qadamw_step": qadamw,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
