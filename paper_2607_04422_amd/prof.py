"""Summaries of rocprofv3 output for the product kernels (text for a profile record).

    python -m paper_2607_04422_amd.prof stats DIR            kernel-time table from a
        ``rocprofv3 --kernel-trace --stats --output-format csv -d DIR`` run
    python -m paper_2607_04422_amd.prof traffic FETCH_DIR WRITE_DIR
        HBM bytes per launch of each kernel from two ``--pmc FETCH_SIZE`` /
        ``--pmc WRITE_SIZE`` runs of ``bench.py --probe``, each counter scaled by
        what it reads for the plain device copy that run ends with
    python -m paper_2607_04422_amd.prof counters DIR [DIR ...]
        SQ/GRBM counters of the product kernels from ``--pmc`` runs of
        ``bench.py --probe`` (each directory one pass), with the derived ratios:
        matrix-core busy fraction, VALU and binary64 instructions per MFMA, LDS
        bank-conflict cycles per LDS instruction, dependency-wait share
    python -m paper_2607_04422_amd.prof lds DIR
        conflict cycles per LDS instruction of each kernel of a
        ``--pmc SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT`` run (the calibration
        program ``probes/lds_banks.hip``)

The traffic record carries the SHA-256 of the NVFP4 product source, so that a
reader (bench.py) can tell whether it still describes the kernel in the tree.
"""
from __future__ import annotations

import collections
import csv
import glob
import hashlib
import os
import re
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
GEMM_SOURCE = os.path.join(HERE, "csrc", "gemm_fp4.hip")
COPY_KERNEL = "copyBuffer"


def source_sha256(path: str = GEMM_SOURCE) -> str:
    with open(path, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()


def short_name(name: str) -> str:
    """`void fp4r::k_gemm_fp4<2, 4, 2, 1, 2>(...)` -> `fp4r::k_gemm_fp4<2, 4, 2, 1, 2>`."""
    name = name.strip().strip('"')
    if name.startswith("void "):
        name = name[5:]
    name = name.replace("(anonymous namespace)::", "")
    depth = 0
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return name[:i]
    return name


def _one(pattern: str) -> str:
    hits = sorted(glob.glob(pattern))
    if not hits:
        raise FileNotFoundError(pattern)
    return hits[0]


def stats(directory: str):
    """[(kernel, calls, total_us, average_us, percent)] from a --stats csv, largest first."""
    path = _one(os.path.join(directory, "*kernel_stats.csv"))
    rows = []
    with open(path) as fh:
        for r in csv.DictReader(fh):
            rows.append((short_name(r["Name"]), int(r["Calls"]), float(r["TotalDurationNs"]) / 1e3,
                         float(r["AverageNs"]) / 1e3, float(r["Percentage"])))
    return sorted(rows, key=lambda t: -t[2])


def per_dispatch(directory: str, counter: str):
    """{kernel: [value per dispatch]} (KiB for FETCH_SIZE / WRITE_SIZE)."""
    path = _one(os.path.join(directory, "*counter_collection.csv"))
    out = collections.OrderedDict()
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != counter:
                continue
            out.setdefault(short_name(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
    return out


def traffic(fetch_dir: str, write_dir: str, copy_bytes: int):
    """Per kernel: mean KiB per dispatch of both counters and calibrated bytes per launch."""
    fe = per_dispatch(fetch_dir, "FETCH_SIZE")
    wr = per_dispatch(write_dir, "WRITE_SIZE")
    copy_f = sum(sum(v) for k, v in fe.items() if COPY_KERNEL in k) * 1024.0
    copy_w = sum(sum(v) for k, v in wr.items() if COPY_KERNEL in k) * 1024.0
    if copy_f <= 0 or copy_w <= 0:
        raise ValueError("no copy-kernel dispatch in the counter runs")
    kf, kw = copy_bytes / copy_f, copy_bytes / copy_w
    rows = []
    for k in fe:
        if k not in wr or COPY_KERNEL in k:
            continue
        f = sum(fe[k]) / len(fe[k])
        w = sum(wr[k]) / len(wr[k])
        rows.append((k, len(fe[k]), f, w, (f * kf + w * kw) * 1024.0))
    return kf, kw, rows


# MI355X: 8 XCDs (GRBM_GUI_ACTIVE is summed over them), 256 CUs x 4 SIMDs
N_XCD = 8
N_SIMD = 1024


def counters(dirs):
    """{kernel: {counter: mean per dispatch}} over every counter of every directory."""
    out = collections.OrderedDict()
    for d in dirs:
        path = _one(os.path.join(d, "*counter_collection.csv"))
        acc = collections.OrderedDict()
        with open(path) as fh:
            for r in csv.DictReader(fh):
                k = short_name(r["Kernel_Name"])
                acc.setdefault(k, collections.defaultdict(list))[r["Counter_Name"]].append(float(r["Counter_Value"]))
        for k, cs in acc.items():
            dst = out.setdefault(k, {})
            for c, v in cs.items():
                dst.setdefault(c, sum(v) / len(v))
    return out


def derived(c: dict) -> dict:
    """Ratios from one kernel's counter means (missing inputs give no entry)."""
    d = {}

    def have(*names):
        return all(n in c and c[n] is not None for n in names)

    if have("SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE") and c["GRBM_GUI_ACTIVE"] > 0:
        d["mfma_busy"] = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (c["GRBM_GUI_ACTIVE"] / N_XCD * N_SIMD)
    if have("SQ_INSTS_VALU", "SQ_INSTS_MFMA") and c["SQ_INSTS_MFMA"] > 0:
        d["valu_per_mfma"] = c["SQ_INSTS_VALU"] / c["SQ_INSTS_MFMA"]
    if have("SQ_INSTS_VALU_ADD_F64", "SQ_INSTS_MFMA") and c["SQ_INSTS_MFMA"] > 0:
        d["add_f64_per_mfma"] = c["SQ_INSTS_VALU_ADD_F64"] / c["SQ_INSTS_MFMA"]
    if have("SQ_INSTS_VALU_CVT", "SQ_INSTS_MFMA") and c["SQ_INSTS_MFMA"] > 0:
        d["cvt_per_mfma"] = c["SQ_INSTS_VALU_CVT"] / c["SQ_INSTS_MFMA"]
    if have("SQ_INSTS_LDS", "SQ_INSTS_MFMA") and c["SQ_INSTS_MFMA"] > 0:
        d["lds_per_mfma"] = c["SQ_INSTS_LDS"] / c["SQ_INSTS_MFMA"]
    if have("SQ_LDS_BANK_CONFLICT", "SQ_INSTS_LDS") and c["SQ_INSTS_LDS"] > 0:
        d["lds_conflict_per_inst"] = c["SQ_LDS_BANK_CONFLICT"] / c["SQ_INSTS_LDS"]
    if have("SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES") and c["SQ_WAVE_CYCLES"] > 0:
        d["wait_share"] = c["SQ_WAIT_INST_ANY"] / c["SQ_WAVE_CYCLES"]
    if have("SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES") and c["SQ_VALU_MFMA_BUSY_CYCLES"] > 0:
        d["valu_coexec_share_of_mfma"] = c["SQ_VALU_MFMA_COEXEC_CYCLES"] / c["SQ_VALU_MFMA_BUSY_CYCLES"]
    return d


DERIVED_COLS = ("mfma_busy", "valu_per_mfma", "add_f64_per_mfma", "cvt_per_mfma", "lds_per_mfma",
                "lds_conflict_per_inst", "wait_share", "valu_coexec_share_of_mfma")


def _counters_md(dirs) -> str:
    cs = counters(dirs)
    keep = [k for k in cs if "k_gemm" in k or "k_encode" in k]
    lines = ["| kernel | " + " | ".join(DERIVED_COLS) + " |", "|---" * (len(DERIVED_COLS) + 1) + "|"]
    for k in keep:
        d = derived(cs[k])
        lines.append(f"| `{k}` | " + " | ".join(f"{d[c]:.3f}" if c in d else "" for c in DERIVED_COLS) + " |")
    lines += ["", "Counter means per dispatch:", ""]
    names = sorted({n for k in keep for n in cs[k]})
    lines.append("| counter | " + " | ".join(f"`{k}`" for k in keep) + " |")
    lines.append("|---" * (len(keep) + 1) + "|")
    for n in names:
        lines.append(f"| {n} | " + " | ".join(f"{cs[k][n]:.4g}" if n in cs[k] else "" for k in keep) + " |")
    lines += ["", f"gemm_fp4_source_sha256: {source_sha256()}"]
    return "\n".join(lines)


def _lds_md(directory: str) -> str:
    cs = counters([directory])
    lines = ["| kernel | SQ_INSTS_LDS | SQ_LDS_BANK_CONFLICT | conflict cycles per LDS instruction |",
             "|---|---|---|---|"]
    for k, c in cs.items():
        n, b = c.get("SQ_INSTS_LDS", 0.0), c.get("SQ_LDS_BANK_CONFLICT", 0.0)
        lines.append(f"| `{k}` | {n:.6g} | {b:.6g} | {b / n if n else 0.0:.2f} |")
    return "\n".join(lines)


def _stats_md(directory: str) -> str:
    lines = ["| kernel | calls | total us | average us | % |", "|---|---|---|---|---|"]
    for k, n, tot, avg, pct in stats(directory):
        if len(k) > 100:   # library kernels (hipBLASLt Cijk_*, torch) named by their first characters
            k = k[:60] + "..."
        lines.append(f"| `{k}` | {n} | {tot:.1f} | {avg:.1f} | {pct:.2f} |")
    return "\n".join(lines)


def _traffic_md(fetch_dir: str, write_dir: str, copy_bytes: int) -> str:
    kf, kw, rows = traffic(fetch_dir, write_dir, copy_bytes)
    lines = [f"calibration: plain copy of {copy_bytes} bytes; FETCH_SIZE factor {kf:.4f}, "
             f"WRITE_SIZE factor {kw:.4f}", "",
             "| kernel | dispatches | FETCH_SIZE KiB/dispatch | WRITE_SIZE KiB/dispatch | HBM bytes/launch (calibrated) |",
             "|---|---|---|---|---|"]
    for k, n, f, w, b in rows:
        lines.append(f"| `{k}` | {n} | {f:.1f} | {w:.1f} | {b:.4g} |")
    # the update product's tile configurations together (bench.py's figure is per launch
    # over every update launch)
    upd = [r for r in rows if r[0].startswith("fp4r::k_gemm_fp4<2")]
    if upd:
        n = sum(r[1] for r in upd)
        mean = sum(r[1] * r[4] for r in upd) / n
        lines += ["", f"update_product_traffic_bytes_per_launch: {mean:.6g}",
                  f"gemm_fp4_source_sha256: {source_sha256()}"]
    return "\n".join(lines)


def read_update_traffic(path: str):
    """Bytes per launch of the update product from a traffic record, or None when the
    record is missing or was taken from a different version of the product source."""
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"update_product_traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    h = re.search(r"gemm_fp4_source_sha256:\s*([0-9a-f]{64})", text)
    if not m or not h or h.group(1) != source_sha256():
        return None
    return float(m.group(1))


def main(argv):
    if len(argv) >= 2 and argv[0] == "stats":
        print(_stats_md(argv[1]))
    elif len(argv) >= 2 and argv[0] == "counters":
        print(_counters_md(argv[1:]))
    elif len(argv) >= 2 and argv[0] == "lds":
        print(_lds_md(argv[1]))
    elif len(argv) >= 3 and argv[0] == "traffic":
        copy_bytes = int(argv[3]) if len(argv) > 3 else 256 << 20
        print(_traffic_md(argv[1], argv[2], copy_bytes))
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
