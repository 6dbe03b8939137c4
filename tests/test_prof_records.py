"""Host logic of the profile records (paper_2607_04422_amd/prof.py) on synthetic
rocprofv3 CSV files: kernel-name shortening, the kernel-time table order, the
traffic calibration against the plain copy, the update product's bytes per launch
over its tile forms, and the source-hash guard bench.py relies on."""
import csv
import os

import pytest

from paper_2607_04422_amd import prof


def _write(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(header)
        w.writerows(rows)


def _counters(d, counter, per_kernel):
    rows = []
    for name, vals in per_kernel.items():
        for v in vals:
            rows.append([name, counter, v])
    _write(os.path.join(d, "run_counter_collection.csv"), ["Kernel_Name", "Counter_Name", "Counter_Value"], rows)


UPD_W = "void fp4r::k_gemm_fp4<2, 2, 2, 2, 2, 2>(fp4r::GemmFp4Args, int, int, long, fp4r::GemmFin)"
UPD_N = "void fp4r::k_gemm_fp4<2, 4, 2, 1, 2, 4>(fp4r::GemmFp4Args, int, int, long, fp4r::GemmFin)"
COPY = "__amd_rocclr_copyBuffer"


def test_short_name_keeps_template_arguments():
    assert prof.short_name(UPD_W) == "fp4r::k_gemm_fp4<2, 2, 2, 2, 2, 2>"
    assert prof.short_name('"void fp4r::k_encode_x2(float const*)"') == "fp4r::k_encode_x2"


def test_stats_sorted_by_total_time(tmp_path):
    d = str(tmp_path / "kt")
    _write(os.path.join(d, "run_kernel_stats.csv"),
           ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage"],
           [["void a(int)", 2, 2000, 1000, 20.0], ["void b(int)", 1, 8000, 8000, 80.0]])
    rows = prof.stats(d)
    assert [r[0] for r in rows] == ["b", "a"]
    assert rows[0][2] == pytest.approx(8.0) and rows[1][3] == pytest.approx(1.0)


def test_traffic_calibration_and_update_mean_over_tile_forms(tmp_path, monkeypatch):
    fd, wd = str(tmp_path / "f"), str(tmp_path / "w")
    copy_bytes = 1 << 20
    # the counters read half of the copy's bytes for FETCH_SIZE and all of them for WRITE_SIZE
    _counters(fd, "FETCH_SIZE", {COPY: [copy_bytes / 2 / 1024], UPD_W: [100.0, 100.0, 100.0], UPD_N: [40.0]})
    _counters(wd, "WRITE_SIZE", {COPY: [copy_bytes / 1024], UPD_W: [10.0, 10.0, 10.0], UPD_N: [4.0]})
    kf, kw, rows = prof.traffic(fd, wd, copy_bytes)
    assert kf == pytest.approx(2.0) and kw == pytest.approx(1.0)
    got = {r[0]: r for r in rows}
    assert got["fp4r::k_gemm_fp4<2, 2, 2, 2, 2, 2>"][4] == pytest.approx((100 * 2 + 10) * 1024)
    text = prof._traffic_md(fd, wd, copy_bytes)
    mean = (3 * (100 * 2 + 10) + (40 * 2 + 4)) * 1024 / 4
    line = [ln for ln in text.splitlines() if ln.startswith("update_product_traffic_bytes_per_launch:")][0]
    assert float(line.split(":")[1]) == pytest.approx(mean, rel=1e-5)
    # the record is read back only while the product source is unchanged
    rec = tmp_path / "record.md"
    rec.write_text(text + "\n")
    assert prof.read_update_traffic(str(rec)) == pytest.approx(mean, rel=1e-5)
    monkeypatch.setattr(prof, "source_sha256", lambda path=prof.GEMM_SOURCE: "0" * 64)
    assert prof.read_update_traffic(str(rec)) is None


def test_counter_ratios(tmp_path):
    d = str(tmp_path / "sq")
    rows = []
    for c, v in (("SQ_INSTS_VALU", 170.0), ("SQ_INSTS_MFMA", 10.0), ("SQ_VALU_MFMA_BUSY_CYCLES", 320.0),
                 ("GRBM_GUI_ACTIVE", 8 * 1000.0), ("SQ_INSTS_LDS", 16.0), ("SQ_LDS_BANK_CONFLICT", 0.0)):
        rows.append([UPD_W, c, v])
    _write(os.path.join(d, "run_counter_collection.csv"), ["Kernel_Name", "Counter_Name", "Counter_Value"], rows)
    c = prof.counters([d])["fp4r::k_gemm_fp4<2, 2, 2, 2, 2, 2>"]
    r = prof.derived(c)
    assert r["valu_per_mfma"] == pytest.approx(17.0)
    assert r["mfma_busy"] == pytest.approx(320.0 / (1000.0 * 1024))
    assert r["lds_per_mfma"] == pytest.approx(1.6)
    assert r["lds_conflict_per_inst"] == 0.0
