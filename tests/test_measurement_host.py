"""Host checks of the measurement tooling: the rocprofv3 summary arithmetic
(paper_1809_02839_amd/profiling.py) on synthetic counter files, the
staleness gate of bench.py's `traffic` entry, and bench.py's refusal of
more than one GPU. No GPU is used."""
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_1809_02839_amd import profiling  # noqa: E402

GEMM = "void spx::(anonymous namespace)::gemm_bf16_kernel<3, 4, false, 128, 1>(spx::(anonymous namespace)::KArgs)"
UPD = "spx::(anonymous namespace)::fused_update_partials_kernel(float*, float*)"
NEG = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda>(int, float*)"


def _counter_csv(path, rows):
    os.makedirs(path, exist_ok=True)
    fields = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    with open(os.path.join(path, "p_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(fields, r)))


def test_short_name_strips_namespaces_and_arguments():
    assert profiling.short_name(GEMM) == "gemm_bf16_kernel<3, 4, false, 128, 1>"
    assert profiling.short_name(UPD) == "fused_update_partials_kernel"
    assert profiling.short_name("plain_kernel") == "plain_kernel"


def test_traffic_scales_each_counter_by_the_calibration_copy(tmp_path):
    calib = 256 << 20
    # the calibration copy reads 4 KiB-counts per KiB moved for FETCH (factor 1/4) and 1:1 for WRITE
    fetch = [(1, NEG, "FETCH_SIZE", calib / 1024 * 4, 0, 1),
             (2, GEMM, "FETCH_SIZE", 1000.0, 0, 1), (2, GEMM, "FETCH_SIZE", 500.0, 0, 1),   # summed per dispatch
             (3, GEMM, "FETCH_SIZE", 3000.0, 0, 1)]
    write = [(1, NEG, "WRITE_SIZE", calib / 1024, 0, 1),
             (2, GEMM, "WRITE_SIZE", 100.0, 0, 1), (3, GEMM, "WRITE_SIZE", 300.0, 0, 1)]
    _counter_csv(tmp_path / "f", fetch)
    _counter_csv(tmp_path / "w", write)
    rows, f_read, f_write = profiling.traffic_table(str(tmp_path / "f"), str(tmp_path / "w"), calib, "neg")
    assert f_read == pytest.approx(0.25) and f_write == pytest.approx(1.0)
    (r,) = rows
    assert r["kernel"] == "gemm_bf16_kernel<3, 4, false, 128, 1>" and r["dispatches"] == 2
    assert r["fetch_kib"] == pytest.approx(2250.0) and r["write_kib"] == pytest.approx(200.0)
    assert r["bytes"] == pytest.approx(2250.0 * 1024 * 0.25 + 200.0 * 1024)

    md = tmp_path / "t.md"
    profiling.write_traffic(str(md), rows, f_read, f_write, calib, "t", "cmd")
    digest, table = profiling.read_traffic(str(md))
    assert digest == profiling.source_digest()
    assert table == {"gemm_bf16_kernel<3, 4, false, 128, 1>": pytest.approx(round(r["bytes"]))}


def test_mfma_busy_is_normalised_by_dispatch_duration(tmp_path):
    dur = 50_000   # ns
    busy = 0.3 * dur * 1e-9 * profiling.NOMINAL_CLOCK_HZ * profiling.SIMDS
    _counter_csv(tmp_path / "c", [(7, GEMM, "SQ_VALU_MFMA_BUSY_CYCLES", busy, 1000, 1000 + dur),
                                  (7, GEMM, "GRBM_GUI_ACTIVE", 123.0, 1000, 1000 + dur)])
    means = profiling.counter_means(str(tmp_path / "c"))
    n, cs = means["gemm_bf16_kernel<3, 4, false, 128, 1>"]
    assert n == 1 and cs[profiling.DURATION] == dur
    md = tmp_path / "m.md"
    profiling.write_counters([str(tmp_path / "c")], str(md), "t", "cmd")
    last = [line for line in md.read_text().splitlines() if line.startswith("| gemm")][0]
    assert last.rstrip(" |").split("|")[-1].strip() == "30.0"


def test_kernel_stats_table_is_sorted_by_total_time(tmp_path):
    p = tmp_path / "s.csv"
    with open(p, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs"])
        w.writerow([UPD, 10, 100, 10.0, 10.0, 9, 11])
        w.writerow([GEMM, 10, 900, 90.0, 90.0, 80, 100])
    md = tmp_path / "s.md"
    profiling.write_stats(str(p), str(md), "t", "cmd", "notes")
    body = [line for line in md.read_text().splitlines() if line.startswith("| ") and not line.startswith("| kernel |")]
    assert body[0].startswith("| gemm_bf16_kernel<3, 4, false, 128, 1>") and body[1].startswith("| fused_update")


def test_traffic_entry_is_null_once_the_kernel_sources_change(monkeypatch):
    import bench
    fam = "gemm_bf16_kernel<3, 4, false, 128, 1>"
    real = bench.traffic_per_launch("vgg_conv", fam)
    assert real is None or real > 0
    monkeypatch.setattr(profiling, "source_digest", lambda: "0" * 16)
    assert bench.traffic_per_launch("vgg_conv", fam) is None
    assert bench.traffic_per_launch("no_such_workload", fam) is None


def test_family_roof_takes_the_slower_of_the_two_roofs():
    import bench
    # 1 GFLOP and 100 MB in 0.1 ms: 0.4 us at the MFMA peak, 12.5 us at the HBM peak -> HBM
    b, ach, peak, unit, t = bench.family_roof({"flops_total": 1e9, "bytes_total": 1e8, "ms_total": 0.1}, 2500.0)
    assert (b, unit, peak) == ("hbm", "GB/s", bench.PEAK_HBM_GBPS)
    assert ach == pytest.approx(1000.0) and t == pytest.approx(1e8 / 8e12 * 1e3)
    # 100 GFLOP and 10 MB: 40 us at the MFMA peak, 1.25 us at the HBM peak -> MFMA
    b, ach, peak, unit, t = bench.family_roof({"flops_total": 1e11, "bytes_total": 1e7, "ms_total": 0.1}, 2500.0)
    assert (b, unit) == ("mfma", "TFLOP/s") and ach == pytest.approx(1000.0) and t == pytest.approx(0.04)
    # a pass with no flops is always HBM-bound
    assert bench.family_roof({"flops_total": 0.0, "bytes_total": 8e6, "ms_total": 0.002}, 2500.0)[0] == "hbm"


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_of_a_family_with_two_kernels_is_dispatch_weighted(monkeypatch):
    import bench
    table = {"fused_update_kernel": (3, 60.0), "fused_update_partials_kernel": (1, 100.0),
             "gemm_bf16_kernel<2, 5, true, 64, 1>": (4, 7.0), "gemm_bf16_kernel<2, 5, true, 128, 1>": (2, 9.0)}
    monkeypatch.setattr(profiling, "read_traffic", lambda path, with_dispatches=False: ("d" * 16, table))
    monkeypatch.setattr(profiling, "source_digest", lambda: "d" * 16)
    assert bench.traffic_per_launch("vgg_conv", "fused_update") == 70   # (3 * 60 + 100) / 4
    # a GEMM family is one instantiation
    assert bench.traffic_per_launch("vgg_conv", "gemm_bf16_kernel<2, 5, true, 64, 1>") == 7
