"""Host-side checks of bench.py's helpers (no GPU): the counter summary's
calibration arithmetic, the traffic file's source-hash and configuration
gate, the refusal of more than one GPU, and the CPU-baseline leg."""

import csv
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _counter_csv(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for disp, name, val in rows:
            w.writerow({"Dispatch_Id": disp, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": val})


def test_pmc_summary_scales_by_the_calibration_copy(tmp_path):
    calib_kib = bench.CALIB_BYTES / 1024
    copy = "void at::native::vectorized_elementwise_kernel<4, MulFunctor<float> >"
    # the copy reads half its bytes on FETCH_SIZE (scale 2) and all on WRITE_SIZE (scale 1);
    # two dispatches of one kernel, each counted in two partial rows that must be summed
    _counter_csv(tmp_path / "f", "FETCH_SIZE", [(1, "vbq_mv_kernel<1>", 100.0), (1, "vbq_mv_kernel<1>", 50.0),
                                                 (2, "vbq_mv_pair_kernel<8>", 250.0), (3, copy, calib_kib / 2),
                                                 (4, "other_kernel", 1e9)])
    _counter_csv(tmp_path / "w", "WRITE_SIZE", [(1, "vbq_mv_kernel<1>", 4.0), (2, "vbq_mv_pair_kernel<8>", 6.0),
                                                 (3, copy, calib_kib), (4, "other_kernel", 7.0)])
    s = bench.pmc_summary(str(tmp_path / "f"), str(tmp_path / "w"))
    assert s["launches"] == 2
    assert s["fetch_scale"] == pytest.approx(2.0) and s["write_scale"] == pytest.approx(1.0)
    assert s["fetch_bytes_per_launch"] == pytest.approx(2.0 * 200.0 * 1024)
    assert s["write_bytes_per_launch"] == pytest.approx(5.0 * 1024)
    assert s["hbm_bytes_per_launch"] == round(2.0 * 200.0 * 1024 + 5.0 * 1024)
    assert s["per_kernel"] == {"vbq_mv_kernel<1>": {"launches": 1, "hbm_bytes_per_launch": round(2.0 * 150 * 1024 + 4 * 1024)},
                               "vbq_mv_pair_kernel<8>": {"launches": 1,
                                                         "hbm_bytes_per_launch": round(2.0 * 250 * 1024 + 6 * 1024)}}
    q = bench.pmc_summary(str(tmp_path / "f"), str(tmp_path / "w"), kernel="other_kernel", sources=bench.QAT_SOURCES)
    assert q["launches"] == 1 and q["kernel_source_sha256"] == bench.kernel_source_hash(bench.QAT_SOURCES)


def test_traffic_file_is_gated_by_hash_and_config(tmp_path, monkeypatch):
    summ = {"launches": 3, "fetch_kib_per_launch_raw": 1.0, "write_kib_per_launch_raw": 1.0, "copy_fetch_kib": 1.0,
            "copy_write_kib": 1.0, "fetch_scale": 2.0, "write_scale": 1.0, "fetch_bytes_per_launch": 10.0,
            "write_bytes_per_launch": 5.0, "hbm_bytes_per_launch": 15, "kernel_source_sha256": bench.kernel_source_hash()}
    path = str(tmp_path / "traffic.md")
    summ["per_kernel"] = {"vbq_mv_pair_kernel<8,1>": {"launches": 2, "hbm_bytes_per_launch": 20}}
    bench.write_traffic_file(path, summ)
    monkeypatch.setattr(bench, "TRAFFIC_FILE", path)
    assert bench.measured_traffic(bench.TRAFFIC_CONFIG) == 15
    assert bench.measured_traffic_per_kernel(bench.TRAFFIC_CONFIG) == {"vbq_mv_pair_kernel<8,1>": 20}
    assert bench.measured_traffic("workload 4, M 1, widths mixed") is None  # another configuration
    summ["kernel_source_sha256"] = "0" * 64                                 # another kernel source
    bench.write_traffic_file(path, summ)
    assert bench.measured_traffic(bench.TRAFFIC_CONFIG) is None
    qpath = str(tmp_path / "qat.md")
    summ["kernel_source_sha256"] = bench.kernel_source_hash(bench.QAT_SOURCES)
    bench.write_qat_traffic_file(qpath, summ)
    assert bench.measured_traffic(bench.QAT_TRAFFIC_CONFIG, qpath, bench.QAT_TRAFFIC_CONFIG, bench.QAT_SOURCES) == 15
    assert bench.measured_traffic(bench.QAT_TRAFFIC_CONFIG, qpath, bench.QAT_TRAFFIC_CONFIG) is None


@pytest.mark.parametrize("extra", [[], ["--qat"]])
def test_more_than_one_gpu_is_refused(extra):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", *extra],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_qat_cpu_baseline_leg():
    from paper_2607_02893_amd import synth
    n = 3000
    W, logits, noise = synth.selection_inputs(n, part=5)
    out = bench.qat_cpu_baseline(W, logits, noise, 0.5, n, budget_s=0.5)
    assert out["kind"] == "oracle" and out["unit"] == "ms/step" and out["value"] > 0
    assert out["cores"] >= 1 and str(n) in out["sample"]
    assert bench.QAT_BYTES_PER_GROUP == 256 + 256 + 16 + 16 + 16 + 1
    assert np.isfinite(out["value"])


def test_profiler_kernel_names_match_the_library_names():
    """rocprofv3 prints template arguments with spaces and the default argument;
    the per-kernel traffic is keyed by vbq_kernel_name's form."""
    assert bench.canonical_kernel("void (anonymous namespace)::vbq_mv_kernel<1, 16, -1>(unsigned short const*, "
                                  "unsigned char const*)") == "vbq_mv_kernel<1,16>"
    assert bench.canonical_kernel("(anonymous namespace)::vbq_mv_kernel<1, 8, 2>(x)") == "vbq_mv_kernel<1,8,2>"
    assert bench.canonical_kernel("vbq_mv_pair_kernel<16, 1>(a, b)") == "vbq_mv_pair_kernel<16,1>"
