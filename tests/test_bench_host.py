"""Host logic of bench.py: the counter summaries behind profiles/ and the
one-GPU contract, on synthetic rocprofv3 CSV rows (no GPU)."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _disp(i, kernel, counters, dur_ns, t0=0):
    return [{"Dispatch_Id": i, "Kernel_Name": kernel, "Counter_Name": c, "Counter_Value": v,
             "Start_Timestamp": t0, "End_Timestamp": t0 + dur_ns} for c, v in counters.items()]


def test_summarize_counters_units(tmp_path):
    # one GEMM dispatch: 1e6 MOPS (x 512 FLOP) in 10 us; 8000 GRBM cycles over
    # 8 XCDs; L2 counters split over two per-channel rows that must be summed
    k = "void fo::(anonymous namespace)::gemm_kernel<0, 6, true>(fo::GemmDesc)"
    m = tmp_path / "m.csv"
    _write(m, _disp(1, k, {"SQ_INSTS_VALU_MFMA_MOPS_BF16": 1e6, "GRBM_GUI_ACTIVE": 8000.0}, 10_000))
    l2 = tmp_path / "l2.csv"
    rows = _disp(7, k, {"TCC_HIT": 300.0, "TCC_MISS": 100.0, "TCC_BUSY": 64000.0, "GRBM_GUI_ACTIVE": 8000.0},
                 10_000)
    rows += _disp(7, k, {"TCC_HIT": 300.0, "TCC_MISS": 100.0}, 10_000)
    rows += _disp(8, "__amd_rocclr_copyBuffer", {"TCC_HIT": 1.0, "TCC_MISS": 1.0}, 5_000)
    _write(l2, rows)
    table = bench.summarize_counters([str(m), str(l2)])
    lines = table.splitlines()
    assert len(lines) == 3, table  # header, rule, the GEMM (the copy is filtered out)
    cells = [c.strip() for c in lines[2].strip("|").split("|")]
    assert cells[0] == "`gemm_kernel<0, 6, true>`"
    assert cells[1] == "1"  # dispatches per pass
    assert float(cells[2]) == pytest.approx(10.0)  # us
    tflops = 1e6 * 512 / 10e-6 / 1e12
    assert float(cells[3]) == pytest.approx(tflops, abs=0.5)
    assert float(cells[4]) == pytest.approx(100 * tflops / bench.PEAK_BF16_TFLOPS, abs=0.05)
    assert float(cells[5]) == pytest.approx(800.0)  # L2 requests, both rows
    assert float(cells[6]) == pytest.approx(0.75)  # hit rate
    assert float(cells[8]) == pytest.approx(64000.0 / 128 / (8000.0 / 8), abs=0.005)  # L2 busy


def test_summarize_pmc_scales_by_calibration_copy(tmp_path):
    kname = "void fo::(anonymous namespace)::gemm_comp_dma_kernel<3, 2, fo::(anonymous namespace)::DmaRKc>(fo::GemmDesc)"
    copy = "__amd_rocclr_copyBuffer"
    f = tmp_path / "f.csv"
    w = tmp_path / "w.csv"
    gib_kib = bench.CALIB_BYTES / 1024
    # FETCH_SIZE reads about half the copied bytes on this GPU (the factor is about 2)
    _write(f, _disp(1, copy, {"FETCH_SIZE": gib_kib / 2 + 10}, 1) + _disp(2, kname, {"FETCH_SIZE": 1000.0}, 1))
    _write(w, _disp(1, copy, {"WRITE_SIZE": gib_kib}, 1) + _disp(2, kname, {"WRITE_SIZE": 500.0}, 1))
    out = bench.summarize_pmc(str(f), str(w))
    fac = gib_kib / (gib_kib / 2 + 10)
    assert out["calibration"]["FETCH_SIZE"]["factor"] == pytest.approx(fac, abs=1e-5)
    assert out["calibration"]["WRITE_SIZE"]["factor"] == pytest.approx(1.0)
    k = out["kernels"]["gemm_comp_dma_kernel<3>"]
    assert k["read_bytes_per_launch"] == pytest.approx(1000 * 1024 * fac, abs=1e-5 * 1000 * 1024 + 1)
    assert k["write_bytes_per_launch"] == 500 * 1024
    assert len(k["source_sha256"]) == 64


def test_committed_traffic_summary_is_well_formed():
    with open(bench.TRAFFIC_FILE) as fh:
        s = json.load(fh)
    for name, (prefix, files) in bench.TRAFFIC_KERNELS.items():
        k = s["kernels"][name]
        assert abs(k["bytes_per_launch"] - k["read_bytes_per_launch"] - k["write_bytes_per_launch"]) <= 1
        for f in files:
            assert os.path.exists(os.path.join(ROOT, f)), f


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_padded_dense_count():
    # the padded-dense transformer step: 1.773 TFLOP at B = 32, L = 128 (every
    # sequence full, no first-token pruning), and it scales linearly in B
    f = bench.padded_bert_flops(32, 128)
    assert f == pytest.approx(1.7734e12, rel=1e-4)
    assert bench.padded_bert_flops(64, 128) == 2 * f
    # one layer's forward matmuls alone: 24 d^2 L per sequence (ffn = 4 d)
    d, L = 768, 128
    one = bench.padded_bert_flops(1, L, layers=1) - 3 * 2 * (d * d + 2 * d) + 2 * L * 3 * d * d
    assert one == 3 * (24 * d * d * L + 4 * d * L * L)
