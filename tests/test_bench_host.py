"""Host-side checks of bench.py: the single-GPU guard and the rocprofv3 summary that turns
FETCH_SIZE / WRITE_SIZE counters into HBM bytes per launch (scaled by what the same
counters read for a 512 MiB device copy).  No GPU is involved."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _write(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


@pytest.mark.parametrize("leg", ["fwd", "bwd"])
def test_summary_scales_counters_by_the_copy(tmp_path, leg):
    kname = bench.KERNELS[leg][0]
    prof = tmp_path / "prof"
    # three launches of the workload's grid (durations 10, 12, 14 us) and one tiny launch that
    # the summary must leave out
    trace = [["void fla::%s_kernel<false>(x)" % kname, "3468", 1000, 11000],
             ["void fla::%s_kernel<false>(x)" % kname, "3468", 20000, 32000],
             ["void fla::%s_kernel<false>(x)" % kname, "3468", 40000, 54000],
             ["void fla::%s_kernel<false>(x)" % kname, "1", 60000, 60500]]
    _write(str(prof / "trace" / "run_kernel_trace.csv"), ["Kernel_Name", "Grid_Size_X", "Start_Timestamp",
                                                          "End_Timestamp"], trace)
    _write(str(prof / "trace" / "run_kernel_stats.csv"), ["Name", "Calls", "TotalDurationNs", "AverageNs",
                                                          "Percentage"], [[kname, 4, 36500, 9125, 100.0]])
    # counters in KiB per dispatch, split over two rows (two XCD groups) for dispatch 7; the
    # 512 MiB copy reads FETCH_SIZE = 256 MiB (half the bytes) and WRITE_SIZE = 512 MiB
    hdr = ["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"]
    _write(str(prof / "fetch_size" / "run_counter_collection.csv"), hdr,
           [[7, kname, 887808, "FETCH_SIZE", 1000.0], [7, kname, 887808, "FETCH_SIZE", 500.0],
            [9, "__amd_rocclr_copyBuffer", 1 << 20, "FETCH_SIZE", 262144.0]])
    _write(str(prof / "write_size" / "run_counter_collection.csv"), hdr,
           [[7, kname, 887808, "WRITE_SIZE", 2000.0],
            [9, "__amd_rocclr_copyBuffer", 1 << 20, "WRITE_SIZE", 524288.0]])
    # matrix-core pass: MOPS and busy cycles summed over two rows, GRBM_GUI_ACTIVE their max
    _write(str(prof / "mfma" / "run_counter_collection.csv"), hdr,
           [[7, kname, 887808, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 1000.0],
            [7, kname, 887808, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 3000.0],
            [7, kname, 887808, "SQ_VALU_MFMA_BUSY_CYCLES", 204800.0],
            [7, kname, 887808, "SQ_VALU_MFMA_BUSY_CYCLES", 204800.0],
            [7, kname, 887808, "GRBM_GUI_ACTIVE", 1600.0], [7, kname, 887808, "GRBM_GUI_ACTIVE", 2000.0],
            [8, kname, 887808, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 4000.0],
            [8, kname, 887808, "SQ_VALU_MFMA_BUSY_CYCLES", 409600.0], [8, kname, 887808, "GRBM_GUI_ACTIVE", 2000.0],
            [11, kname, 512, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 8.0],   # a one-token launch: left out
            [11, kname, 512, "SQ_VALU_MFMA_BUSY_CYCLES", 4.0], [11, kname, 512, "GRBM_GUI_ACTIVE", 9000.0]])
    out = tmp_path / "out"
    bench.summarize(str(prof), "synthetic", "rocprofv3 ...", leg, out_dir=str(out))
    rec = json.loads((out / os.path.basename(bench.traffic_path(leg, "synthetic"))).read_text())
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    assert rec["bytes_per_launch"] == int(1500 * 1024 * 2.0 + 2000 * 1024)
    assert rec["avg_duration_us"] == pytest.approx(12.0)   # the tiny launch is not averaged in
    assert rec["kernel_hash"] == bench.kernel_hash(leg)
    assert rec["mfma_flop_per_launch"] == pytest.approx(4000 * 512)
    assert rec["mfma_busy"] == pytest.approx(409600 / (2000 / 8 * 1024))
    md = (out / ("%s_synthetic.md" % kname)).read_text()
    assert "3 dispatches" in md and "rocprofv3 ..." in md


def test_roofline_follows_arithmetic_intensity():
    # 120 FLOP/B (full 16 x 16 windows): below the 312.5 FLOP/B ridge, HBM-bound
    r = bench.roofline(48e9, 400e6, 100.0, 123)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["traffic"] == 123
    assert r["achieved"] == pytest.approx(4000.0) and r["frac"] == pytest.approx(0.5)
    # 512 FLOP/B (1024-token windows): matrix-core bound
    r = bench.roofline(512e9, 1e9, 1000.0, None)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s" and r["achieved"] == pytest.approx(512.0)
    assert r["frac"] == pytest.approx(512.0 / 2500.0)


def test_cycle_summary_splits_cold_and_warm_calls_and_scales_counters(tmp_path):
    prof = tmp_path / "prof"
    ch, ca, co = ("void fla::(anonymous namespace)::cycle_scan_chunks<32>(fla::CycleArgs)",
                  "fla::(anonymous namespace)::cycle_scan_carries(fla::CycleArgs)",
                  "void fla::(anonymous namespace)::cycle_scan_outputs<32>(fla::CycleArgs)")
    flush = "void at::native::reduce_kernel<512, 1>(x)"
    # one cold call (after the flush: 30, 4, 40 us) and one warm call (20, 2, 30 us)
    trace = [[flush, "1", 0, 500], [ch, "3072", 1000, 31000], [ca, "96", 31000, 35000], [co, "3072", 35000, 75000],
             [ch, "3072", 80000, 100000], [ca, "96", 100000, 102000], [co, "3072", 102000, 132000]]
    _write(str(prof / "trace" / "run_kernel_trace.csv"), ["Kernel_Name", "Grid_Size_X", "Start_Timestamp",
                                                          "End_Timestamp"], trace)
    hdr = ["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"]
    # FETCH_SIZE of the copy reads half its 512 MiB: every fetch figure is scaled by 2
    _write(str(prof / "fetch_size" / "run_counter_collection.csv"), hdr,
           [[1, ch, 196608, "FETCH_SIZE", 1000.0], [1, ch, 196608, "FETCH_SIZE", 1000.0],
            [9, "__amd_rocclr_copyBuffer", 1 << 20, "FETCH_SIZE", 262144.0]])
    _write(str(prof / "write_size" / "run_counter_collection.csv"), hdr,
           [[3, co, 196608, "WRITE_SIZE", 4000.0],
            [9, "__amd_rocclr_copyBuffer", 1 << 20, "WRITE_SIZE", 524288.0]])
    out = tmp_path / "out"
    bench.summarize_cycle(str(prof), "rocprofv3 ... -- python3 bench.py", str(out))
    text = (out / "cycle_scan_cyclescan_img4096.md").read_text()
    assert "| cycle_scan_chunks<32> | 1 | 30.00 | 1 | 20.00 | %.1f | - |" % (2000 * 1024 * 2 / 1e6) in text
    assert "| cycle_scan_carries | 1 | 4.00 | 1 | 2.00 | - | - |" in text
    assert "| cycle_scan_outputs<32> | 1 | 40.00 | 1 | 30.00 | - | %.1f |" % (4000 * 1024 / 1e6) in text
    assert "| sum (one call) | | 74.00 | | 52.00 | | |" in text
    assert "Kernel source hash: %s" % bench.kernel_hash("cycle") in text


def test_parse_sclk_takes_the_marked_level():
    text = "0: 500Mhz \n1: 1888Mhz *\n2: 2400Mhz \n"
    assert bench.parse_sclk(text) == 1888
    assert bench.parse_sclk("0: 500Mhz \n1: 2400Mhz \n") is None
    assert bench.parse_sclk("") is None


def test_clock_sampler_without_sysfs_gives_none(monkeypatch):
    import glob
    monkeypatch.setattr(glob, "glob", lambda pattern: [])
    s = bench.ClockSampler()
    with s:
        pass
    assert s.median() is None
