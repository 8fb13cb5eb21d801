"""The benchmark's host-side arithmetic without a GPU: the step statistic,
the split of GEMM durations by what ran beside them, and the one-GPU guard."""
import csv
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_step_statistic_drops_warmup_and_the_slowest_five_percent(bench):
    """Sec. VII-B's per-iteration statistic: 10 warm-up steps out, then the
    slowest 5% of the rest (2 of 40), then the mean."""
    steps = [1000.0] * 10 + [100.0 + k for k in range(38)] + [500.0, 900.0]
    assert bench.trimmed_mean(steps) == pytest.approx(sum(100.0 + k for k in range(38)) / 38)
    # fewer than 20 kept steps drop none; a list no longer than the warm-up is averaged whole
    assert bench.trimmed_mean([5.0] * 10 + [1.0, 3.0]) == pytest.approx(2.0)
    assert bench.trimmed_mean([4.0, 6.0]) == pytest.approx(5.0)


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_gemm_split_by_what_ran_beside(bench, tmp_path):
    """GEMMs overlapping a pack launch, a sums launch or a device-to-host copy
    are counted apart from those that ran alone, with the time each group adds
    over the median of the lone ones."""
    us = 1000  # the traces are in ns
    gemms = [(k * 600 * us, k * 600 * us + 500 * us) for k in range(100)]
    gemms = [(a, b + (50 * us if 20 <= k < 25 else 0) + (5 * us if 40 <= k < 60 else 0) + (20 * us if 70 <= k < 72 else 0))
             for k, (a, b) in enumerate(gemms)]
    rows = [(a, b, "Cijk_Alik_Bljk_BBS_gemm") for a, b in gemms]
    rows.append((20 * 600 * us, 25 * 600 * us, "sums_run_kernel(ckpt::Args)"))
    rows.append((70 * 600 * us, 72 * 600 * us, "void ckpt::tile_kernel<0, false, 256, 2, true, true>(ckpt::Args)"))
    _write(tmp_path / "x_kernel_trace.csv", ["Start_Timestamp", "End_Timestamp", "Kernel_Name"], rows)
    _write(tmp_path / "x_memory_copy_trace.csv", ["Start_Timestamp", "End_Timestamp", "Direction"],
           [(40 * 600 * us, 60 * 600 * us - 1, "MEMORY_COPY_DEVICE_TO_HOST"),
            (80 * 600 * us, 90 * 600 * us, "MEMORY_COPY_HOST_TO_DEVICE")])
    table = bench.gemm_inflation(str(tmp_path), "test")
    lines = {ln.split("|")[1].strip(): [c.strip() for c in ln.split("|")[2:-1]]
             for ln in table.splitlines() if ln.startswith("| beside") or ln.startswith("| alone")}
    assert "100 GEMM dispatches, 1 pack launches, 1 sums launches, 1 device-to-host copies" in table
    assert lines["beside_pack"][:2] == ["2", "520.0"] and lines["beside_pack"][3] == "+4.00%"
    assert lines["beside_sums"][:2] == ["5", "550.0"] and lines["beside_sums"][4] == "0.2"
    assert lines["beside_d2h"][:2] == ["20", "505.0"] and lines["beside_d2h"][3] == "+1.00%"
    assert lines["alone"][:2] == ["73", "500.0"]  # the host-to-device copy does not count


def test_d2h_per_snapshot_from_a_copy_trace(bench, tmp_path):
    """Each timed snapshot's D2H rate from the memory-copy trace groups one
    copy per chunk group (here four 256 MiB groups per snapshot, packed in one
    launch, so groups and launches differ), after the warm-up snapshots."""
    ms = 1_000_000  # ns
    rows = []
    for k in range(5):  # 2 warm-up + 3 timed snapshots, 100 ms apart
        t = k * 100 * ms
        for g in range(4):  # four 5 ms copies back to back, then the 8-byte counter copies (short)
            rows.append((t + g * 5 * ms, t + (g + 1) * 5 * ms, "MEMORY_COPY_DEVICE_TO_HOST"))
            rows.append((t + (g + 1) * 5 * ms, t + (g + 1) * 5 * ms + 2000, "MEMORY_COPY_DEVICE_TO_HOST"))
    _write(tmp_path / "x_memory_copy_trace.csv", ["Start_Timestamp", "End_Timestamp", "Direction"], rows)
    b = {"steps": 3, "warmup": 2, "roofline": {"launches": 3}, "config": {"image_bytes": 20 * ms,
                                                                        "groups_per_snapshot": 4}}
    rates, med = bench.timed_d2h_from_trace(str(tmp_path), b)
    assert rates == [pytest.approx(1.0)] * 3 and med == pytest.approx(1.0)  # 20e6 bytes in 20 ms = 1 GB/s


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 2 and "one GPU" in (r.stdout + r.stderr)
