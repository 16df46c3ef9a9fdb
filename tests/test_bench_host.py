"""Host logic of the benchmark's measurement plumbing (no GPU): the kernel
source hash ignores comments but not code, a stored traffic record is used
only while that hash and the kernel-relevant launch options match, byte
counters are scaled by the calibration copy, and trace summaries keep the
requested dispatch window."""
import csv
import json
import os

import pytest

import bench

COUNTER_COLS = ["Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
TRACE_COLS = ["Kernel_Name", "Start_Timestamp", "End_Timestamp"]


def _csv(path, cols, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(cols)
        w.writerows(rows)


@pytest.fixture
def fake_root(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int f(int x) { return x + 1; }  // one\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setitem(bench.KERNEL_SOURCES, "fused_pool_kernel", ["k.hip"])
    (tmp_path / "profiles").mkdir()
    return tmp_path


def test_kernel_hash_ignores_comments_not_code(fake_root):
    h0 = bench.kernel_hash()
    (fake_root / "k.hip").write_text("/* block\n comment */ int f(int x) {\n  return x + 1;   // other words\n}\n")
    assert bench.kernel_hash() == h0
    (fake_root / "k.hip").write_text("int f(int x) { return x + 2; }\n")
    assert bench.kernel_hash() != h0


def test_traffic_record_needs_matching_hash_and_options(fake_root, monkeypatch):
    monkeypatch.setitem(bench.PLAN_OPTS, "wl", {"table_major": 2, "consumer_wgs": 1024})
    rec = {"workload": "wl", "kernel": "fused_pool_kernel", "kernel_hash": bench.kernel_hash(),
           "plan_options": {"table_major": 2}, "hbm_bytes_per_launch": 123}
    (fake_root / "profiles" / "traffic_wl.json").write_text(json.dumps(rec))
    # consumer-only options do not change the pooling kernel
    assert bench.traffic_record("wl")["hbm_bytes_per_launch"] == 123
    monkeypatch.setitem(bench.PLAN_OPTS, "wl", {"table_major": 1})
    assert bench.traffic_record("wl") is None
    monkeypatch.setitem(bench.PLAN_OPTS, "wl", {"table_major": 2})
    (fake_root / "k.hip").write_text("int f(int x) { return x - 1; }\n")
    assert bench.traffic_record("wl") is None
    assert bench.traffic_record("absent") is None


def test_traffic_scales_counters_by_the_calibration_copy(fake_root, tmp_path):
    # FETCH_SIZE reads half the bytes for the 1 GiB copy (factor 2), WRITE_SIZE all of them.
    gib_kib = (1 << 30) / 1024
    fetch = [("fused_pool_kernel", "FETCH_SIZE", v, 0, 1) for v in (1000.0, 1000.0, 1300.0)]  # the median, not the mean
    fetch += [("copy_kernel", "FETCH_SIZE", gib_kib / 2, 0, 1)] * 2
    write = [("fused_pool_kernel", "WRITE_SIZE", v, 0, 1) for v in (50.0, 50.0)]
    write += [("copy_kernel", "WRITE_SIZE", gib_kib, 0, 1)] * 2
    _csv(str(tmp_path / "f" / "vm" / "1_counter_collection.csv"), COUNTER_COLS, fetch)
    _csv(str(tmp_path / "w" / "vm" / "2_counter_collection.csv"), COUNTER_COLS, write)
    r = bench.traffic(str(tmp_path / "f"), str(tmp_path / "w"), "dlrm")
    assert r["fetch_kib_raw"] == 1000.0 and r["write_kib_raw"] == 50.0
    assert r["fetch_scale"] == 2.0 and r["write_scale"] == 1.0
    assert r["fetch_bytes"] == 2000 * 1024 and r["write_bytes"] == 50 * 1024
    assert r["hbm_bytes_per_launch"] == 2050 * 1024
    assert r["kernel_hash"] == bench.kernel_hash()


def test_summarize_keeps_the_dispatch_window(tmp_path):
    # kernel A: five dispatches of 1, 2, 3, 4, 5 us (timestamps in ns), B: one of 10 us
    rows = [("A", 1000 * i, 1000 * i + 1000 * (i + 1)) for i in range(5)] + [("B", 0, 10_000)]
    _csv(str(tmp_path / "t" / "vm" / "9_kernel_trace.csv"), TRACE_COLS, rows)
    out = bench.summarize(str(tmp_path / "t"), "2:4")
    line = next(l for l in out.splitlines() if l.startswith("A "))
    calls, mean, median, mn = line.split()[1:]
    assert (int(calls), float(mean), float(median), float(mn)) == (3, 3.0, 3.0, 2.0)
    assert not any(l.startswith("B ") for l in out.splitlines())  # B has no dispatch 2
    full = bench.summarize(str(tmp_path / "t"))
    assert any(l.startswith("B ") and l.split()[1] == "1" for l in full.splitlines())


def test_roofline_claims_and_fractions():
    """Zipf workloads state their HBM efficiency on distinct-row bytes (with
    the counter bytes beside them); uniform ones on algorithmic bytes."""
    import bench
    r = bench.roofline("large", alg=8_000_000_000, unique_bytes=4_000_000_000, fused_ms=1.0,
                       traffic_bytes=6_000_000_000)
    assert r["claim"] == "frac_unique_rows"
    assert (r["frac"], r["frac_unique_rows"], r["frac_counter"]) == (1.0, 0.5, 0.75)
    assert r["achieved"] == 8000.0 and r["peak"] == 8000.0 and r["traffic"] == 6_000_000_000
    r = bench.roofline("dlrm", alg=4_000_000_000, unique_bytes=3_900_000_000, fused_ms=1.0, traffic_bytes=None)
    assert r["claim"] == "frac" and r["frac"] == 0.5 and r["frac_counter"] is None
    assert bench.HEADLINE == "large" and set(bench.SECONDARY) | {bench.HEADLINE} == {"tiny", "dlrm", "skewed",
                                                                                      "large", "mixed"}


def test_more_than_one_gpu_is_refused_with_a_message():
    """The benchmark runs on one GPU: --gpus N > 1 exits with status 2 and
    says why, before touching a GPU."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.abspath(bench.__file__), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and "--gpus 2" in r.stderr
