"""Host logic of bench.py (no GPU): the one-GPU guard, the source hash that
keys the traffic record, the rocprofv3 counter summary, and the oracle
baseline's fields."""
from __future__ import annotations

import csv
import json
import os
import subprocess
import sys

import bench
from paper_2609_26368_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_source_hash_ignores_comments_and_spacing(tmp_path, monkeypatch):
    for p in bench.KERNEL_SOURCES:
        (tmp_path / p).parent.mkdir(parents=True, exist_ok=True)
        (tmp_path / p).write_text("int f(int x) {\n  return x + 1;  // one more\n}\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_source_hash()
    first = tmp_path / bench.KERNEL_SOURCES[0]
    first.write_text("/* a block\n comment */ int f(int x)   {\n\n  return x + 1;  // changed text\n}\n")
    assert bench.kernel_source_hash() == h0
    first.write_text("int f(int x) {\n  return x + 2;\n}\n")
    assert bench.kernel_source_hash() != h0


def _counter_dir(path, rows):
    """rows: (dispatch id, kernel name, counter, value per instance, instances)"""
    path.mkdir(parents=True)
    with open(path / "run_counter_collection.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for d, name, counter, value, inst in rows:
            for _ in range(inst):
                w.writerow([d, name, counter, value])


def test_traffic_summary_calibrates_by_the_copy(tmp_path, monkeypatch):
    fa = "void hs2::k_fa_ring<4, 4, 32, 2, 2, false, 128>(hs2::FaArgs)"
    other = "hs2::k_sel_filter(hs2::SelArgs)"
    copy = "__amd_rocclr_copyBuffer"
    # the copy of COPY_BYTES reads back half its bytes (in KiB) through FETCH_SIZE, all through WRITE_SIZE
    kib = bench.COPY_BYTES / 1024
    _counter_dir(tmp_path / "cf", [(1, copy, "FETCH_SIZE", kib / 2 / 4, 4), (2, "small", "FETCH_SIZE", 1.0, 1)])
    _counter_dir(tmp_path / "cw", [(1, copy, "WRITE_SIZE", kib / 8, 8)])
    # two dispatches of the FA kernel (summed over counter instances, averaged over dispatches)
    _counter_dir(tmp_path / "f", [(1, fa, "FETCH_SIZE", 100.0, 4), (2, fa, "FETCH_SIZE", 300.0, 4),
                                  (3, other, "FETCH_SIZE", 7.0, 1)])
    _counter_dir(tmp_path / "w", [(1, fa, "WRITE_SIZE", 10.0, 2), (2, fa, "WRITE_SIZE", 10.0, 2)])
    out = tmp_path / "traffic_{workload}.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out))
    bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"), str(tmp_path / "cw"), "wl")
    rec = json.loads((tmp_path / "traffic_wl.json").read_text())
    assert rec["copy_kernel"] == copy
    assert abs(rec["fetch_factor"] - 2.0) < 1e-12 and abs(rec["write_factor"] - 1.0) < 1e-12
    assert rec["kernel"].startswith("void hs2::k_fa_ring")
    assert rec["fetch_bytes_per_launch"] == (4 * 100.0 + 4 * 300.0) / 2 * 1024 * 2.0
    assert rec["write_bytes_per_launch"] == 20.0 * 1024
    assert rec["bytes_per_launch"] == rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]
    assert rec["source_hash"] == bench.kernel_source_hash()


def test_cpu_baseline_fields():
    w = W.Workload("tiny", 1, 300, 2, 8, 2, 128, 32, 16, 1)
    inp = W.make_inputs(w, seed=3)
    r = bench.cpu_baseline(w, inp, 0.4)
    assert set(r) == {"value", "unit", "cores", "kind", "sample", "cpu_model", "cpu_count", "single_thread"}
    assert r["kind"] == "oracle" and r["unit"] == "tokens/s"
    assert r["value"] > 0 and r["cores"] >= 1
    assert r["cpu_count"] == os.cpu_count()
    assert isinstance(r["cpu_model"], str)
    one = r["single_thread"]
    assert one["cores"] == 1 and one["unit"] == "tokens/s" and one["value"] > 0


def test_cpu_model_is_the_lscpu_model_name():
    m = bench.cpu_model()
    if os.path.exists("/proc/cpuinfo") and "model name" in open("/proc/cpuinfo").read():
        assert m and "\n" not in m


def test_kv_copies_rotation_rule():
    gib = 1 << 30
    assert bench.kv_copies_for(int(1.07e9), "rotate", 0) == 4          # 4 copies of the 128K chunk cache
    assert bench.kv_copies_for(4 * 1024 * 1024, "rotate", 0) == 512    # small caches: at least 2 GiB in all
    assert bench.kv_copies_for(1024, "rotate", 0) == 1024              # capped
    assert bench.kv_copies_for(4 * gib, "rotate", 0) == 4
    assert bench.kv_copies_for(int(1.07e9), "warm", 0) == 1
    assert bench.kv_copies_for(int(1.07e9), "flush", 0) == 1
    assert bench.kv_copies_for(int(1.07e9), "rotate", 7) == 7
