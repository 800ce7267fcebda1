"""Host-side checks of bench.py's contract (CPU): a request for more than one GPU
is refused with a message before anything touches a device, and the HBM-traffic
figure of the roofline is reported only for the split-kernel source that its
rocprofv3 counters were taken on."""
import json
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

REC = os.path.join(ROOT, "profiles", "split_mfma_kernel_traffic.json")


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_exits_with_a_message(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "one GPU" in r.stderr
    assert r.stdout == ""  # no JSON line


def test_traffic_record_is_the_scaled_counter_sum():
    rec = json.load(open(REC))
    t = (rec["fetch_size_kib_per_dispatch"] * rec["fetch_scale"]
         + rec["write_size_kib_per_dispatch"] * rec["write_scale"]) * 1024
    # the stored KiB figures are rounded to 0.01 KiB
    assert abs(rec["traffic_bytes_per_launch"] - t) <= 0.005 * 1024 * (rec["fetch_scale"] + rec["write_scale"]) + 1
    # the calibration read 1 GiB through FETCH_SIZE at the stated scale
    assert rec["fetch_scale"] in (1.0, 2.0) and rec["write_scale"] == 1.0
    # every page is read at least once: HBM bytes at or above the algorithmic bytes
    # of the bench workload's split launch (1.2206e9 B of INT2 pages)
    assert rec["traffic_bytes_per_launch"] >= 1.22e9


def test_traffic_only_for_the_source_it_was_measured_on(tmp_path, monkeypatch):
    rec = json.load(open(REC))
    os.makedirs(tmp_path / "profiles")
    src = tmp_path / rec["source"]
    os.makedirs(src.parent)
    shutil.copy(os.path.join(ROOT, rec["source"]), src)
    import hashlib
    rec["source_sha256"] = hashlib.sha256(src.read_bytes()).hexdigest()
    (tmp_path / "profiles" / "split_mfma_kernel_traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.split_traffic() == rec["traffic_bytes_per_launch"]
    src.write_bytes(src.read_bytes() + b"\n// changed\n")  # the kernel changed since
    assert bench.split_traffic() is None
    os.remove(tmp_path / "profiles" / "split_mfma_kernel_traffic.json")  # no record
    assert bench.split_traffic() is None
