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
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert set(rec["workloads"]) >= {"qwen3_8b_b64_ctx32k", "qwen3_32b_b128_ctx32k",
                                     "longctx_b16_h96x8_ctx128k"}
    for name, w in rec["workloads"].items():
        t = (w["fetch_size_kib_per_dispatch"] * rec["fetch_scale"]
             + w["write_size_kib_per_dispatch"] * rec["write_scale"]) * 1024
        # the stored KiB figures are rounded to 0.01 KiB
        assert abs(w["traffic_bytes_per_launch"] - t) <= 0.005 * 1024 * 3 + 1, name
        # every page is read at least once: HBM bytes at or above the algorithmic bytes
        assert w["traffic_bytes_per_launch"] >= w["algorithmic_bytes_per_launch"], name


def test_algorithmic_bytes_of_the_record_match_the_workloads():
    import numpy as np
    import workloads as W
    rec = json.load(open(REC))
    for idx in (2, 3, 4):
        cfg = W.config(idx)
        lens = cfg.lens.astype(np.int64)
        pages = int(np.sum((lens + 63) // 64))
        alg = int(lens.sum()) * cfg.Hkv * 96 + pages * 4 + cfg.B * 4
        assert rec["workloads"][cfg.name]["algorithmic_bytes_per_launch"] == alg


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
    w = "qwen3_8b_b64_ctx32k"
    assert bench.split_traffic(w) == rec["workloads"][w]["traffic_bytes_per_launch"]
    assert bench.split_traffic("no_such_workload") is None
    src.write_bytes(src.read_bytes() + b"\n// changed\n")  # the kernel changed since
    assert bench.split_traffic(w) is None
    os.remove(tmp_path / "profiles" / "split_mfma_kernel_traffic.json")  # no record
    assert bench.split_traffic(w) is None
