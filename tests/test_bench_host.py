"""Host-side checks of bench.py (no GPU): the one-GPU rule, the metric's
workload, the algorithmic byte count, and that a counter record taken for
another kernel source is not reported as the current kernel's traffic."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads as wl  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_metric_workload_shape():
    """6 cameras x 118 depth bins x 32x88 features, C = 80 fp32, 360x360 BEV."""
    w = wl.make("nuscenes", seed=0)
    assert w.P.shape == (1, 6, 118, 32, 88) and w.P.dtype == np.float32
    assert w.F.shape == (1, 6, 32, 88, 80) and w.F.dtype == np.float32
    assert w.rig.n_cells == 360 * 360
    # P, F read once and the fp32 map written once
    assert bench.algorithmic_bytes(w) == 4 * (6 * 118 * 32 * 88 + 6 * 32 * 88 * 80 + 360 * 360 * 80)


def test_traffic_only_for_the_current_kernel(tmp_path, monkeypatch):
    rec = {"kernel_sha256_16": bench.kernel_hash(),
           "workloads": {"nuscenes": {"hbm_bytes_per_launch": 123}}}
    path = tmp_path / "traffic.json"
    path.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    assert bench.load_traffic("nuscenes") == 123
    assert bench.load_traffic("highres") is None
    rec["kernel_sha256_16"] = "0" * 16
    path.write_text(json.dumps(rec))
    assert bench.load_traffic("nuscenes") is None


def test_committed_traffic_record_is_well_formed():
    with open(bench.TRAFFIC_FILE) as fh:
        rec = json.load(fh)
    assert len(rec["kernel_sha256_16"]) == 16
    entry = rec["workloads"]["nuscenes"]
    assert entry["hbm_bytes_per_launch"] == entry["read_bytes"] + entry["write_bytes"]
    assert os.path.exists(os.path.join(ROOT, entry["summary"]))


def test_traffic_hash_covers_every_forward_source(tmp_path):
    """An edit to any file that shapes the forward's traffic (kernels, device
    helpers, constants, plan layout, build flags) changes the hash, so a
    stale counter record is not reported as current."""
    names = {os.path.basename(p) for p in bench.FORWARD_SOURCES}
    assert {"forward.hip", "device.h", "internal.h", "plan.hip", "build.py"} <= names
    copies = []
    for p in bench.FORWARD_SOURCES:
        q = tmp_path / os.path.basename(p)
        q.write_bytes(open(p, "rb").read())
        copies.append(str(q))
    base = bench.kernel_hash(copies)
    for q in copies:
        orig = open(q, "rb").read()
        open(q, "wb").write(orig + b" ")
        assert bench.kernel_hash(copies) != base, q
        open(q, "wb").write(orig)
    assert bench.kernel_hash(copies) == base
