"""Host-side checks of bench.py's contract (no GPU): the one-GPU refusal, and
the counter record it reports only for the kernel sources it was measured on."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_traffic_record_matches_the_sources():
    # Every committed record was taken on the current sources of its kernel.
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    for key, r in rec.items():
        cfg, dt = key.split(":")
        got = bench.measured_traffic(cfg, dt, 2)
        assert got == r["fetch_bytes"] + r["write_bytes"], key
        # counter traffic is at least the compulsory bytes
        assert got >= 0.99 * r["algorithmic_bytes"], key


def test_traffic_record_dropped_when_a_source_changes(tmp_path, monkeypatch):
    # A copy of the tree in which one source of the c2 kernel differs by a byte.
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    r = rec["c2:f32"]
    os.makedirs(tmp_path / "profiles")
    for f in r["source_files"]:
        dst = tmp_path / f
        os.makedirs(dst.parent, exist_ok=True)
        data = open(os.path.join(ROOT, f), "rb").read()
        dst.write_bytes(data)
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps({"c2:f32": r}))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("c2", "f32", 2) == r["fetch_bytes"] + r["write_bytes"]
    first = tmp_path / r["source_files"][0]
    first.write_bytes(first.read_bytes() + b"\n")
    assert bench.measured_traffic("c2", "f32", 2) is None
    # and never for a kernel family the record does not describe
    assert bench.measured_traffic("c2", "f32", 1) is None


@pytest.mark.parametrize("cfg", ["c2", "c3", "c4", "c5"])
def test_no_record_for_unknown_workloads(cfg):
    assert bench.measured_traffic(cfg + "x", "f32", 2) is None
