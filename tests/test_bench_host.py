"""Host-side checks of bench.py's contract (no GPU): the one-GPU refusal, and
the counter record it reports only for the kernel sources it was measured on."""
import hashlib
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


def test_traffic_records_are_well_formed():
    # Every committed record names its kernel and sources; bench.py reports it
    # only while those sources are the ones it was measured on.
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    for key, r in rec.items():
        cfg, dt = key.split(":")
        for f in ("kernel", "source_files", "source_sha256", "fetch_bytes", "write_bytes",
                  "algorithmic_bytes", "commands"):
            assert f in r, (key, f)
        # counter traffic is at least the compulsory bytes
        assert r["fetch_bytes"] + r["write_bytes"] >= 0.99 * r["algorithmic_bytes"], key
        got = bench.measured_traffic(cfg, dt, 2)
        assert got in (None, r["fetch_bytes"] + r["write_bytes"]), key


def sources_hash(root, files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(root, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def test_traffic_record_dropped_when_a_source_changes(tmp_path, monkeypatch):
    # A copy of the tree holding one record taken on exactly these sources,
    # then one source of the kernel differs by a byte.
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    r = dict(rec["c2:f32"])
    os.makedirs(tmp_path / "profiles")
    for f in r["source_files"]:
        dst = tmp_path / f
        os.makedirs(dst.parent, exist_ok=True)
        data = open(os.path.join(ROOT, f), "rb").read()
        dst.write_bytes(data)
    r["source_sha256"] = sources_hash(str(tmp_path), r["source_files"])
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
