"""bench.py's contract checks that need no GPU: one GPU only, with a message."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("path", ["chamfer", "mesh", "p2s", "emd"])
def test_more_than_one_gpu_exits_with_a_message(path):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2",
                        "--path", path], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def test_forward_fractions_follow_their_definitions(tmp_path, monkeypatch):
    """The three roofline fractions of a cd_forward time: credited 9 flop per
    directed pair-evaluation (2 B N M), executed 10 flop per computed distance
    (B N M), and the VALU issue fraction from a counter record with the
    current sources' sha (none when the sha differs)."""
    import json
    import bench
    B, N, M, ms = 16, 16384, 16384, 0.5
    peak = 157.3e12
    rec = {"kernel_source_sha256": bench._sources_sha256(bench.FORWARD_SOURCES),
           "workloads": {"w": {"lane_ops_per_call": 3.0e10}}}
    credited, executed, issue = bench.forward_fractions(B, N, M, ms, rec, "w")
    assert abs(credited - 9 * 2 * B * N * M / 5e-4 / peak) < 1e-12
    assert abs(executed - 10 * B * N * M / 5e-4 / peak) < 1e-12
    assert abs(executed / credited - 10 / 18) < 1e-12
    assert abs(issue - 3.0e10 / (5e-4 * 2.4e9 * 256 * 128)) < 1e-12
    assert bench.forward_fractions(B, N, M, ms, rec, "other")[2] is None
    assert bench.forward_fractions(B, N, M, ms, None, "w")[2] is None
    # A record taken at other sources is ignored.
    path = tmp_path / "rec.json"
    path.write_text(json.dumps(dict(rec, kernel_source_sha256="0" * 64)))
    monkeypatch.setattr(bench, "VALU_RECORD", str(path))
    assert bench.valu_record() is None
    path.write_text(json.dumps(rec))
    assert bench.valu_record()["workloads"]["w"]["lane_ops_per_call"] == 3.0e10


def test_committed_records_name_their_sources():
    """The committed counter records carry the sha256 of the sources they were
    taken at, and the library sha is stable and covers the sources."""
    import json
    import bench
    for name in ("counters_cd_forward_valu.json", "traffic_mesh_b16_n16384.json"):
        with open(os.path.join(ROOT, "profiles", name)) as f:
            rec = json.load(f)
        assert len(rec["kernel_source_sha256"]) == 64
    a, b = bench.library_sources_sha256(), bench.library_sources_sha256()
    assert a == b and len(a) == 64
    assert isinstance(bench.cpu_model(), str) and bench.cpu_model()
