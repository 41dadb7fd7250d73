"""The parts of bench.py's contract that need no GPU: more than one GPU is
refused with a message, and the stored HBM traffic of the score kernel is
reported only for the workload it was measured on and only while the score
kernel's sources are the ones the counters were taken on."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)


def _stored():
    kv = {}
    with open(bench.TRAFFIC_FILE) as fh:
        for line in fh:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    return kv


def test_traffic_is_gated_by_workload_size_and_source(monkeypatch):
    kv = _stored()
    n = int(kv["candidates"])
    monkeypatch.setattr(bench, "score_source_digest", lambda: kv["score_source_sha256"])
    assert bench.measured_traffic(kv["workload"], n) == float(kv["hbm_bytes_per_launch"])
    assert bench.measured_traffic(kv["workload"], n + 1) is None
    assert bench.measured_traffic("another", n) is None
    monkeypatch.setattr(bench, "score_source_digest", lambda: "0" * 64)
    assert bench.measured_traffic(kv["workload"], n) is None


def test_stored_traffic_is_near_the_algorithmic_bytes():
    # FETCH_SIZE + WRITE_SIZE per launch against 9 bytes per candidate: the
    # kernel moves its output once (a few percent for coefficients and partial
    # lines), never a re-read of its own output
    kv = _stored()
    ratio = float(kv["hbm_bytes_per_launch"]) / float(kv["algorithmic_bytes_per_launch"])
    assert 1.0 <= ratio < 1.1
    assert int(kv["algorithmic_bytes_per_launch"]) == 9 * int(kv["candidates"])
