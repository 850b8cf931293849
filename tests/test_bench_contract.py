"""bench.py's host-side contract: one GPU only, and the HBM traffic read from a counter
summary only while that summary was taken on the current fingerprint source."""

import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _summary(path, sha):
    with open(path, "w") as f:
        f.write("# test summary\n")
        f.write(f"fingerprint source sha256 prefix: {sha}\n")
        f.write("fp FETCH_SIZE KiB per dispatch: 1000.0\n")
        f.write("fp WRITE_SIZE KiB per dispatch: 10.0\n")
        f.write("copy fetch scale: 2.0\n")
        f.write("copy write scale: 1.0\n")


def test_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    p = tmp_path / "pmc.txt"
    monkeypatch.setattr(bench, "PROFILE_PMC", {"decoder7b": str(p)})
    _summary(p, bench.source_digest())
    assert bench.pmc_traffic("decoder7b") == int(1000.0 * 1024 * 2.0 + 10.0 * 1024 * 1.0)
    assert bench.pmc_traffic("random16") is None  # no counter summary for that workload
    _summary(p, "0" * 16)
    assert bench.pmc_traffic("decoder7b") is None


def test_committed_profiles_parse():
    for path in bench.PROFILE_PMC.values():
        kv = {}
        for line in open(path):
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
        for key in ("fingerprint source sha256 prefix", "fp FETCH_SIZE KiB per dispatch",
                    "fp WRITE_SIZE KiB per dispatch", "copy fetch scale", "copy write scale"):
            assert key in kv, (path, key)
        float(kv["fp FETCH_SIZE KiB per dispatch"])
        float(kv["copy fetch scale"])


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
