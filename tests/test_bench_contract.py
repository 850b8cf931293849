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


def test_block_lengths_follow_the_payload_geometry():
    """The exposure figures weigh blocks by their byte lengths: full blocks, the short
    last block of each payload, none for an empty payload."""

    class B:  # the host-side fields of a Batch
        pass

    import numpy as np
    b = B()
    b.block_bytes = 4096
    b.host_len = np.array([0, 1, 4096, 4097, 10000, 0, 8192], dtype=np.uint64)
    nb = [(int(n) + 4095) // 4096 for n in b.host_len]
    b.host_first = np.concatenate([[0], np.cumsum(nb)]).astype(np.uint64)
    b.n_blocks = int(b.host_first[-1])
    want = [1, 4096, 4096, 1, 4096, 4096, 1808, 4096, 4096]
    assert bench.block_lengths(b).tolist() == want
    assert int(bench.block_lengths(b).sum()) == int(b.host_len.sum())
