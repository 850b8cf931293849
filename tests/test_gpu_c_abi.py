"""The C ABI used from plain C (tests/c_abi/detect.c: hipMalloc'd buffers, a HIP stream,
no torch): fingerprint -> insert -> lookup -> compaction on four payloads, its printed
outputs compared with the oracle on the same bytes."""

import os
import subprocess

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

BINARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "detect")
BLOCK = 65536


def payloads():
    """The bytes detect.c builds (see its header comment)."""
    lens = [(1 << 20) + 17, 4096, 100000, 4096]
    out = []
    for p, n in enumerate(lens):
        i = np.arange(n, dtype=np.uint64)
        v = ((i * np.uint64(2654435761) + np.uint64(p * 40503)) & np.uint64(0xFFFFFFFF)) >> np.uint64(11)
        out.append((v & np.uint64(0xFF)).astype(np.uint8))
    out[2][:BLOCK] = out[0][:BLOCK]
    out[3][:] = out[1]
    return out


def test_plain_c_caller_matches_oracle():
    if not os.path.exists(BINARY):
        pytest.fail(f"{BINARY} is not built; run __graft_entry__.build()")
    print("[gpu-case] c abi detect", flush=True)
    res = subprocess.run([BINARY], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    lines = res.stdout.splitlines()
    n = int(lines[0].split()[1])
    blocks = [ln.split() for ln in lines[1:1 + n]]
    digests = np.array([int(b[2], 16) for b in blocks], np.uint64)
    status = np.array([int(b[3]) for b in blocks], np.uint8)
    ref = np.array([int(b[4]) for b in blocks], np.uint64)
    _, count, _, nbytes = lines[1 + n].split()
    misses = np.array([int(ln.split()[1]) for ln in lines[2 + n:]], np.uint64)

    p = payloads()
    table = oracle.Table()
    first, _ = oracle.batch_digests(p[:1], BLOCK)
    table.insert(first, np.arange(first.size, dtype=np.uint64) + 1000)
    want = oracle.run(p, BLOCK, table)
    assert n == want["digests"].size
    assert np.array_equal(digests, want["digests"])
    assert np.array_equal(status, want["status"])
    assert np.array_equal(ref, want["ref"])
    assert int(count) == want["miss_count"] and int(nbytes) == want["miss_bytes"]
    assert np.array_equal(misses, want["miss_idx"])
    # payload 0's blocks and payload 2's first block are held; payload 3 repeats payload 1
    assert (status == 1).sum() == first.size + 1 and (status == 2).sum() == 1
