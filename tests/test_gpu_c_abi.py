"""The C ABI used from plain C (hipMalloc'd buffers, a HIP stream, no torch):
tests/c_abi/detect.c runs fingerprint -> insert -> lookup -> compaction on four payloads,
tests/c_abi/remap.c the address-remap calls; their printed outputs are compared with the
oracle on the same inputs."""

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


REMAP_BINARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "remap")


def test_plain_c_remap_matches_oracle():
    """tests/c_abi/remap.c: the weight-sharing case of two chunks of one client allocation
    mapped into two server allocations, a later overlapping addition refused, probes
    translated before and after the allocation is freed; everything printed equals the
    oracle."""
    from oracle import remap as oremap
    if not os.path.exists(REMAP_BINARY):
        pytest.fail(f"{REMAP_BINARY} is not built; run __graft_entry__.build()")
    print("[gpu-case] c abi remap", flush=True)
    res = subprocess.run([REMAP_BINARY], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    by_tag = {}
    for ln in res.stdout.splitlines():
        f = ln.split()
        by_tag.setdefault(f[0], []).append(f[1:])
    va = (3 << 40) + 0x4000
    m = oremap.RemapMap(64)
    st, counts = m.update(add_start=[va, va + 0x3000, 4 << 40], add_len=[0x3000, 0x500, 16],
                          add_target=[0x7F0000000000, 0x7F8000001000, 1 << 20])
    st_c, counts_c = m.update(add_start=[va + 0x100], add_len=[8], add_target=[5])
    probe = [va, va + 0x2FFF, va + 0x3000, va + 0x3004, va + 0x3500, va - 1, (4 << 40) + 15, (4 << 40) + 16,
             (1 << 64) - 1]
    before = m.translate(probe)
    _, counts_f = m.update(rem_start=[va], rem_len=[0x4000])
    after = m.translate(probe)
    assert tuple(int(x) for x in by_tag["add"][0]) == counts == (3, 3, 0, 0)
    assert [int(x[1]) for x in by_tag["status"]] == st.tolist()
    assert tuple(int(x) for x in by_tag["clash"][0]) == (*counts_c, oremap.OVERLAP) and st_c[0] == oremap.OVERLAP
    assert [int(x[1], 16) for x in by_tag["before"]] == before.tolist()
    assert before[3] == 0x7F8000001000 + 4
    assert tuple(int(x) for x in by_tag["free"][0]) == counts_f == (1, 0, 2, 0)
    assert [int(x[1], 16) for x in by_tag["after"]] == after.tolist()
