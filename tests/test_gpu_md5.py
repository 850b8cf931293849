"""GPU parity of the paper's identifier (MD5 of a payload's first 1024 bits,
Appendix discussion), and its exposure next to full-content block digests."""

import hashlib

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23115_amd as g
import workloads as W
from gpu_util import keys_to_device, run_path, say, to_device, u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def gpu_md5(payloads, prefix, min_len=1024, skew=0):
    arena, offs, lens = W.pack(payloads, skew=skew)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, 4096)
    d, k, e = g.md5_prefix(batch, prefix, min_len)
    torch.cuda.synchronize()
    return u64(d).reshape(-1, 2).view(np.uint8).reshape(-1, 16), u64(k), e.cpu().numpy()


@pytest.mark.parametrize("prefix", [128, 64, 1000, 0])
@pytest.mark.parametrize("skew", [0, 1, 6])
def test_md5_prefix_lengths(prefix, skew):
    rng = np.random.default_rng(900 + prefix + skew)
    lens = list(range(0, 140)) + [183, 184, 191, 192, 1023, 1024, 1025, 5000, 70000]
    payloads = [np.frombuffer(rng.bytes(n), np.uint8) for n in lens]
    say("md5 prefix", prefix, "skew", skew)
    d, k, e = gpu_md5(payloads, prefix, skew=skew)
    ed, ek, ee = oracle.md5_prefix(payloads, prefix)
    assert np.array_equal(d, ed) and np.array_equal(k, ek) and np.array_equal(e, ee)
    for i, p in enumerate(payloads[::17]):
        assert d[i * 17].tobytes() == hashlib.md5(p[:prefix].tobytes()).digest()


def test_md5_prefix_small_copies_full():
    sc = W.SmallCopies()
    say("md5 prefix small copies")
    batch = g.Batch.from_arena(to_device(sc.arena), sc.offsets, sc.sizes, 4096)
    d, k, e = g.md5_prefix(batch)
    torch.cuda.synchronize()
    ed, ek, ee = oracle.md5_prefix(sc.payloads())
    assert np.array_equal(u64(d).reshape(-1, 2).view(np.uint8).reshape(-1, 16), ed)
    assert np.array_equal(u64(k), ek) and np.array_equal(e.cpu().numpy(), ee)


def test_prefix_identifier_misses_late_changes():
    """Payloads updated only past their first 128 bytes: the prefix identifier still
    matches the table (the server would restore stale bytes), the block digests do not."""
    rng = np.random.default_rng(950)
    block = 65536
    base = [np.frombuffer(rng.bytes(int(n)), np.uint8).copy() for n in rng.integers(2000, 300000, 40)]
    updated = [b.copy() for b in base]
    changed = rng.choice(40, 10, replace=False)
    for i in changed.tolist():
        pos = int(rng.integers(128, updated[i].size))
        updated[i][pos] ^= 0x01
    # table keyed by the prefix identifier of the base payloads
    _, base_keys, _ = oracle.md5_prefix(base)
    table = g.Cache(1 << 10)
    table.insert(keys_to_device(base_keys), keys_to_device(np.arange(40, dtype=np.uint64)))
    arena, offs, lens = W.pack(updated)
    d_arena = to_device(arena)
    batch = g.Batch.from_arena(d_arena, offs, lens, block)
    say("md5 prefix exposure")
    _, keys, _ = g.md5_prefix(batch)
    st, _ = table.lookup(keys)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == g.HIT_CACHE).all()  # every payload, changed or not, "hits"
    # the block-digest path, with a table of the base payloads' block digests
    bd, _ = oracle.batch_digests(base, block)
    btable = g.Cache(1 << 12)
    btable.insert(keys_to_device(bd), keys_to_device(np.arange(bd.size, dtype=np.uint64)))
    gpu = run_path(batch, btable)
    otable = oracle.Table()
    otable.insert(bd, np.arange(bd.size, dtype=np.uint64))
    want = oracle.run(updated, block, otable)
    assert np.array_equal(gpu["status"], want["status"]) and gpu["miss_count"] == want["miss_count"]
    first = batch.host_first
    missed_payloads = {s for s in range(40) for gi in range(int(first[s]), int(first[s + 1]))
                       if gpu["status"][gi] == g.MISS}
    assert missed_payloads == set(changed.tolist())
