"""Seeded workloads: deterministic, of the stated shapes, and with the planted truth
the oracle must reproduce (end-to-end pins of the oracle at workload scale).

The full-size 16 MiB and ResNet-50 workloads run here; the 7B decoder (13.5 GB),
100k small copies and the 40 GB bf16 set are checked at reduced sizes built by the
same generators (the full sizes run in the GPU suite).
"""

import math

import numpy as np

import oracle
import workloads as W


def test_generators_are_deterministic():
    a = W.random16_payload()
    b = W.random16_payload()
    assert a.size == 16 << 20 and np.array_equal(a, b)
    assert np.array_equal(W.resnet50_tensor(5), W.resnet50_tensor(5))
    d = W.Decoder(layers=10, d=128, ffn=344, vocab=500)
    assert np.array_equal(d.payload(d.perturbed[0]), d.payload(d.perturbed[0]))


def test_shapes():
    shapes = W.resnet50_shapes()
    assert len(shapes) == 161
    assert sum(math.prod(s) for _, s in shapes) == 25_557_032
    d = W.Decoder()
    assert len(d.shapes) == 291
    assert sum(d.nbytes) == 13_476_831_232
    assert len(d.perturbed) == 21 and d.perturbed_layers.size == 3
    blocks = sum(oracle.num_blocks(n, W.DECODER_BLOCK) for n in d.nbytes)
    assert blocks == 12_917
    assert sum(oracle.num_blocks(d.nbytes[i], W.DECODER_BLOCK) for i in d.perturbed) == 1_158
    large = W.LargeSet()
    assert large.sizes.size == 2000 and int(large.sizes.sum()) == 40_000_000_000
    assert (large.sizes % 2 == 0).all()


def test_random16_passes():
    block = W.RANDOM16_BLOCK
    p = W.random16_payload()
    table = oracle.Table()
    r1 = oracle.run([p], block, table)
    assert (r1["status"] == oracle.MISS).all() and r1["miss_count"] == 256
    assert table.insert(r1["digests"], np.arange(256, dtype=np.uint64)) == 256
    r2 = oracle.run([p], block, table)
    assert (r2["status"] == oracle.HIT_CACHE).all()
    q, chosen = W.random16_rerandomized(p)
    r3 = oracle.run([q], block, table)
    assert r3["miss_idx"].tolist() == chosen.tolist()
    assert r3["miss_count"] == 64 and r3["miss_bytes"] == 64 * block


def test_resnet50_truth():
    block = W.RESNET_BLOCK
    payloads = W.resnet50_payloads()
    assert sum(p.size for p in payloads) == 51_114_064
    first, _ = oracle.geometry([p.size for p in payloads], block)
    assert int(first[-1]) == 895
    cached = W.resnet50_cached_tensors()
    table = oracle.Table()
    for t in cached.tolist():
        d, _ = oracle.payload_digests(payloads[t], block)
        table.insert(d, np.full(d.size, t, np.uint64))
    res = oracle.run(payloads, block, table)
    expect = np.zeros(int(first[-1]), np.uint8)
    for t in cached.tolist():
        expect[int(first[t]):int(first[t + 1])] = oracle.HIT_CACHE
    assert np.array_equal(res["status"], expect)


def test_decoder_truth_reduced():
    block = 64 << 10
    d = W.Decoder(layers=10, d=256, ffn=688, vocab=1000)
    base = [d.base(i) for i in range(len(d.shapes))]
    pay = [d.payload(i) for i in range(len(d.shapes))]
    table = oracle.Table()
    bd, _ = oracle.batch_digests(base, block)
    table.insert(bd, np.arange(bd.size, dtype=np.uint64))
    res = oracle.run(pay, block, table)
    first, _ = oracle.geometry([p.size for p in pay], block)
    expect = np.full(int(first[-1]), oracle.HIT_CACHE, np.uint8)
    for i in d.perturbed:
        expect[int(first[i]):int(first[i + 1])] = oracle.MISS
    assert np.array_equal(res["status"], expect)
    # unperturbed blocks reference their own base position
    hit = res["status"] == oracle.HIT_CACHE
    assert np.array_equal(res["ref"][hit], np.flatnonzero(hit).astype(np.uint64))


def test_small_copies_truth_reduced():
    sc = W.SmallCopies(n=2000)
    payloads = sc.payloads()
    res = oracle.run(payloads, W.SMALL_BLOCK, oracle.Table())
    first, _ = oracle.geometry([p.size for p in payloads], W.SMALL_BLOCK)
    # global block index of every full leaf, in batch order
    full_g = []
    for s, p in enumerate(payloads):
        full_g.extend(int(first[s]) + k for k in range(p.size // 4096))
    full_g = np.array(full_g)
    # root of each planted copy chain
    root = np.arange(full_g.size)
    for t, s in zip(sc.targets.tolist(), sc.sources.tolist()):
        root[t] = root[s]
    expect_status = np.zeros(int(first[-1]), np.uint8)
    expect_ref = np.arange(int(first[-1]), dtype=np.uint64)
    expect_status[full_g[sc.targets]] = oracle.HIT_BATCH
    expect_ref[full_g[sc.targets]] = full_g[root[sc.targets]]
    assert np.array_equal(res["status"], expect_status)
    assert np.array_equal(res["ref"], expect_ref)
    assert res["miss_count"] == int(first[-1]) - sc.targets.size


def test_large_set_truth_reduced():
    block = 256 << 10
    ls = W.LargeSet(n=12, total=24_000_000, lo=1 << 20, hi=8 << 20)
    payloads = [ls.tensor(i) for i in range(12)]
    digests, _ = oracle.batch_digests(payloads, block)
    n = digests.size
    rand = ls.random_digests(5000)
    assert not np.isin(rand, digests).any()
    chosen = ls.cached_blocks(n)
    table = oracle.Table()
    table.insert(rand, np.zeros(rand.size, np.uint64))
    table.insert(digests[chosen], chosen.astype(np.uint64))
    res = oracle.run(payloads, block, table)
    expect = np.zeros(n, np.uint8)
    expect[chosen] = oracle.HIT_CACHE
    assert np.array_equal(res["status"], expect)
    assert np.array_equal(res["ref"][chosen], chosen.astype(np.uint64))


def test_write_logs_recipe():
    """The first-write logs: deterministic, grouped by allocation, every write inside its
    allocation, and all three kinds of write present (sub-ranges, whole allocations,
    repeats of an earlier write of the same allocation)."""
    a = W.WriteLogs(n_alloc=300)
    b = W.WriteLogs(n_alloc=300)
    assert np.array_equal(a.addr, b.addr) and np.array_equal(a.length, b.length)
    rf = a.region_first.astype(np.int64)
    assert rf[0] == 0 and rf[-1] == a.addr.size and np.all(np.diff(rf) >= 1) and np.all(np.diff(rf) <= 64)
    whole = repeats = 0
    for r in range(300):
        base = (r + 1) << 36
        ad = a.addr[rf[r]:rf[r + 1]].astype(np.int64)
        ln = a.length[rf[r]:rf[r + 1]].astype(np.int64)
        size = int((ad + ln).max() - base)
        assert np.all(ad >= base) and np.all(ad + ln <= base + (16 << 20))
        seen = set()
        for x, n in zip(ad.tolist(), ln.tolist()):
            whole += x == base and n == size
            repeats += (x, n) in seen
            seen.add((x, n))
    assert whole > 0 and repeats > 0
