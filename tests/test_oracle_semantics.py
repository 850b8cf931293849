"""The oracle's geometry, lookup (with in-batch first occurrence), insert and
compaction, pinned by brute force that never hashes: payloads are sliced into
blocks directly, and hits are decided on the raw block BYTES.

Sec. 4.1.2: a payload whose identifier the server already holds sends only
(hash, size); otherwise its bytes travel. Within one batch a block whose bytes
already travelled earlier in the batch need not travel again.
"""

import numpy as np

import oracle


def brute_blocks(payloads, block):
    out = []
    for p in payloads:
        for b0 in range(0, len(p), block):
            out.append(bytes(p[b0:b0 + block]))
    return out


def test_geometry_brute_force():
    rng = np.random.default_rng(31)
    for block in (4096, 65536):
        lens = [int(x) for x in rng.integers(0, 5 * block, size=40)] + [0, 0, block, 1]
        first, blen = oracle.geometry(lens, block)
        expect_len = []
        expect_first = [0]
        for n in lens:
            cnt = 0
            for b0 in range(0, n, block):
                expect_len.append(min(block, n - b0))
                cnt += 1
            expect_first.append(expect_first[-1] + cnt)
        assert first.tolist() == expect_first
        assert blen.tolist() == expect_len


def _random_batch(rng, pool, n_payloads, block):
    payloads = []
    for _ in range(n_payloads):
        k = int(rng.integers(0, 5))
        parts = [pool[int(rng.integers(0, len(pool)))] for _ in range(k)]
        tail = rng.bytes(int(rng.integers(0, 3)) * 700)  # sometimes a short last block
        payloads.append(np.frombuffer(b"".join(parts) + tail, np.uint8))
    return payloads


def test_lookup_and_compaction_brute_force():
    block = 4096
    rng = np.random.default_rng(32)
    for trial in range(30):
        pool = [rng.bytes(block) for _ in range(6)]
        payloads = _random_batch(rng, pool, 8, block)
        blocks = brute_blocks(payloads, block)
        # table: some pool blocks, stored under their oracle digest with an arbitrary value
        cached = {pool[i]: 1000 + i for i in range(len(pool)) if rng.random() < 0.4}
        table = oracle.Table()
        keys = [int(oracle.payload_digests(np.frombuffer(b, np.uint8), block)[0][0]) for b in cached]
        table.insert(np.array(keys, np.uint64), np.array(list(cached.values()), np.uint64))
        res = oracle.run(payloads, block, table)
        # brute force on bytes
        first = {}
        exp_status, exp_ref = [], []
        for g, b in enumerate(blocks):
            if b in cached:
                exp_status.append(1)
                exp_ref.append(cached[b])
            elif b in first:
                exp_status.append(2)
                exp_ref.append(first[b])
            else:
                first[b] = g
                exp_status.append(0)
                exp_ref.append(g)
        assert res["status"].tolist() == exp_status, trial
        assert res["ref"].tolist() == exp_ref, trial
        miss = [g for g, s in enumerate(exp_status) if s == 0]
        assert res["miss_idx"].tolist() == miss
        assert res["miss_count"] == len(miss)
        assert res["miss_bytes"] == sum(len(blocks[g]) for g in miss)


def test_replayed_batch_is_all_hits():
    block = 65536
    rng = np.random.default_rng(33)
    payload = np.frombuffer(rng.bytes(10 * block + 123), np.uint8)
    table = oracle.Table()
    res1 = oracle.run([payload], block, table)
    assert (res1["status"] == oracle.MISS).all()
    n = res1["digests"].size
    assert table.insert(res1["digests"], np.arange(n, dtype=np.uint64)) == n
    res2 = oracle.run([payload], block, table)
    assert (res2["status"] == oracle.HIT_CACHE).all()
    assert res2["ref"].tolist() == list(range(n))
    assert res2["miss_count"] == 0 and res2["miss_bytes"] == 0


def test_insert_brute_force_dict():
    rng = np.random.default_rng(34)
    table = oracle.Table()
    ref = {}
    special = np.array([0, 2**64 - 1, 1, 2**63], dtype=np.uint64)
    for _ in range(20):
        keys = np.concatenate([rng.integers(0, 50, size=30, dtype=np.uint64), special[rng.integers(0, 4, 3)]])
        vals = rng.integers(0, 2**64, size=keys.size, dtype=np.uint64, endpoint=False)
        n_new = table.insert(keys, vals)
        exp_new = 0
        for k, v in zip(keys.tolist(), vals.tolist()):
            if k not in ref:
                ref[k] = v
                exp_new += 1
        assert n_new == exp_new
        assert sorted(ref) == table.keys.tolist()
        present, got = table.get(np.array(list(ref), np.uint64))
        assert present.all()
        assert got.tolist() == [ref[k] for k in ref]


def test_lookup_special_keys():
    table = oracle.Table()
    table.insert(np.array([0, 2**64 - 1], np.uint64), np.array([7, 9], np.uint64))
    d = np.array([2**64 - 1, 5, 0, 5, 2**64 - 2, 2**64 - 2], np.uint64)
    st, ref = oracle.lookup(d, table)
    assert st.tolist() == [1, 0, 1, 2, 0, 2]
    assert ref.tolist() == [9, 1, 7, 1, 4, 4]


def test_empty_batch():
    st, ref = oracle.lookup(np.zeros(0, np.uint64), oracle.Table())
    assert st.size == 0 and ref.size == 0
    idx, cnt, nb = oracle.compact(st, np.zeros(0, np.uint64))
    assert idx.size == 0 and cnt == 0 and nb == 0
