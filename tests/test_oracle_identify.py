"""The oracle's free-time weight identification (Sec. 4.1.1) pinned by brute force on
raw bytes: a block matches iff its recorded bytes equal its current bytes; an
allocation is weights iff it has recorded payloads and all of their blocks match."""

import numpy as np

import oracle


def brute(recorded, current, block, region_first):
    match, first = [], []
    for r, c in zip(recorded, current):
        fd = oracle.NO_DIFF
        for j, b0 in enumerate(range(0, len(r), block)):
            same = bytes(r[b0:b0 + block]) == bytes(c[b0:b0 + block])
            match.append(1 if same else 0)
            if not same and fd == oracle.NO_DIFF:
                fd = j
        first.append(fd)
    weight = []
    for a, b in zip(region_first[:-1], region_first[1:]):
        weight.append(1 if b > a and all(first[s] == oracle.NO_DIFF for s in range(a, b)) else 0)
    return match, first, weight


def test_identify_against_bytes():
    rng = np.random.default_rng(51)
    block = 8192
    for trial in range(20):
        lens = [int(x) for x in rng.integers(0, 5 * block, 12)]
        recorded = [np.frombuffer(rng.bytes(n), np.uint8).copy() for n in lens]
        current = [r.copy() for r in recorded]
        for c in current:  # some payloads change in place after the write
            if c.size and rng.random() < 0.3:
                c[int(rng.integers(0, c.size))] ^= 0x40
        cuts = sorted(set(int(x) for x in rng.integers(0, len(lens) + 1, 4)))
        region_first = [0] + cuts + [len(lens)]
        rec_digests, _ = oracle.batch_digests(recorded, block)
        m, f, w = oracle.identify_weights(rec_digests, current, block, region_first)
        em, ef, ew = brute(recorded, current, block, region_first)
        assert m.tolist() == em, trial
        assert f.tolist() == ef, trial
        assert w.tolist() == ew, trial


def test_unchanged_allocation_is_weights_and_empty_is_not():
    rng = np.random.default_rng(52)
    p = [np.frombuffer(rng.bytes(70000), np.uint8)]
    d, _ = oracle.batch_digests(p, 65536)
    m, f, w = oracle.identify_weights(d, p, 65536, [0, 1, 1])
    assert m.tolist() == [1, 1] and f.tolist() == [oracle.NO_DIFF] and w.tolist() == [1, 0]
