"""Pins for the oracle's first-write rule (Sec. 4.1.1: where an address range is
written several times, only the first host-to-device write counts) and its leaf-level
identification, against brute force on raw bytes and addresses.

Brute force keeps, for every address of a small space, the index of the first write
covering it (painting the writes in reverse time order), and reads each write's pieces
off as the maximal runs of addresses it owns."""

import numpy as np
import pytest

import oracle


def brute_pieces(addr, length, region_first):
    pw, po, pl, first = [], [], [], [0]
    for r in range(len(region_first) - 1):
        w0, w1 = region_first[r], region_first[r + 1]
        owner = {}
        for j in reversed(range(w0, w1)):  # earlier writes paint over later ones
            for x in range(addr[j], addr[j] + length[j]):
                owner[x] = j
        for j in range(w0, w1):
            xs = sorted(x for x, o in owner.items() if o == j)
            runs = []
            for x in xs:
                if runs and runs[-1][1] == x:
                    runs[-1][1] = x + 1
                else:
                    runs.append([x, x + 1])
            for lo, hi in runs:
                pw.append(j), po.append(lo - addr[j]), pl.append(hi - lo)
        first.append(len(pw))
    return pw, po, pl, first


def random_log(rng, n_regions, space=300):
    addr, length, region_first = [], [], [0]
    for _ in range(n_regions):
        k = int(rng.integers(0, 12))
        base = int(rng.integers(0, 1000)) * 1000
        for _ in range(k):
            kind = rng.random()
            if kind < 0.1 and addr:  # repeat an earlier write of this allocation exactly
                j = int(rng.integers(region_first[-1], len(addr))) if len(addr) > region_first[-1] else None
                if j is not None:
                    addr.append(addr[j]), length.append(length[j])
                    continue
            lo = base + int(rng.integers(0, space))
            n = 0 if kind < 0.15 else int(rng.integers(1, space // 2))
            addr.append(lo), length.append(n)
        region_first.append(len(addr))
    return addr, length, region_first


def test_pieces_against_painted_addresses():
    rng = np.random.default_rng(61)
    for trial in range(200):
        addr, length, rf = random_log(rng, int(rng.integers(1, 5)))
        pw, po, pl, first, status = oracle.first_write_pieces(addr, length, rf)
        bw, bo, bl, bf = brute_pieces(addr, length, rf)
        assert pw.tolist() == bw and po.tolist() == bo and pl.tolist() == bl, trial
        assert first.tolist() == bf, trial
        assert (status == oracle.FW_OK).all()


def test_closed_cases():
    # disjoint writes: each owns itself, whole
    pw, po, pl, first, _ = oracle.first_write_pieces([0, 100, 50], [50, 10, 50], [0, 3])
    assert (pw.tolist(), po.tolist(), pl.tolist()) == ([0, 1, 2], [0, 0, 0], [50, 10, 50])
    # a write inside an earlier one owns nothing; one over the end of an earlier one owns its tail
    pw, po, pl, first, _ = oracle.first_write_pieces([0, 10, 90], [100, 20, 30], [0, 3])
    assert (pw.tolist(), po.tolist(), pl.tolist()) == ([0, 2], [0, 10], [100, 20])
    # a later write over two earlier ones owns the gap between them and its two ends
    pw, po, pl, first, _ = oracle.first_write_pieces([10, 40, 0], [10, 10, 60], [0, 3])
    assert (pw.tolist(), po.tolist(), pl.tolist()) == ([0, 1, 2, 2, 2], [0, 0, 0, 20, 50], [10, 10, 10, 20, 10])
    # allocations do not see each other's writes; an empty allocation has no pieces
    pw, po, pl, first, _ = oracle.first_write_pieces([0, 0], [8, 8], [0, 1, 1, 2])
    assert (pw.tolist(), first.tolist()) == ([0, 1], [0, 1, 1, 2])


def test_refusals():
    top = 2**64 - 1
    # reaching the last address exactly is valid; one byte further is not
    pw, po, pl, first, st = oracle.first_write_pieces([top - 9, top - 9], [9, 10], [0, 1, 2])
    assert st.tolist() == [oracle.FW_OK, oracle.FW_INVALID] and first.tolist() == [0, 1, 1]
    _, _, _, first, st = oracle.first_write_pieces(list(range(5)), [1] * 5, [0, 3, 5], max_writes=2)
    assert st.tolist() == [oracle.FW_TOO_MANY, oracle.FW_OK] and first.tolist() == [0, 0, 2]


def test_pieces_cover_the_union_once():
    rng = np.random.default_rng(62)
    for _ in range(50):
        addr, length, rf = random_log(rng, 1, space=5000)
        pw, po, pl, _, _ = oracle.first_write_pieces(addr, length, rf)
        starts = [addr[int(w)] + int(o) for w, o in zip(pw, po)]
        spans = sorted(zip(starts, [s + int(n) for s, n in zip(starts, pl)]))
        assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))  # disjoint
        union = set()
        for a, n in zip(addr, length):
            union.update(range(a, a + n))
        assert sum(int(n) for n in pl) == len(union)


def test_first_write_identification_against_bytes():
    """Digests of the owned pieces, recorded from the bytes each write carried and
    compared with the allocation's current bytes, decide weights exactly when every
    written byte still equals its first writer's byte."""
    rng = np.random.default_rng(63)
    block = 8192
    for trial in range(40):
        size = int(rng.integers(1, 4)) * 20000
        n = int(rng.integers(1, 8))
        addr = [int(rng.integers(0, size - 1)) for _ in range(n)]
        length = [int(rng.integers(0, size - a + 1)) for a in addr]
        data = [np.frombuffer(rng.bytes(m), np.uint8) for m in length]
        if n > 1 and rng.random() < 0.4:  # a later write repeats an earlier one's bytes
            addr[-1], length[-1], data[-1] = addr[0], length[0], data[0].copy()
        mem = np.zeros(size, np.uint8)
        for a, d in zip(addr, data):
            mem[a:a + d.size] = d
        first_byte = {}
        for j in reversed(range(n)):
            for i in range(length[j]):
                first_byte[addr[j] + i] = data[j][i]
        if rng.random() < 0.5 and first_byte:  # something changes one written byte later
            x = sorted(first_byte)[int(rng.integers(0, len(first_byte)))]
            mem[x] ^= 0x5A
        expect = int(bool(first_byte) and all(mem[x] == v for x, v in first_byte.items()))
        pw, po, pl, first, _ = oracle.first_write_pieces(addr, length, [0, n])
        recorded = [data[int(w)][int(o):int(o) + int(m)] for w, o, m in zip(pw, po, pl)]
        current = [mem[addr[int(w)] + int(o):addr[int(w)] + int(o) + int(m)] for w, o, m in zip(pw, po, pl)]
        rec, _ = oracle.batch_digests(recorded, block)
        _, _, weight = oracle.identify_weights(rec, current, block, first)
        assert weight.tolist() == [expect], trial


def brute_leaves(recorded, current, block):
    per = block // 4096
    match, first = [], []
    for r, c in zip(recorded, current):
        fd = oracle.NO_DIFF
        nb = (len(r) + block - 1) // block
        for b in range(nb):
            for k in range(per):
                lo = b * block + k * 4096
                hi = min(lo + 4096, (b + 1) * block, len(r))
                same = lo >= hi or bytes(r[lo:hi]) == bytes(c[lo:hi])
                match.append(1 if same else 0)
                if not same and fd == oracle.NO_DIFF:
                    fd = b * per + k
        first.append(fd)
    return match, first


@pytest.mark.parametrize("block", [4096, 16384, 65536])
def test_identify_leaves_against_bytes(block):
    rng = np.random.default_rng(64 + block)
    for trial in range(15):
        lens = [int(x) for x in rng.integers(0, 3 * block + 5000, 10)]
        recorded = [np.frombuffer(rng.bytes(n), np.uint8).copy() for n in lens]
        current = [r.copy() for r in recorded]
        for c in current:
            if c.size and rng.random() < 0.4:
                c[int(rng.integers(0, c.size))] ^= 0x11
        cuts = sorted(set(int(x) for x in rng.integers(0, len(lens) + 1, 3)))
        region_first = [0] + cuts + [len(lens)]
        _, rec_leaves = oracle.batch_digests(recorded, block, with_leaves=True)
        m, f, w = oracle.identify_leaves(rec_leaves, current, block, region_first)
        em, ef = brute_leaves(recorded, current, block)
        assert m.tolist() == em, trial
        assert f.tolist() == ef, trial
        _, _, wb = oracle.identify_weights(oracle.batch_digests(recorded, block)[0], current, block, region_first)
        assert w.tolist() == wb.tolist(), trial  # same verdict as the block-level check
