"""Pins for the oracle's address-remap interval map (Gleam Sec. 4.1.3, Weight Chunk Sharing;
Appendix, Implementation Details, Virtual Memory Map).

The map's rules are pinned against a brute force that keeps every interval as the
Python set of the addresses it covers, on an address space small enough to check
every address, plus the edge cases of the 64-bit space that brute force cannot reach.
"""

import random

import numpy as np
import pytest

from oracle import remap

TOP = (1 << 64) - 1


class Brute:
    """Every interval as (start, length, target); meetings tested on address sets."""

    def __init__(self, capacity):
        self.capacity = capacity
        self.items = []

    @staticmethod
    def cover(s, n):
        return set(range(s, s + n))

    def update(self, removals, additions):
        survivors = [iv for iv in self.items
                     if not any(self.cover(iv[0], iv[1]) & self.cover(d, n) for d, n in removals)]
        status = []
        for s, n, t in additions:
            status.append(remap.INVALID if n == 0 or s + n > TOP or t + n > TOP else remap.ADDED)
        for i, (s, n, t) in enumerate(additions):
            if status[i] != remap.ADDED:
                continue
            mine = self.cover(s, n)
            hit = any(mine & self.cover(v[0], v[1]) for v in survivors)
            hit |= any(mine & self.cover(additions[j][0], additions[j][1])
                       for j in range(len(additions)) if j != i and status[j] != remap.INVALID)
            if hit:
                status[i] = remap.OVERLAP
        taken = [a for a, st in zip(additions, status) if st == remap.ADDED]
        if len(survivors) + len(taken) > self.capacity:
            status = [remap.FULL if st == remap.ADDED else st for st in status]
            return status, (len(self.items), 0, 0, sum(st != remap.ADDED for st in status))
        removed = len(self.items) - len(survivors)
        self.items = sorted(survivors + taken)
        return status, (len(self.items), len(taken), removed, len(additions) - len(taken))

    def translate(self, p):
        for s, n, t in self.items:
            if s <= p < s + n:
                return t + (p - s)
        return remap.UNMAPPED


def test_overlap_counts_match_pairwise():
    rng = np.random.default_rng(5)
    for _ in range(50):
        a = rng.integers(0, 100, (rng.integers(0, 20), 2))
        b = rng.integers(0, 100, (rng.integers(0, 20), 2))
        a.sort(axis=1)
        b.sort(axis=1)
        got = remap.overlap_counts(a[:, 0], a[:, 1], b[:, 0], b[:, 1]) if len(a) else []
        want = [sum(1 for f2, l2 in b if f2 <= l1 and l2 >= f1) for f1, l1 in a]
        assert list(got) == want


@pytest.mark.parametrize("seed", range(6))
def test_random_updates_match_brute_force(seed):
    rng = random.Random(seed)
    space = 48
    cap = rng.choice([4, 8, 64])
    m, bf = remap.RemapMap(cap), Brute(cap)
    for step in range(150):
        removals = [(rng.randrange(space), rng.randrange(0, 10)) for _ in range(rng.randrange(0, 3))]
        additions = [(rng.randrange(space), rng.randrange(0, 7), rng.randrange(1000, 2000))
                     for _ in range(rng.randrange(0, 6))]
        st, counts = m.update([r[0] for r in removals], [r[1] for r in removals],
                              [a[0] for a in additions], [a[1] for a in additions], [a[2] for a in additions])
        st_b, counts_b = bf.update(removals, additions)
        assert list(st) == st_b, (seed, step)
        assert tuple(counts) == counts_b, (seed, step)
        s, n, t = m.export()
        assert list(zip(s.tolist(), n.tolist(), t.tolist())) == bf.items
        got = m.translate(np.arange(space + 8, dtype=np.uint64))
        assert got.tolist() == [bf.translate(p) for p in range(space + 8)]
        # invariants: sorted by start, disjoint, non-empty, within capacity
        assert np.all(n > 0) and len(m) <= cap
        assert np.all(s[1:] >= s[:-1] + n[:-1])


def test_paper_two_chunks_in_one_allocation():
    """Sec. 4.1.3's case: two chunks written into one client allocation find their
    shareable copies in two different server allocations."""
    task, base = 3, 0x4000
    va = (task << 40) + base
    pos1, pos2 = 0x7F00_0000_0000, 0x7F80_0000_1000
    m = remap.RemapMap(16)
    st, counts = m.update(add_start=[va, va + 0x3000], add_len=[0x3000, 0x500], add_target=[pos1, pos2])
    assert st.tolist() == [remap.ADDED] * 2 and counts == (2, 2, 0, 0)
    probes = [va, va + 0x2FFF, va + 0x3000, va + 0x3004, va + 0x34FF, va + 0x3500, va - 1,
              ((task + 1) << 40) + base]
    assert m.translate(probes).tolist() == [pos1, pos1 + 0x2FFF, pos2, pos2 + 4, pos2 + 0x4FF,
                                            remap.UNMAPPED, remap.UNMAPPED, remap.UNMAPPED]
    # freeing the client allocation removes both mappings, and only them
    m.update(add_start=[(4 << 40)], add_len=[16], add_target=[1 << 20])
    st, counts = m.update(rem_start=[va], rem_len=[0x4000])
    assert counts == (1, 0, 2, 0)
    assert m.translate([va + 0x3004, 4 << 40]).tolist() == [remap.UNMAPPED, 1 << 20]


def test_edges_of_the_address_space():
    m = remap.RemapMap(8)
    st, _ = m.update(add_start=[0, TOP - 5, TOP - 3, 100, 200, 300],
                     add_len=[1, 5, 4, 0, 8, 8],
                     add_target=[TOP - 1, 7, 9, 1, TOP - 8, TOP - 7])
    # [TOP-5, TOP) ends exactly at 2^64 - 1; [TOP-3, TOP+1) wraps; length 0; target
    # + length = 2^64 - 1 is allowed, 2^64 is not (the last translation would be UNMAPPED)
    assert st.tolist() == [remap.ADDED, remap.ADDED, remap.INVALID, remap.INVALID, remap.ADDED,
                           remap.INVALID]
    assert m.translate([0, 1, TOP - 5, TOP - 1, TOP, 207]).tolist() == [
        TOP - 1, remap.UNMAPPED, 7, 11, remap.UNMAPPED, TOP - 1]
    # a removal whose end passes 2^64 is clipped and still removes the top interval
    st, counts = m.update(rem_start=[TOP - 2], rem_len=[TOP])
    assert counts == (2, 0, 1, 0)
    # an empty removal removes nothing, even inside an interval
    _, counts = m.update(rem_start=[203], rem_len=[0])
    assert counts == (2, 0, 0, 0)


def test_clashes_are_refused_on_both_sides():
    m = remap.RemapMap(8)
    m.update(add_start=[100], add_len=[10], add_target=[5000])
    st, counts = m.update(add_start=[109, 120, 125, 140, 150, 150], add_len=[2, 6, 10, 5, 3, 3],
                          add_target=[1, 2, 3, 4, 5, 6])
    # 109 meets the survivor; 120 and 125 meet each other; 140 is clear; the two 150s clash
    assert st.tolist() == [remap.OVERLAP, remap.OVERLAP, remap.OVERLAP, remap.ADDED, remap.OVERLAP,
                           remap.OVERLAP]
    assert counts == (2, 1, 0, 5)
    # adjacent intervals do not meet
    st, _ = m.update(add_start=[110, 90], add_len=[30, 10], add_target=[1, 2])
    assert st.tolist() == [remap.ADDED, remap.ADDED]


def test_remove_and_readd_in_one_call_replaces_a_mapping():
    m = remap.RemapMap(4)
    m.update(add_start=[0, 64], add_len=[64, 64], add_target=[1000, 2000])
    st, counts = m.update(rem_start=[10], rem_len=[1], add_start=[0], add_len=[32], add_target=[9000])
    assert st.tolist() == [remap.ADDED] and counts == (2, 1, 1, 0)
    assert m.translate([5, 40, 70]).tolist() == [9005, remap.UNMAPPED, 2006]


def test_full_changes_nothing():
    m = remap.RemapMap(3)
    m.update(add_start=[0, 10], add_len=[5, 5], add_target=[100, 200])
    before = m.export()
    st, counts = m.update(rem_start=[0], rem_len=[1], add_start=[20, 30, 40, 40],
                          add_len=[1, 1, 1, 0], add_target=[1, 2, 3, 4])
    # 1 survivor + 3 additions > 3: nothing happens, the removal included
    assert st.tolist() == [remap.FULL] * 3 + [remap.INVALID]
    assert counts == (2, 0, 0, 4)
    for a, b in zip(before, m.export()):
        assert np.array_equal(a, b)
    st, counts = m.update(rem_start=[0], rem_len=[1], add_start=[20, 30], add_len=[1, 1], add_target=[1, 2])
    assert counts == (3, 2, 1, 0)
