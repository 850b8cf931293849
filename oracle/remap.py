"""Address-remap interval map: the oracle's definition.

TEST INFRASTRUCTURE ONLY (the package docstring says who may use it). It shares no
code with the GPU library.

Gleam, Sec. 4.1.3 (Weight Chunk Sharing): two host-to-device chunks written into one
client allocation may each find their shareable copy inside a different server
allocation, so the server keeps a virtual memory layer that maps ranges of client device
addresses onto the positions of those copies. Appendix, Implementation Details (Virtual
Memory Map): each task gets its own virtual address space of 1 TB, and the mappings are
kept in a red-black tree; the calls whose arguments carry device pointers are
translated through it.

Here the map is a set of disjoint, non-empty intervals [start, start + length), each
with a target. A pointer p inside an interval translates to target + (p - start); a
pointer outside every interval is unmapped. A task's space is a range of the
64-bit key space (e.g. task t owns [t * 2^40, (t + 1) * 2^40)), so one map holds
every task.

One batched update applies removals, then additions:
  1. every interval that shares at least one address with a non-empty removal range
     [d, d + dlen) (clipped at 2^64) is removed whole;
  2. an addition is INVALID if its length is 0 or if start + length or
     target + length exceeds 2^64 - 1 (so no translation equals UNMAPPED);
  3. a valid addition is an OVERLAP if it shares an address with a surviving interval
     or with another valid addition of the same call (both of two clashing additions
     are refused: the result does not depend on their order);
  4. if the survivors and the remaining additions exceed the capacity, the call
     changes nothing and those additions are FULL;
  5. otherwise the map becomes the survivors plus the remaining additions (ADDED).
"""

from __future__ import annotations

import numpy as np

ADDED, INVALID, OVERLAP, FULL = 0, 1, 2, 3
UNMAPPED = (1 << 64) - 1
_TOP = (1 << 64) - 1


def _u64(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.uint64).reshape(-1))


def overlap_counts(first, last, other_first, other_last) -> np.ndarray:
    """For each closed interval [first[i], last[i]], how many of the closed intervals
    [other_first[j], other_last[j]] share an address with it.

    Interval b meets a iff b.first <= a.last and b.last >= a.first. Every b with
    b.last < a.first also has b.first <= a.last, so the count is
    #{b.first <= a.last} - #{b.last < a.first}: two counts over sorted arrays."""
    of = np.sort(_u64(other_first))
    ol = np.sort(_u64(other_last))
    n_first_le = np.searchsorted(of, _u64(last), side="right")
    n_last_lt = np.searchsorted(ol, _u64(first), side="left")
    return (n_first_le - n_last_lt).astype(np.int64)


class RemapMap:
    """The interval map, kept as three arrays sorted by start (the order a tree walk
    would visit). `capacity` bounds the number of intervals."""

    def __init__(self, capacity: int):
        self.capacity = int(capacity)
        self.start = np.zeros(0, np.uint64)
        self.length = np.zeros(0, np.uint64)
        self.target = np.zeros(0, np.uint64)

    def __len__(self):
        return int(self.start.size)

    def update(self, rem_start=(), rem_len=(), add_start=(), add_len=(), add_target=()):
        """Apply one batched update. Returns (status u8[n_add], counts) with counts =
        (intervals after, added, removed, refused)."""
        rs, rl = _u64(rem_start), _u64(rem_len)
        a_s, a_l, a_t = _u64(add_start), _u64(add_len), _u64(add_target)
        assert rs.size == rl.size and a_s.size == a_l.size == a_t.size
        n_add = a_s.size

        # 1. removals: every interval meeting a non-empty range goes
        keep = np.ones(len(self), bool)
        if rs.size and len(self):
            nz = rl > 0
            r_first, r_len = rs[nz], rl[nz]
            # last address of [d, d + dlen), clipped at the top of the 64-bit space
            # (Python integers, so the sum cannot wrap)
            r_last = _u64([min(d + n - 1, _TOP) for d, n in zip(r_first.tolist(), r_len.tolist())])
            if r_first.size:
                # (an interval in the map never reaches past the top, so this cannot wrap)
                last = self.start + (self.length - np.uint64(1))
                keep = overlap_counts(self.start, last, r_first, r_last) == 0
        n_removed = int((~keep).sum())
        s_start, s_len, s_target = self.start[keep], self.length[keep], self.target[keep]

        # 2. invalid additions: empty, or reaching past the top of the 64-bit space at
        # either end (Python integers, so the sums cannot wrap)
        status = np.full(n_add, ADDED, np.uint8)
        for i, (s0, n, t0) in enumerate(zip(a_s.tolist(), a_l.tolist(), a_t.tolist())):
            if n == 0 or s0 + n > _TOP or t0 + n > _TOP:
                status[i] = INVALID
        valid = status == ADDED

        # 3. overlaps with survivors and with the other valid additions
        if valid.any():
            v_first = a_s[valid]
            v_last = v_first + (a_l[valid] - np.uint64(1))
            clash = overlap_counts(v_first, v_last, s_start, s_start + (s_len - np.uint64(1))) > 0
            # each valid addition meets itself once
            clash |= overlap_counts(v_first, v_last, v_first, v_last) > 1
            idx = np.flatnonzero(valid)
            status[idx[clash]] = OVERLAP
        take = status == ADDED
        n_take = int(take.sum())

        # 4. capacity: all or nothing
        if s_start.size + n_take > self.capacity:
            status[take] = FULL
            refused = int((status != ADDED).sum())
            return status, (len(self), 0, 0, refused)

        # 5. the new map, sorted by start
        start = np.concatenate([s_start, a_s[take]])
        order = np.argsort(start, kind="stable")
        self.start = start[order]
        self.length = np.concatenate([s_len, a_l[take]])[order]
        self.target = np.concatenate([s_target, a_t[take]])[order]
        return status, (len(self), n_take, n_removed, n_add - n_take)

    def translate(self, addrs) -> np.ndarray:
        """target + (p - start) for the interval holding p, else UNMAPPED."""
        p = _u64(addrs)
        out = np.full(p.size, UNMAPPED, np.uint64)
        if not len(self) or not p.size:
            return out
        # the last interval whose start is <= p is the only one that can hold p
        i = np.searchsorted(self.start, p, side="right") - 1
        ok = i >= 0
        j = np.where(ok, i, 0)
        inside = ok & (p - self.start[j] < self.length[j])
        out[inside] = self.target[j][inside] + (p[inside] - self.start[j][inside])
        return out

    def export(self):
        """The intervals in start order: (start, length, target)."""
        return self.start.copy(), self.length.copy(), self.target.copy()
