"""The oracle's table lifecycle (Sec. 4.1.3: LRU eviction of the shared cache) pinned
against a plain dict simulation written directly from the rules: new entries start at
stamp 0, a touch raises a present key's stamp to the epoch, eviction drops the entries
with the smallest (stamp, key), erase drops the named keys, export is key order."""

import numpy as np

import oracle


class DictLRU:
    def __init__(self):
        self.d = {}

    def insert(self, keys, vals):
        new = 0
        for k, v in zip(keys.tolist(), vals.tolist()):
            if k not in self.d:
                self.d[k] = [v, 0]
                new += 1
        return new

    def touch(self, keys, epochs):
        hit = 0
        for k, e in zip(keys.tolist(), epochs.tolist()):
            if k in self.d:
                self.d[k][1] = max(self.d[k][1], e)
                hit += 1
        return hit

    def evict(self, keep):
        order = sorted(self.d, key=lambda k: (self.d[k][1], k))
        gone = order[:max(0, len(order) - keep)]
        for k in gone:
            del self.d[k]
        return gone

    def erase(self, keys):
        n = 0
        for k in set(keys.tolist()):
            if k in self.d:
                del self.d[k]
                n += 1
        return n


def test_lifecycle_against_dict():
    rng = np.random.default_rng(71)
    t, ref = oracle.Table(), DictLRU()
    special = np.array([0, 2**64 - 1], np.uint64)
    for step in range(60):
        op = step % 4
        if op == 0:
            keys = np.concatenate([rng.integers(0, 400, 50, dtype=np.uint64), special[rng.integers(0, 2, 2)]])
            vals = rng.integers(0, 2**63, keys.size, dtype=np.uint64)
            assert t.insert(keys, vals) == ref.insert(keys, vals)
        elif op == 1:
            keys = rng.integers(0, 450, 80, dtype=np.uint64)
            epochs = rng.integers(1, 1000, keys.size, dtype=np.uint64)
            assert t.touch(keys, epochs) == ref.touch(keys, epochs)
        elif op == 2 and step % 8 == 2:
            keep = int(rng.integers(0, len(ref.d) + 5))
            assert t.evict(keep).tolist() == ref.evict(keep)
        else:
            keys = rng.integers(0, 450, 30, dtype=np.uint64)
            assert t.erase(keys) == ref.erase(keys)
        k, v, st = t.export()
        assert k.tolist() == sorted(ref.d)
        assert v.tolist() == [ref.d[x][0] for x in sorted(ref.d)]
        assert st.tolist() == [ref.d[x][1] for x in sorted(ref.d)]
