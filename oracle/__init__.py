"""Reference oracle for weight-cache hit detection.

TEST INFRASTRUCTURE ONLY. This package is the plain, slow, obviously correct CPU
definition of what the GPU library computes. Only the test suite, the package's
smoke check and the benchmark's CPU-baseline leg may import it; the GPU library
never does, and shares no code with it.

The method (Gleam, Sec. 4.1.2 "Hash-based Weight Chunk Retrieval"): the server
holds a set of hash identifiers of weight chunks it already has; each incoming
host-to-device payload is hashed from its source bytes, and only payloads whose
identifier is not in the set must send their bytes; a hit sends only the
identifier and size, and the server restores the bytes locally. Sec. 4.1.1 and
4.1.3 add that chunks later found to be weights are kept for reuse.

The oracle computes, per fixed-size block of each payload:
  geometry      -- blocks and leaves restart at every payload start
  digests       -- XXH64 (seed 0) per 4 KiB leaf, bottom-up pairwise tree per
                   block (gleam_oracle.c)
  lookup        -- HIT_CACHE if the digest is in the table (value = the table's);
                   else HIT_BATCH if an earlier block of the same batch has the
                   same digest (ref = the earliest such block); else MISS
  compaction    -- the ascending list of MISS blocks, their count and bytes
  insert        -- set semantics; an existing key is never overwritten; among
                   equal keys of one insert batch the lowest index's value wins

The fingerprint is C (gleam_oracle.c) because the oracle must digest tens of GB;
everything after it is numpy. remap.py holds the address-remap interval map of the
weight-sharing layer (Sec. 4.1.3; Appendix, Implementation Details, Virtual Memory Map).
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gleam_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

MISS, HIT_CACHE, HIT_BATCH = 0, 1, 2
LEAF_BYTES = 4096


def build() -> str:
    """Compile gleam_oracle.c into liboracle.so next to it (plain gcc, no SIMD flags)."""
    tmp = _LIB_PATH + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-shared", "-fPIC",
                           _SRC, "-o", tmp, "-lm"])
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    u64, u32, p = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p
    lib.oracle_xxh64.argtypes = [p, u64, u64]
    lib.oracle_xxh64.restype = u64
    lib.oracle_node.argtypes = [u64, u64]
    lib.oracle_node.restype = u64
    lib.oracle_tree.argtypes = [p, u64]
    lib.oracle_tree.restype = u64
    lib.oracle_blocks.argtypes = [p, u64, u32, u32, u64, u64, p, p]
    lib.oracle_blocks.restype = ctypes.c_int
    lib.oracle_md5.argtypes = [p, u64, p]
    lib.oracle_md5.restype = None
    _lib = lib
    return lib


def _as_u8(data) -> np.ndarray:
    if isinstance(data, (bytes, bytearray, memoryview)):
        return np.frombuffer(bytes(data), dtype=np.uint8)
    arr = np.ascontiguousarray(data)
    if arr.dtype != np.uint8:
        arr = arr.view(np.uint8).reshape(-1)
    return arr.reshape(-1)


# --------------------------------------------------------------------------- #
# Fingerprints (C)
# --------------------------------------------------------------------------- #
def xxh64(data, seed: int = 0) -> int:
    """XXH64 of `data` with `seed` (the xxHash specification's 64-bit algorithm)."""
    arr = _as_u8(data)
    return int(_load().oracle_xxh64(arr.ctypes.data if arr.size else None, arr.size, seed))


def node(left: int, right: int) -> int:
    """Tree node: XXH64(LE64(left) || LE64(right), seed 0). The paper hashes a chunk's
    bytes as its identifier (Sec. 4.1.2); folding leaf digests pairwise is this path's
    reading for blocks larger than one leaf."""
    return int(_load().oracle_node(left, right))


def tree(digests) -> int:
    """Block identifier from its leaf digests (Sec. 4.1.2 identifier, leaf-tree reading):
    bottom-up pairwise tree over >= 1 leaf digests; an odd last element moves up
    unchanged; a single leaf's digest is the block's."""
    work = np.array(digests, dtype=np.uint64)
    if work.size == 0:
        raise ValueError("a block has at least one leaf")
    return int(_load().oracle_tree(work.ctypes.data, work.size))


def num_blocks(length: int, block_bytes: int) -> int:
    return (int(length) + block_bytes - 1) // block_bytes


def payload_digests(payload, block_bytes: int, leaf_bytes: int = LEAF_BYTES,
                    with_leaves: bool = False, first_block: int = 0, count: int | None = None):
    """Block digests (and optionally padded leaf digests) of one payload: Sec. 4.1.1's
    payload (the bytes of one host-to-device copy) cut into blocks from its start, each
    identified by the hash of its bytes (Sec. 4.1.2).

    Returns (block_digests u64[count], leaf_digests u64[count, block/leaf] or None).
    """
    arr = _as_u8(payload)
    nblk = num_blocks(arr.size, block_bytes)
    if count is None:
        count = nblk - first_block
    blk = np.zeros(count, dtype=np.uint64)
    per = block_bytes // leaf_bytes
    leaves = np.zeros((count, per), dtype=np.uint64) if with_leaves else None
    if count:
        rc = _load().oracle_blocks(arr.ctypes.data, arr.size, leaf_bytes, block_bytes, first_block, count,
                                   blk.ctypes.data, leaves.ctypes.data if with_leaves else None)
        if rc != 0:
            raise ValueError(f"oracle_blocks failed with {rc}")
    return blk, leaves


def geometry(seg_lens, block_bytes: int):
    """Per-batch geometry: blk_first[S+1] (exclusive prefix of blocks per payload)
    and blk_len[n_blocks] (bytes of each block; only a payload's last block is short).
    Blocks restart at every payload start, since the decision is per host-to-device
    copy (Sec. 4.1.1, 4.1.2); a zero-length payload has no blocks."""
    lens = np.asarray(seg_lens, dtype=np.uint64).reshape(-1)
    nblk = [num_blocks(n, block_bytes) for n in lens.tolist()]
    blk_first = np.zeros(len(nblk) + 1, dtype=np.uint64)
    blk_first[1:] = np.cumsum(np.array(nblk, dtype=np.uint64))
    blk_len = np.full(int(blk_first[-1]), block_bytes, dtype=np.uint64)
    for s, n in enumerate(lens.tolist()):
        if nblk[s]:
            blk_len[int(blk_first[s + 1]) - 1] = n - (nblk[s] - 1) * block_bytes
    return blk_first, blk_len


def batch_digests(payloads, block_bytes: int, with_leaves: bool = False, threads: int = 1,
                  blocks_per_task: int | None = None):
    """Digests of every block of a batch, in batch order (payload-major, then offset).

    `threads` > 1 hands independent block ranges to a thread pool; each range is
    still one plain call of the oracle above.
    """
    lens = [int(_as_u8(p).size) for p in payloads]
    blk_first, _ = geometry(lens, block_bytes)
    n = int(blk_first[-1])
    per = block_bytes // LEAF_BYTES
    blk = np.zeros(n, dtype=np.uint64)
    leaves = np.zeros((n, per), dtype=np.uint64) if with_leaves else None
    if blocks_per_task is None:
        blocks_per_task = max(1, (64 << 20) // block_bytes)
    tasks = []
    for s, p in enumerate(payloads):
        nb = int(blk_first[s + 1] - blk_first[s])
        for j0 in range(0, nb, blocks_per_task):
            tasks.append((s, j0, min(blocks_per_task, nb - j0)))

    def run(task):
        s, j0, cnt = task
        b, lv = payload_digests(payloads[s], block_bytes, with_leaves=with_leaves, first_block=j0, count=cnt)
        g0 = int(blk_first[s]) + j0
        blk[g0:g0 + cnt] = b
        if with_leaves:
            leaves[g0:g0 + cnt] = lv

    if threads <= 1:
        for t in tasks:
            run(t)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(run, tasks))
    return blk, leaves


# --------------------------------------------------------------------------- #
# Table, lookup, compaction (numpy)
# --------------------------------------------------------------------------- #
class Table:
    """The server's identifier set: a map from u64 digest to u64 value, with a last-use
    stamp per entry for LRU eviction (Sec. 4.1.3).

    Every u64 is a valid key (no reserved value). New entries get stamp 0.
    """

    def __init__(self):
        self.keys = np.zeros(0, dtype=np.uint64)   # sorted
        self.vals = np.zeros(0, dtype=np.uint64)
        self.stamps = np.zeros(0, dtype=np.uint64)

    def __len__(self):
        return int(self.keys.size)

    def _set(self, k, v, t):
        order = np.argsort(k, kind="stable")
        self.keys, self.vals, self.stamps = k[order], v[order], t[order]

    def insert(self, keys, vals) -> int:
        """Sec. 4.1.2 and 4.1.3: identified chunks join the server's identifier set.
        Insert in batch order: a key already present keeps its value; among equal keys
        of this batch the lowest index wins (the paper is silent on both; these are the
        readings taken). Returns the number of new keys."""
        keys = np.asarray(keys, dtype=np.uint64).reshape(-1)
        vals = np.asarray(vals, dtype=np.uint64).reshape(-1)
        if keys.size != vals.size:
            raise ValueError("keys and vals differ in length")
        if keys.size == 0:
            return 0
        uniq, first = np.unique(keys, return_index=True)       # first = lowest index per key
        new = ~self.contains(uniq)
        add_k, add_v = uniq[new], vals[first[new]]
        self._set(np.concatenate([self.keys, add_k]), np.concatenate([self.vals, add_v]),
                  np.concatenate([self.stamps, np.zeros(add_k.size, np.uint64)]))
        return int(add_k.size)

    def contains(self, keys) -> np.ndarray:
        keys = np.asarray(keys, dtype=np.uint64).reshape(-1)
        if self.keys.size == 0:
            return np.zeros(keys.size, dtype=bool)
        pos = np.searchsorted(self.keys, keys)
        pos_c = np.minimum(pos, self.keys.size - 1)
        return (pos < self.keys.size) & (self.keys[pos_c] == keys)

    def get(self, keys) -> tuple[np.ndarray, np.ndarray]:
        """(present mask, value where present else 0)."""
        keys = np.asarray(keys, dtype=np.uint64).reshape(-1)
        present = self.contains(keys)
        out = np.zeros(keys.size, dtype=np.uint64)
        if present.any():
            out[present] = self.vals[np.searchsorted(self.keys, keys[present])]
        return present, out

    # -- lifecycle (Sec. 4.1.3: LRU eviction keeps the cache bounded) --------------- #
    def touch(self, keys, epochs) -> int:
        """Sec. 4.1.3 (LRU over the shared pool): record a use. Stamp present keys with
        max(stamp, epoch). Returns how many keys (with repetition) were present."""
        keys = np.asarray(keys, dtype=np.uint64).reshape(-1)
        epochs = np.broadcast_to(np.asarray(epochs, dtype=np.uint64), keys.shape)
        present = self.contains(keys)
        pos = np.searchsorted(self.keys, keys[present])
        np.maximum.at(self.stamps, pos, epochs[present])
        return int(present.sum())

    def evict(self, keep: int) -> np.ndarray:
        """Sec. 4.1.3 LRU eviction: keep the `keep` most recently used entries. Entries are
        ordered by (stamp, key) ascending (ties in last use: smaller key first, a reading)
        and the first len - keep are removed. Returns them in that order."""
        n_evict = max(0, len(self) - int(keep))
        order = np.lexsort((self.keys, self.stamps))   # primary: stamp, secondary: key
        gone = order[:n_evict]
        evicted = self.keys[gone].copy()
        mask = np.ones(len(self), dtype=bool)
        mask[gone] = False
        self.keys, self.vals, self.stamps = self.keys[mask], self.vals[mask], self.stamps[mask]
        return evicted

    def erase(self, keys) -> int:
        """Sec. 4.1.3: chunks leave the shared pool. Remove the given keys that are
        present. Returns how many entries went."""
        keys = np.unique(np.asarray(keys, dtype=np.uint64).reshape(-1))
        gone = self.contains(keys)
        mask = ~np.isin(self.keys, keys[gone])
        self.keys, self.vals, self.stamps = self.keys[mask], self.vals[mask], self.stamps[mask]
        return int(gone.sum())

    def export(self):
        """(keys, vals, stamps) sorted by key: the identifier set a server ships at
        connect time (Sec. 4.1.2), also a checkpoint of the table."""
        return self.keys.copy(), self.vals.copy(), self.stamps.copy()


def lookup(digests, table: Table):
    """status u8[n] and ref u64[n] for a batch of block digests (Sec. 4.1.2: a held
    identifier means only the identifier and size travel; any other chunk sends its
    bytes; the paper is silent on a chunk repeated inside one batch, and the reading
    taken is that only its earliest copy travels).

    HIT_CACHE (1): digest in the table; ref = its value.
    HIT_BATCH (2): otherwise, an earlier block g0 < g has the same digest; ref = the
                   smallest such g0 (itself a MISS).
    MISS (0):      otherwise; ref = g.
    The table is not modified.
    """
    d = np.asarray(digests, dtype=np.uint64).reshape(-1)
    n = d.size
    status = np.zeros(n, dtype=np.uint8)
    ref = np.zeros(n, dtype=np.uint64)
    if n == 0:
        return status, ref
    present, val = table.get(d)
    _, first, inverse = np.unique(d, return_index=True, return_inverse=True)
    g0 = first[inverse.reshape(-1)].astype(np.uint64)
    g = np.arange(n, dtype=np.uint64)
    status[present] = HIT_CACHE
    ref[present] = val[present]
    batch = ~present & (g0 < g)
    status[batch] = HIT_BATCH
    ref[batch] = g0[batch]
    miss = ~present & (g0 == g)
    ref[miss] = g[miss]
    return status, ref


def compact(status, blk_len=None):
    """The bytes that must still travel (Sec. 4.1.2: on a miss the full chunk is sent):
    ascending MISS block indices, their count, and (given blk_len) their total bytes."""
    st = np.asarray(status, dtype=np.uint8).reshape(-1)
    idx = np.flatnonzero(st == MISS).astype(np.uint64)
    nbytes = None
    if blk_len is not None:
        nbytes = int(np.asarray(blk_len, dtype=np.uint64)[idx].sum(dtype=np.uint64))
    return idx, int(idx.size), nbytes


def run(payloads, block_bytes: int, table: Table, threads: int = 1):
    """The whole decision of Sec. 4.1.2 for one batch: digests -> lookup -> compaction."""
    digests, _ = batch_digests(payloads, block_bytes, threads=threads)
    _, blk_len = geometry([_as_u8(p).size for p in payloads], block_bytes)
    status, ref = lookup(digests, table)
    miss_idx, miss_count, miss_bytes = compact(status, blk_len)
    return {"digests": digests, "status": status, "ref": ref, "miss_idx": miss_idx,
            "miss_count": miss_count, "miss_bytes": miss_bytes}


# --------------------------------------------------------------------------- #
# Weight identification at free time (Sec. 4.1.1)
# --------------------------------------------------------------------------- #
NO_DIFF = 2**64 - 1


def identify_weights(recorded_digests, current_payloads, block_bytes: int, region_first, threads: int = 1):
    """Sec. 4.1.1: an allocation ("block" in the paper) holds weights only if every
    payload recorded at its first host-to-device write still has the same bytes when
    the allocation is freed. The recorded payloads are compared block by block through
    their digests: recorded at write time vs. computed now from the current bytes.

    recorded_digests : u64[n_blocks] block digests of the payloads as written
    current_payloads : the same payloads' current bytes (same lengths)
    region_first     : u64[R+1]; payloads of allocation r are [region_first[r], region_first[r+1])

    Returns (block_match u8[n_blocks], first_diff u64[S] = index within the payload of
    its first differing block or 2^64-1, region_weight u8[R]); an allocation with no
    recorded payload is not identified as weights.
    """
    rec = np.asarray(recorded_digests, dtype=np.uint64).reshape(-1)
    cur, _ = batch_digests(current_payloads, block_bytes, threads=threads)
    if cur.size != rec.size:
        raise ValueError("recorded digests do not match the payloads' geometry")
    block_match = (cur == rec).astype(np.uint8)
    lens = [_as_u8(p).size for p in current_payloads]
    blk_first, _ = geometry(lens, block_bytes)
    first_diff = np.full(len(lens), NO_DIFF, dtype=np.uint64)
    for s in range(len(lens)):
        bad = np.flatnonzero(block_match[int(blk_first[s]):int(blk_first[s + 1])] == 0)
        if bad.size:
            first_diff[s] = bad[0]
    rf = np.asarray(region_first, dtype=np.uint64).reshape(-1)
    region_weight = np.zeros(rf.size - 1, dtype=np.uint8)
    for r in range(rf.size - 1):
        segs = first_diff[int(rf[r]):int(rf[r + 1])]
        region_weight[r] = 1 if segs.size and (segs == NO_DIFF).all() else 0
    return block_match, first_diff, region_weight


def identify_leaves(recorded_leaf_digests, current_payloads, block_bytes: int, region_first, threads: int = 1):
    """identify_weights at leaf granularity (Sec. 4.1.1's consistency check, located to
    the first 4 KiB leaf that changed). The recorded leaf digests are laid out as
    batch_digests(with_leaves=True) gives them: u64[n_blocks, block/leaf], slots past a
    short block's last leaf 0.

    Returns (leaf_match u8[n_blocks * block/leaf]: 1 where the recorded and current slot
    agree, slots without a leaf included; first_diff_leaf u64[S] = index within the
    payload of its first changed leaf or 2^64-1; region_weight u8[R] as in
    identify_weights)."""
    rec = np.asarray(recorded_leaf_digests, dtype=np.uint64).reshape(-1)
    _, cur = batch_digests(current_payloads, block_bytes, with_leaves=True, threads=threads)
    cur = cur.reshape(-1)
    if cur.size != rec.size:
        raise ValueError("recorded leaf digests do not match the payloads' geometry")
    leaf_match = (cur == rec).astype(np.uint8)
    per = block_bytes // LEAF_BYTES
    lens = [_as_u8(p).size for p in current_payloads]
    blk_first, _ = geometry(lens, block_bytes)
    first_diff = np.full(len(lens), NO_DIFF, dtype=np.uint64)
    for s in range(len(lens)):
        # slot order within a payload is leaf order: block-major, then leaf
        bad = np.flatnonzero(leaf_match[int(blk_first[s]) * per:int(blk_first[s + 1]) * per] == 0)
        if bad.size:
            first_diff[s] = bad[0]
    rf = np.asarray(region_first, dtype=np.uint64).reshape(-1)
    region_weight = np.zeros(rf.size - 1, dtype=np.uint8)
    for r in range(rf.size - 1):
        segs = first_diff[int(rf[r]):int(rf[r + 1])]
        region_weight[r] = 1 if segs.size and (segs == NO_DIFF).all() else 0
    return leaf_match, first_diff, region_weight


FW_OK, FW_TOO_MANY, FW_INVALID = 0, 1, 2
_TOP64 = (1 << 64) - 1


def first_write_pieces(addr, length, region_first, max_writes: int | None = None):
    """Sec. 4.1.1: where an address range is written several times, only the first
    host-to-device write counts. Writes are listed in time order; the writes of
    allocation r are [region_first[r], region_first[r+1]). A write owns the bytes of
    [addr, addr + len) that no earlier write of its allocation covers; a piece is a
    maximal run of bytes owned by one write.

    Returns (piece_write u64[P], piece_offset u64[P] (from the write's start),
    piece_len u64[P], region_piece_first u64[R+1], region_status u8[R]), pieces ordered
    by allocation, then write, then address. An allocation with a write reaching past
    the top of the 64-bit address space (addr + len > 2^64 - 1) is refused
    (FW_INVALID, no pieces); with max_writes given, so is one with more writes than
    that (FW_TOO_MANY).
    """
    a = [int(x) for x in np.asarray(addr, dtype=np.uint64).reshape(-1)]
    n = [int(x) for x in np.asarray(length, dtype=np.uint64).reshape(-1)]
    rf = [int(x) for x in np.asarray(region_first, dtype=np.uint64).reshape(-1)]
    pw, po, pl = [], [], []
    first = [0]
    status = []
    for r in range(len(rf) - 1):
        w0, w1 = rf[r], rf[r + 1]
        if any(a[j] + n[j] > _TOP64 for j in range(w0, w1)):
            status.append(FW_INVALID)
            first.append(len(pw))
            continue
        if max_writes is not None and w1 - w0 > max_writes:
            status.append(FW_TOO_MANY)
            first.append(len(pw))
            continue
        covered = []  # the union of the earlier writes: sorted, disjoint [lo, hi)
        for j in range(w0, w1):
            lo, hi = a[j], a[j] + n[j]
            if lo == hi:
                continue
            # the gaps of `covered` inside [lo, hi), in address order
            at = lo
            for c_lo, c_hi in covered:
                if c_hi <= at or c_lo >= hi:
                    continue
                if c_lo > at:
                    pw.append(j), po.append(at - lo), pl.append(c_lo - at)
                at = max(at, c_hi)
            if at < hi:
                pw.append(j), po.append(at - lo), pl.append(hi - at)
            # merge [lo, hi) into the union
            merged = []
            for c_lo, c_hi in covered:
                if c_hi < lo or c_lo > hi:
                    merged.append((c_lo, c_hi))
                else:
                    lo, hi = min(lo, c_lo), max(hi, c_hi)
            merged.append((lo, hi))
            covered = sorted(merged)
        status.append(FW_OK)
        first.append(len(pw))
    u = lambda v: np.array(v, dtype=np.uint64)
    return u(pw), u(po), u(pl), u(first), np.array(status, dtype=np.uint8)


# --------------------------------------------------------------------------- #
# The paper's identifier: MD5 of a payload's first 1024 bits (Appendix discussion)
# --------------------------------------------------------------------------- #
def md5(data) -> bytes:
    """MD5 (RFC 1321) of `data`."""
    arr = _as_u8(data)
    out = np.zeros(16, dtype=np.uint8)
    _load().oracle_md5(arr.ctypes.data if arr.size else None, arr.size, out.ctypes.data)
    return out.tobytes()


def md5_prefix(payloads, prefix_bytes: int = 128, min_len: int = 1024):
    """Per payload: MD5 of its first min(len, prefix_bytes) bytes (u8[S, 16]), the table
    key = the digest's first 8 bytes as a little-endian u64, and whether the paper would
    build a cache entry for it (only payloads longer than min_len bytes)."""
    S = len(payloads)
    digests = np.zeros((S, 16), dtype=np.uint8)
    eligible = np.zeros(S, dtype=np.uint8)
    for s, p in enumerate(payloads):
        arr = _as_u8(p)
        digests[s] = np.frombuffer(md5(arr[:prefix_bytes]), np.uint8)
        eligible[s] = 1 if arr.size > min_len else 0
    keys = digests[:, :8].copy().view("<u8").reshape(-1).astype(np.uint64)
    return digests, keys, eligible


# --------------------------------------------------------------------------- #
# Sender-side plan, packing and the receiver's restore (Sec. 4.1.2)
# --------------------------------------------------------------------------- #
PLAN_DTYPE = np.dtype([("block", "<u8"), ("payload", "<u8"), ("offset", "<u8"), ("ident", "<u8"),
                       ("length", "<u4"), ("kind", "<u4")])


def _round16(n: int) -> int:
    return (int(n) + 15) // 16 * 16


def send_plan(payload_lens, block_bytes: int, digests, status, ref):
    """Sec. 4.1.2: a block whose identifier the server holds sends (hash, size); a block
    repeating an earlier block of the batch sends (that block, size); any other block
    sends its bytes. One record per block, in batch order:
        kind MISS      -> ident = offset of its bytes in the packed send buffer, where
                          every block starts at a multiple of 16 bytes
        kind HIT_CACHE -> ident = the block digest
        kind HIT_BATCH -> ident = the earlier block's index
    Returns (records, totals = [miss blocks, cache-hit blocks, batch-hit blocks, packed bytes])."""
    blk_first, blk_len = geometry(payload_lens, block_bytes)
    n = int(blk_first[-1])
    digests = np.asarray(digests, dtype=np.uint64).reshape(-1)
    status = np.asarray(status, dtype=np.uint8).reshape(-1)
    ref = np.asarray(ref, dtype=np.uint64).reshape(-1)
    rec = np.zeros(n, dtype=PLAN_DTYPE)
    packed = 0
    for s in range(len(payload_lens)):
        for j in range(int(blk_first[s + 1] - blk_first[s])):
            gidx = int(blk_first[s]) + j
            r = rec[gidx]
            r["block"], r["payload"], r["offset"] = gidx, s, j * block_bytes
            r["length"], r["kind"] = int(blk_len[gidx]), int(status[gidx])
            if status[gidx] == MISS:
                r["ident"] = packed
                packed += _round16(blk_len[gidx])
            elif status[gidx] == HIT_CACHE:
                r["ident"] = digests[gidx]
            else:
                r["ident"] = ref[gidx]
            rec[gidx] = r
    totals = np.array([(status == MISS).sum(), (status == HIT_CACHE).sum(), (status == HIT_BATCH).sum(), packed],
                      dtype=np.uint64)
    return rec, totals


def pack_misses(payloads, records, packed_bytes: int) -> np.ndarray:
    """The send buffer: every MISS block's bytes at its planned offset (zero padding)."""
    out = np.zeros(int(packed_bytes), dtype=np.uint8)
    for r in records[records["kind"] == MISS]:
        p = _as_u8(payloads[int(r["payload"])])
        o, ln = int(r["offset"]), int(r["length"])
        out[int(r["ident"]):int(r["ident"]) + ln] = p[o:o + ln]
    return out
