"""The oracle's block digest (leaf split + bottom-up pairwise tree) pinned from outside.

Pins:
  * the node function equals the library's XXH64 of the 16-byte little-endian pair;
  * the bottom-up rule (odd last element promoted) equals the recursive
    largest-power-of-two split of RFC 6962 section 2.1 for every n up to 300 --
    a different formulation, written here with the library's hash, so a wrong
    pairing order or promotion rule in the oracle shows up;
  * closed forms for one to five leaves;
  * whole payloads against a pure-Python split + recursive tree (library hash),
    over partial leaves, partial blocks and several block sizes;
  * invariants: equal bytes give equal digests; a flipped bit, or two leaves
    swapped, change the block digest.
"""

import struct

import numpy as np
import pytest
import xxhash

import oracle


def lib_node(a, b):
    return xxhash.xxh64_intdigest(struct.pack("<QQ", a, b))


def split_tree(d):
    """RFC 6962-style: left subtree = the largest power of two strictly below n."""
    n = len(d)
    if n == 1:
        return d[0]
    k = 1
    while k * 2 < n:
        k *= 2
    return lib_node(split_tree(d[:k]), split_tree(d[k:]))


def ref_payload(payload: bytes, block: int, leaf: int = 4096):
    out = []
    for b0 in range(0, len(payload), block):
        blk = payload[b0:b0 + block]
        leaves = [xxhash.xxh64_intdigest(blk[l0:l0 + leaf]) for l0 in range(0, len(blk), leaf)]
        out.append(split_tree(leaves))
    return out


@pytest.mark.parametrize("a,b", [(0, 0), (1, 2), (2, 1), (2**64 - 1, 0), (0x0123456789ABCDEF, 2**63)])
def test_node_is_hash_of_le_pair(a, b):
    assert oracle.node(a, b) == lib_node(a, b)


def test_node_order_matters():
    assert oracle.node(1, 2) != oracle.node(2, 1)


def test_bottom_up_equals_recursive_split():
    rng = np.random.default_rng(21)
    for n in range(1, 301):
        d = [int(x) for x in rng.integers(0, 2**64, size=n, dtype=np.uint64)]
        assert oracle.tree(d) == split_tree(d), n


def test_closed_forms():
    l = [0x1111, 0x2222, 0x3333, 0x4444, 0x5555]
    n = lib_node
    assert oracle.tree(l[:1]) == l[0]
    assert oracle.tree(l[:2]) == n(l[0], l[1])
    assert oracle.tree(l[:3]) == n(n(l[0], l[1]), l[2])
    assert oracle.tree(l[:4]) == n(n(l[0], l[1]), n(l[2], l[3]))
    assert oracle.tree(l[:5]) == n(n(n(l[0], l[1]), n(l[2], l[3])), l[4])


@pytest.mark.parametrize("block", [4096, 65536, 1 << 20, 2 << 20])
def test_payloads_against_pure_python(block):
    rng = np.random.default_rng(22 + block)
    lengths = [0, 1, 100, 4095, 4096, 4097, 8292, block - 1, block, block + 1, 3 * block + 777]
    for ln in lengths:
        data = rng.bytes(ln)
        got, _ = oracle.payload_digests(np.frombuffer(data, np.uint8), block)
        assert [int(x) for x in got] == ref_payload(data, block), (block, ln)


def test_leaf_digest_padding():
    rng = np.random.default_rng(23)
    data = np.frombuffer(rng.bytes(65536 + 5000), np.uint8)
    blk, leaves = oracle.payload_digests(data, 65536, with_leaves=True)
    assert leaves.shape == (2, 16)
    assert int(leaves[1, 0]) == xxhash.xxh64_intdigest(data[65536:65536 + 4096].tobytes())
    assert int(leaves[1, 1]) == xxhash.xxh64_intdigest(data[65536 + 4096:].tobytes())
    assert not leaves[1, 2:].any()
    assert int(blk[1]) == lib_node(int(leaves[1, 0]), int(leaves[1, 1]))


def test_invariants():
    rng = np.random.default_rng(24)
    a = np.frombuffer(rng.bytes(1 << 20), np.uint8).copy()
    d, _ = oracle.payload_digests(a, 1 << 20)
    d2, _ = oracle.payload_digests(a.copy(), 1 << 20)
    assert d[0] == d2[0]
    b = a.copy()
    b[123457] ^= 0x10
    assert oracle.payload_digests(b, 1 << 20)[0][0] != d[0]
    c = a.copy()
    c[0:4096], c[4096:8192] = a[4096:8192], a[0:4096]
    assert oracle.payload_digests(c, 1 << 20)[0][0] != d[0]


def test_one_leaf_block_is_leaf_digest():
    rng = np.random.default_rng(25)
    data = np.frombuffer(rng.bytes(3 * 4096 + 17), np.uint8)
    blk, _ = oracle.payload_digests(data, 4096)
    for j in range(4):
        assert int(blk[j]) == xxhash.xxh64_intdigest(data[j * 4096:(j + 1) * 4096].tobytes())
