"""The oracle's leaf fingerprint (XXH64, seed 0) pinned to values from outside it.

Pins: the published XXH64 vectors in tests/golden/xxh64_published.txt, and the
installed `xxhash` package (an independent implementation the oracle does not
call) on every tail path: lengths 0..129 cover the <32-byte branch and every
mix of 8-, 4- and 1-byte tail steps; 4095/4096/4097 the leaf edges.
"""

import os

import numpy as np
import pytest
import xxhash

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "xxh64_published.txt")


def _published():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            text, seed, digest, _src = line.rstrip("\n").split("\t")
            rows.append((text.strip('"').encode(), int(seed), int(digest, 16)))
    return rows


@pytest.mark.parametrize("data,seed,expected", _published())
def test_published_vectors(data, seed, expected):
    assert oracle.xxh64(data, seed) == expected


@pytest.mark.parametrize("seed", [0, 1, 2**64 - 1])
def test_all_tail_paths_against_library(seed):
    rng = np.random.default_rng(11)
    for n in list(range(0, 130)) + [255, 256, 1000, 4095, 4096, 4097, 65536]:
        data = rng.bytes(n)
        assert oracle.xxh64(data, seed) == xxhash.xxh64_intdigest(data, seed), n


def test_random_lengths_against_library():
    rng = np.random.default_rng(12)
    for _ in range(300):
        n = int(rng.integers(0, 8193))
        data = rng.bytes(n)
        assert oracle.xxh64(data) == xxhash.xxh64_intdigest(data), n


def test_single_bit_flip_changes_digest():
    rng = np.random.default_rng(13)
    base = bytearray(rng.bytes(4096))
    d0 = oracle.xxh64(bytes(base))
    for pos in (0, 1, 7, 31, 32, 2047, 4095):
        for bit in (0, 7):
            b = bytearray(base)
            b[pos] ^= 1 << bit
            assert oracle.xxh64(bytes(b)) != d0


def test_planted_mistake_is_caught():
    """A dropped tail step (a plausible bug) must disagree with the library."""
    data = bytes(range(37))  # 32-byte stripe + 4-byte word + 1 byte
    good = xxhash.xxh64_intdigest(data)
    assert oracle.xxh64(data) == good
    assert oracle.xxh64(data[:36]) != good
