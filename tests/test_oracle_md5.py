"""The oracle's MD5 (the paper's identifier: MD5 of a chunk's first 1024 bits,
Appendix discussion) pinned to the RFC 1321 test suite and to Python's hashlib
(an independent implementation the oracle never calls), over every padding case."""

import hashlib
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "md5_rfc1321.txt")


def _suite():
    rows = []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        text, digest = line.rstrip("\n").split("\t")
        rows.append((text.strip('"').encode(), digest))
    return rows


@pytest.mark.parametrize("data,digest", _suite())
def test_rfc1321_suite(data, digest):
    assert oracle.md5(data).hex() == digest


def test_every_padding_case_against_hashlib():
    rng = np.random.default_rng(61)
    for n in list(range(0, 200)) + [1000, 4096, 65537]:
        data = rng.bytes(n)
        assert oracle.md5(data) == hashlib.md5(data).digest(), n


def test_prefix_keys_and_eligibility():
    rng = np.random.default_rng(62)
    payloads = [np.frombuffer(rng.bytes(n), np.uint8) for n in (0, 5, 128, 129, 1024, 1025, 5000)]
    d, keys, elig = oracle.md5_prefix(payloads)
    for i, p in enumerate(payloads):
        h = hashlib.md5(p[:128].tobytes()).digest()
        assert d[i].tobytes() == h
        assert int(keys[i]) == int.from_bytes(h[:8], "little")
    assert elig.tolist() == [0, 0, 0, 0, 0, 1, 1]
    # a payload that differs only after its first 128 bytes has the same prefix identifier
    a = payloads[-1].copy()
    b = a.copy()
    b[4000] ^= 1
    da, _, _ = oracle.md5_prefix([a, b])
    assert da[0].tobytes() == da[1].tobytes()
    assert oracle.payload_digests(a, 4096)[0][0] != oracle.payload_digests(b, 4096)[0][0]
