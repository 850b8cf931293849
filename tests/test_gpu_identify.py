"""GPU parity of free-time weight identification (Sec. 4.1.1): block matches, each
payload's first changed block and each allocation's verdict equal the oracle's, and
the byte-level truth (which payloads were changed after being written)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23115_amd as g
import workloads as W
from gpu_util import host_threads, keys_to_device, say, to_device, u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def run_identify(arena, offs, lens, block, recorded, region_first):
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    m, f, w = g.identify_weights(batch, keys_to_device(recorded), region_first)
    torch.cuda.synchronize()
    return m.cpu().numpy(), u64(f), w.cpu().numpy()


@pytest.mark.parametrize("block", [4096, 65536, 1 << 20, 2 << 20])
def test_identify_random_regions(block):
    rng = np.random.default_rng(800 + block.bit_length())
    lens = [int(x) for x in rng.integers(0, 4 * block, 60)] + [0, 1, 4096, block]
    rng.shuffle(lens)
    written = [np.frombuffer(rng.bytes(n), np.uint8).copy() for n in lens]
    current = [w.copy() for w in written]
    changed = set()
    for i, c in enumerate(current):
        if c.size and rng.random() < 0.25:  # in-place updates after the write
            for _ in range(int(rng.integers(1, 4))):
                c[int(rng.integers(0, c.size))] ^= 1 << int(rng.integers(0, 8))
            changed.add(i)
    cuts = sorted(set(int(x) for x in rng.integers(0, len(lens) + 1, 12)))
    region_first = np.array([0] + cuts + [len(lens)], np.uint64)
    recorded, _ = oracle.batch_digests(written, block)
    arena, offs, lens_a = W.pack(current)
    say("identify block", block, "payloads", len(lens), "regions", region_first.size - 1)
    m, f, w = run_identify(arena, offs, lens_a, block, recorded, region_first)
    em, ef, ew = oracle.identify_weights(recorded, current, block, region_first)
    assert np.array_equal(m, em) and np.array_equal(f, ef) and np.array_equal(w, ew)
    # byte-level truth: a payload shows a difference iff it was changed
    assert {i for i in range(len(lens)) if f[i] != oracle.NO_DIFF} == {i for i in changed if current[i].size}


def test_identify_unaligned_and_empty_regions():
    rng = np.random.default_rng(850)
    block = 65536
    written = [np.frombuffer(rng.bytes(int(n)), np.uint8).copy() for n in rng.integers(1, 200000, 30)]
    current = [w.copy() for w in written]
    current[4][100] ^= 1
    current[17][-1] ^= 0x80
    region_first = np.array([0, 0, 5, 5, 12, 20, 30, 30], np.uint64)
    recorded, _ = oracle.batch_digests(written, block)
    arena, offs, lens = W.pack(current, skew=3)
    say("identify unaligned")
    m, f, w = run_identify(arena, offs, lens, block, recorded, region_first)
    em, ef, ew = oracle.identify_weights(recorded, current, block, region_first)
    assert np.array_equal(m, em) and np.array_equal(f, ef) and np.array_equal(w, ew)
    assert w.tolist() == [0, 0, 0, 1, 0, 1, 0]


@pytest.mark.timeout(900)
def test_identify_decoder7b_full():
    """Allocations = embedding, each layer, head; the payload is the base weights as
    written, the device holds the rank-16-updated layers: exactly those 3 layers'
    allocations are not weights, and every block of their 7 matrices changed."""
    threads = host_threads()
    dec = W.Decoder()
    block = W.DECODER_BLOCK
    say("identify decoder7b generate")
    arena, offs, lens = dec.arena(perturbed=True, threads=threads)
    current = [arena[int(o):int(o) + int(n)] for o, n in zip(offs, lens)]
    recorded, _ = oracle.batch_digests(current, block, threads=threads)
    first = oracle.geometry(lens, block)[0]
    for i in dec.perturbed:
        bd, _ = oracle.payload_digests(dec.base(i), block)
        recorded[int(first[i]):int(first[i + 1])] = bd
    # allocation boundaries: [embed], [layer l tensors] x 32, [final norm, lm head]
    region_first = np.array([0] + [1 + 9 * l for l in range(33)] + [len(lens)], np.uint64)
    say("identify decoder7b gpu", int(lens.sum()), "bytes")
    m, f, w = run_identify(arena, offs, lens, block, recorded, region_first)
    em, ef, ew = oracle.identify_weights(recorded, current, block, region_first, threads=threads)
    assert np.array_equal(m, em) and np.array_equal(f, ef) and np.array_equal(w, ew)
    bad_regions = {int(l) + 1 for l in dec.perturbed_layers}
    assert {r for r in range(w.size) if w[r] == 0} == bad_regions
    assert all(f[i] == 0 for i in dec.perturbed)


@pytest.mark.parametrize("block", [4096, 1 << 20])
def test_identify_payloads_changed_throughout(block):
    """Payloads whose every leaf changed (a layer rewritten in place) next to unchanged and
    partly changed ones, payload boundaries inside waves: leaf matches, first changed
    leaves and verdicts equal the oracle's; and a 256 MiB payload changed throughout is
    compared within a small multiple of the time of an unchanged one (with one atomic per
    changed leaf on the payload's word it took 15x as long)."""
    rng = np.random.default_rng(9100 + block.bit_length())
    lens = [3 << 20, 5000, 1 << 20, 4096, 777, 2 << 20]
    written = [np.frombuffer(rng.bytes(n), np.uint8).copy() for n in lens]
    current = [np.frombuffer(rng.bytes(n), np.uint8).copy() if i % 2 == 0 else w.copy()
               for i, (n, w) in enumerate(zip(lens, written))]
    current[3][100] ^= 1
    region_first = np.array([0, 2, 4, len(lens)], np.uint64)
    _, rec = oracle.batch_digests(written, block, with_leaves=True)
    arena, offs, lens_a = W.pack(current)
    batch = g.Batch.from_arena(to_device(arena), offs, lens_a, block)
    say("identify changed throughout", block)
    m, f, w = g.identify_leaves(batch, keys_to_device(rec.reshape(-1)), region_first)
    torch.cuda.synchronize()
    em, ef, ew = oracle.identify_leaves(rec, current, block, region_first)
    assert np.array_equal(m.cpu().numpy(), em)
    assert np.array_equal(u64(f), ef)
    assert np.array_equal(w.cpu().numpy(), ew)
    if block != 4096:
        return
    big = torch.randint(0, 256, (256 << 20,), dtype=torch.uint8, device="cuda")
    other = torch.randint(0, 256, (256 << 20,), dtype=torch.uint8, device="cuda")
    cur = g.Batch.from_arena(big, [0], [big.numel()], block)
    times = {}
    for label, src in (("changed", other), ("same", big)):
        rb = g.Batch.from_arena(src, [0], [src.numel()], block)
        leaves = torch.empty(rb.n_blocks * rb.leaves_per_block, dtype=torch.int64, device="cuda")
        g.fp_chunks(rb, leaf_out=leaves)
        ws = g.workspace(leaves.numel() + 1)
        for _ in range(3):
            g.identify_leaves(cur, leaves, [0, 1], ws=ws)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(5):
            g.identify_leaves(cur, leaves, [0, 1], ws=ws)
        b.record()
        torch.cuda.synchronize()
        times[label] = a.elapsed_time(b) / 5
    assert times["changed"] < 3 * times["same"] + 0.05, times
