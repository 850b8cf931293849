"""GPU parity of the rest of free-time weight identification (Sec. 4.1.1):

- gleam_first_writes: the pieces each recorded write owns (only the first write of an
  address counts) equal the oracle's, piece for piece, with the per-allocation starts
  and statuses, including the limits (2,048 writes per allocation, the top of the
  address space);
- the whole first-write check on the GPU: the pieces digested from the payloads as they
  land, then from the allocations at free time, decide weights exactly as painting every
  written byte with its first writer does;
- gleam_identify_leaves: leaf matches, each payload's first changed leaf and the
  allocations' verdicts equal the oracle's (at the full 7B-decoder size too)."""

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


def gpu_pieces(addr, length, region_first):
    pw, po, pl, first, status = g.first_writes(np.asarray(addr, np.uint64), np.asarray(length, np.uint64),
                                               np.asarray(region_first, np.uint64))
    torch.cuda.synchronize()
    first = u64(first)
    n = int(first[-1])
    return u64(pw)[:n], u64(po)[:n], u64(pl)[:n], first, status.cpu().numpy()


def check_pieces(addr, length, region_first, what):
    got = gpu_pieces(addr, length, region_first)
    want = oracle.first_write_pieces(addr, length, region_first, max_writes=2048)
    for a, b, name in zip(got, want, ("write", "offset", "length", "region first", "status")):
        assert np.array_equal(a, b), f"{what}: {name} differs"
    return got


def random_log(rng, n_regions, max_writes, span):
    addr, length, rf = [], [], [0]
    for _ in range(n_regions):
        k = int(rng.integers(0, max_writes + 1))
        base = int(rng.integers(0, 2**40)) << 12
        for _ in range(k):
            u = rng.random()
            if u < 0.05:
                addr.append(base + int(rng.integers(0, span))), length.append(0)
            elif u < 0.15 and len(addr) > rf[-1]:  # repeat an earlier write of this allocation
                j = int(rng.integers(rf[-1], len(addr)))
                addr.append(addr[j]), length.append(length[j])
            else:
                lo = int(rng.integers(0, span))
                addr.append(base + lo), length.append(int(rng.integers(1, max(2, span // 4))))
        rf.append(len(addr))
    return addr, length, rf


@pytest.mark.parametrize("seed,n_regions,max_writes,span", [(0, 1, 8, 100), (1, 50, 20, 1000), (2, 300, 60, 1 << 20),
                                                             (3, 20, 400, 5000), (4, 4, 2048, 1 << 16),
                                                             (5, 4097, 3, 1000), (6, 70_000, 2, 100)])
def test_pieces_random_logs(seed, n_regions, max_writes, span):
    rng = np.random.default_rng(7000 + seed)
    addr, length, rf = random_log(rng, n_regions, max_writes, span)
    say("first writes", seed, "writes", len(addr), "allocations", n_regions)
    check_pieces(addr, length, rf, f"seed {seed}")


def test_pieces_one_wave_boundary():
    """Allocations of 63, 64 and 65 writes (64 is the most a one-wave workgroup takes), each
    also with a write past the top of the address space, between small ones."""
    rng = np.random.default_rng(7100)
    addr, length, rf = [], [], [0]
    for k in (63, 64, 65, 1, 64, 65, 0, 63):
        for bad in (False, True):
            base = int(rng.integers(0, 2**40)) << 12
            for j in range(k):
                addr.append(base + int(rng.integers(0, 3000))), length.append(int(rng.integers(0, 700)))
            if bad and k:
                addr[-1], length[-1] = 2**64 - 5, 5 + int(rng.integers(1, 4))
            rf.append(len(addr))
    say("first writes one-wave boundary", "writes", len(addr))
    *_, status = check_pieces(addr, length, rf, "one-wave boundary")
    assert status.tolist() == [g.FW_OK, g.FW_INVALID] * 6 + [g.FW_OK, g.FW_OK, g.FW_OK, g.FW_INVALID]


def test_pieces_one_wave_shapes():
    """Allocations of at most 64 writes in the shapes that stress the one-wave pass: 64
    nested writes (each one byte wider on the left), 64 identical writes, 64 touching
    writes end to start, 64 zero-length writes at one address, zero-length writes at the
    ends of others, writes growing and then shrinking around one point, and a write at the
    top of the address space."""
    top = 2**64 - 1
    logs = [
        ([1000 - j for j in range(64)], [100 + j for j in range(64)]),
        ([5000] * 64, [300] * 64),
        ([10_000 + 7 * j for j in range(64)], [7] * 64),
        ([777] * 64, [0] * 64),
        ([100, 100, 200, 200, 150], [100, 0, 0, 50, 0]),
        ([500 - j for j in range(32)] + [470 + j for j in range(32)], [2 * j + 1 for j in range(32)] + [40 - j for j in range(32)]),
        ([top - 100, top - 50, top - 100], [100, 50, 10]),
    ]
    addr, length, rf = [], [], [0]
    for a, l in logs:
        addr += a
        length += l
        rf.append(len(addr))
    say("first writes one-wave shapes")
    *_, status = check_pieces(addr, length, rf, "one-wave shapes")
    assert (status == g.FW_OK).all()


def test_pieces_wide_address_spans():
    """Allocations whose writes do not share their top 7 address bits (spread over the
    whole 64-bit space, or straddling a multiple of 2^57), of one wave's size and larger,
    beside ones that do."""
    rng = np.random.default_rng(7500)
    addr, length, rf = [], [], [0]
    for k in (1, 5, 40, 64, 100, 64, 30):
        for kind in ("spread", "straddle", "narrow"):
            for _ in range(k):
                if kind == "spread":
                    a = int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2))
                    n = int(rng.integers(0, min(2**62, 2**64 - 1 - a) + 1))
                elif kind == "straddle":
                    a = (5 << 57) - 3000 + int(rng.integers(0, 6000))
                    n = int(rng.integers(0, 4000))
                else:
                    a = (9 << 57) + int(rng.integers(0, 6000))
                    n = int(rng.integers(0, 4000))
                addr.append(a), length.append(n)
            rf.append(len(addr))
    say("first writes wide spans", "writes", len(addr))
    *_, status = check_pieces(addr, length, rf, "wide spans")
    assert (status == g.FW_OK).all()


def test_pieces_many_large_allocations():
    """Allocations of over 64 writes (more than one wave takes) in every chunk of a call,
    so each workgroup takes several in turn (some refused, some small ones between them)."""
    rng = np.random.default_rng(7200)
    addr, length, rf = [], [], [0]
    for r in range(600):
        k = int(rng.integers(65, 90)) if r % 7 else int(rng.integers(0, 64))
        a, l, _ = random_log_k(rng, k, 4000)
        if r % 11 == 5 and k:
            a[-1], l[-1] = 2**64 - 3, 4
        addr += a
        length += l
        rf.append(len(addr))
    say("first writes many large", "writes", len(addr))
    check_pieces(addr, length, rf, "many large")


def test_pieces_over_a_million_allocations():
    """Over a million allocations: chunks of 4,116, so each wave takes about 257 in turn,
    the larger ones are found in five rounds per chunk and each chunk's scan and move take
    five rounds; most have zero to two writes, some over 64."""
    rng = np.random.default_rng(7300)
    n_regions = (1 << 20) + 5000
    k = rng.integers(0, 3, size=n_regions)
    big = rng.choice(n_regions, size=40, replace=False)
    k[big] = rng.integers(65, 130, size=40)
    rf = np.zeros(n_regions + 1, np.uint64)
    rf[1:] = np.cumsum(k)
    n = int(rf[-1])
    region = np.repeat(np.arange(n_regions, dtype=np.uint64), k)
    addr = (region << np.uint64(24)) + rng.integers(0, 5000, size=n).astype(np.uint64)
    length = rng.integers(0, 3000, size=n).astype(np.uint64)
    say("first writes", n_regions, "allocations", n, "writes")
    check_pieces(addr, length, rf, "over a million allocations")


def random_log_k(rng, k, span):
    """One allocation of exactly k writes within [base, base + span)."""
    base = int(rng.integers(0, 2**40)) << 12
    addr, length = [], []
    for _ in range(k):
        if length and rng.random() < 0.1:
            j = int(rng.integers(0, len(addr)))
            addr.append(addr[j]), length.append(length[j])
        else:
            addr.append(base + int(rng.integers(0, span))), length.append(int(rng.integers(0, span // 3)))
    return addr, length, [0, k]


def test_pieces_edges():
    top = 2**64 - 1
    # disjoint, nested, spanning, empty allocations, an allocation ending at the top of the
    # address space, one past it, one with 2,048 writes and one with 2,049
    addr = [0, 100, 50, 10, 40, 0, top - 9, top - 9, 5, 5]
    length = [50, 10, 50, 10, 10, 60, 9, 10, 0, 0]
    rf = [0, 3, 3, 6, 7, 8, 10]
    nested = list(range(2048, 0, -1))  # each write starts one byte before the previous one
    addr += nested
    length += [4096] * 2048
    rf.append(len(addr))
    addr += list(range(2049))
    length += [1] * 2049
    rf.append(len(addr))
    say("first writes edges")
    _, _, _, _, status = check_pieces(addr, length, rf, "edges")
    assert status.tolist() == [g.FW_OK, g.FW_OK, g.FW_OK, g.FW_OK, g.FW_INVALID, g.FW_OK, g.FW_OK, g.FW_TOO_MANY]


def test_reused_outputs_and_workspace():
    """Calls sharing outputs and workspace (sized for the largest) give each log's pieces,
    the later, smaller log too."""
    rng = np.random.default_rng(7400)
    logs = [random_log(rng, 400, 90, 1 << 16), random_log(rng, 37, 20, 3000)]
    n = max(len(a) for a, _, _ in logs)
    n_regions = max(len(rf) - 1 for _, _, rf in logs)
    bufs = g.first_writes_outputs(n, n_regions)
    ws = g.first_writes_workspace(n, n_regions)
    for k, (addr, length, rf) in enumerate(logs):
        say("first writes reused buffers", k, "writes", len(addr))
        pw, po, pl, first, status = g.first_writes(np.asarray(addr, np.uint64), np.asarray(length, np.uint64),
                                                   np.asarray(rf, np.uint64), out=bufs, ws=ws)
        torch.cuda.synchronize()
        want = oracle.first_write_pieces(addr, length, rf, max_writes=2048)
        m = len(rf) - 1
        first = u64(first)[:m + 1]
        p = int(first[-1])
        got = (u64(pw)[:p], u64(po)[:p], u64(pl)[:p], first, status.cpu().numpy()[:m])
        for a, b, name in zip(got, want, ("write", "offset", "length", "region first", "status")):
            assert np.array_equal(a, b), f"log {k}: {name} differs"


def test_no_writes_and_no_allocations():
    say("first writes empty")
    pw, po, pl, first, status = gpu_pieces([], [], [0, 0, 0])
    assert first.tolist() == [0, 0, 0] and status.tolist() == [0, 0]
    pw, po, pl, first, status = gpu_pieces([], [], [0])
    assert first.tolist() == [0]


@pytest.mark.parametrize("block", [4096, 65536])
def test_first_write_identification_end_to_end(block):
    """Allocations on the device receive overlapping writes in order; at each write's
    landing its owned pieces are digested from its payload, and at free time the same
    pieces are digested from the allocation. The verdicts equal painting every written
    byte with its first writer's byte and comparing with the allocation's bytes."""
    rng = np.random.default_rng(7100 + block)
    n_alloc = 24
    sizes = [int(rng.integers(1, 40)) * 10_000 for _ in range(n_alloc)]
    allocs = [torch.zeros(s, dtype=torch.uint8, device="cuda") for s in sizes]
    writes = []  # (allocation, offset, payload bytes) in time order, grouped by allocation
    rf = [0]
    for a, size in enumerate(sizes):
        for _ in range(int(rng.integers(0, 9))):
            off = int(rng.integers(0, size))
            n = int(rng.integers(0, size - off + 1))
            if writes and writes[-1][0] == a and rng.random() < 0.3:  # the same bytes again
                off, data = writes[-1][1], writes[-1][2]
            else:
                data = np.frombuffer(rng.bytes(n), np.uint8)
            writes.append((a, off, data))
        rf.append(len(writes))
    # payloads as they arrive (the sources), and the allocations after every write
    src, src_offs, src_lens = W.pack([w[2] for w in writes])
    d_src = to_device(src)
    for a, off, data in writes:
        if data.size:
            allocs[a][off:off + data.size] = to_device(data)
    dst_addr = np.array([allocs[a].data_ptr() + off for a, off, _ in writes], np.uint64)
    lens = np.array([w[2].size for w in writes], np.uint64)
    say("first-write identification", block, "writes", len(writes))
    pw, po, pl, first, status = gpu_pieces(dst_addr, lens, rf)
    assert (status == g.FW_OK).all()
    # recorded: the pieces of each payload, digested from the source bytes
    rec_batch = g.Batch(np.uint64(d_src.data_ptr()) + src_offs[pw] + po, pl, block, keepalive=d_src)
    recorded = g.fp_chunks(rec_batch).clone()
    # later, in-place changes to some allocations
    host_alloc = [t.cpu().numpy() for t in allocs]
    for a in range(n_alloc):
        if rng.random() < 0.3:
            x = int(rng.integers(0, sizes[a]))
            allocs[a][x] ^= 0x24
            host_alloc[a][x] ^= 0x24
    cur_batch = g.Batch(dst_addr[pw] + po, pl, block)
    _, _, weight = g.identify_weights(cur_batch, recorded, first)
    torch.cuda.synchronize()
    # byte truth: every written byte equals its first writer's byte
    expect = []
    for a in range(n_alloc):
        first_byte = {}
        for w in reversed(range(rf[a], rf[a + 1])):
            _, off, data = writes[w]
            for i in range(data.size):
                first_byte[off + i] = data[i]
        ok = bool(first_byte) and all(host_alloc[a][x] == v for x, v in first_byte.items())
        expect.append(1 if ok else 0)
    assert weight.cpu().numpy().tolist() == expect
    assert 0 < sum(expect) < n_alloc


@pytest.mark.parametrize("block", [4096, 16384, 1 << 20])
def test_identify_leaves_random_regions(block):
    rng = np.random.default_rng(7200 + block.bit_length())
    lens = [int(x) for x in rng.integers(0, 3 * block + 9000, 50)] + [0, 1, 4096, 4097, block]
    rng.shuffle(lens)
    written = [np.frombuffer(rng.bytes(n), np.uint8).copy() for n in lens]
    current = [w.copy() for w in written]
    for c in current:
        if c.size and rng.random() < 0.3:
            for _ in range(int(rng.integers(1, 3))):
                c[int(rng.integers(0, c.size))] ^= 1 << int(rng.integers(0, 8))
    cuts = sorted(set(int(x) for x in rng.integers(0, len(lens) + 1, 10)))
    region_first = np.array([0] + cuts + [len(lens)], np.uint64)
    _, rec_leaves = oracle.batch_digests(written, block, with_leaves=True)
    arena, offs, lens_a = W.pack(current, skew=int(rng.integers(0, 8)))
    batch = g.Batch.from_arena(to_device(arena), offs, lens_a, block)
    say("identify leaves", block)
    m, f, w = g.identify_leaves(batch, keys_to_device(rec_leaves.reshape(-1)), region_first)
    torch.cuda.synchronize()
    em, ef, ew = oracle.identify_leaves(rec_leaves, current, block, region_first)
    assert np.array_equal(m.cpu().numpy(), em)
    assert np.array_equal(u64(f), ef)
    assert np.array_equal(w.cpu().numpy(), ew)


@pytest.mark.timeout(900)
def test_identify_leaves_decoder7b_full():
    """The 13.5 GB decoder written as the base weights, 3 layers updated in place: the
    first changed leaf of each updated matrix is its first leaf, and the verdicts are
    the block-level ones."""
    threads = host_threads()
    dec = W.Decoder()
    block = W.DECODER_BLOCK
    say("identify leaves decoder7b generate")
    arena, offs, lens = dec.arena(perturbed=True, threads=threads)
    current = [arena[int(o):int(o) + int(n)] for o, n in zip(offs, lens)]
    _, rec = oracle.batch_digests(current, block, with_leaves=True, threads=threads)
    first = oracle.geometry(lens, block)[0]
    for i in dec.perturbed:
        _, lv = oracle.payload_digests(dec.base(i), block, with_leaves=True)
        rec[int(first[i]):int(first[i + 1])] = lv
    region_first = np.array([0] + [1 + 9 * l for l in range(33)] + [len(lens)], np.uint64)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    say("identify leaves decoder7b gpu")
    m, f, w = g.identify_leaves(batch, keys_to_device(rec.reshape(-1)), region_first)
    torch.cuda.synchronize()
    em, ef, ew = oracle.identify_leaves(rec, current, block, region_first, threads=threads)
    assert np.array_equal(m.cpu().numpy(), em)
    assert np.array_equal(u64(f), ef)
    assert np.array_equal(w.cpu().numpy(), ew)
    assert {r for r in range(ew.size) if ew[r] == 0} == {int(l) + 1 for l in dec.perturbed_layers}
    assert all(u64(f)[i] == 0 for i in dec.perturbed)
