"""GPU parity: every output of the library's kernels equals the oracle's, bit for
bit, on the same seeded inputs (integer work: no tolerance).

Sizes span several workgroups and end in ragged tails; edge cases cover empty
batches, zero-length and one-byte payloads, every tail path of the leaf hash,
unaligned payload starts, every block size from 4 KiB to 16 MiB (one leaf per
block up to 4096 leaves per block), keys 0 and 2^64-1, duplicate keys, multi-tile
compaction and table capacity errors."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23115_amd as g
import workloads as W
from gpu_util import assert_same, host_threads, keys_to_device, run_path, say, to_device, u64

pytestmark = pytest.mark.gpu

TAIL_LENGTHS = [1, 2, 3, 4, 5, 7, 8, 9, 15, 16, 31, 32, 33, 37, 63, 64, 100, 255, 4095, 4096, 4097, 8191, 8192]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def oracle_path(payloads, block, table):
    res = oracle.run(payloads, block, table, threads=host_threads())
    _, leaves = oracle.batch_digests(payloads, block, with_leaves=True, threads=host_threads())
    res["leaves"] = leaves
    return res


def make_payloads(rng, block, extra=()):
    lens = TAIL_LENGTHS + [block - 1, block, block + 1, 2 * block + 12345, 3 * block] + list(extra)
    lens += [0, 0]
    order = rng.permutation(len(lens))
    return [np.frombuffer(rng.bytes(int(lens[i])), np.uint8) for i in order]


@pytest.mark.parametrize("block", [4096 << k for k in range(13)])
def test_digests_every_block_size(block):
    rng = np.random.default_rng(100 + block.bit_length())
    payloads = make_payloads(rng, block)
    arena, offs, lens = W.pack(payloads, align=256)
    say("digests block", block, "payloads", len(payloads), "bytes", int(lens.sum()))
    d_arena = to_device(arena)
    batch = g.Batch.from_arena(d_arena, offs, lens, block)
    table = g.Cache(1 << 10)
    gpu = run_path(batch, table, with_leaves=True)
    ref = oracle_path(payloads, block, oracle.Table())
    assert_same(gpu, ref, f"block {block}")
    assert np.array_equal(gpu["leaves"], ref["leaves"])


@pytest.mark.parametrize("skew", [1, 2, 3, 4, 8, 12])
@pytest.mark.parametrize("block", [4096, 65536, 256 << 10, 1 << 20, 2 << 20, 16 << 20])
def test_unaligned_payload_starts(skew, block):
    rng = np.random.default_rng(200 + skew + block.bit_length())
    payloads = make_payloads(rng, block)
    arena, offs, lens = W.pack(payloads, align=256, skew=skew)
    say("unaligned skew", skew, "block", block)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    gpu = run_path(batch, g.Cache(1 << 10), with_leaves=True)
    ref = oracle_path(payloads, block, oracle.Table())
    assert_same(gpu, ref, f"skew {skew}")
    assert np.array_equal(gpu["leaves"], ref["leaves"])


@pytest.mark.parametrize("block", [4096, 65536, 1 << 20])
def test_mixed_alignment_in_one_wave(block):
    """Payloads at 16-byte aligned, 8-byte, odd and 2-byte starts side by side, so waves
    mix them."""
    rng = np.random.default_rng(250 + block.bit_length())
    payloads = make_payloads(rng, block, extra=[5000, 12000, 4096 * 3])
    lens = np.array([p.size for p in payloads], np.uint64)
    offs = np.zeros(len(payloads), np.uint64)
    pos = 0
    for i, n in enumerate(lens.tolist()):
        start = ((pos + 255) // 256) * 256 + (0, 8, 3, 2)[i % 4]
        offs[i] = start
        pos = start + n
    arena = np.zeros(pos + 512, np.uint8)
    for p, o in zip(payloads, offs.tolist()):
        arena[o:o + p.size] = p
    say("mixed alignment block", block)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    gpu = run_path(batch, g.Cache(1 << 10), with_leaves=True)
    ref = oracle_path(payloads, block, oracle.Table())
    assert_same(gpu, ref, "mixed alignment")
    assert np.array_equal(gpu["leaves"], ref["leaves"])


@pytest.mark.parametrize("block", [4096, 65536])
def test_many_empty_payloads_between_small_ones(block):
    # runs of up to 150 zero-length payloads: a wave's blocks then lie more than 64
    # payloads past its first block's payload, and the batch has over 64^2 payloads
    rng = np.random.default_rng(900 + block)
    payloads = []
    for _ in range(120):
        payloads += [np.zeros(0, np.uint8)] * int(rng.integers(0, 151))
        payloads.append(np.frombuffer(rng.bytes(int(rng.integers(1, 3 * block))), np.uint8))
    arena, offs, lens = W.pack(payloads)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    assert batch.n_seg > 64 * 64
    say("many empty payloads", block, batch.n_seg, batch.n_blocks)
    gpu = run_path(batch, g.Cache(1 << 10))
    assert_same(gpu, oracle_path(payloads, block, oracle.Table()), "empty runs")


def mixed_layout_payloads(rng, block, min_slots):
    """Payloads of every layout the kernels distinguish (full and contiguous, short,
    empty, odd-aligned starts) until the batch has at least `min_slots` leaf slots."""
    payloads, offsets, slots, pos = [], [], 0, 0
    while slots < min_slots:
        kind = int(rng.integers(0, 4))
        n = [int(rng.integers(8, 20)) * block, int(rng.integers(1, block)), 0, int(rng.integers(1, 3 * block))][kind]
        pos = (pos + 255) // 256 * 256 + (int(rng.integers(1, 16)) if kind == 3 else 0)
        payloads.append(np.frombuffer(rng.bytes(n), np.uint8))
        offsets.append(pos)
        pos += n
        slots += -(-n // block) * (block // 4096)
    arena = np.zeros(pos + 16, np.uint8)
    for o, p in zip(offsets, payloads):
        arena[o:o + p.size] = p
    return payloads, arena, np.array(offsets, np.uint64), np.array([p.size for p in payloads], np.uint64)


# Batches of blocks up to 64 KiB and at most 65,536 leaf slots use the four-lanes-per-leaf
# kernel; larger ones the two-lanes-per-leaf kernel. Same layouts on both sides.
@pytest.mark.parametrize("block", [4096, 8192, 32768, 65536])
@pytest.mark.parametrize("min_slots", [60_000, 70_000])
def test_both_small_block_kernels_on_mixed_layouts(block, min_slots):
    rng = np.random.default_rng(950 + block + min_slots)
    payloads, arena, offs, lens = mixed_layout_payloads(rng, block, min_slots)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    slots = batch.n_blocks * (block // 4096)
    assert (slots <= 65_536) == (min_slots == 60_000)
    say("mixed layouts", block, slots)
    gpu = run_path(batch, g.Cache(1 << 15), with_leaves=True)
    assert_same(gpu, oracle_path(payloads, block, oracle.Table()), "mixed layouts")


def test_random16_three_passes():
    block = W.RANDOM16_BLOCK
    p = W.random16_payload()
    say("random16 pass 1")
    d_p = to_device(p)
    batch = g.Batch.from_arena(d_p, [0], [p.size], block)
    table = g.Cache(1 << 10)
    otable = oracle.Table()
    gpu1 = run_path(batch, table, with_leaves=True)
    ref1 = oracle_path([p], block, otable)
    assert_same(gpu1, ref1, "pass 1")
    assert np.array_equal(gpu1["leaves"], ref1["leaves"])
    assert gpu1["miss_count"] == 256
    say("random16 insert")
    vals = torch.arange(256, dtype=torch.int64, device="cuda")
    n_new = table.insert(gpu1["_device_digests"], vals)
    assert int(n_new.item()) == 256 == otable.insert(ref1["digests"], np.arange(256, dtype=np.uint64))
    say("random16 pass 2a")
    gpu2 = run_path(batch, table)
    ref2 = oracle_path([p], block, otable)
    assert_same(gpu2, ref2, "pass 2a")
    assert (gpu2["status"] == g.HIT_CACHE).all()
    q, chosen = W.random16_rerandomized(p)
    say("random16 pass 2b")
    batch_q = g.Batch.from_arena(to_device(q), [0], [q.size], block)
    gpu3 = run_path(batch_q, table)
    ref3 = oracle_path([q], block, otable)
    assert_same(gpu3, ref3, "pass 2b")
    assert gpu3["miss_idx"].tolist() == chosen.tolist()


@pytest.mark.parametrize("block", [65536, 1 << 20])
def test_single_payload_above_4gib(block):
    # byte offsets past 2^32 and leaf indices past 2^20 in one payload (4.5 GiB plus a
    # short last block, 16 bytes into its buffer): the streamed path's offset arithmetic
    rng = np.random.default_rng(990)
    n = (9 << 29) + 12345
    host = np.empty(n + 16, np.uint8)
    step = 1 << 26  # fill in 64 MiB pieces, each with its own bytes
    for o in range(0, host.size, step):
        k = min(step, host.size - o)
        host[o:o + k] = np.frombuffer(rng.bytes(k), np.uint8)
    payload = host[16:16 + n]
    say("payload above 4 GiB", block)
    batch = g.Batch.from_arena(to_device(host), [16], [n], block)
    d = g.fp_chunks(batch)
    torch.cuda.synchronize()
    want, _ = oracle.batch_digests([payload], block, threads=host_threads())
    assert np.array_equal(u64(d), want)


def test_repeated_runs_identical():
    block = 65536
    rng = np.random.default_rng(300)
    pool = [rng.bytes(block) for _ in range(8)]
    payloads = [np.frombuffer(b"".join(pool[int(i)] for i in rng.integers(0, 8, 40)) + rng.bytes(777), np.uint8)
                for _ in range(10)]
    arena, offs, lens = W.pack(payloads)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    table = g.Cache(1 << 12)
    say("determinism x10")
    first = run_path(batch, table)
    for _ in range(9):
        again = run_path(batch, table)
        assert_same(again, first, "repeat")
    ref = oracle_path(payloads, block, oracle.Table())
    assert_same(first, ref, "vs oracle")
    assert (first["status"] == g.HIT_BATCH).sum() > 100


@pytest.mark.parametrize("block", [4096, 65536, 1 << 20])
def test_digests_do_not_depend_on_batch_position(block):
    """A payload's block digests are a function of its bytes alone: the same payloads
    hashed alone (the small-batch kernel), in shuffled order, behind 70,000 tiny payloads
    (past that kernel's 65,536-slot limit, so the two-lane kernel and another wave packing)
    and at shifted start offsets (the unaligned load path) all agree, and with the
    oracle."""
    rng = np.random.default_rng(7 + block.bit_length())
    payloads = make_payloads(rng, block, extra=[5 * block + 77])
    ref, _ = oracle.batch_digests(payloads, block, threads=host_threads())
    def per_payload(digests, lens, idx):
        f, _ = oracle.geometry(lens, block)
        return [digests[int(f[i]):int(f[i + 1])] for i in idx]

    want = per_payload(ref, [p.size for p in payloads], range(len(payloads)))
    tiny = [np.frombuffer(rng.bytes(int(n)), np.uint8) for n in rng.integers(1, 300, 70_000)]
    order = rng.permutation(len(payloads))
    layouts = {
        "shuffled": ([payloads[i] for i in order], list(order), 0, 0),
        "behind 70,000 tiny payloads": (tiny + [payloads[i] for i in order], list(order), len(tiny), 0),
        "offset 5": (payloads, list(range(len(payloads))), 0, 5),
    }
    for name, (batch_payloads, idx, skip, skew) in layouts.items():
        arena, offs, lens = W.pack(batch_payloads, align=256, skew=skew)
        say("position independence", block, name)
        batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
        d = u64(g.fp_chunks(batch))
        got = per_payload(d, lens, range(skip, skip + len(idx)))
        for k, i in enumerate(idx):
            assert np.array_equal(got[k], want[i]), f"{name}: payload {i}"
    for i in (0, len(payloads) // 2, len(payloads) - 1):
        arena, offs, lens = W.pack([payloads[i]], align=256)
        say("position independence", block, "alone", i)
        batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
        assert np.array_equal(u64(g.fp_chunks(batch)), want[i]), f"alone: payload {i}"


@pytest.mark.parametrize("block", [4096, 65536])
@pytest.mark.parametrize("avg_slots", [55, 70])
def test_large_batches_either_side_of_the_kernel_choice(block, avg_slots):
    """Past 65,536 leaf slots, blocks of up to 64 KiB go to the four-lanes-per-leaf kernel
    when payloads average at least 64 slots, else to the two-lanes one: batches of 1,400
    payloads averaging about 55 or 70 slots (random tails, some empty payloads, a 3-byte skew);
    every block and leaf digest equals the oracle's."""
    rng = np.random.default_rng(5100 + avg_slots + block.bit_length())
    n = 1400
    leaves = rng.integers(avg_slots // 2, 3 * avg_slots // 2 + 1, n)
    lens = leaves * 4096 - rng.integers(0, 4096, n)
    lens[rng.choice(n, 20, replace=False)] = 0
    payloads = [np.frombuffer(rng.bytes(int(m)), np.uint8) for m in lens]
    arena, offs, blens = W.pack(payloads, align=256, skew=3)
    batch = g.Batch.from_arena(to_device(arena), offs, blens, block)
    slots = batch.n_blocks * batch.leaves_per_block
    assert slots > 65536
    say("kernel choice: slots per payload", slots / batch.n_seg, "block", block)
    d, lv = g.fp_chunks(batch, with_leaves=True)
    want, wleaves = oracle.batch_digests(payloads, block, with_leaves=True, threads=host_threads())
    assert np.array_equal(u64(d), want)
    assert np.array_equal(u64(lv), wleaves.reshape(-1))


@pytest.mark.parametrize("skew", [0, 3, 16])
def test_4k_blocks_past_the_small_batch_limit(skew):
    """4 KiB blocks past the small-batch kernel's 65,536 slots, every tail length: 80,000
    payloads of lengths 0 (between the others), 1, 31..33, 511..513, 1000, 2048,
    4095..4097, 8192, 9000 and 12289, at aligned and unaligned starts, leaf digests on;
    every digest equals the oracle's."""
    rng = np.random.default_rng(4242 + skew)
    n = 80_000
    lens = rng.choice(np.array([0, 1, 31, 32, 33, 511, 512, 513, 1000, 2048, 4095, 4096, 4097, 8192, 9000, 12289]),
                      n, p=[0.05] + [0.95 / 15] * 15).astype(np.int64)
    payloads = [np.frombuffer(rng.bytes(int(m)), np.uint8) for m in lens]
    arena, offs, blens = W.pack(payloads, align=256, skew=skew)
    say("4 KiB blocks past the small-batch limit, skew", skew, "payloads", n)
    batch = g.Batch.from_arena(to_device(arena), offs, blens, 4096)
    assert batch.n_blocks > 65536
    d, lv = g.fp_chunks(batch, with_leaves=True)
    want, wleaves = oracle.batch_digests(payloads, 4096, with_leaves=True, threads=host_threads())
    assert np.array_equal(u64(d), want)
    assert np.array_equal(u64(lv), wleaves.reshape(-1))


@pytest.mark.parametrize("block,skew", [(8192, 0), (16384, 5), (32768, 3)])
def test_last_slots_four_lanes(block, skew):
    """Past 65,536 leaf slots with small payloads, the two-lanes kernel hands the batch's
    last 16,384 slots to workgroups of four lanes per leaf: 50,000 small copies (64 B to
    24 KiB, planted repeats) in blocks of 2-8 leaves, so payloads straddle the hand-over;
    every block and leaf digest equals the oracle's."""
    sc = W.SmallCopies(n=50_000, lo=64, hi=24576, workload=41, skew=skew)
    payloads = sc.payloads()
    batch = g.Batch.from_arena(to_device(sc.arena), sc.offsets, sc.sizes, block)
    slots = batch.n_blocks * batch.leaves_per_block
    assert slots > 65536 and slots < 64 * batch.n_seg
    say("last slots four lanes", block, "skew", skew, "slots", slots)
    d, lv = g.fp_chunks(batch, with_leaves=True)
    want, wleaves = oracle.batch_digests(payloads, block, with_leaves=True, threads=host_threads())
    assert np.array_equal(u64(d), want)
    assert np.array_equal(u64(lv), wleaves.reshape(-1))


@pytest.mark.parametrize("seed", range(24))
def test_randomized_batches(seed):
    """Seeded random batch geometries: block size 4 KiB..16 MiB, 1..4000 payloads whose
    lengths mix empty, tiny, leaf- and block-edge and multi-block sizes, repeated
    payloads, an optional skew of every start, a table holding a random part of the
    digests; every output (digests, leaf digests, status, ref, miss list, count, bytes)
    equals the oracle's."""
    rng = np.random.default_rng(90_000 + seed)
    block = 4096 << int(rng.integers(0, 13))
    n = int(rng.choice([1, 7, 64, 300, 1500, 4000]))
    budget = 48 << 20
    edges = np.array([0, 1, 31, 32, 33, 4095, 4096, 4097, block - 1, block, block + 1, 2 * block + 17])
    kind = rng.integers(0, 3, n)
    lens = np.where(kind == 0, rng.choice(edges, n),
                    np.where(kind == 1, rng.integers(0, 8192, n), rng.integers(0, 3 * block + 1, n)))
    lens = np.minimum(lens, budget // n)
    payloads = [np.frombuffer(rng.bytes(int(m)), np.uint8) for m in lens]
    for i in rng.integers(0, n, n // 10):  # some payloads repeat an earlier one
        j = int(rng.integers(0, n))
        payloads[int(i)] = payloads[j].copy()
    skew = int(rng.choice([0, 0, 0, 4, 8, 13]))
    arena, offs, blens = W.pack(payloads, align=256, skew=skew)
    say("randomized batch", seed, "block", block, "payloads", n, "bytes", int(blens.sum()), "skew", skew)
    batch = g.Batch.from_arena(to_device(arena), offs, blens, block)
    dig, _ = oracle.batch_digests(payloads, block, threads=host_threads())
    held = np.unique(dig[rng.random(dig.size) < 0.3]) if dig.size else np.zeros(0, np.uint64)
    table, otable = g.Cache(1 << 16), oracle.Table()
    if held.size:
        vals = rng.integers(0, 2**63, held.size, dtype=np.uint64)
        table.insert(keys_to_device(held), keys_to_device(vals))
        otable.insert(held, vals)
    gpu = run_path(batch, table, with_leaves=True)
    ref = oracle_path(payloads, block, otable)
    assert_same(gpu, ref, f"seed {seed}")
    assert np.array_equal(gpu["leaves"], ref["leaves"])


def test_lookup_special_keys_and_duplicates():
    rng = np.random.default_rng(400)
    pool = np.concatenate([rng.integers(0, 2**64, 500, dtype=np.uint64, endpoint=False),
                           np.array([0, 2**64 - 1, 1, 2**63], np.uint64)])
    keys = pool[rng.integers(0, pool.size, 20000)]
    cached = pool[rng.choice(pool.size, 200, replace=False)]
    cached = np.concatenate([cached, np.array([0, 2**64 - 1], np.uint64)])
    cvals = rng.integers(0, 2**64, cached.size, dtype=np.uint64, endpoint=False)
    say("lookup special keys")
    table = g.Cache(1 << 12)
    n_new = table.insert(keys_to_device(cached), keys_to_device(cvals))
    ot = oracle.Table()
    assert int(n_new.item()) == ot.insert(cached, cvals)
    status, ref = table.lookup(keys_to_device(keys))
    torch.cuda.synchronize()
    est, eref = oracle.lookup(keys, ot)
    assert np.array_equal(status.cpu().numpy(), est)
    assert np.array_equal(u64(ref), eref)
    assert {0, 1, 2} <= set(est.tolist())


def test_insert_lowest_index_wins_and_existing_kept():
    rng = np.random.default_rng(500)
    table, ot = g.Cache(1 << 12, max_load=0.9), oracle.Table()
    for rnd in range(5):
        keys = rng.integers(0, 300, 700).astype(np.uint64)
        keys[rng.integers(0, 700, 5)] = 2**64 - 1
        keys[rng.integers(0, 700, 5)] = 0
        vals = rng.integers(0, 2**64, 700, dtype=np.uint64, endpoint=False)
        say("insert round", rnd)
        n_new = table.insert(keys_to_device(keys), keys_to_device(vals))
        assert int(n_new.item()) == ot.insert(keys, vals)
        probe = np.concatenate([np.arange(0, 310, dtype=np.uint64), np.array([2**64 - 1], np.uint64)])
        st, ref = table.lookup(keys_to_device(probe))
        torch.cuda.synchronize()
        est, eref = oracle.lookup(probe, ot)
        assert np.array_equal(st.cpu().numpy(), est)
        assert np.array_equal(u64(ref), eref)


@pytest.mark.parametrize("seed", range(16))
def test_randomized_table_rounds(seed):
    """Seeded random table rounds: capacity 16..2^16 slots filled towards max_load 0.9 in
    several inserts (duplicates inside a call, keys already present, keys 0 and 2^64-1,
    keys clustered on a few home slots so probe runs are long and wrap past the table's
    end), each followed by a lookup of present, absent and repeated keys with batch sizes
    on both sides of the single-workgroup limit (4096); new-key counts, statuses and refs
    equal the oracle's after every round."""
    rng = np.random.default_rng(7700 + seed)
    cap = 1 << int(rng.integers(4, 17))
    table, ot = g.Cache(cap, max_load=0.9), oracle.Table()
    limit = int(0.9 * cap)
    bits = cap.bit_length() - 1
    for rnd in range(6):
        room = limit - table.key_bound()  # the host bound counts every key of a call
        if room <= 0:
            break
        n = int(rng.integers(1, min(room, 3000) + 1))
        pool = np.concatenate([rng.integers(0, 2**64 - 1, n, dtype=np.uint64, endpoint=True),
                               colliding_keys(rng, max(1, n // 4), bits)])
        keys = rng.choice(pool, n)
        keys[rng.random(n) < 0.02] = 0
        keys[rng.random(n) < 0.02] = 2**64 - 1
        if len(ot):
            old_keys, _, _ = ot.export()
            pick = rng.random(n) < 0.2
            keys[pick] = rng.choice(old_keys, int(pick.sum()))
        vals = rng.integers(0, 2**64 - 1, n, dtype=np.uint64, endpoint=True)
        say("table round seed", seed, "cap", cap, "round", rnd, "n", n)
        n_new = table.insert(keys_to_device(keys), keys_to_device(vals))
        assert int(n_new.item()) == ot.insert(keys, vals)
        stored, _, _ = ot.export()
        m = int(rng.choice([17, 4095, 4096, 4097, 9000]))
        probe = np.concatenate([rng.choice(stored, m // 2), rng.integers(0, 2**64 - 1, m - m // 2,
                                                                         dtype=np.uint64, endpoint=True)])
        probe = probe[rng.permutation(probe.size)]
        st, ref = table.lookup(keys_to_device(probe))
        torch.cuda.synchronize()
        est, eref = oracle.lookup(probe, ot)
        assert np.array_equal(st.cpu().numpy(), est), f"round {rnd}: status"
        assert np.array_equal(u64(ref), eref), f"round {rnd}: ref"


GOLDEN = 0x9E3779B97F4A7C15  # the multiplier of the library's slot hash (Fibonacci hashing)


def colliding_keys(rng, count, top_bits):
    """`count` distinct keys whose Fibonacci hash has the same top `top_bits` bits, so all
    of them start probing at one slot of a 2**top_bits-slot table."""
    inv = pow(GOLDEN, -1, 2**64)
    home = int(rng.integers(0, 2**top_bits))
    low = rng.choice(2**(64 - top_bits) - 1, count, replace=False) + 1
    return np.array([((home << (64 - top_bits) | int(v)) * inv) % 2**64 for v in low], np.uint64)


# Lookups of up to 4,096 keys dedup in one workgroup's LDS table of 8,192 slots; larger
# ones in a workspace table of a power of two >= 2n slots.
@pytest.mark.parametrize("n_keys,repeats,filler", [(8, 5, 0), (24, 3, 0), (40, 1, 0), (40, 4, 3_900),
                                                   (40, 4, 10_000), (30, 3, 20_000)])
def test_dedup_collisions_with_duplicates(n_keys, repeats, filler):
    # the colliding keys all start probing at one slot of the dedup table the lookup uses,
    # duplicates interleaved at random (and random filler keys): the lowest index must win
    rng = np.random.default_rng(800 + n_keys + filler)
    n = n_keys * repeats + filler
    if n <= 4_096:
        bits = 13
    else:
        cap = 64
        while cap < 2 * n:
            cap *= 2
        bits = cap.bit_length() - 1
    distinct = colliding_keys(rng, n_keys, bits)
    keys = np.concatenate([np.repeat(distinct, repeats),
                           rng.integers(0, 2**64, filler, dtype=np.uint64, endpoint=False)])
    keys = keys[rng.permutation(keys.size)]
    say("dedup collisions", n_keys, repeats, filler)
    table, ot = g.Cache(1 << 16), oracle.Table()
    status, ref = table.lookup(keys_to_device(keys))
    torch.cuda.synchronize()
    est, eref = oracle.lookup(keys, ot)
    assert np.array_equal(status.cpu().numpy(), est)
    assert np.array_equal(u64(ref), eref)
    vals = np.arange(keys.size, dtype=np.uint64) + 1000
    n_new = table.insert(keys_to_device(keys), keys_to_device(vals))
    assert int(n_new.item()) == ot.insert(keys, vals) == np.unique(keys).size
    st2, ref2 = table.lookup(keys_to_device(keys))
    torch.cuda.synchronize()
    est2, eref2 = oracle.lookup(keys, ot)
    assert np.array_equal(st2.cpu().numpy(), est2) and np.array_equal(u64(ref2), eref2)


@pytest.mark.parametrize("kind", ["one_partition", "one_key", "two_partitions_with_hits"])
def test_lookup_skewed_keys(kind):
    """Lookups of 9,000-16,384 keys (the three-launch path) with skewed keys: 16,384
    distinct keys that agree in bits 40-43, one key repeated 16,384 times, and keys
    drawn from two such groups with half of them cached and repeats, against the
    oracle."""
    rng = np.random.default_rng(870)
    n = 16_384
    if kind == "one_partition":
        keys = rng.integers(0, 2**64, n, dtype=np.uint64, endpoint=False)
        keys = (keys & ~np.uint64(0xF << 40)) | np.uint64(7 << 40)
        keys = np.unique(keys)[:n]
        keys = keys[rng.permutation(keys.size)]
        cached = keys[: keys.size // 4]
    elif kind == "one_key":
        keys = np.full(n, 0x123456789ABCDEF0, np.uint64)
        cached = np.zeros(0, np.uint64)
    else:
        pool = rng.integers(0, 2**64, 3000, dtype=np.uint64, endpoint=False)
        pool = (pool & ~np.uint64(0xF << 40)) | (np.uint64(3 << 40) * (pool & np.uint64(1)).astype(np.uint64))
        pool = np.concatenate([pool, np.array([0, 2**64 - 1], np.uint64)])
        keys = pool[rng.integers(0, pool.size, 9000)]
        cached = pool[rng.choice(pool.size, pool.size // 2, replace=False)]
    cvals = rng.integers(0, 2**64, cached.size, dtype=np.uint64, endpoint=False)
    say("lookup skewed keys", kind, keys.size)
    table, ot = g.Cache(1 << 15), oracle.Table()
    if cached.size:
        table.insert(keys_to_device(cached), keys_to_device(cvals))
        ot.insert(cached, cvals)
    status, ref = table.lookup(keys_to_device(keys))
    torch.cuda.synchronize()
    est, eref = oracle.lookup(keys, ot)
    assert np.array_equal(status.cpu().numpy(), est)
    assert np.array_equal(u64(ref), eref)


@pytest.mark.parametrize("n", [4_095, 4_096, 4_097, 16_384, 16_385])
def test_lookup_at_single_workgroup_limit(n):
    rng = np.random.default_rng(850 + n)
    pool = np.concatenate([rng.integers(0, 2**64, n // 3, dtype=np.uint64, endpoint=False),
                           np.array([0, 2**64 - 1], np.uint64)])
    keys = pool[rng.integers(0, pool.size, n)]
    cached = np.concatenate([pool[rng.choice(pool.size, pool.size // 2, replace=False)],
                             np.array([2**64 - 1], np.uint64)])
    cvals = rng.integers(0, 2**64, cached.size, dtype=np.uint64, endpoint=False)
    say("lookup limit", n)
    table, ot = g.Cache(1 << 15), oracle.Table()
    table.insert(keys_to_device(cached), keys_to_device(cvals))
    ot.insert(cached, cvals)
    status, ref = table.lookup(keys_to_device(keys))
    torch.cuda.synchronize()
    est, eref = oracle.lookup(keys, ot)
    assert np.array_equal(status.cpu().numpy(), est)
    assert np.array_equal(u64(ref), eref)
    assert {0, 1, 2} <= set(est.tolist())


def test_capacity_is_enforced():
    table = g.Cache(16, max_load=0.5)  # at most 8 keys
    k = keys_to_device(np.arange(9, dtype=np.uint64))
    with pytest.raises(g.GleamError) as e:
        table.insert(k, k)
    assert e.value.status == g.E_CAPACITY
    table.insert(k[:8], k[:8])
    with pytest.raises(g.GleamError):
        table.insert(k[8:], k[8:])
    assert table.key_bound() == 8
    st, ref = table.lookup(k)
    torch.cuda.synchronize()
    assert st.cpu().numpy().tolist() == [1] * 8 + [0]


def short_block_batch(rng, n, block=4096):
    """A batch of n blocks whose payloads end in short blocks."""
    lens = []
    left = n
    while left:
        k = int(min(left, rng.integers(1, 6)))
        lens.append((k - 1) * block + int(rng.integers(1, block + 1)))
        left -= k
    batch = g.Batch(np.full(len(lens), 0, np.uint64), lens, block)
    assert batch.n_blocks == n
    return batch, lens


def check_compaction(status, d_status, batch, lens, block=4096):
    counters = torch.full((2,), -1, dtype=torch.int64, device="cuda")
    miss_idx, counters = g.miss_compact(d_status, batch, counters=counters)
    torch.cuda.synchronize()
    c = u64(counters)
    _, blen = oracle.geometry(lens, block)
    eidx, ecnt, ebytes = oracle.compact(status, blen)
    assert int(c[0]) == ecnt and int(c[1]) == ebytes
    assert np.array_equal(u64(miss_idx)[:ecnt], eidx)


# one workgroup up to 65,536 statuses (16,384 per round), tiles of 2,048 above: two
# launches up to 1,024 tiles (2,097,152 statuses), three beyond
@pytest.mark.parametrize("n", [1, 63, 2047, 2048, 2049, 3 * 2048 + 17, 16_383, 16_384, 16_385, 65_536, 65_537,
                               100_003, 2_097_152, 2_097_153, 2_500_001])
def test_compaction_tiles(n):
    rng = np.random.default_rng(600 + n)
    status = rng.choice(np.array([0, 1, 2], np.uint8), n, p=[0.3, 0.5, 0.2])
    # a batch whose geometry has n blocks with short last blocks
    block = 4096
    lens = []
    left = n
    while left:
        k = int(min(left, rng.integers(1, 6)))
        lens.append((k - 1) * block + int(rng.integers(1, block + 1)))
        left -= k
    batch = g.Batch(np.full(len(lens), 0, np.uint64), lens, block)
    assert batch.n_blocks == n
    say("compaction n", n)
    check_compaction(status, to_device(status), batch, lens)


@pytest.mark.parametrize("offset", [1, 3, 8])
def test_compaction_status_at_odd_address(offset):
    rng = np.random.default_rng(650 + offset)
    n = 40_000
    status = rng.choice(np.array([0, 1, 2], np.uint8), n, p=[0.4, 0.4, 0.2])
    batch, lens = short_block_batch(rng, n)
    say("compaction status offset", offset)
    buf = torch.zeros(n + 16, dtype=torch.uint8, device="cuda")
    d_status = buf[offset:offset + n]
    d_status.copy_(torch.from_numpy(status).to("cuda"))
    check_compaction(status, d_status, batch, lens)


# few blocks but over 65,536 payloads (zero-length ones between): the tiled path. 30,000
# blocks: one payload per byte-total thread; 100,000 (300,000 payloads): more payloads
# than the 1,024 byte-total workgroups cover in one step; 10 blocks: those workgroups
# capped by the workspace's 64 scratch words.
@pytest.mark.parametrize("n", [30_000, 100_000, 10])
def test_compaction_more_payloads_than_small_path(n):
    rng = np.random.default_rng(660 + n)
    status = rng.choice(np.array([0, 1, 2], np.uint8), n, p=[0.5, 0.3, 0.2])
    lens = []
    empties = 2 if n > 1_000 else 7_000
    for _ in range(n):  # one short block each, then empty payloads
        lens += [int(rng.integers(1, 4097))] + [0] * empties
    batch = g.Batch(np.full(len(lens), 0, np.uint64), lens, 4096)
    assert batch.n_blocks == n and batch.n_seg > 65_536
    say("compaction payloads", batch.n_seg)
    check_compaction(status, to_device(status), batch, lens)


def test_empty_inputs():
    say("empty batch")
    batch = g.Batch([], [], 65536)
    assert batch.n_blocks == 0
    d = g.fp_chunks(batch)
    assert d.numel() == 0
    table = g.Cache(64)
    st, ref = table.lookup(d)
    miss_idx, counters = g.miss_compact(st, batch)
    torch.cuda.synchronize()
    assert u64(counters).tolist() == [0, 0]
    # zero-length payloads between non-empty ones
    rng = np.random.default_rng(700)
    payloads = [np.zeros(0, np.uint8), np.frombuffer(rng.bytes(5000), np.uint8), np.zeros(0, np.uint8)]
    arena, offs, lens = W.pack(payloads)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, 4096)
    gpu = run_path(batch, table)
    assert_same(gpu, oracle_path(payloads, 4096, oracle.Table()), "zero-length")


def test_compaction_of_only_empty_payloads_beyond_small_path():
    """70,000 zero-length payloads: no blocks, so no statuses, and the byte total is
    wanted. The count and the byte total are still written (both 0)."""
    batch = g.Batch(np.zeros(70_000, np.uint64), np.zeros(70_000, np.uint64), 65536)
    assert batch.n_blocks == 0 and batch.n_seg > 65_536
    say("compaction of 70,000 empty payloads")
    status = torch.empty(1, dtype=torch.uint8, device="cuda")[:0]
    counters = torch.full((2,), -1, dtype=torch.int64, device="cuda")
    g.miss_compact(status, batch, counters=counters)
    torch.cuda.synchronize()
    assert u64(counters).tolist() == [0, 0]


@pytest.mark.parametrize("n", [1_000, 10_000, 100_000])  # one-workgroup and grid lookups; both compactions
def test_optional_outputs_absent(n):
    """Lookup without the ref output and compaction without a batch (no byte total) give
    the same statuses and miss lists as with them."""
    rng = np.random.default_rng(1500 + n)
    pool = rng.integers(0, 2**64, n // 2, dtype=np.uint64, endpoint=False)
    keys = pool[rng.integers(0, pool.size, n)]
    table, ot = g.Cache(1 << 17), oracle.Table()
    cached = pool[: pool.size // 3]
    table.insert(keys_to_device(cached), keys_to_device(cached))
    ot.insert(cached, cached)
    say("optional outputs", n)
    st_noref, ref_none = table.lookup(keys_to_device(keys), want_ref=False)
    assert ref_none is None
    miss_idx, counters = g.miss_compact(st_noref)  # no batch: count only
    torch.cuda.synchronize()
    est, _ = oracle.lookup(keys, ot)
    eidx, ecnt, _ = oracle.compact(est)
    assert np.array_equal(st_noref.cpu().numpy(), est)
    assert int(u64(counters)[0]) == ecnt
    assert np.array_equal(u64(miss_idx)[:ecnt], eidx)


def test_batch_from_tensors():
    """Payloads given as torch tensors (several dtypes, contiguous slices at odd byte
    offsets): the digests are those of each tensor's bytes."""
    torch.manual_seed(1600)
    base = torch.randint(-128, 127, (300_000,), dtype=torch.int8, device="cuda")
    tensors = [torch.randn(257, 129, device="cuda").to(torch.float16),
               torch.randn(70_000, device="cuda").to(torch.bfloat16),
               torch.randn(33, 1000, device="cuda"),
               base[3:200_003],          # contiguous, 3 bytes into its storage
               base[100_001:100_001],    # empty
               torch.arange(5, dtype=torch.int64, device="cuda")]
    say("batch from tensors")
    batch = g.Batch.from_tensors(tensors, 65536)
    d = g.fp_chunks(batch)
    torch.cuda.synchronize()
    payloads = [t.cpu().contiguous().view(torch.uint8).numpy() if t.numel() else np.zeros(0, np.uint8)
                for t in tensors]
    want, _ = oracle.batch_digests(payloads, 65536)
    assert np.array_equal(u64(d), want)
    with pytest.raises(ValueError):
        g.Batch.from_tensors([torch.zeros(8, 8, device="cuda").t()], 65536)


def test_binding_refuses_tensors_the_kernels_would_misread():
    batch = g.Batch.from_arena(torch.zeros(1 << 16, dtype=torch.uint8, device="cuda"), [0], [1 << 16], 4096)
    table = g.Cache(1 << 10)
    keys = torch.zeros(16, dtype=torch.int64, device="cuda")
    with pytest.raises(ValueError):  # wrong dtype
        g.fp_chunks(batch, out=torch.zeros(16, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):  # too short
        g.fp_chunks(batch, out=torch.zeros(8, dtype=torch.int64, device="cuda"))
    with pytest.raises(ValueError):  # not contiguous
        table.lookup(torch.zeros(16, 2, dtype=torch.int64, device="cuda")[:, 0])
    with pytest.raises(ValueError):  # host memory
        table.insert(keys.cpu(), keys)
    with pytest.raises(ValueError):  # status must be u8
        g.miss_compact(torch.zeros(16, dtype=torch.int64, device="cuda"))
    arena = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError):  # a payload past the arena's end
        g.Batch.from_arena(arena, [4000], [200], 4096)
    with pytest.raises(ValueError):  # an offset past the end
        g.Batch.from_arena(arena, [5000], [0], 4096)
    with pytest.raises(ValueError):  # not contiguous
        g.Batch.from_arena(torch.zeros(64, 2, dtype=torch.uint8, device="cuda")[:, 0], [0], [8], 4096)
    assert g.Batch.from_arena(arena, [4000], [96], 4096).n_blocks == 1  # ends exactly at the end


@pytest.mark.parametrize("layout", ["runs", "scattered", "special"])
def test_lookup_and_insert_of_heavily_repeated_keys(layout):
    """Batches dominated by one key, as zero-filled tensors make them: long runs of it
    (lanes of one workgroup and of many), the same key scattered one per workgroup among
    distinct keys, and the keys 0 and 2^64-1 repeated. Statuses, refs and insert counts
    equal the oracle's, and the lookup of 262,144 equal keys stays within a small multiple
    of the lookup of as many distinct keys (with one device-wide compare-and-swap per
    key it took 36x as long)."""
    rng = np.random.default_rng({"runs": 450, "scattered": 451, "special": 452}[layout])
    n = 262_144
    hot = np.uint64(0x5DEECE66D1234567)
    keys = rng.integers(0, 2**64, n, dtype=np.uint64, endpoint=False)
    if layout == "runs":
        keys[:] = hot
        keys[rng.integers(0, n, 300)] = rng.integers(0, 2**64, 300, dtype=np.uint64, endpoint=False)
    elif layout == "scattered":
        keys[::256] = hot
        keys[7::512] = hot
    else:
        keys[: n // 2] = 2**64 - 1
        keys[n // 2:] = 0
    cached = np.array([keys[1], np.uint64(12345)], np.uint64)
    table, ot = g.Cache(1 << 20, max_load=0.5), oracle.Table()
    table.insert(keys_to_device(cached), keys_to_device(np.array([7, 8], np.uint64)))
    ot.insert(cached, np.array([7, 8], np.uint64))
    say("repeated keys", layout)
    d = keys_to_device(keys)
    status, ref = table.lookup(d)
    torch.cuda.synchronize()
    est, eref = oracle.lookup(keys, ot)
    assert np.array_equal(status.cpu().numpy(), est)
    assert np.array_equal(u64(ref), eref)
    fresh, ofresh = g.Cache(1 << 20, max_load=0.5), oracle.Table()
    vals = np.arange(n, dtype=np.uint64)
    n_new = fresh.insert(d, keys_to_device(vals))
    assert int(n_new.item()) == ofresh.insert(keys, vals)
    k, v, _, c = fresh.export()
    torch.cuda.synchronize()
    ek, ev, _ = ofresh.export()
    assert np.array_equal(u64(k)[:int(c.item())], ek) and np.array_equal(u64(v)[:int(c.item())], ev)
    if layout == "runs":
        distinct = keys_to_device(rng.integers(0, 2**64, n, dtype=np.uint64, endpoint=False))
        ws = g.workspace(n)
        st = torch.empty(n, dtype=torch.uint8, device="cuda")

        def timed(x):
            for _ in range(3):
                table.lookup(x, status=st, ws=ws)
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(5):
                table.lookup(x, status=st, ws=ws)
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) / 5

        t_hot, t_distinct = timed(d), timed(distinct)
        assert t_hot < 4 * t_distinct + 0.05, (t_hot, t_distinct)
