"""GPU parity of gleam_detect, the one-call decision (one kernel for a small batch):
every output -- digests, statuses, refs, the miss list, its count and bytes -- equals
the oracle's bit for bit, and equals what gleam_fp_chunks -> gleam_cache_lookup ->
gleam_miss_compact write, on both sides of every size limit of the one-kernel path
(65,536 leaf slots, 4,096 blocks, 64 KiB blocks) and of its one-wave / four-wave
choice (512 blocks)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23115_amd as g
import workloads as W
from gpu_util import host_threads, keys_to_device, run_path, say, to_device, u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def detect_outputs(batch, table, want_ref=True, out=None):
    res = g.detect(batch, table, out=out, want_ref=want_ref)
    torch.cuda.synchronize()
    n = batch.n_blocks
    c = u64(res.counters)
    o = {"digests": u64(res.digests)[:n], "status": res.status[:n].cpu().numpy(),
         "ref": u64(res.ref)[:n] if res.ref is not None else None,
         "miss_count": int(c[0]), "miss_bytes": int(c[1])}
    o["miss_idx"] = u64(res.miss_idx)[:o["miss_count"]]
    return o


def check(batch, payloads, table, ot, what, want_ref=True):
    """detect == oracle, and detect == the three calls."""
    got = detect_outputs(batch, table, want_ref)
    ref = oracle.run(payloads, batch.block_bytes, ot, threads=host_threads())
    for k in ("digests", "status", "miss_idx"):
        assert np.array_equal(got[k], ref[k]), f"{what}: {k} differs from the oracle"
    if want_ref:
        assert np.array_equal(got["ref"], ref["ref"]), f"{what}: ref differs from the oracle"
    assert got["miss_count"] == ref["miss_count"] and got["miss_bytes"] == ref["miss_bytes"], what
    three = run_path(batch, table)
    for k in ("digests", "status", "miss_idx"):
        assert np.array_equal(got[k], three[k]), f"{what}: {k} differs from the three calls"
    assert (got["miss_count"], got["miss_bytes"]) == (three["miss_count"], three["miss_bytes"]), what
    return got


def tables_from(payloads, block, which, capacity=1 << 14):
    """A GPU table and an oracle table holding the digests of the payloads in `which`
    (computed by the oracle), with value = payload index."""
    keys, vals = [np.zeros(0, np.uint64)], [np.zeros(0, np.uint64)]
    for i in which:
        d, _ = oracle.payload_digests(payloads[i], block)
        keys.append(d)
        vals.append(np.full(d.size, i, np.uint64))
    keys, vals = np.concatenate(keys), np.concatenate(vals)
    t, ot = g.Cache(capacity), oracle.Table()
    if keys.size:
        t.insert(keys_to_device(keys), keys_to_device(vals))
        ot.insert(keys, vals)
    return t, ot


def test_random16_three_passes():
    """16 MiB of random bytes, 64 KiB blocks: empty table (256 MISS), then after the
    insert the same bytes (256 HIT_CACHE), then 64 re-randomised blocks (64 MISS)."""
    p = W.random16_payload()
    p2, chosen = W.random16_rerandomized(p)
    block = 1 << 16
    d_p, d_p2 = to_device(p), to_device(p2)
    b1 = g.Batch.from_arena(d_p, [0], [p.size], block)
    b2 = g.Batch.from_arena(d_p2, [0], [p2.size], block)
    t, ot = g.Cache(1 << 10), oracle.Table()
    say("detect random16 pass 1")
    r1 = check(b1, [p], t, ot, "pass 1")
    assert r1["miss_count"] == 256
    vals = np.arange(256, dtype=np.uint64)
    t.insert(keys_to_device(r1["digests"]), keys_to_device(vals))
    ot.insert(r1["digests"], vals)
    say("detect random16 pass 2a")
    assert check(b1, [p], t, ot, "pass 2a")["miss_count"] == 0
    say("detect random16 pass 2b")
    r3 = check(b2, [p2], t, ot, "pass 2b")
    assert np.array_equal(r3["miss_idx"], np.sort(chosen))


def test_resnet50():
    block = W.RESNET_BLOCK
    payloads = W.resnet50_payloads()
    cached = W.resnet50_cached_tensors()
    t, ot = tables_from(payloads, block, cached.tolist())
    arena, offs, lens = W.pack(payloads)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    say("detect resnet50", batch.n_blocks, "blocks")
    got = check(batch, payloads, t, ot, "resnet50")
    assert int((got["status"] == g.HIT_CACHE).sum()) == 471


@pytest.mark.parametrize("block", [4096, 8192, 16384, 32768, 65536, 131072])
@pytest.mark.parametrize("skew", [0, 3])
def test_mixed_layouts(block, skew):
    """Short, long, empty and repeated payloads at a byte skew; half of them cached."""
    rng = np.random.default_rng(9100 + block + skew)
    lens = [0, 1, 7, 31, 32, 33, 100, 4095, 4096, 4097, block - 1, block, block + 1, 2 * block + 77,
            3 * block, 0, 12345]
    payloads = [np.frombuffer(rng.bytes(n), np.uint8) for n in lens]
    payloads += [payloads[11].copy(), payloads[13].copy(), payloads[8].copy()]  # repeats in the batch
    arena, offs, lens = W.pack(payloads, align=64, skew=skew)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    t, ot = tables_from(payloads, block, range(0, len(payloads), 2))
    say("detect mixed", block, skew, batch.n_blocks, "blocks")
    got = check(batch, payloads, t, ot, f"mixed {block} skew {skew}")
    assert (got["status"] == g.HIT_BATCH).any()


# around the one-wave / four-wave choice (512 blocks) and the one-kernel limits
# (4,096 blocks; 65,536 leaf slots = 4,096 blocks of 64 KiB)
@pytest.mark.parametrize("n_blocks,block", [(1, 4096), (511, 4096), (512, 4096), (513, 4096), (4095, 4096),
                                            (4096, 4096), (4097, 4096), (4096, 65536), (4097, 65536)])
def test_size_limits(n_blocks, block):
    rng = np.random.default_rng(9300 + n_blocks + block)
    # payloads of 1-3 blocks, last one short, with some repeats
    payloads, total = [], 0
    while total < n_blocks:
        k = int(min(rng.integers(1, 4), n_blocks - total))
        n = (k - 1) * block + int(rng.integers(1, block + 1))
        if payloads and rng.random() < 0.1 and payloads[-1].size == n:
            payloads.append(payloads[-1].copy())
        else:
            payloads.append(np.frombuffer(rng.bytes(n), np.uint8))
        total += k
    arena, offs, lens = W.pack(payloads)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    assert batch.n_blocks == n_blocks
    t, ot = tables_from(payloads, block, range(1, len(payloads), 3))
    say("detect size limit", n_blocks, block)
    check(batch, payloads, t, ot, f"{n_blocks} blocks of {block}")


def test_small_copies_prefix():
    """The first 3,000 of the 100k small copies (planted repeats, 4 KiB blocks)."""
    sc = W.SmallCopies(n=3_000)
    payloads = sc.payloads()
    batch = g.Batch.from_arena(to_device(sc.arena), sc.offsets, sc.sizes, W.SMALL_BLOCK)
    say("detect small copies", batch.n_blocks, "blocks")
    got = check(batch, payloads, g.Cache(1 << 10), oracle.Table(), "small copies")
    assert int((got["status"] == g.HIT_BATCH).sum()) == sc.targets.size


@pytest.mark.parametrize("n", [1, 4096, 4097, 65536])
def test_single_payload_per_call(n):
    """One host-to-device copy per call (what a per-copy interceptor would issue)."""
    rng = np.random.default_rng(9500 + n)
    p = np.frombuffer(rng.bytes(n), np.uint8)
    batch = g.Batch.from_arena(to_device(p), [0], [n], 4096)
    say("detect one payload", n)
    check(batch, [p], g.Cache(64), oracle.Table(), f"one payload of {n}")


def test_calls_in_a_row_reuse_the_workspace_and_skip_ref():
    """Back-to-back calls on one stream with one set of outputs and workspace, the later
    batches smaller; then without the ref output."""
    rng = np.random.default_rng(9600)
    big = [np.frombuffer(rng.bytes(int(n)), np.uint8) for n in rng.integers(1, 200_000, 40)]
    small = big[:5]
    arena, offs, lens = W.pack(big)
    d_arena = to_device(arena)
    b_big = g.Batch.from_arena(d_arena, offs, lens, 16384)
    b_small = g.Batch.from_arena(d_arena, offs[:5], lens[:5], 16384)
    out = g.Detect(b_big)
    t = g.Cache(1 << 10)
    say("detect calls in a row")
    for _ in range(3):
        g.detect(b_big, t, out=out)
        g.detect(b_small, t, out=out)
    torch.cuda.synchronize()
    want = oracle.run(small, 16384, oracle.Table(), threads=host_threads())
    n = b_small.n_blocks
    assert np.array_equal(u64(out.digests)[:n], want["digests"])
    assert np.array_equal(out.status[:n].cpu().numpy(), want["status"])
    assert np.array_equal(u64(out.ref)[:n], want["ref"])
    c = u64(out.counters)
    assert (int(c[0]), int(c[1])) == (want["miss_count"], want["miss_bytes"])
    assert np.array_equal(u64(out.miss_idx)[:want["miss_count"]], want["miss_idx"])
    check(b_big, big, t, oracle.Table(), "no ref", want_ref=False)


def test_empty_batches():
    t = g.Cache(64)
    for lens in ([], [0], [0] * 70_000):
        batch = g.Batch(np.zeros(len(lens), np.uint64), lens, 65536)
        out = g.Detect(batch)
        out.counters.fill_(-1)
        say("detect empty batch", len(lens))
        g.detect(batch, t, out=out)
        torch.cuda.synchronize()
        assert u64(out.counters).tolist() == [0, 0]


def test_paths_alternate_on_one_workspace():
    """One prepared workspace serves a three-kernel batch (planted repeats), a one-kernel
    batch, then the first again: a dedup slot left behind by a call would show as a wrong
    repeat or reference in the next."""
    rng = np.random.default_rng(9700)
    base = [np.frombuffer(rng.bytes(int(n)), np.uint8) for n in rng.integers(1, 60_000, 600)]
    big = base + [base[i].copy() for i in rng.integers(0, len(base), 200)]  # repeats in the batch
    arena, offs, lens = W.pack(big)
    d_arena = to_device(arena)
    b_big = g.Batch.from_arena(d_arena, offs, lens, 4096)
    b_small = g.Batch.from_arena(d_arena, offs[:40], lens[:40], 4096)
    assert b_big.n_blocks > 4096 and b_small.n_blocks <= 4096
    t, ot = tables_from(big, 4096, range(0, 600, 7))
    out = g.Detect(b_big)
    for i, (b, p) in enumerate([(b_big, big), (b_small, big[:40]), (b_big, big), (b_big, big)]):
        say("detect alternating", i, b.n_blocks)
        got = detect_outputs(b, t, out=out)
        want = oracle.run(p, 4096, ot, threads=host_threads())
        for k in ("digests", "status", "ref", "miss_idx"):
            assert np.array_equal(got[k], want[k]), f"call {i}: {k}"
        assert (got["miss_count"], got["miss_bytes"]) == (want["miss_count"], want["miss_bytes"]), i


def test_beyond_the_three_kernel_limit():
    """2,100,000 blocks of 4 KiB (past 2,097,152: the three calls' kernels run) drawn from
    4,000 distinct blocks, so most repeat; then a three-kernel batch on the same workspace."""
    rng = np.random.default_rng(9800)
    n_blk, per = 2_100_000, 100_000
    pool = rng.integers(0, 256, (4000, 4096), dtype=np.uint8)
    pick = rng.integers(0, pool.shape[0], n_blk)
    arena = pool[pick].reshape(-1)
    offs = np.arange(0, n_blk, per, dtype=np.uint64) * 4096
    lens = np.full(offs.size, per * 4096, np.uint64)
    lens[-1] = (n_blk - per * (offs.size - 1)) * 4096 - 123  # a short last block
    payloads = [arena[int(o):int(o) + int(n)] for o, n in zip(offs, lens)]
    d_arena = to_device(arena)
    batch = g.Batch.from_arena(d_arena, offs, lens, 4096)
    assert batch.n_blocks == n_blk
    t, ot = g.Cache(1 << 13), oracle.Table()
    keys = oracle.batch_digests([pool[i] for i in range(0, 4000, 3)], 4096)[0]
    t.insert(keys_to_device(keys), keys_to_device(keys))
    ot.insert(keys, keys)
    out = g.Detect(batch)
    say("detect past the three-kernel limit", n_blk)
    got = detect_outputs(batch, t, out=out)
    want = oracle.run(payloads, 4096, ot, threads=host_threads())
    for k in ("digests", "status", "ref", "miss_idx"):
        assert np.array_equal(got[k], want[k]), k
    assert (got["miss_count"], got["miss_bytes"]) == (want["miss_count"], want["miss_bytes"])
    sub_b = g.Batch.from_arena(d_arena, [offs[0], 4096 * 7], [9000 * 4096, 5000 * 4096 + 1], 4096)
    say("detect after the limit, three kernels", sub_b.n_blocks)
    got = detect_outputs(sub_b, t, out=out)
    want = oracle.run([arena[:9000 * 4096], arena[4096 * 7:4096 * 7 + 5000 * 4096 + 1]], 4096, ot,
                      threads=host_threads())
    for k in ("digests", "status", "ref", "miss_idx"):
        assert np.array_equal(got[k], want[k]), k
    assert (got["miss_count"], got["miss_bytes"]) == (want["miss_count"], want["miss_bytes"])


@pytest.mark.parametrize("block", [4096, 65536])
def test_large_payloads_four_lanes(block):
    """Past the one-kernel limits with payloads of at least 64 leaf slots on average (the
    fingerprint then runs four lanes per leaf): 300 payloads of 0.5-1.5 MiB with short
    last blocks, some blocks planted as copies of earlier ones."""
    rng = np.random.default_rng(9900 + block)
    sizes = rng.integers(1 << 19, 3 << 19, 300)
    payloads = [bytearray(rng.bytes(int(n))) for n in sizes]
    for _ in range(200):  # block-aligned copies of earlier blocks
        i, j = sorted(rng.integers(0, len(payloads), 2))
        bi = int(rng.integers(0, len(payloads[i]) // block))
        bj = int(rng.integers(0, len(payloads[j]) // block))
        if (i, bi) != (j, bj):
            payloads[j][bj * block:(bj + 1) * block] = payloads[i][bi * block:(bi + 1) * block]
    payloads = [np.frombuffer(bytes(p), np.uint8) for p in payloads]
    arena, offs, lens = W.pack(payloads)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    slots = batch.n_blocks * (block // 4096)
    assert slots > 65536 and slots // 64 >= len(payloads)
    t, ot = tables_from(payloads, block, range(0, len(payloads), 5), capacity=1 << 16)
    say("detect large payloads", block, batch.n_blocks, "blocks")
    got = check(batch, payloads, t, ot, f"large payloads, {block} blocks")
    assert (got["status"] == g.HIT_BATCH).any()


@pytest.mark.parametrize("seed", range(16))
def test_randomized_batches_detect(seed):
    """Seeded random batches through gleam_detect, on both sides of its one-kernel limits:
    block size 4-256 KiB, 1-3000 payloads of empty, tiny, leaf- and block-edge and
    multi-block lengths, repeated payloads, an optional skew, a table holding a random part
    of the digests; every output equals the oracle's and the three calls'."""
    rng = np.random.default_rng(97_000 + seed)
    block = 4096 << int(rng.integers(0, 7))
    n = int(rng.choice([1, 9, 120, 900, 3000]))
    edges = np.array([0, 1, 31, 32, 33, 4095, 4096, 4097, block - 1, block, block + 1, 2 * block + 17])
    kind = rng.integers(0, 3, n)
    lens = np.where(kind == 0, rng.choice(edges, n),
                    np.where(kind == 1, rng.integers(0, 8192, n), rng.integers(0, 3 * block + 1, n)))
    lens = np.minimum(lens, (96 << 20) // n)
    payloads = [np.frombuffer(rng.bytes(int(m)), np.uint8) for m in lens]
    for i in rng.integers(0, n, n // 8):
        payloads[int(i)] = payloads[int(rng.integers(0, n))].copy()
    skew = int(rng.choice([0, 0, 3, 8]))
    arena, offs, blens = W.pack(payloads, align=256, skew=skew)
    batch = g.Batch.from_arena(to_device(arena), offs, blens, block)
    say("randomized detect", seed, "block", block, "payloads", n, "blocks", batch.n_blocks, "skew", skew)
    dig, _ = oracle.batch_digests(payloads, block, threads=host_threads())
    held = np.unique(dig[rng.random(dig.size) < 0.3]) if dig.size else np.zeros(0, np.uint64)
    t, ot = g.Cache(1 << 16), oracle.Table()
    if held.size:
        vals = rng.integers(0, 2**63, held.size, dtype=np.uint64)
        t.insert(keys_to_device(held), keys_to_device(vals))
        ot.insert(held, vals)
    check(batch, payloads, t, ot, f"seed {seed}")
