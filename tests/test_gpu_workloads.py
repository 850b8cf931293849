"""GPU parity at the workloads' full sizes, in the launch configuration bench.py times:
every block digest, status, ref and the miss list/count/bytes equal the oracle's, and
the planted truth holds. The oracle computes every output (it digests tens of GB in
seconds across host threads), so nothing is sampled.

Table contents on both sides come from the oracle's digests (never from the GPU path).
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23115_amd as g
import workloads as W
from gpu_util import assert_same, detect_path, host_threads, keys_to_device, run_path, say, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def gpu_table(capacity, keys, vals, max_load=0.7):
    t = g.Cache(capacity, max_load=max_load)
    if len(keys):
        t.insert(keys_to_device(keys), keys_to_device(vals))
    return t


def test_resnet50_full():
    block = W.RESNET_BLOCK
    payloads = W.resnet50_payloads()
    cached = W.resnet50_cached_tensors()
    ot = oracle.Table()
    keys, vals = [], []
    for t in cached.tolist():
        d, _ = oracle.payload_digests(payloads[t], block)
        keys.append(d)
        vals.append(np.full(d.size, t, np.uint64))
    keys, vals = np.concatenate(keys), np.concatenate(vals)
    ot.insert(keys, vals)
    arena, offs, lens = W.pack(payloads)
    say("resnet50 full", int(lens.sum()), "bytes")
    batch = g.Batch.from_arena(to_device(arena), offs, lens, block)
    gpu = run_path(batch, gpu_table(1 << 12, keys, vals), with_leaves=True)
    ref = oracle.run(payloads, block, ot, threads=host_threads())
    assert_same(gpu, ref, "resnet50")
    assert_same(detect_path(batch, gpu_table(1 << 12, keys, vals)), ref, "resnet50 detect")
    _, leaves = oracle.batch_digests(payloads, block, with_leaves=True, threads=host_threads())
    assert np.array_equal(gpu["leaves"], leaves)
    first = batch.host_first
    expect = np.zeros(batch.n_blocks, np.uint8)
    for t in cached.tolist():
        expect[int(first[t]):int(first[t + 1])] = g.HIT_CACHE
    assert np.array_equal(gpu["status"], expect)


@pytest.mark.parametrize("skew,n", [(0, 100_000), (5, 20_000)])
def test_small_copies(skew, n):
    sc = W.SmallCopies(n=n, skew=skew)
    payloads = sc.payloads()
    say("small copies n", n, "skew", skew, "bytes", int(sc.sizes.sum()))
    batch = g.Batch.from_arena(to_device(sc.arena), sc.offsets, sc.sizes, W.SMALL_BLOCK)
    gpu = run_path(batch, g.Cache(1 << 10))
    ref = oracle.run(payloads, W.SMALL_BLOCK, oracle.Table(), threads=host_threads())
    assert_same(gpu, ref, "small copies")
    say("small copies detect n", n, "skew", skew)
    assert_same(detect_path(batch, g.Cache(1 << 10)), ref, "small copies detect")
    assert int((gpu["status"] == g.HIT_BATCH).sum()) == sc.targets.size
    assert gpu["miss_count"] == batch.n_blocks - sc.targets.size


@pytest.mark.timeout(900)
def test_decoder7b_full():
    threads = host_threads()
    dec = W.Decoder()
    block = W.DECODER_BLOCK
    say("decoder7b generate")
    arena, offs, lens = dec.arena(perturbed=True, threads=threads)
    payloads = [arena[int(o):int(o) + int(n)] for o, n in zip(offs, lens)]
    # the table: oracle digests of the base weights (payload bytes where unperturbed)
    digests, _ = oracle.batch_digests(payloads, block, threads=threads)
    first = oracle.geometry(lens, block)[0]
    base_digests = digests.copy()
    for i in dec.perturbed:
        bd, _ = oracle.payload_digests(dec.base(i), block)
        base_digests[int(first[i]):int(first[i + 1])] = bd
    ot = oracle.Table()
    bidx = np.arange(base_digests.size, dtype=np.uint64)
    ot.insert(base_digests, bidx)
    say("decoder7b gpu path", int(lens.sum()), "bytes")
    d_arena = to_device(arena)
    batch = g.Batch.from_arena(d_arena, offs, lens, block)
    gpu = run_path(batch, gpu_table(1 << 15, base_digests, bidx))
    status, ref = oracle.lookup(digests, ot)
    _, blen = oracle.geometry(lens, block)
    midx, mcnt, mbytes = oracle.compact(status, blen)
    want = {"digests": digests, "status": status, "ref": ref, "miss_idx": midx, "miss_count": mcnt,
            "miss_bytes": mbytes}
    assert_same(gpu, want, "decoder7b")
    say("decoder7b detect")
    assert_same(detect_path(batch, gpu_table(1 << 15, base_digests, bidx)), want, "decoder7b detect")
    assert mcnt == 1158 and int((status == g.HIT_CACHE).sum()) == 11759


@pytest.mark.timeout(1200)
def test_large_bf16_40gb():
    threads = host_threads()
    ls = W.LargeSet()
    block = W.LARGE_BLOCK
    say("large bf16 generate 40 GB")
    arena, offs, lens = ls.arena(threads=threads)
    payloads = [arena[int(o):int(o) + int(n)] for o, n in zip(offs, lens)]
    digests, _ = oracle.batch_digests(payloads, block, threads=threads)
    n = digests.size
    rand = ls.random_digests()
    chosen = ls.cached_blocks(n)
    assert not np.isin(rand, digests).any()
    keys = np.concatenate([rand, digests[chosen]])
    vals = np.concatenate([np.zeros(rand.size, np.uint64), chosen.astype(np.uint64)])
    ot = oracle.Table()
    ot.insert(keys, vals)
    say("large bf16 gpu path", n, "blocks")
    d_arena = to_device(arena)
    del arena
    batch = g.Batch.from_arena(d_arena, offs, lens, block)
    table = gpu_table(1 << 25, keys, vals, max_load=0.65)
    gpu = run_path(batch, table)
    status, ref = oracle.lookup(digests, ot)
    _, blen = oracle.geometry(lens, block)
    midx, mcnt, mbytes = oracle.compact(status, blen)
    want = {"digests": digests, "status": status, "ref": ref, "miss_idx": midx, "miss_count": mcnt,
            "miss_bytes": mbytes}
    assert_same(gpu, want, "large bf16")
    say("large bf16 detect")
    assert_same(detect_path(batch, table), want, "large bf16 detect")
    expect = np.zeros(n, np.uint8)
    expect[chosen] = g.HIT_CACHE
    assert np.array_equal(gpu["status"], expect)
