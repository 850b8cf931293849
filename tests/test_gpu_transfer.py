"""GPU parity of the transfer around the decision (Sec. 4.1.2): the send plan and the
packed buffer equal the oracle's, and the receiver rebuilds every payload byte for byte
from the plan, the packed bytes and the copies it holds."""

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


def check_round_trip(payloads, block, held_blocks, skew=0):
    """held_blocks: byte strings the receiver already holds (one block each)."""
    # the receiver's held copies, in device memory; table values = their addresses
    pool = to_device(np.frombuffer(b"".join(held_blocks), np.uint8).copy()) if held_blocks else None
    table = g.Cache(1 << 12)
    otable = oracle.Table()
    if held_blocks:
        keys = np.concatenate([oracle.payload_digests(np.frombuffer(b, np.uint8), block)[0] for b in held_blocks])
        addrs = np.array([pool.data_ptr() + i * block for i in range(len(held_blocks))], np.uint64)
        table.insert(keys_to_device(keys), keys_to_device(addrs))
        otable.insert(keys, addrs)
    arena, offs, lens = W.pack(payloads, skew=skew)
    src = g.Batch.from_arena(to_device(arena), offs, lens, block)
    d = g.fp_chunks(src)
    status, ref = table.lookup(d)
    records, totals = g.send_plan(src, d, status, ref)
    torch.cuda.synchronize()
    tot = u64(totals)
    packed = torch.zeros(max(int(tot[3]), 1), dtype=torch.uint8, device="cuda")
    g.pack_misses(src, records, packed)
    # oracle side
    res = oracle.run(payloads, block, otable)
    erec, etot = oracle.send_plan([p.size for p in payloads], block, res["digests"], res["status"], res["ref"])
    epacked = oracle.pack_misses(payloads, erec, int(etot[3]))
    rec = g.records_to_numpy(records)
    assert np.array_equal(tot, etot)
    assert np.array_equal(rec, erec)
    assert np.array_equal(packed.cpu().numpy()[:int(tot[3])], epacked)
    # receiver: fresh zeroed destinations with the same geometry
    dst_arena, doffs, dlens = W.pack([np.zeros(p.size, np.uint8) for p in payloads], skew=(skew + 5) % 16)
    d_dst = to_device(dst_arena)
    dst = g.Batch.from_arena(d_dst, doffs, dlens, block)
    g.restore_blocks(dst, records, packed, held=ref)
    torch.cuda.synchronize()
    out = d_dst.cpu().numpy()
    for p, o in zip(payloads, doffs.tolist()):
        assert np.array_equal(out[o:o + p.size], p)
    return tot


@pytest.mark.parametrize("block,skew", [(4096, 0), (65536, 0), (65536, 3), (1 << 20, 0), (2 << 20, 8)])
def test_plan_pack_restore(block, skew):
    rng = np.random.default_rng(1100 + block.bit_length() + skew)
    pool = [rng.bytes(block) for _ in range(10)]
    payloads = []
    for _ in range(30):
        parts = [pool[int(i)] for i in rng.integers(0, 10, int(rng.integers(0, 5)))]
        payloads.append(np.frombuffer(b"".join(parts) + rng.bytes(int(rng.integers(0, block))), np.uint8))
    payloads += [np.zeros(0, np.uint8), np.frombuffer(rng.bytes(17), np.uint8)]
    say("transfer block", block, "skew", skew)
    tot = check_round_trip(payloads, block, pool[:4], skew)
    assert tot[0] > 0 and tot[1] > 0 and tot[2] > 0


@pytest.mark.timeout(900)
def test_transfer_decoder7b_full():
    """Sender: the perturbed payload against a table of the base weights whose values are
    the addresses of the receiver's base copy; receiver: rebuild all 13.5 GB."""
    threads = host_threads()
    dec = W.Decoder()
    block = W.DECODER_BLOCK
    say("transfer decoder7b generate")
    arena, offs, lens = dec.arena(perturbed=True, threads=threads)
    base_arena, _, _ = dec.arena(perturbed=False, threads=threads)
    d_pay = to_device(arena)
    d_base = to_device(base_arena)
    del base_arena
    src = g.Batch.from_arena(d_pay, offs, lens, block)
    base = g.Batch.from_arena(d_base, offs, lens, block)
    bd = g.fp_chunks(base)
    addrs = torch.from_numpy(np.array([d_base.data_ptr() + int(o) + j * block
                                       for o, n in zip(offs, lens) for j in range(-(-int(n) // block))],
                                      np.uint64).view(np.int64)).to("cuda")
    table = g.Cache(1 << 15)
    table.insert(bd, addrs)
    say("transfer decoder7b plan/pack/restore")
    d = g.fp_chunks(src)
    status, ref = table.lookup(d)
    records, totals = g.send_plan(src, d, status, ref)
    torch.cuda.synchronize()
    tot = u64(totals)
    assert tot.tolist() == [1158, 11759, 0, 1158 * block]
    packed = torch.empty(int(tot[3]), dtype=torch.uint8, device="cuda")
    g.pack_misses(src, records, packed)
    dst_t = torch.zeros_like(d_pay)
    dst = g.Batch.from_arena(dst_t, offs, lens, block)
    g.restore_blocks(dst, records, packed, held=ref)
    torch.cuda.synchronize()
    assert torch.equal(dst_t, d_pay)
    # the plan against the oracle on the host
    payloads = [arena[int(o):int(o) + int(n)] for o, n in zip(offs, lens)]
    ot = oracle.Table()
    ot.insert(g.as_u64(bd), g.as_u64(addrs))
    res = oracle.run(payloads, block, ot, threads=threads)
    erec, etot = oracle.send_plan(lens, block, res["digests"], res["status"], res["ref"])
    assert np.array_equal(g.records_to_numpy(records), erec) and np.array_equal(tot, etot)


def test_malformed_records_are_skipped():
    """Records that the kernels' own checks reject are skipped: a payload index past the
    batch, a block running past its payload's end, packed bytes past the buffer (also
    with an offset that would wrap 2^64), and an unknown kind. Every other block is
    packed and restored as planned."""
    rng = np.random.default_rng(77)
    block = 4096
    payloads = [np.frombuffer(rng.bytes(n), np.uint8) for n in (3 * block, 2 * block + 100, block, 5000)]
    payloads.append(payloads[0].copy())  # repeats payload 0: HIT_BATCH blocks
    arena, offs, lens = W.pack(payloads)
    src = g.Batch.from_arena(to_device(arena), offs, lens, block)
    d = g.fp_chunks(src)
    status, ref = g.Cache(1 << 10).lookup(d)
    records, totals = g.send_plan(src, d, status, ref)
    torch.cuda.synchronize()
    rec = g.records_to_numpy(records).copy()
    n_packed = int(u64(totals)[3])
    miss = np.flatnonzero(rec["kind"] == g.MISS)
    batch_rep = np.flatnonzero(rec["kind"] == g.HIT_BATCH)
    assert miss.size >= 5 and batch_rep.size >= 2
    bad = {}
    r = rec.copy()
    r["payload"][miss[0]] = len(payloads) + 3            # no such payload
    r["offset"][miss[1]] = int(lens[r["payload"][miss[1]]]) - 10  # runs past the payload's end
    r["ident"][miss[2]] = n_packed - 8                    # packed bytes past the buffer
    r["ident"][miss[3]] = (1 << 64) - 8                   # ... with a wrapping offset
    r["kind"][batch_rep[0]] = 7                           # unknown kind
    for k, i in enumerate((miss[0], miss[1], miss[2], miss[3], batch_rep[0])):
        bad[int(i)] = k
    d_rec = torch.from_numpy(r.view(np.uint8).copy()).to("cuda")
    say("malformed records: pack")
    packed = torch.zeros(max(n_packed, 1), dtype=torch.uint8, device="cuda")
    g.pack_misses(src, d_rec, packed)
    dst_arena, doffs, dlens = W.pack([np.zeros(p.size, np.uint8) for p in payloads])
    d_dst = to_device(dst_arena)
    dst = g.Batch.from_arena(d_dst, doffs, dlens, block)
    say("malformed records: restore")
    g.restore_blocks(dst, d_rec, packed, held=None)
    torch.cuda.synchronize()
    got_packed = packed.cpu().numpy()
    out = d_dst.cpu().numpy()
    for i in range(rec.size):
        p, o, n, kind = int(rec["payload"][i]), int(rec["offset"][i]), int(rec["length"][i]), int(rec["kind"][i])
        got = out[int(doffs[p]) + o:int(doffs[p]) + o + n]
        if i in bad:
            assert not got.any(), f"record {i} should have been skipped"
        elif kind == g.MISS:
            ident = int(rec["ident"][i])
            assert np.array_equal(got_packed[ident:ident + n], payloads[p][o:o + n]), f"packed block {i}"
            assert np.array_equal(got, payloads[p][o:o + n]), f"restored block {i}"
        elif kind == g.HIT_BATCH and int(rec["ident"][i]) not in bad:
            assert np.array_equal(got, payloads[p][o:o + n]), f"repeated block {i}"
        # a HIT_BATCH block repeating a skipped MISS gets that block's unwritten packed
        # bytes or nothing; either way it stays inside its own payload


@pytest.mark.parametrize("block", [4096, 1 << 20])
def test_connect_protocol_with_separate_tables(block):
    """The paper's flow (Sec. 4.1.2) with a client and a server table:
    1. at connect the server sends its identifier set (export of its table, whose values
       are the device addresses of the blocks it holds);
    2. the client builds its own table from those identifiers, fingerprints its
       payloads, looks them up, plans and packs;
    3. the server resolves each HIT_CACHE digest it receives through its own table
       (digest -> address of its copy) and rebuilds every payload."""
    rng = np.random.default_rng(5150 + block.bit_length())
    pool = [rng.bytes(block) for _ in range(8)]
    payloads = []
    for _ in range(20):
        parts = [pool[int(i)] for i in rng.integers(0, 8, int(rng.integers(0, 4)))]
        payloads.append(np.frombuffer(b"".join(parts) + rng.bytes(int(rng.integers(0, block))), np.uint8))
    # server: holds pool[:5]; table value = device address of the held copy
    held = to_device(np.frombuffer(b"".join(pool[:5]), np.uint8).copy())
    skeys = np.concatenate([oracle.payload_digests(np.frombuffer(b, np.uint8), block)[0] for b in pool[:5]])
    saddr = np.array([held.data_ptr() + i * block for i in range(5)], np.uint64)
    server = g.Cache(1 << 10)
    server.insert(keys_to_device(skeys), keys_to_device(saddr))
    say("connect protocol: export", block)
    keys, _, _, count = server.export()
    torch.cuda.synchronize()
    shipped = keys[:int(count.item())].clone()  # the identifier set sent at connect
    # client: its own table holds only the identifiers
    client = g.Cache(1 << 10)
    client.insert(shipped, torch.zeros_like(shipped))
    arena, offs, lens = W.pack(payloads)
    src = g.Batch.from_arena(to_device(arena), offs, lens, block)
    d = g.fp_chunks(src)
    status, ref = client.lookup(d)
    records, totals = g.send_plan(src, d, status, ref)
    torch.cuda.synchronize()
    tot = u64(totals)
    assert tot[1] > 0 and tot[0] > 0
    packed = torch.zeros(max(int(tot[3]), 1), dtype=torch.uint8, device="cuda")
    g.pack_misses(src, records, packed)
    # server: digest -> held address for the HIT_CACHE records
    rec = g.records_to_numpy(records)
    idents = keys_to_device(rec["ident"].astype(np.uint64))
    sstatus, saddr_of = server.lookup(idents)
    torch.cuda.synchronize()
    hc = rec["kind"] == g.HIT_CACHE
    assert np.all(sstatus.cpu().numpy()[hc] == g.HIT_CACHE)  # the server holds every block the client skipped
    dst_arena, doffs, dlens = W.pack([np.zeros(p.size, np.uint8) for p in payloads], skew=3)
    d_dst = to_device(dst_arena)
    dst = g.Batch.from_arena(d_dst, doffs, dlens, block)
    say("connect protocol: restore", block)
    g.restore_blocks(dst, records, packed, held=saddr_of)
    torch.cuda.synchronize()
    out = d_dst.cpu().numpy()
    for p, o in zip(payloads, doffs.tolist()):
        assert np.array_equal(out[o:o + p.size], p)
    # bytes that crossed the network: the packed MISS blocks, not the held ones
    assert int(tot[3]) < int(lens.sum())
