"""The binding on a stream other than torch's current one: every call's own allocations
and fills run on the stream its kernels run on, so results do not depend on which
stream torch considers current, and a counter the binding zeroes is zeroed before the
kernel that writes it (not after, on another stream)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23115_amd as g
import workloads as W
from gpu_util import host_threads, keys_to_device, say, to_device, u64

pytestmark = pytest.mark.gpu

BLOCK = 65536


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def payloads(seed):
    rng = np.random.default_rng(seed)
    lens = [0, 1, 31, 4095, 4097, BLOCK - 1, BLOCK, 3 * BLOCK + 12345, 200_000]
    out = [np.frombuffer(rng.bytes(n), np.uint8) for n in lens]
    out.append(out[7].copy())  # a repeat: HIT_BATCH blocks
    return out


def run_on(stream, batch, table, remap, probe):
    """Every output allocated by the binding, on `stream` (None: torch's current)."""
    d = g.fp_chunks(batch, stream=stream)
    st, ref = table.lookup(d, stream=stream)
    idx, cnt = g.miss_compact(st, batch, stream=stream)
    md5, _, _ = g.md5_prefix(batch, stream=stream)
    tr = remap.translate(probe, stream=stream)
    match, _, weight = g.identify_weights(batch, d, [0, batch.n_seg], stream=stream)
    return d, st, ref, idx, cnt, md5, tr, match, weight


def host(outs):
    h = [u64(t) if t.dtype == torch.int64 else t.cpu().numpy() for t in outs]
    h[3] = h[3][:int(h[4][0])]  # the miss list is valid up to the miss count only
    return h


@pytest.mark.parametrize("kind", ["stream", "handle"])
def test_side_stream_matches_current_stream(kind):
    p = payloads(2100)
    arena, offs, lens = W.pack(p)
    batch = g.Batch.from_arena(to_device(arena), offs, lens, BLOCK)
    table = g.Cache(1 << 12)
    first = g.fp_chunks(g.Batch.from_arena(to_device(arena), offs[:3], lens[:3], BLOCK))
    table.insert(first, torch.arange(first.numel(), dtype=torch.int64, device="cuda"))
    remap = g.Remap(64)
    remap.update(add_start=keys_to_device(np.array([1 << 40], np.uint64)),
                 add_len=keys_to_device(np.array([1 << 20], np.uint64)),
                 add_target=keys_to_device(np.array([7 << 32], np.uint64)))
    probe = keys_to_device(np.array([(1 << 40) + 5, (1 << 40) - 1, (1 << 40) + (1 << 20)], np.uint64))
    torch.cuda.synchronize()
    say("streams", kind)
    want = host(run_on(None, batch, table, remap, probe))
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    got = host(run_on(side if kind == "stream" else side.cuda_stream, batch, table, remap, probe))
    side.synchronize()
    for a, b in zip(got, want):
        assert np.array_equal(a, b)
    # and the path itself against the oracle
    t = oracle.Table()
    fd, _ = oracle.batch_digests(p[:3], BLOCK)
    t.insert(fd, np.arange(fd.size, dtype=np.uint64))
    res = oracle.run(p, BLOCK, t, threads=host_threads())
    assert np.array_equal(want[0], res["digests"]) and np.array_equal(want[1], res["status"])
    assert int(want[4][0]) == res["miss_count"] and int(want[4][1]) == res["miss_bytes"]
    assert want[6].tolist() == [(7 << 32) + 5, g.UNMAPPED, g.UNMAPPED]
    assert want[7].all() and want[8].tolist() == [1]


def test_binding_zeroed_counters_precede_the_kernel():
    """Torch's current stream is kept busy with a long read while compaction and the
    calibration read run on a side stream with counters the binding creates: the zeroing
    must be ordered before the kernel that writes them."""
    rng = np.random.default_rng(2200)
    n = 40_000
    status = rng.choice(np.array([0, 1, 2], np.uint8), n, p=[0.4, 0.4, 0.2])
    lens = []
    left = n
    while left:
        k = int(min(left, rng.integers(1, 4)))
        lens.append((k - 1) * 4096 + int(rng.integers(1, 4097)))
        left -= k
    batch = g.Batch(np.zeros(len(lens), np.uint64), lens, 4096)
    d_status = to_device(status)
    src = torch.randint(0, 256, (1 << 20,), dtype=torch.uint8, device="cuda")
    busy = torch.empty(1 << 31, dtype=torch.uint8, device="cuda")
    want_sink = u64(g.read_stream(src))[0]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    say("zeroed counters behind a busy current stream")
    for _ in range(3):
        g.read_stream(busy, sink=torch.zeros(1, dtype=torch.int64, device="cuda"))  # current stream: ~0.3 ms
        _, counters = g.miss_compact(d_status, batch, stream=side)
        sink = g.read_stream(src, stream=side)
        side.synchronize()
        torch.cuda.synchronize()
        _, blen = oracle.geometry(lens, 4096)
        _, ecnt, ebytes = oracle.compact(status, blen)
        assert u64(counters).tolist() == [ecnt, ebytes]
        assert u64(sink)[0] == want_sink


def test_preload_then_calls_work():
    """gleam_preload loads every source file's GPU code on the device; the calls work
    after it as before, and calling it again is harmless."""
    say("preload")
    g.preload()
    g.preload()
    buf = torch.randint(0, 256, (1 << 20,), dtype=torch.uint8, device="cuda")
    batch = g.Batch.from_arena(buf, [0], [buf.numel()], 65536)
    d = g.fp_chunks(batch)
    torch.cuda.synchronize()
    want, _ = oracle.batch_digests([buf.cpu().numpy()], 65536)
    assert np.array_equal(g.as_u64(d), want)
