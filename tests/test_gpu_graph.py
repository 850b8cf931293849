"""The detect path (fingerprint -> lookup -> compaction) captured once in a HIP graph and
replayed: every replay equals an eager run, with eager work and synchronisations between
replays, and a replay after the payload bytes change in place sees the new bytes. Every
step is a plain kernel launch (clears are fill kernels, nothing allocates or syncs), so
the calls are capture-safe."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23115_amd as g
import workloads as W
from gpu_util import say, u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


class Path:
    def __init__(self, batch, table):
        n = batch.n_blocks
        self.batch, self.table = batch, table
        self.d = torch.empty(n, dtype=torch.int64, device="cuda")
        self.st = torch.empty(n, dtype=torch.uint8, device="cuda")
        self.ref = torch.empty(n, dtype=torch.int64, device="cuda")
        self.idx = torch.empty(n, dtype=torch.int64, device="cuda")
        self.cnt = torch.zeros(2, dtype=torch.int64, device="cuda")
        self.ws = g.workspace(n)

    def run(self):
        g.fp_chunks(self.batch, out=self.d)
        self.table.lookup(self.d, status=self.st, ref=self.ref, ws=self.ws)
        g.miss_compact(self.st, self.batch, miss_idx=self.idx, counters=self.cnt, ws=self.ws)

    def snapshot(self):
        torch.cuda.synchronize()
        c = u64(self.cnt)
        return (u64(self.d).copy(), self.st.cpu().numpy().copy(), u64(self.ref).copy(),
                u64(self.idx)[:int(c[0])].copy(), c.copy())


def same(a, b):
    return all(np.array_equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("which", ["random16", "resnet50"])
def test_graph_replays_match_eager(which):
    if which == "random16":
        p = W.random16_payload()
        payloads, block = [p], W.RANDOM16_BLOCK
    else:
        payloads, block = W.resnet50_payloads(), W.RESNET_BLOCK
    arena, offs, lens = W.pack(payloads)
    d_arena = torch.from_numpy(arena).to("cuda")
    batch = g.Batch.from_arena(d_arena, offs, lens, block)
    table = g.Cache(1 << 12)
    half = g.Batch.from_arena(d_arena, offs[: len(offs) // 2 + 1], lens[: len(lens) // 2 + 1], block)
    table.insert(g.fp_chunks(half), torch.arange(half.n_blocks, dtype=torch.int64, device="cuda"))
    path = Path(batch, table)
    other = Path(batch, table)
    say("graph", which, "eager")
    path.run()
    eager = path.snapshot()
    # capture on a side stream (warm-up done above)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            path.run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for i in range(5):
        say("graph", which, "replay", i)
        for t in (path.d, path.st, path.ref, path.idx, path.cnt):
            t.fill_(-1 if t.dtype != torch.uint8 else 7)
        graph.replay()
        assert same(path.snapshot(), eager), f"replay {i}"
        other.run()  # eager work between replays
        assert same(other.snapshot(), eager)
    # new bytes in place: the replay sees them
    arena2 = arena.copy()
    arena2[int(offs[0]):int(offs[0]) + 100] ^= 0x5A
    d_arena.copy_(torch.from_numpy(arena2))
    graph.replay()
    replayed = path.snapshot()
    other.run()
    assert same(replayed, other.snapshot())
    ot = oracle.Table()
    hd, _ = oracle.batch_digests([arena[int(o):int(o) + int(n)] for o, n in zip(offs[: len(offs) // 2 + 1],
                                                                            lens[: len(lens) // 2 + 1])], block)
    ot.insert(hd, np.arange(hd.size, dtype=np.uint64))
    want = oracle.run([arena2[int(o):int(o) + int(n)] for o, n in zip(offs, lens)], block, ot)
    assert np.array_equal(replayed[0], want["digests"]) and np.array_equal(replayed[1], want["status"])
    assert int(replayed[4][0]) == want["miss_count"] and int(replayed[4][1]) == want["miss_bytes"]
