"""GPU parity of the address-remap map (Sec. 4.1.3, Weight Chunk Sharing; Appendix,
Implementation Details, Virtual Memory Map): after every update the statuses, counts and exported intervals equal the
oracle's bit for bit, and so does the translation of every probed address."""

import numpy as np
import pytest
import torch

import paper_2607_23115_amd as g
import workloads
from gpu_util import keys_to_device, say, u64
from oracle import remap as oremap

pytestmark = pytest.mark.gpu

TOP = (1 << 64) - 1


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def dev(a) -> torch.Tensor:
    return keys_to_device(np.asarray(a, dtype=np.uint64).reshape(-1))


def update_both(m, om, rem=((), ()), add=((), (), ())):
    rs, rl = (np.asarray(x, np.uint64) for x in rem)
    a_s, a_l, a_t = (np.asarray(x, np.uint64) for x in add)
    st, counts = m.update(dev(rs) if rs.size else None, dev(rl) if rs.size else None,
                          dev(a_s) if a_s.size else None, dev(a_l) if a_s.size else None,
                          dev(a_t) if a_s.size else None)
    torch.cuda.synchronize()
    est, ecounts = om.update(rs, rl, a_s, a_l, a_t)
    return st.cpu().numpy(), tuple(int(c) for c in u64(counts)), est, tuple(ecounts)


def assert_map(m, om, what):
    s, n, t, c = m.export()
    torch.cuda.synchronize()
    k = int(c.item())
    es, en, et = om.export()
    assert k == es.size, f"{what}: count"
    assert np.array_equal(u64(s)[:k], es), f"{what}: starts"
    assert np.array_equal(u64(n)[:k], en), f"{what}: lengths"
    assert np.array_equal(u64(t)[:k], et), f"{what}: targets"


def probes(om, rng, n_random, space):
    """Random addresses plus every interval's first, last, one-past-last and one-before."""
    s, n, _ = om.export()
    edge = np.concatenate([s, s + n - np.uint64(1), s + n, s - np.uint64(1)]) if s.size else np.zeros(0, np.uint64)
    rnd = rng.integers(0, space, n_random, dtype=np.uint64)
    return np.concatenate([edge, rnd, np.array([0, TOP, TOP - 1], np.uint64)])


def assert_translate(m, om, addrs, what):
    got = u64(m.translate(dev(addrs)))
    torch.cuda.synchronize()
    assert np.array_equal(got, om.translate(addrs)), f"{what}: translation"


@pytest.mark.parametrize("cap,space", [(1, 64), (16, 128), (200, 2000), (5000, 40000)])
def test_random_update_sequence(cap, space):
    rng = np.random.default_rng(cap)
    m, om = g.Remap(cap), oremap.RemapMap(cap)
    for step in range(40):
        n_del = int(rng.integers(0, 1 + max(2, cap // 20)))
        n_add = int(rng.integers(0, 1 + max(4, cap // 4)))
        maxlen = max(4, space // max(cap, 1))
        rem = (rng.integers(0, space, n_del, dtype=np.uint64), rng.integers(0, 2 * maxlen, n_del, dtype=np.uint64))
        add = (rng.integers(0, space, n_add, dtype=np.uint64), rng.integers(0, maxlen, n_add, dtype=np.uint64),
               rng.integers(0, 1 << 62, n_add, dtype=np.uint64))
        say("remap sequence cap", cap, "step", step, "n_del", n_del, "n_add", n_add)
        st, counts, est, ecounts = update_both(m, om, rem, add)
        assert np.array_equal(st, est), f"step {step}: statuses"
        assert counts == ecounts, f"step {step}: counts"
        assert_map(m, om, f"step {step}")
        assert_translate(m, om, probes(om, rng, 500, space + 16), f"step {step}")


def test_edges_of_the_address_space():
    say("remap edges")
    m, om = g.Remap(8), oremap.RemapMap(8)
    add = ([0, TOP - 5, TOP - 3, 100, 200, 300, TOP, 50], [1, 5, 4, 0, 8, 8, 1, TOP],
           [TOP - 1, 7, 9, 1, TOP - 8, TOP - 7, 0, 0])
    st, counts, est, ecounts = update_both(m, om, add=add)
    assert np.array_equal(st, est) and counts == ecounts
    assert st.tolist() == [0, 0, 1, 1, 0, 1, 1, 1]
    assert_translate(m, om, np.array([0, 1, TOP - 5, TOP - 1, TOP, 207, 199, 208], np.uint64), "edges")
    # removal clipped at 2^64; empty removal; removal of everything
    for rem in (([TOP - 2], [TOP]), ([203], [0]), ([0], [TOP])):
        st, counts, est, ecounts = update_both(m, om, rem=rem)
        assert counts == ecounts, rem
        assert_map(m, om, f"removal {rem}")


def test_no_op_update_and_empty_map():
    say("remap no-op")
    m, om = g.Remap(4), oremap.RemapMap(4)
    st, counts, est, ecounts = update_both(m, om)
    assert counts == ecounts == (0, 0, 0, 0)
    assert_translate(m, om, np.array([0, 5, TOP], np.uint64), "empty")
    update_both(m, om, add=([10], [5], [1000]))
    st, counts, est, ecounts = update_both(m, om, rem=([100], [5]))
    assert counts == ecounts == (1, 0, 0, 0)


def test_full_leaves_the_map_unchanged():
    say("remap full")
    m, om = g.Remap(3), oremap.RemapMap(3)
    update_both(m, om, add=([0, 10], [5, 5], [100, 200]))
    st, counts, est, ecounts = update_both(m, om, rem=([0], [1]), add=([20, 30, 40, 40], [1, 1, 1, 0], [1, 2, 3, 4]))
    assert st.tolist() == est.tolist() == [3, 3, 3, 1]
    assert counts == ecounts == (2, 0, 0, 4)
    assert_map(m, om, "after FULL")


def test_paper_two_chunks_in_one_allocation():
    """Sec. 4.1.3: two chunks of one client allocation map into two server allocations."""
    say("remap paper case")
    va = (3 << 40) + 0x4000
    pos1, pos2 = 0x7F00_0000_0000, 0x7F80_0000_1000
    m, om = g.Remap(16), oremap.RemapMap(16)
    st, counts, est, ecounts = update_both(m, om, add=([va, va + 0x3000], [0x3000, 0x500], [pos1, pos2]))
    assert st.tolist() == [0, 0]
    probe = np.array([va, va + 0x2FFF, va + 0x3000, va + 0x3004, va + 0x34FF, va + 0x3500, va - 1], np.uint64)
    got = u64(m.translate(dev(probe)))
    assert got.tolist() == [pos1, pos1 + 0x2FFF, pos2, pos2 + 4, pos2 + 0x4FF, TOP, TOP]


def test_many_tasks_workload():
    """256 tasks (the 7B decoder, ResNet-50 and the 2,000-tensor set) mapped at once, 2^20
    pointers translated, then tasks freed and new ones loaded in one update."""
    tasks = workloads.RemapTasks(256)
    start, length, target = tasks.intervals()
    cap = 1 << 18
    m, om = g.Remap(cap), oremap.RemapMap(cap)
    say("remap tasks: load", start.size, "intervals")
    st, counts, est, ecounts = update_both(m, om, add=(start, length, target))
    assert counts == ecounts and counts[1] == start.size
    assert_map(m, om, "tasks loaded")
    ptr = tasks.pointers(1 << 20)
    say("remap tasks: translate", ptr.size)
    assert_translate(m, om, ptr, "tasks")
    # free 16 tasks (their whole 1 TB spaces) and load the intervals of 16 others shifted
    # into the freed spaces
    gone = np.arange(0, 256, 16)
    rem = (gone.astype(np.uint64) << np.uint64(40), np.full(gone.size, 1 << 40, np.uint64))
    s2, l2, t2 = tasks.intervals(gone + 1)
    s2 = s2 - np.uint64(1 << 40)
    say("remap tasks: replace", gone.size, "tasks")
    st, counts, est, ecounts = update_both(m, om, rem=rem, add=(s2, l2, t2))
    assert np.array_equal(st, est) and counts == ecounts
    assert counts[1] == s2.size and counts[2] > 0
    assert_map(m, om, "tasks replaced")
    assert_translate(m, om, ptr, "tasks replaced")


@pytest.mark.parametrize("count", [4097, 8191, 8192, 8193, 16_384, 16_385, 24_577])
def test_fence_strides(count):
    """Translation searches a fence of every S-th start (S = ceil(count / 8192)) first:
    probe every interval edge at counts around the stride changes, then shrink the map."""
    rng = np.random.default_rng(count)
    start = np.sort(rng.choice(1 << 30, count, replace=False).astype(np.uint64)) * np.uint64(4)
    length = rng.integers(1, 5, count, dtype=np.uint64)
    target = rng.integers(0, 1 << 62, count, dtype=np.uint64)
    m, om = g.Remap(count), oremap.RemapMap(count)
    say("remap fence: count", count)
    st, counts, est, ecounts = update_both(m, om, add=(start, length, target))
    assert counts == ecounts and counts[0] == count
    assert_translate(m, om, probes(om, rng, 10_000, 1 << 33), f"fence {count}")
    keep = start[::1000]
    st, counts, est, ecounts = update_both(m, om, rem=([0], [1 << 33]), add=(keep, length[::1000], target[::1000]))
    assert counts == ecounts and counts[0] == keep.size
    assert_translate(m, om, probes(om, rng, 10_000, 1 << 33), f"fence {count} shrunk")


@pytest.mark.parametrize("n_add,n_del", [(1, 1), (2047, 2048), (2048, 2049), (2049, 5), (3000, 2047),
                                         (16_384, 16_385), (16_385, 3)])
def test_one_workgroup_and_batched_updates(n_add, n_del):
    """Batches of up to 2048 removals or additions run in one workgroup, larger ones
    through the radix sort and scans: both sides of the switch, with clashes, invalid
    additions and empty removal ranges mixed in."""
    rng = np.random.default_rng(n_add * 7 + n_del)
    space = 1 << 20
    m, om = g.Remap(1 << 14), oremap.RemapMap(1 << 14)
    base = (rng.choice(space // 64, 4000, replace=False).astype(np.uint64) * np.uint64(64),
            rng.integers(1, 64, 4000, dtype=np.uint64), rng.integers(0, 1 << 62, 4000, dtype=np.uint64))
    update_both(m, om, add=base)
    for step in range(3):
        rem = (rng.integers(0, space, n_del, dtype=np.uint64), rng.integers(0, 200, n_del, dtype=np.uint64))
        a_len = rng.integers(0, 300, n_add, dtype=np.uint64)
        add = (rng.integers(0, space, n_add, dtype=np.uint64), a_len, rng.integers(0, 1 << 62, n_add,
                                                                                   dtype=np.uint64))
        say("remap switch-over n_add", n_add, "n_del", n_del, "step", step)
        st, counts, est, ecounts = update_both(m, om, rem, add)
        assert np.array_equal(st, est), f"step {step}: statuses"
        assert counts == ecounts, f"step {step}: counts"
        assert_map(m, om, f"step {step}")
        assert_translate(m, om, probes(om, rng, 2000, space), f"step {step}")


def test_beyond_one_grid_pass():
    """More candidates than one pass of the capped grid (8192 x 256 lanes)."""
    n = 3_000_000
    rng = np.random.default_rng(77)
    start = np.sort(rng.choice(1 << 40, n, replace=False).astype(np.uint64)) * np.uint64(8)
    length = rng.integers(1, 9, n, dtype=np.uint64)
    target = rng.integers(0, 1 << 60, n, dtype=np.uint64)
    perm = rng.permutation(n)
    m, om = g.Remap(1 << 22), oremap.RemapMap(1 << 22)
    say("remap grid-stride: add", n)
    st, counts, est, ecounts = update_both(m, om, add=(start[perm], length[perm], target[perm]))
    assert np.array_equal(st, est) and counts == ecounts
    say("remap grid-stride: remove 1/3 and add overlapping")
    rem = (start[::3], np.ones(start[::3].size, np.uint64))
    add = (start[1::5] + np.uint64(4), np.full(start[1::5].size, 2, np.uint64),
           np.zeros(start[1::5].size, np.uint64))
    st, counts, est, ecounts = update_both(m, om, rem=rem, add=add)
    assert np.array_equal(st, est) and counts == ecounts
    assert_map(m, om, "grid-stride")
    probe = np.concatenate([start[:: 7], start[::11] + np.uint64(5), rng.integers(0, 1 << 43, 10**5,
                                                                                  dtype=np.uint64)])
    assert_translate(m, om, probe, "grid-stride")


def test_translate_replays_in_a_graph():
    """Translation enqueues one kernel launch and reads the map's own count, so a captured
    graph sees later updates on every replay."""
    say("remap graph")
    m, om = g.Remap(64), oremap.RemapMap(64)
    update_both(m, om, add=([0, 100], [50, 50], [1000, 5000]))
    addrs = dev(np.arange(0, 200, 3, dtype=np.uint64))
    out = torch.empty(addrs.numel(), dtype=torch.int64, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        m.translate(addrs, out=out, stream=s)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=s):
            m.translate(addrs, out=out, stream=s)
    torch.cuda.synchronize()
    host = np.arange(0, 200, 3, dtype=np.uint64)
    for k in range(3):
        out.fill_(0)
        update_both(m, om, add=([200 + 10 * k], [5], [7]))
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(u64(out), om.translate(host)), f"replay {k}"


def test_binding_refusals():
    say("remap refusals")
    m = g.Remap(4)
    with pytest.raises(ValueError):
        m.update(add_start=dev([1, 2]), add_len=dev([1]), add_target=dev([1, 2]))
    with pytest.raises(ValueError):
        m.translate(torch.zeros(4, dtype=torch.int32, device="cuda"))
    with pytest.raises(g.GleamError) as e:
        m.update(add_start=dev([1]), add_len=dev([1]), add_target=dev([1]),
                 ws=torch.empty(256, dtype=torch.uint8, device="cuda"))
    assert e.value.status == g.E_WORKSPACE
    m.close()
    with pytest.raises(g.GleamError):
        m.translate(dev([1]))


def test_update_replays_in_a_graph():
    """gleam_remap_update with batches past the one-workgroup size (so through the radix
    sort and scans) captured once: it clears a region and maps new intervals inside it,
    so every replay gives the same map, whatever eager updates outside the region did in
    between; statuses, counts, export and translation equal the oracle's each time."""
    rng = np.random.default_rng(2400)
    space, region = 1 << 24, (1 << 22, 1 << 23)
    m, om = g.Remap(1 << 15), oremap.RemapMap(1 << 15)
    n0 = 6000
    base_s = np.sort(rng.choice(space // 256, n0, replace=False).astype(np.uint64)) * np.uint64(256)
    update_both(m, om, add=(base_s, rng.integers(1, 256, n0, dtype=np.uint64),
                            rng.integers(0, 1 << 60, n0, dtype=np.uint64)))
    n_del, n_add = 3000, 2500
    r_s = np.sort(rng.choice(np.arange(region[0], region[1], 1024, dtype=np.uint64), n_del, replace=False))
    rem = (r_s, np.full(n_del, 1024, np.uint64))
    a_s = rng.choice(r_s, n_add, replace=False) + rng.integers(0, 512, n_add, dtype=np.uint64)
    add = (a_s, rng.integers(1, 256, n_add, dtype=np.uint64), rng.integers(0, 1 << 60, n_add, dtype=np.uint64))
    d = [dev(x) for x in (*rem, *add)]
    status = torch.empty(n_add, dtype=torch.uint8, device="cuda")
    counts = torch.empty(4, dtype=torch.int64, device="cuda")
    ws = m.update_workspace(n_add, n_del)

    def update_call():
        g._check(g.lib.gleam_remap_update(m.handle, g._ptr(d[0]), g._ptr(d[1]), n_del, g._ptr(d[2]), g._ptr(d[3]),
                                          g._ptr(d[4]), n_add, g._ptr(status), g._ptr(counts), g._ptr(ws),
                                          ws.numel(), g._stream(None)))

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side), torch.cuda.graph(graph, stream=side):
        update_call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for k in range(3):
        say("remap update graph replay", k)
        status.fill_(0xEE)
        counts.fill_(-1)
        graph.replay()
        torch.cuda.synchronize()
        est, ecounts = om.update(*rem, *add)
        assert np.array_equal(status.cpu().numpy(), est), f"replay {k}: statuses"
        got = tuple(int(c) for c in u64(counts))
        assert got[:len(ecounts)] == tuple(ecounts), f"replay {k}: counts"
        assert_map(m, om, f"replay {k}")
        assert_translate(m, om, probes(om, rng, 3000, space), f"replay {k}")
        # eager work between replays, outside the region
        out_s = rng.integers(region[1], space, 100, dtype=np.uint64)
        update_both(m, om, rem=(out_s, np.full(100, 300, np.uint64)),
                    add=(out_s + np.uint64(50), np.full(100, 10, np.uint64), np.full(100, k, np.uint64)))
