"""GPU parity of the table lifecycle (Sec. 4.1.3: LRU eviction of the shared cache;
Sec. 4.1.2: the identifier set shipped at connect): every export, eviction order,
count and lookup equals the oracle's after each operation of a random sequence."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23115_amd as g
from gpu_util import keys_to_device, say, u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def exported(table):
    k, v, s, c = table.export()
    torch.cuda.synchronize()
    n = int(c.item())
    return u64(k)[:n], u64(v)[:n], u64(s)[:n]


def assert_table(table, ot, what):
    k, v, s = exported(table)
    ek, ev, es = ot.export()
    assert np.array_equal(k, ek), f"{what}: keys"
    assert np.array_equal(v, ev), f"{what}: values"
    assert np.array_equal(s, es), f"{what}: stamps"


def test_random_lifecycle_sequence():
    rng = np.random.default_rng(1000)
    table, ot = g.Cache(1024, max_load=0.9), oracle.Table()
    special = np.array([0, 2**64 - 1], np.uint64)
    for step in range(80):
        op = ["insert", "touch", "touch1", "evict", "erase", "lookup"][step % 6]
        say("lifecycle step", step, op)
        if op == "insert":
            keys = np.concatenate([rng.integers(0, 600, 60, dtype=np.uint64), special[rng.integers(0, 2, 2)]])
            vals = rng.integers(0, 2**64, keys.size, dtype=np.uint64, endpoint=False)
            try:
                n_new = table.insert(keys_to_device(keys), keys_to_device(vals))
            except g.GleamError as e:
                assert e.status == g.E_CAPACITY
                continue
            assert int(n_new.item()) == ot.insert(keys, vals)
        elif op in ("touch", "touch1"):
            keys = np.concatenate([rng.integers(0, 650, 90, dtype=np.uint64), special])
            if op == "touch":
                ep = rng.integers(1, 10_000, keys.size, dtype=np.uint64)
                hit = table.touch(keys_to_device(keys), epochs=keys_to_device(ep))
            else:
                ep = np.full(keys.size, step * 100 + 7, np.uint64)
                hit = table.touch(keys_to_device(keys), epoch=int(ep[0]))
            assert int(hit.item()) == ot.touch(keys, ep)
        elif op == "evict":
            keep = int(rng.integers(0, len(ot) + 3))
            ev, counts = table.evict(keep)
            torch.cuda.synchronize()
            want = ot.evict(keep)
            c = u64(counts)
            assert int(c[0]) == want.size and int(c[1]) == len(ot)
            assert np.array_equal(u64(ev)[:want.size], want)
        elif op == "erase":
            keys = np.concatenate([rng.integers(0, 650, 40, dtype=np.uint64), special[:1]])
            counts = table.erase(keys_to_device(keys))
            torch.cuda.synchronize()
            c = u64(counts)
            assert int(c[0]) == ot.erase(keys) and int(c[1]) == len(ot)
            table.set_key_bound(int(c[1]))
        else:
            probe = np.concatenate([np.arange(0, 660, dtype=np.uint64), special])
            st, ref = table.lookup(keys_to_device(probe))
            torch.cuda.synchronize()
            est, eref = oracle.lookup(probe, ot)
            assert np.array_equal(st.cpu().numpy(), est) and np.array_equal(u64(ref), eref)
        assert_table(table, ot, f"step {step} {op}")


def test_evict_large_table_and_restore():
    rng = np.random.default_rng(1001)
    n = 1_000_000
    keys = rng.integers(0, 2**64, n, dtype=np.uint64, endpoint=False)
    vals = np.arange(n, dtype=np.uint64)
    table, ot = g.Cache(1 << 21, max_load=0.6), oracle.Table()
    say("lifecycle large insert")
    table.insert(keys_to_device(keys), keys_to_device(vals))
    ot.insert(keys, vals)
    ep = rng.integers(0, 50, n, dtype=np.uint64)  # many equal stamps: ties go by key
    table.touch(keys_to_device(keys), epochs=keys_to_device(ep))
    ot.touch(keys, ep)
    say("lifecycle large evict")
    ev, counts = table.evict(n // 2)
    torch.cuda.synchronize()
    want = ot.evict(n // 2)
    assert np.array_equal(u64(ev)[:want.size], want)
    assert_table(table, ot, "after evict")
    # checkpoint: export, rebuild a fresh table from it, export again
    k, v, s = exported(table)
    fresh = g.Cache(1 << 21, max_load=0.6)
    fresh.insert(keys_to_device(k), keys_to_device(v))
    fresh.touch(keys_to_device(k), epochs=keys_to_device(s))
    k2, v2, s2 = exported(fresh)
    assert np.array_equal(k, k2) and np.array_equal(v, v2) and np.array_equal(s, s2)


def test_maintenance_workspace_checked():
    table = g.Cache(64)
    small = torch.empty(256, dtype=torch.uint8, device="cuda")
    with pytest.raises(g.GleamError) as e:
        table.evict(1, ws=small)
    assert e.value.status == g.E_WORKSPACE
    with pytest.raises(g.GleamError):
        table.set_key_bound(10)  # cannot raise the bound above 0


GOLDEN = 0x9E3779B97F4A7C15
GOLDEN_INV = pow(GOLDEN, -1, 1 << 64)


def keys_at_homes(rng, homes, log2_cap):
    """Keys whose table home slot (top log2_cap bits of key * GOLDEN) is the given one:
    crowded homes make long clusters of linear probing."""
    shift = 64 - log2_cap
    out = []
    for h in homes:
        r = int(rng.integers(0, 1 << 62)) & ((1 << shift) - 1)
        out.append((((int(h) << shift) | r) * GOLDEN_INV) % (1 << 64))
    return np.array(out, np.uint64)


def test_erase_long_clusters():
    """Keys crowded onto a few home slots (clusters of hundreds of slots, wrapping past
    the table's end), erased a few at a time: after each erase the export, counts and
    lookups equal the oracle's."""
    rng = np.random.default_rng(1002)
    log2_cap = 12
    homes = np.concatenate([rng.integers(0, 1 << log2_cap, 300), np.full(200, (1 << log2_cap) - 3),
                            np.full(150, 17)])
    keys = np.unique(keys_at_homes(rng, homes, log2_cap))
    vals = rng.integers(0, 2**64, keys.size, dtype=np.uint64, endpoint=False)
    table, ot = g.Cache(1 << log2_cap, max_load=0.5), oracle.Table()
    table.insert(keys_to_device(keys), keys_to_device(vals))
    ot.insert(keys, vals)
    ep = rng.integers(1, 1000, keys.size, dtype=np.uint64)
    table.touch(keys_to_device(keys), epochs=keys_to_device(ep))
    ot.touch(keys, ep)
    for rnd in range(6):
        pick = keys[rng.random(keys.size) < 0.15]
        absent = rng.integers(0, 2**64, 20, dtype=np.uint64, endpoint=False)
        erase = np.concatenate([pick, absent, pick[:5]])  # repeats too
        say("erase long clusters round", rnd, erase.size)
        counts = table.erase(keys_to_device(erase))
        torch.cuda.synchronize()
        c = u64(counts)
        assert int(c[0]) == ot.erase(erase) and int(c[1]) == len(ot)
        assert_table(table, ot, f"round {rnd}")
        probe = np.concatenate([keys, absent])
        st, ref = table.lookup(keys_to_device(probe))
        torch.cuda.synchronize()
        est, eref = oracle.lookup(probe, ot)
        assert np.array_equal(st.cpu().numpy(), est) and np.array_equal(u64(ref), eref)
        # put half of them back, so later rounds erase from a changed layout
        back = pick[::2]
        bv = rng.integers(0, 2**64, back.size, dtype=np.uint64, endpoint=False)
        table.set_key_bound(int(c[1]))
        table.insert(keys_to_device(back), keys_to_device(bv))
        ot.insert(back, bv)


def test_erase_few_keys_from_large_table():
    """1,000 present and 100 absent keys out of 2.5M entries in 2^22 slots."""
    rng = np.random.default_rng(1003)
    n = 2_500_000
    keys = rng.integers(0, 2**64, n, dtype=np.uint64, endpoint=False)
    vals = np.arange(n, dtype=np.uint64)
    table, ot = g.Cache(1 << 22, max_load=0.65), oracle.Table()
    say("erase large insert")
    table.insert(keys_to_device(keys), keys_to_device(vals))
    ot.insert(keys, vals)
    erase = np.concatenate([keys[rng.choice(n, 1000, replace=False)],
                            rng.integers(0, 2**64, 100, dtype=np.uint64, endpoint=False)])
    say("erase large erase")
    counts = table.erase(keys_to_device(erase))
    torch.cuda.synchronize()
    c = u64(counts)
    assert int(c[0]) == ot.erase(erase) == 1000 and int(c[1]) == len(ot)
    assert_table(table, ot, "after erase")


@pytest.mark.parametrize("log2_cap,n,keeps", [(13, 5_000, (4_000, 1_234, 1, 0)),
                                             (17, 50_000, (40_000, 12_345, 1, 0))])
def test_evict_full_width_stamps_and_export_order(log2_cap, n, keeps):
    """Stamps spread over all 64 bits (every digit of the two-word sort key matters), the
    keys 0 and 2^64-1 present; a table the one-workgroup sort orders (2^13 slots) and one
    of several sort tiles (2^17): eviction order and export equal the oracle's."""
    rng = np.random.default_rng(1002 + log2_cap)
    keys = rng.integers(0, 2**64, n, dtype=np.uint64, endpoint=False)
    keys[:2] = [0, 2**64 - 1]
    vals = rng.integers(0, 2**64, n, dtype=np.uint64, endpoint=False)
    table, ot = g.Cache(1 << log2_cap, max_load=0.7), oracle.Table()
    table.insert(keys_to_device(keys), keys_to_device(vals))
    ot.insert(keys, vals)
    ep = rng.integers(0, 2**64, n, dtype=np.uint64, endpoint=False)
    ep[::3] = ep[0]  # a third share one stamp
    ep[1::7] >>= np.uint64(40)
    table.touch(keys_to_device(keys), epochs=keys_to_device(ep))
    ot.touch(keys, ep)
    say("lifecycle full-width stamps")
    assert_table(table, ot, "before evict")
    for keep in keeps:
        ev, counts = table.evict(keep)
        torch.cuda.synchronize()
        want = ot.evict(keep)
        assert u64(counts).tolist() == [want.size, len(ot)]
        assert np.array_equal(u64(ev)[:want.size], want)
        assert_table(table, ot, f"after evict to {keep}")


@pytest.mark.parametrize("log2_cap", [13, 14])
def test_sort_skips_shared_digits(log2_cap):
    """Keys that differ only in their top byte (seven of the export's eight digit passes
    move nothing), all stamps equal (every stamp pass moves nothing), tables of 0, 1 and
    2 entries (no pass moves anything): the orders still equal the oracle's, in the
    one-workgroup sort (2^13 slots) and the tiled one (2^14 slots plus the side slot)."""
    rng = np.random.default_rng(1003 + log2_cap)
    base = np.uint64(0x0012_3456_789A_BCDE)
    tops = rng.choice(256, 200, replace=False).astype(np.uint64)
    cases = {"top byte": base | (tops << np.uint64(56)), "empty": np.zeros(0, np.uint64),
             "one": np.array([7], np.uint64), "two": np.array([2**64 - 1, 0], np.uint64)}
    for what, keys in cases.items():
        say("lifecycle shared digits", log2_cap, what)
        table, ot = g.Cache(1 << log2_cap, max_load=0.5), oracle.Table()
        if keys.size:
            vals = rng.integers(0, 2**64, keys.size, dtype=np.uint64, endpoint=False)
            table.insert(keys_to_device(keys), keys_to_device(vals))
            ot.insert(keys, vals)
            ep = np.full(keys.size, 99, np.uint64)
            table.touch(keys_to_device(keys), epochs=keys_to_device(ep))
            ot.touch(keys, ep)
        assert_table(table, ot, what)
        keep = keys.size // 2
        ev, counts = table.evict(keep)
        torch.cuda.synchronize()
        want = ot.evict(keep)
        assert u64(counts).tolist() == [want.size, len(ot)], what
        assert np.array_equal(u64(ev)[:want.size], want), what
        assert_table(table, ot, f"{what} after evict")


def test_touch_of_heavily_repeated_keys():
    """262,144 copies of a few keys with distinct epochs, as the blocks of zero-filled
    tensors give (runs, and one key scattered across workgroups): each stamp is the
    largest epoch of its key's copies, the count is the oracle's, and the touch stays
    within a small multiple of a touch of as many distinct keys (with one device-wide
    atomic per copy it took 50x as long)."""
    rng = np.random.default_rng(1004)
    n = 262_144
    hot = np.array([0x1234567, 0, 2**64 - 1, 99], np.uint64)
    keys = np.full(n, hot[0], np.uint64)
    keys[::256] = hot[1]
    keys[5::512] = hot[2]
    keys[n // 2: n // 2 + 1000] = hot[3]
    table, ot = g.Cache(1 << 12, max_load=0.5), oracle.Table()
    present = np.concatenate([hot[:3], np.array([7, 8], np.uint64)])
    table.insert(keys_to_device(present), keys_to_device(np.arange(present.size, dtype=np.uint64)))
    ot.insert(present, np.arange(present.size, dtype=np.uint64))
    ep = rng.permutation(n).astype(np.uint64) + np.uint64(1)
    say("touch repeated keys")
    hit = table.touch(keys_to_device(keys), epochs=keys_to_device(ep))
    torch.cuda.synchronize()
    assert int(hit.item()) == ot.touch(keys, ep)
    assert_table(table, ot, "after touch")
    # timing against distinct keys (kernel time: epochs prepared beforehand)
    dk = rng.integers(0, 2**63, n, dtype=np.uint64)
    big = g.Cache(1 << 20, max_load=0.5)
    d_dk, d_hot = keys_to_device(dk), keys_to_device(keys)
    big.insert(d_dk, keys_to_device(np.arange(n, dtype=np.uint64)))
    big.insert(keys_to_device(hot), keys_to_device(np.arange(hot.size, dtype=np.uint64)))
    eps = [keys_to_device(ep + np.uint64(n * i)) for i in range(8)]

    def timed(d):
        for e in eps[:3]:
            big.touch(d, epochs=e)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for e in eps[3:]:
            big.touch(d, epochs=e)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / 5

    t_hot, t_distinct = timed(d_hot), timed(d_dk)
    assert t_hot < 4 * t_distinct + 0.05, (t_hot, t_distinct)
