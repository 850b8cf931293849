"""The workspace-free lookup (gleam_cache_lookup_noalloc) against gleam_cache_lookup.

Both calls go through the C ABI on the same keys and table; statuses and refs must be
equal byte for byte (and equal to the oracle's). Calls follow each other on one stream,
the later ones smaller, so stale scratch contents from an earlier call would show."""

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


def _keys(rng, n, distinct):
    pool = rng.integers(0, 2**64, distinct, dtype=np.uint64, endpoint=False)
    pool[:2] = [0, 2**64 - 1]  # the two special keys
    return pool, pool[rng.integers(0, pool.size, n)]


def test_noalloc_lookup_matches_workspace_lookup_on_calls_in_a_row():
    rng = np.random.default_rng(4242)
    pool, _ = _keys(rng, 1, 400_000)
    table, ot = g.Cache(1 << 20), oracle.Table()
    cached = pool[::3]
    table.insert(keys_to_device(cached), keys_to_device(cached))
    ot.insert(cached, cached)
    # the largest call allowed, then smaller ones (the last on the one-workgroup path)
    for n in (g.lookup_noalloc_max_keys(), 250_000, 4_097, 3_000):
        keys = pool[rng.integers(0, pool.size, n)]
        d_keys = keys_to_device(keys)
        say("noalloc lookup", n)
        st_ws, ref_ws = table.lookup(d_keys)
        st_na = torch.full((n,), 0x77, dtype=torch.uint8, device="cuda")
        ref_na = torch.full((n,), -5, dtype=torch.int64, device="cuda")
        table.lookup_noalloc(d_keys, st_na, ref_na)
        torch.cuda.synchronize()
        assert torch.equal(st_na, st_ws), f"n={n}: statuses differ from gleam_cache_lookup"
        assert torch.equal(ref_na, ref_ws), f"n={n}: refs differ from gleam_cache_lookup"
        est, eref = oracle.lookup(keys, ot)
        assert np.array_equal(st_na.cpu().numpy(), est)
        assert np.array_equal(u64(ref_na), eref)


def test_noalloc_lookup_refuses_more_keys_than_its_scratch():
    table = g.Cache(64)
    n = g.lookup_noalloc_max_keys() + 1
    keys = torch.zeros(n, dtype=torch.int64, device="cuda")
    status = torch.zeros(n, dtype=torch.uint8, device="cuda")
    say("noalloc lookup refusal", n)
    with pytest.raises(g.GleamError) as e:
        table.lookup_noalloc(keys, status)
    assert e.value.status == g.E_UNSUPPORTED
    torch.cuda.synchronize()
    assert int(status.sum()) == 0  # nothing was enqueued
