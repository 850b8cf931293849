"""Helpers for the GPU parity tests: run the library's path on device tensors and
bring results back as host numpy arrays. The oracle side is computed separately,
by the tests, from the same host bytes."""

from __future__ import annotations

import os
import sys

import numpy as np
import torch

import paper_2607_23115_amd as g


def say(*args) -> None:
    """Name the case before each GPU step (flushed, so a failing box still shows it)."""
    print("[gpu-case]", *args, flush=True)
    sys.stdout.flush()


def host_threads() -> int:
    """Oracle threads: the affinity mask, capped by the job's stated CPU share."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    try:
        share = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        share = 0
    return max(1, min(n, share) if share > 0 else n)


def to_device(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if not a.flags.writeable:  # torch warns on read-only arrays (e.g. views of bytes objects)
        a = a.copy()
    return torch.from_numpy(a).to("cuda")


def u64(t: torch.Tensor) -> np.ndarray:
    return g.as_u64(t)


def keys_to_device(keys: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(keys, dtype=np.uint64).view(np.int64)).to("cuda")


def run_path(batch: g.Batch, table: g.Cache, with_leaves: bool = False):
    """fp -> lookup -> compact on the device; host copies of every output."""
    if with_leaves:
        d, lv = g.fp_chunks(batch, with_leaves=True)
    else:
        d, lv = g.fp_chunks(batch), None
    status, ref = table.lookup(d)
    miss_idx, counters = g.miss_compact(status, batch)
    torch.cuda.synchronize()
    c = u64(counters)
    out = {"digests": u64(d), "status": status.cpu().numpy(), "ref": u64(ref),
           "miss_count": int(c[0]), "miss_bytes": int(c[1]),
           "leaves": u64(lv).reshape(batch.n_blocks, batch.leaves_per_block) if lv is not None else None}
    out["miss_idx"] = u64(miss_idx)[:out["miss_count"]]
    out["_device_digests"] = d
    return out


def detect_path(batch: g.Batch, table: g.Cache, out: g.Detect | None = None):
    """gleam_detect (one call: one kernel for small batches, three for large ones); host
    copies of every output, as run_path returns them."""
    res = g.detect(batch, table, out=out)
    torch.cuda.synchronize()
    n = batch.n_blocks
    c = u64(res.counters)
    o = {"digests": u64(res.digests)[:n], "status": res.status[:n].cpu().numpy(), "ref": u64(res.ref)[:n],
         "miss_count": int(c[0]), "miss_bytes": int(c[1]), "leaves": None}
    o["miss_idx"] = u64(res.miss_idx)[:o["miss_count"]]
    return o


def assert_same(gpu: dict, ref: dict, what: str = "") -> None:
    assert np.array_equal(gpu["digests"], ref["digests"]), f"{what}: digests differ"
    assert np.array_equal(gpu["status"], ref["status"]), f"{what}: status differs"
    assert np.array_equal(gpu["ref"], ref["ref"]), f"{what}: ref differs"
    assert gpu["miss_count"] == ref["miss_count"], f"{what}: miss count"
    assert np.array_equal(gpu["miss_idx"], ref["miss_idx"]), f"{what}: miss list"
    assert gpu["miss_bytes"] == ref["miss_bytes"], f"{what}: miss bytes"
