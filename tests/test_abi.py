"""The C-ABI library on the CPU: it loads, exports every symbol include/gleam.h
declares, and validates arguments on the host before anything would be enqueued.
No call here launches GPU work (every call below fails validation, or is host-only)."""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2607_23115_amd as g

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "gleam.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gleam_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 12
    lib = ctypes.CDLL(g.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(g.EXPORTS) == names


def test_status_strings():
    assert g.lib.gleam_status_string(0) == b"ok"
    assert g.lib.gleam_status_string(-3) == b"workspace too small"
    assert g.lib.gleam_status_string(99) == b"unknown status"


def test_geometry_matches_oracle():
    rng = np.random.default_rng(41)
    for block in (4096, 65536, 1 << 20, 16 << 20):
        lens = np.concatenate([rng.integers(0, 3 * block, 50), [0, 1, block, block + 1]]).astype(np.uint64)
        first = g.geometry(lens, block)
        ofirst, _ = oracle.geometry(lens, block)
        assert np.array_equal(first, ofirst)


def test_geometry_rejects_bad_block():
    with pytest.raises(g.GleamError) as e:
        g.geometry([10], 1000)
    assert e.value.status == g.E_INVALID
    with pytest.raises(g.GleamError):
        g.geometry([10], 32 << 20)


def test_sizes():
    assert g.lib.gleam_cache_bytes(16) == 256 + 16 * 24
    assert g.lib.gleam_cache_bytes(15) == 0
    assert g.lib.gleam_cache_bytes(8) == 0
    ws = [g.workspace_bytes(n) for n in (0, 1, 1000, 10**6)]
    assert all(w % 256 == 0 and w > 0 for w in ws)
    assert ws == sorted(ws)
    # scratch table of >= 2n slots of 16 bytes
    assert g.workspace_bytes(10**6) >= 2 * 10**6 * 8  # >= 2n scratch slots of 8 bytes


def _batch(n_seg=1, n_blocks=1, leaf=4096, block=65536, ptr=256):
    return g._Batch(ptr, ptr, ptr, n_seg, n_blocks, leaf, block)


def _call_fp(b, out=256, leaf=None):
    return g.lib.gleam_fp_chunks(ctypes.byref(b) if b is not None else None, out, leaf, None)


def test_fp_chunks_validation():
    assert _call_fp(None) == g.E_INVALID
    assert _call_fp(_batch(leaf=512)) == g.E_INVALID
    assert _call_fp(_batch(block=3000)) == g.E_INVALID
    assert _call_fp(_batch(block=32 << 20)) == g.E_INVALID
    assert _call_fp(_batch(n_seg=0)) == g.E_INVALID
    assert _call_fp(_batch(), out=None) == g.E_INVALID
    assert _call_fp(_batch(ptr=0)) == g.E_INVALID
    # an empty batch is a no-op that succeeds without touching the device
    assert _call_fp(_batch(n_seg=0, n_blocks=0), out=None) == g.OK


def test_detect_validation():
    det = g.lib.gleam_detect
    ok = _batch(n_blocks=4)
    # batch, table, outputs and workspace are checked before anything is enqueued
    assert det(None, 256, 256, 256, None, 256, 256, None, 256, 1 << 20, None) == g.E_INVALID
    assert det(ctypes.byref(_batch(leaf=512)), 256, 256, 256, None, 256, 256, None, 256, 1 << 20, None) == g.E_INVALID
    assert det(ctypes.byref(ok), None, 256, 256, None, 256, 256, None, 256, 1 << 20, None) == g.E_INVALID
    assert det(ctypes.byref(ok), 256, 256, 256, None, 256, None, None, 256, 1 << 20, None) == g.E_INVALID
    assert det(ctypes.byref(ok), 256, None, 256, None, 256, 256, None, 256, 1 << 20, None) == g.E_INVALID
    assert det(ctypes.byref(ok), 256, 256, None, None, 256, 256, None, 256, 1 << 20, None) == g.E_INVALID
    assert det(ctypes.byref(ok), 256, 256, 256, None, None, 256, None, 256, 1 << 20, None) == g.E_INVALID
    assert det(ctypes.byref(ok), 256, 256, 256, None, 256, 256, None, 256, 16, None) == g.E_WORKSPACE
    assert det(ctypes.byref(ok), 256, 256, 256, None, 256, 256, None, 300, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_last_error() != b""


def test_identify_validation():
    f = g.lib.gleam_identify_weights
    assert f(None, 256, 256, 1, None, None, 256, 256, 1 << 20, None) == g.E_INVALID
    b = _batch()
    assert f(ctypes.byref(b), None, 256, 1, None, None, 256, 256, 1 << 20, None) == g.E_INVALID
    assert f(ctypes.byref(b), 256, None, 1, None, None, 256, 256, 1 << 20, None) == g.E_INVALID
    assert f(ctypes.byref(b), 256, 256, 1, None, None, None, 256, 1 << 20, None) == g.E_INVALID
    assert f(ctypes.byref(b), 256, 256, 1, None, None, 256, 300, 1 << 20, None) == g.E_INVALID
    assert f(ctypes.byref(b), 256, 256, 1, None, None, 256, 256, 64, None) == g.E_WORKSPACE


def test_md5_prefix_validation():
    f = g.lib.gleam_md5_prefix
    b = _batch()
    assert f(None, 128, 1024, 256, None, None, None) == g.E_INVALID
    assert f(ctypes.byref(b), (1 << 20) + 1, 1024, 256, None, None, None) == g.E_INVALID
    assert f(ctypes.byref(b), 128, 1024, None, None, None, None) == g.E_INVALID
    assert f(ctypes.byref(_batch(n_seg=0, n_blocks=0)), 128, 1024, None, None, None, None) == g.OK


def test_transfer_validation():
    b = _batch()
    assert g.lib.gleam_send_plan(None, 256, 256, 256, 256, 256, 256, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_send_plan(ctypes.byref(b), None, 256, 256, 256, 256, 256, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_send_plan(ctypes.byref(b), 256, 256, 256, 256, 256, 256, 16, None) == g.E_WORKSPACE
    assert g.lib.gleam_pack_misses(ctypes.byref(b), None, 256, 16, None) == g.E_INVALID
    assert g.lib.gleam_restore_blocks(ctypes.byref(b), None, 256, 16, None, None) == g.E_INVALID
    assert ctypes.sizeof(ctypes.c_uint64) * 4 + 8 == g.RECORD_BYTES == g.RECORD_DTYPE.itemsize


def test_cache_create_validation():
    h = ctypes.c_void_p()
    assert g.lib.gleam_cache_create(256, 1 << 20, 100, 0.5, ctypes.byref(h), None) == g.E_INVALID  # not pow2
    assert g.lib.gleam_cache_create(257, 1 << 20, 64, 0.5, ctypes.byref(h), None) == g.E_INVALID  # unaligned
    assert g.lib.gleam_cache_create(256, 100, 64, 0.5, ctypes.byref(h), None) == g.E_INVALID      # too small
    assert g.lib.gleam_cache_create(256, 1 << 20, 64, 1.0, ctypes.byref(h), None) == g.E_INVALID  # load
    assert g.lib.gleam_cache_create(None, 1 << 20, 64, 0.5, ctypes.byref(h), None) == g.E_INVALID
    assert g.lib.gleam_cache_create(256, 1 << 20, 64, 0.5, None, None) == g.E_INVALID
    assert g.lib.gleam_cache_destroy(None) == g.OK
    assert g.lib.gleam_cache_key_bound(None) == 2**64 - 1
    assert g.lib.gleam_cache_maint_bytes(None) == 0
    assert g.lib.gleam_cache_touch(None, 256, 1, None, 0, None, None) == g.E_INVALID
    assert g.lib.gleam_cache_evict(None, 0, None, 256, 256, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_cache_erase(None, 256, 1, 256, 256, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_cache_export(None, 256, 256, None, 256, 256, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_cache_set_key_bound(None, 0) == g.E_INVALID


def test_lookup_insert_compact_validation():
    assert g.lib.gleam_cache_lookup(None, 256, 4, 256, None, 256, 1 << 20, None) == g.E_INVALID
    # the workspace-free lookup: a null table is refused before anything touches a device
    assert g.lib.gleam_cache_lookup_noalloc(None, 256, 4, 256, None, None) == g.E_INVALID
    assert g.lookup_noalloc_max_keys() == 1 << 20
    assert g.lib.gleam_cache_insert(None, 256, 256, 4, None, 256, 1 << 20, None) == g.E_INVALID
    # compaction: null count, workspace too small or unaligned, bytes without a batch
    assert g.lib.gleam_miss_compact(256, 10, None, 256, None, None, 256, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_miss_compact(256, 10, None, 256, 256, None, 256, 16, None) == g.E_WORKSPACE
    assert g.lib.gleam_miss_compact(256, 10, None, 256, 256, None, 300, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_miss_compact(256, 10, None, 256, 256, 256, 256, 1 << 20, None) == g.E_INVALID
    b = _batch(n_blocks=11)
    assert g.lib.gleam_miss_compact(256, 10, ctypes.byref(b), 256, 256, 256, 256, 1 << 20, None) == g.E_INVALID
    assert g.lib.gleam_last_error() != b""


def test_remap_validation():
    h = ctypes.c_void_p()
    assert g.lib.gleam_remap_bytes(1) == 256 + 24 + 65536
    assert g.lib.gleam_remap_bytes(1000) == 256 + 24 * 1000 + 65536
    assert g.lib.gleam_remap_bytes(0) == 0
    assert g.lib.gleam_remap_bytes((1 << 31) + 1) == 0
    assert g.lib.gleam_remap_create(256, 1 << 20, 0, ctypes.byref(h), None) == g.E_INVALID      # capacity
    assert g.lib.gleam_remap_create(257, 1 << 20, 64, ctypes.byref(h), None) == g.E_INVALID     # unaligned
    assert g.lib.gleam_remap_create(256, 256 + 24 * 64 + 65535, 64, ctypes.byref(h), None) == g.E_INVALID
    assert g.lib.gleam_remap_create(None, 1 << 20, 64, ctypes.byref(h), None) == g.E_INVALID
    assert g.lib.gleam_remap_create(256, 1 << 20, 64, None, None) == g.E_INVALID
    assert g.lib.gleam_remap_destroy(None) == g.OK
    assert g.lib.gleam_remap_update_bytes(None, 1, 1) == 0
    assert g.lib.gleam_remap_update(None, None, None, 0, None, None, None, 0, None, 256, 256, 1 << 20,
                                    None) == g.E_INVALID
    assert g.lib.gleam_remap_translate(None, 256, 1, 256, None) == g.E_INVALID
    assert g.lib.gleam_remap_export(None, 256, 256, 256, 256, None) == g.E_INVALID
    assert b"gleam_remap_export" in g.lib.gleam_last_error()


def test_counts_beyond_any_workspace_are_refused():
    """n above 2^40 items has no workspace layout (its size would overflow): the call
    returns GLEAM_E_UNSUPPORTED at once, before anything is enqueued."""
    for n in (2**40 + 1, 2**62 + 1, 2**64 - 1):
        assert g.lib.gleam_miss_compact(256, n, None, 256, 256, None, 256, 1 << 20, None) == g.E_UNSUPPORTED
        assert b"2^40" in g.lib.gleam_last_error()
        assert g.lib.gleam_workspace_bytes(n) == 0


def test_binding_refuses_batches_the_kernels_would_misread():
    """A Batch's descriptors and payloads must be GPU memory, and an arena's payloads must
    lie inside it; the binding refuses the rest before any GPU work (runs without a GPU)."""
    import torch
    with pytest.raises(ValueError):
        g.Batch.from_tensors([torch.zeros(16)], 4096)        # host tensor
    with pytest.raises(ValueError):
        g.Batch.from_arena(torch.zeros(64, dtype=torch.uint8), [0], [16], 4096)
    with pytest.raises(ValueError):
        g.Batch([0], [16], 4096, device="cpu")
