"""Python binding of libgleam: GPU cache-hit detection for host-to-device weight payloads.

Argument marshalling only: every step of the path runs in the library's gfx950
kernels (include/gleam.h documents each call). PyTorch supplies device memory
(tensors) and streams. Importing this module fails loudly if libgleam.so has not
been built (python -m paper_2607_23115_amd.build).

    batch = Batch.from_tensors([t0, t1, ...], block_bytes=1 << 20)
    digests = fp_chunks(batch)
    table = Cache(capacity=1 << 15)
    status, ref = table.lookup(digests)
    miss_idx, miss_count, miss_bytes = miss_compact(status, batch)

Every call takes `stream` (a torch stream, a raw hipStream_t handle, or None for torch's
current stream). Tensors a call creates itself (outputs not passed in, workspaces,
zeroed counters) are allocated and filled on that stream, so they are ordered before the
call's kernels and are not reused by torch's allocator while that stream still needs
them. Tensors passed in are the caller's: order them yourself when they come from other
streams. A Cache's or Remap's storage belongs to the stream current at construction;
synchronise the other streams that used it before dropping the object.
"""

from __future__ import annotations

import contextlib
import ctypes
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgleam.so")

OK, E_INVALID, E_CAPACITY, E_WORKSPACE, E_HIP, E_UNSUPPORTED = 0, -1, -2, -3, -4, -5
FW_OK, FW_TOO_MANY, FW_INVALID = 0, 1, 2
MISS, HIT_CACHE, HIT_BATCH = 0, 1, 2
REMAP_ADDED, REMAP_INVALID, REMAP_OVERLAP, REMAP_FULL = 0, 1, 2, 3
UNMAPPED = (1 << 64) - 1
LEAF_BYTES = 4096

EXPORTS = (
    "gleam_batch_geometry", "gleam_fp_chunks", "gleam_cache_bytes", "gleam_cache_create", "gleam_cache_destroy",
    "gleam_cache_key_bound", "gleam_workspace_bytes", "gleam_cache_insert", "gleam_cache_lookup",
    "gleam_miss_compact", "gleam_status_string", "gleam_last_error", "gleam_identify_weights",
    "gleam_md5_prefix", "gleam_cache_maint_bytes", "gleam_cache_touch", "gleam_cache_evict", "gleam_cache_erase",
    "gleam_cache_export", "gleam_cache_set_key_bound", "gleam_send_plan", "gleam_pack_misses",
    "gleam_restore_blocks", "gleam_read_stream", "gleam_remap_bytes", "gleam_remap_create", "gleam_remap_destroy",
    "gleam_remap_update_bytes", "gleam_remap_update", "gleam_remap_translate", "gleam_remap_export",
    "gleam_cache_lookup_noalloc", "gleam_cache_lookup_noalloc_max_keys", "gleam_detect",
    "gleam_detect_ws_init", "gleam_identify_leaves", "gleam_first_writes_ws_bytes", "gleam_first_writes",
    "gleam_cache_erase_bytes", "gleam_detect_workspace_bytes", "gleam_preload",
)


class GleamError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


class _Batch(ctypes.Structure):
    _fields_ = [("seg_addr", ctypes.c_void_p), ("seg_len", ctypes.c_void_p), ("blk_first", ctypes.c_void_p),
                ("n_seg", ctypes.c_uint64), ("n_blocks", ctypes.c_uint64), ("leaf_bytes", ctypes.c_uint32),
                ("block_bytes", ctypes.c_uint32)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libgleam.so is not built at {LIB_PATH}; run python -m paper_2607_23115_amd.build")
    lib = ctypes.CDLL(LIB_PATH)
    u64, u32, vp, st = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_int32
    sz = ctypes.c_size_t
    sigs = {
        "gleam_batch_geometry": ([vp, u64, u32, vp, vp], st),
        "gleam_fp_chunks": ([ctypes.POINTER(_Batch), vp, vp, vp], st),
        "gleam_cache_bytes": ([u64], sz),
        "gleam_cache_create": ([vp, sz, u64, ctypes.c_double, ctypes.POINTER(vp), vp], st),
        "gleam_cache_destroy": ([vp], st),
        "gleam_cache_key_bound": ([vp], u64),
        "gleam_workspace_bytes": ([u64], sz),
        "gleam_cache_insert": ([vp, vp, vp, u64, vp, vp, sz, vp], st),
        "gleam_cache_lookup": ([vp, vp, u64, vp, vp, vp, sz, vp], st),
        "gleam_cache_lookup_noalloc": ([vp, vp, u64, vp, vp, vp], st),
        "gleam_detect": ([ctypes.POINTER(_Batch), vp, vp, vp, vp, vp, vp, vp, vp, sz, vp], st),
        "gleam_detect_ws_init": ([vp, sz, vp], st),
        "gleam_detect_workspace_bytes": ([u64], sz),
        "gleam_identify_leaves": ([ctypes.POINTER(_Batch), vp, vp, u64, vp, vp, vp, vp, sz, vp], st),
        "gleam_first_writes_ws_bytes": ([u64, u64], sz),
        "gleam_first_writes": ([vp, vp, u64, vp, u64, vp, vp, vp, vp, vp, vp, sz, vp], st),
        "gleam_cache_lookup_noalloc_max_keys": ([], sz),
        "gleam_miss_compact": ([vp, u64, ctypes.POINTER(_Batch), vp, vp, vp, vp, sz, vp], st),
        "gleam_identify_weights": ([ctypes.POINTER(_Batch), vp, vp, u64, vp, vp, vp, vp, sz, vp], st),
        "gleam_md5_prefix": ([ctypes.POINTER(_Batch), u32, u64, vp, vp, vp, vp], st),
        "gleam_cache_maint_bytes": ([vp], sz),
        "gleam_cache_touch": ([vp, vp, u64, vp, u64, vp, vp], st),
        "gleam_cache_evict": ([vp, u64, vp, vp, vp, sz, vp], st),
        "gleam_cache_erase": ([vp, vp, u64, vp, vp, sz, vp], st),
        "gleam_cache_erase_bytes": ([u64], sz),
        "gleam_cache_export": ([vp, vp, vp, vp, vp, vp, sz, vp], st),
        "gleam_cache_set_key_bound": ([vp, u64], st),
        "gleam_send_plan": ([ctypes.POINTER(_Batch), vp, vp, vp, vp, vp, vp, sz, vp], st),
        "gleam_pack_misses": ([ctypes.POINTER(_Batch), vp, vp, u64, vp], st),
        "gleam_restore_blocks": ([ctypes.POINTER(_Batch), vp, vp, u64, vp, vp], st),
        "gleam_read_stream": ([vp, u64, vp, vp], st),
        "gleam_remap_bytes": ([u64], sz),
        "gleam_remap_create": ([vp, sz, u64, ctypes.POINTER(vp), vp], st),
        "gleam_remap_destroy": ([vp], st),
        "gleam_remap_update_bytes": ([vp, u64, u64], sz),
        "gleam_remap_update": ([vp, vp, vp, u64, vp, vp, vp, u64, vp, vp, vp, sz, vp], st),
        "gleam_remap_translate": ([vp, vp, u64, vp, vp], st),
        "gleam_remap_export": ([vp, vp, vp, vp, vp, vp], st),
        "gleam_status_string": ([st], ctypes.c_char_p),
        "gleam_preload": ([], st),
        "gleam_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


lib = _load()


def _check(status: int) -> None:
    if status != OK:
        detail = lib.gleam_last_error().decode() or lib.gleam_status_string(status).decode()
        raise GleamError(status, detail)


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor | None, name: str, dtypes, min_numel: int = 0, optional: bool = False):
    """Check a tensor handed to the library: on a GPU, contiguous, of the expected dtype
    and at least min_numel elements (the kernels read and write plain memory)."""
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a tensor on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtypes is not None and t.dtype not in dtypes:
        raise ValueError(f"{name} must be {' or '.join(str(d) for d in dtypes)}, not {t.dtype}")
    if t.numel() < min_numel:
        raise ValueError(f"{name} holds {t.numel()} elements, {min_numel} needed")
    return t


_U64 = (torch.int64,)
_U8 = (torch.uint8,)


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _torch_stream(stream, device) -> torch.cuda.Stream:
    """The torch stream object of a call's stream (None: torch's current stream; a raw
    hipStream_t handle is wrapped)."""
    cur = torch.cuda.current_stream(device)
    if stream is None or (isinstance(stream, torch.cuda.Stream) and stream == cur):
        return cur
    if isinstance(stream, torch.cuda.Stream):
        return stream
    h = int(stream)
    if h == cur.cuda_stream:
        return cur
    if h == 0:
        return torch.cuda.default_stream(device)
    return torch.cuda.ExternalStream(h, device=device)


@contextlib.contextmanager
def _on_stream(stream, device):
    """Run a call's own allocations and fills on the stream its kernels run on, and yield
    that stream's handle. Tensors a call creates (outputs, workspaces, zeroed counters)
    then belong to that stream: a fill is ordered before the kernels that use the memory,
    and the caching allocator does not hand the memory out again before the stream is
    done with it, whichever stream is torch's current one."""
    s = _torch_stream(stream, device)
    with torch.cuda.stream(s):
        yield _stream(s)


def _u64_device(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).to(device)


def preload(device="cuda") -> None:
    """Load the library's GPU code on `device` now (gleam_preload), so that no later
    call pays the lazy code-object load at its first launch."""
    with torch.cuda.device(torch.device(device)):
        _check(lib.gleam_preload())


def lookup_noalloc_max_keys() -> int:
    return int(lib.gleam_cache_lookup_noalloc_max_keys())


def workspace_bytes(n: int) -> int:
    return int(lib.gleam_workspace_bytes(n))


def workspace(n: int, device="cuda") -> torch.Tensor:
    """Device workspace for lookup / insert / compaction of n items."""
    return torch.empty(max(workspace_bytes(n), 256), dtype=torch.uint8, device=device)


def geometry(seg_len, block_bytes: int) -> np.ndarray:
    """blk_first[S+1] for the given payload lengths (the library's host geometry)."""
    lens = np.ascontiguousarray(seg_len, dtype=np.uint64).reshape(-1)
    first = np.zeros(lens.size + 1, dtype=np.uint64)
    _check(lib.gleam_batch_geometry(lens.ctypes.data if lens.size else None, lens.size, block_bytes,
                                    first.ctypes.data, None))
    return first


class Batch:
    """A batch of payloads in device memory: addresses, lengths and block geometry."""

    def __init__(self, seg_addr, seg_len, block_bytes: int, device="cuda", keepalive=None):
        if torch.device(device).type != "cuda":
            raise ValueError("a Batch's descriptors live in GPU memory: device must be a CUDA device")
        addr = np.ascontiguousarray(seg_addr, dtype=np.uint64).reshape(-1)
        lens = np.ascontiguousarray(seg_len, dtype=np.uint64).reshape(-1)
        if addr.size != lens.size:
            raise ValueError("seg_addr and seg_len differ in length")
        self.block_bytes = int(block_bytes)
        self.host_len = lens
        self.host_first = geometry(lens, block_bytes)
        self.n_seg = int(lens.size)
        self.n_blocks = int(self.host_first[-1])
        self.d_addr = _u64_device(addr if addr.size else np.zeros(1, np.uint64), device)
        self.d_len = _u64_device(lens if lens.size else np.zeros(1, np.uint64), device)
        self.d_first = _u64_device(self.host_first, device)
        self.keepalive = keepalive
        self._c = _Batch(self.d_addr.data_ptr(), self.d_len.data_ptr(), self.d_first.data_ptr(), self.n_seg,
                         self.n_blocks, LEAF_BYTES, self.block_bytes)

    @classmethod
    def from_arena(cls, arena: torch.Tensor, offsets, lengths, block_bytes: int) -> "Batch":
        """Payloads at byte offsets of one contiguous GPU tensor; every payload must lie
        inside it (the kernels read exactly those bytes)."""
        if not isinstance(arena, torch.Tensor) or arena.device.type != "cuda" or not arena.is_contiguous():
            raise ValueError("Batch.from_arena needs a contiguous tensor on the GPU")
        offs = np.ascontiguousarray(offsets, dtype=np.uint64).reshape(-1)
        lens = np.ascontiguousarray(lengths, dtype=np.uint64).reshape(-1)
        if offs.size != lens.size:
            raise ValueError("offsets and lengths differ in length")
        size = arena.numel() * arena.element_size()
        if offs.size and (int(offs.max()) > size or np.any(lens > np.uint64(size) - offs)):
            raise ValueError("a payload reaches past the end of the arena")
        return cls(offs + np.uint64(arena.data_ptr()), lens, block_bytes, arena.device, keepalive=arena)

    @classmethod
    def from_tensors(cls, tensors, block_bytes: int) -> "Batch":
        """One payload per contiguous device tensor: its bytes, from data_ptr() for
        numel() * element_size() bytes (a non-contiguous view is refused)."""
        dev = tensors[0].device if tensors else torch.device("cuda")
        for t in tensors:
            if t.device.type != "cuda" or t.device != dev:
                raise ValueError("Batch.from_tensors needs tensors on one GPU")
            if not t.is_contiguous():
                raise ValueError("Batch.from_tensors needs contiguous tensors (call .contiguous() first)")
        addr = [t.data_ptr() for t in tensors]
        lens = [t.numel() * t.element_size() for t in tensors]
        return cls(addr, lens, block_bytes, dev, keepalive=list(tensors))

    @property
    def leaves_per_block(self) -> int:
        return self.block_bytes // LEAF_BYTES

    def c_struct(self) -> _Batch:
        return self._c


def fp_chunks(batch: Batch, out: torch.Tensor | None = None, leaf_out: torch.Tensor | None = None,
              with_leaves: bool = False, stream=None):
    """Block digests (u64 as int64 tensor); optionally padded leaf digests."""
    dev = batch.d_first.device
    with _on_stream(stream, dev) as hs:
        if out is None:
            out = torch.empty(max(batch.n_blocks, 1), dtype=torch.int64, device=dev)
        if with_leaves and leaf_out is None:
            leaf_out = torch.empty(max(batch.n_blocks * batch.leaves_per_block, 1), dtype=torch.int64, device=dev)
        _dev(out, "out", _U64, batch.n_blocks)
        _dev(leaf_out, "leaf_out", _U64, batch.n_blocks * batch.leaves_per_block, optional=True)
        _check(lib.gleam_fp_chunks(ctypes.byref(batch.c_struct()), _ptr(out), _ptr(leaf_out), hs))
    if with_leaves:
        return out[:batch.n_blocks], leaf_out[:batch.n_blocks * batch.leaves_per_block]
    return out[:batch.n_blocks]


class Cache:
    """A device-resident identifier table over a torch-allocated storage tensor."""

    def __init__(self, capacity: int, max_load: float = 0.7, device="cuda", stream=None):
        nbytes = int(lib.gleam_cache_bytes(capacity))
        if nbytes == 0:
            raise GleamError(E_INVALID, f"invalid capacity {capacity}")
        self.capacity = capacity
        self.storage = torch.empty(nbytes, dtype=torch.uint8, device=device)
        h = ctypes.c_void_p()
        _check(lib.gleam_cache_create(_ptr(self.storage), nbytes, capacity, max_load, ctypes.byref(h),
                                      _stream(stream)))
        self._h = h

    @property
    def handle(self) -> ctypes.c_void_p:
        if self._h is None:
            raise GleamError(E_INVALID, "table handle already destroyed")
        return self._h

    def key_bound(self) -> int:
        return int(lib.gleam_cache_key_bound(self.handle))

    def insert(self, keys: torch.Tensor, vals: torch.Tensor, ws: torch.Tensor | None = None,
               n_new: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        n = keys.numel()
        if vals.numel() != n:
            raise ValueError("keys and vals differ in length")
        _dev(keys, "keys", _U64)
        with _on_stream(stream, keys.device) as hs:
            if ws is None:
                ws = workspace(n, keys.device)
            if n_new is None:
                n_new = torch.empty(1, dtype=torch.int64, device=keys.device)
            _dev(vals, "vals", _U64)
            _dev(n_new, "n_new", _U64, 1)
            _dev(ws, "ws", _U8)
            _check(lib.gleam_cache_insert(self.handle, _ptr(keys), _ptr(vals), n, _ptr(n_new), _ptr(ws),
                                          ws.numel(), hs))
        return n_new

    def lookup(self, keys: torch.Tensor, status: torch.Tensor | None = None, ref: torch.Tensor | None = None,
               ws: torch.Tensor | None = None, want_ref: bool = True, stream=None):
        n = keys.numel()
        _dev(keys, "keys", _U64)
        with _on_stream(stream, keys.device) as hs:
            if status is None:
                status = torch.empty(max(n, 1), dtype=torch.uint8, device=keys.device)
            if ref is None and want_ref:
                ref = torch.empty(max(n, 1), dtype=torch.int64, device=keys.device)
            if ws is None:
                ws = workspace(n, keys.device)
            _dev(status, "status", _U8, n)
            _dev(ref, "ref", _U64, n, optional=True)
            _dev(ws, "ws", _U8)
            _check(lib.gleam_cache_lookup(self.handle, _ptr(keys), n, _ptr(status), _ptr(ref), _ptr(ws),
                                          ws.numel(), hs))
        return status[:n], (ref[:n] if ref is not None else None)

    def lookup_noalloc(self, keys: torch.Tensor, status: torch.Tensor, ref: torch.Tensor | None = None,
                       stream=None):
        """lookup() with the library's own scratch instead of a workspace (at most
        lookup_noalloc_max_keys() keys; calls on one GPU must not overlap). The caller
        passes the outputs, so nothing is allocated."""
        n = keys.numel()
        _dev(keys, "keys", _U64)
        _dev(status, "status", _U8, n)
        _dev(ref, "ref", _U64, n, optional=True)
        _check(lib.gleam_cache_lookup_noalloc(self.handle, _ptr(keys), n, _ptr(status), _ptr(ref), _stream(stream)))
        return status[:n], (ref[:n] if ref is not None else None)

    # -- lifecycle ------------------------------------------------------------------ #
    def maint_workspace(self) -> torch.Tensor:
        n = int(lib.gleam_cache_maint_bytes(self.handle))
        if n == 0:
            raise GleamError(E_UNSUPPORTED, "no maintenance workspace for this table")
        return torch.empty(n, dtype=torch.uint8, device=self.storage.device)

    def touch(self, keys: torch.Tensor, epochs: torch.Tensor | None = None, epoch: int = 0, stream=None):
        """Stamp present keys with max(stamp, epoch); returns the device count of present keys."""
        _dev(keys, "keys", _U64)
        _dev(epochs, "epochs", _U64, keys.numel(), optional=True)
        with _on_stream(stream, keys.device) as hs:
            n_touched = torch.empty(1, dtype=torch.int64, device=keys.device)
            _check(lib.gleam_cache_touch(self.handle, _ptr(keys), keys.numel(), _ptr(epochs), epoch,
                                         _ptr(n_touched), hs))
        return n_touched

    def evict(self, keep: int, ws: torch.Tensor | None = None, stream=None):
        """Keep the `keep` most recently used entries: (evicted keys [capacity+1], counts[2])."""
        dev = self.storage.device
        with _on_stream(stream, dev) as hs:
            ws = self.maint_workspace() if ws is None else ws
            evicted = torch.empty(self.capacity + 1, dtype=torch.int64, device=dev)
            counts = torch.empty(2, dtype=torch.int64, device=dev)
            _dev(ws, "ws", _U8)
            _check(lib.gleam_cache_evict(self.handle, keep, _ptr(evicted), _ptr(counts), _ptr(ws), ws.numel(), hs))
        return evicted, counts

    def erase(self, keys: torch.Tensor, ws: torch.Tensor | None = None, stream=None):
        """Remove the given keys that are present: counts int64[2] = {removed, live after}."""
        _dev(keys, "keys", _U64)
        dev = self.storage.device
        with _on_stream(stream, dev) as hs:
            if ws is None:
                nb = int(lib.gleam_cache_erase_bytes(keys.numel()))
                if nb == 0:
                    raise GleamError(E_UNSUPPORTED, "too many keys to erase at once")
                ws = torch.empty(nb, dtype=torch.uint8, device=dev)
            counts = torch.empty(2, dtype=torch.int64, device=dev)
            _dev(ws, "ws", _U8)
            _check(lib.gleam_cache_erase(self.handle, _ptr(keys), keys.numel(), _ptr(counts), _ptr(ws), ws.numel(),
                                         hs))
        return counts

    def export(self, ws: torch.Tensor | None = None, stream=None):
        """(keys, vals, stamps, count) with the first count entries valid, sorted by key."""
        dev = self.storage.device
        with _on_stream(stream, dev) as hs:
            ws = self.maint_workspace() if ws is None else ws
            keys = torch.empty(self.capacity + 1, dtype=torch.int64, device=dev)
            vals = torch.empty_like(keys)
            stamps = torch.empty_like(keys)
            count = torch.empty(1, dtype=torch.int64, device=dev)
            _dev(ws, "ws", _U8)
            _check(lib.gleam_cache_export(self.handle, _ptr(keys), _ptr(vals), _ptr(stamps), _ptr(count),
                                          _ptr(ws), ws.numel(), hs))
        return keys, vals, stamps, count

    def set_key_bound(self, n: int) -> None:
        _check(lib.gleam_cache_set_key_bound(self.handle, n))

    def close(self) -> None:
        if self._h is not None:
            lib.gleam_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Remap:
    """The address-remap map of the weight-sharing layer over a torch-allocated storage
    tensor: disjoint intervals of client device addresses, each mapped onto a target."""

    def __init__(self, capacity: int, device="cuda", stream=None):
        nbytes = int(lib.gleam_remap_bytes(capacity))
        if nbytes == 0:
            raise GleamError(E_INVALID, f"invalid capacity {capacity}")
        self.capacity = capacity
        self.storage = torch.empty(nbytes, dtype=torch.uint8, device=device)
        h = ctypes.c_void_p()
        _check(lib.gleam_remap_create(_ptr(self.storage), nbytes, capacity, ctypes.byref(h), _stream(stream)))
        self._h = h

    @property
    def handle(self) -> ctypes.c_void_p:
        if self._h is None:
            raise GleamError(E_INVALID, "map handle already destroyed")
        return self._h

    def update_workspace(self, n_add: int, n_del: int) -> torch.Tensor:
        n = int(lib.gleam_remap_update_bytes(self.handle, n_add, n_del))
        if n == 0:
            raise GleamError(E_UNSUPPORTED, "no update workspace for these sizes")
        return torch.empty(n, dtype=torch.uint8, device=self.storage.device)

    def update(self, del_start: torch.Tensor | None = None, del_len: torch.Tensor | None = None,
               add_start: torch.Tensor | None = None, add_len: torch.Tensor | None = None,
               add_target: torch.Tensor | None = None, status: torch.Tensor | None = None,
               counts: torch.Tensor | None = None, ws: torch.Tensor | None = None, want_status: bool = True,
               stream=None):
        """Removals, then additions: (status u8[n_add] or None, counts int64[4] =
        {intervals after, added, removed, refused}) on the device."""
        dev = self.storage.device
        n_del = 0 if del_start is None else del_start.numel()
        n_add = 0 if add_start is None else add_start.numel()
        if n_del and (del_len is None or del_len.numel() != n_del):
            raise ValueError("del_start and del_len differ in length")
        if n_add and (add_len is None or add_target is None or add_len.numel() != n_add
                      or add_target.numel() != n_add):
            raise ValueError("add_start, add_len and add_target differ in length")
        for t, name in ((del_start, "del_start"), (del_len, "del_len")):
            _dev(t, name, _U64, n_del, optional=n_del == 0)
        for t, name in ((add_start, "add_start"), (add_len, "add_len"), (add_target, "add_target")):
            _dev(t, name, _U64, n_add, optional=n_add == 0)
        live = (lambda t, n: _ptr(t) if n else None)
        with _on_stream(stream, dev) as hs:
            if status is None and want_status:
                status = torch.empty(max(n_add, 1), dtype=torch.uint8, device=dev)
            if counts is None:
                counts = torch.empty(4, dtype=torch.int64, device=dev)
            if ws is None:
                ws = self.update_workspace(n_add, n_del)
            _dev(status, "status", _U8, n_add, optional=True)
            _dev(counts, "counts", _U64, 4)
            _dev(ws, "ws", _U8)
            _check(lib.gleam_remap_update(self.handle, live(del_start, n_del), live(del_len, n_del), n_del,
                                          live(add_start, n_add), live(add_len, n_add), live(add_target, n_add),
                                          n_add, _ptr(status), _ptr(counts), _ptr(ws), ws.numel(), hs))
        return (status[:n_add] if status is not None else None), counts

    def translate(self, addr: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """target + (p - start) for each address inside an interval, else UNMAPPED (-1)."""
        n = addr.numel()
        _dev(addr, "addr", _U64)
        with _on_stream(stream, addr.device) as hs:
            if out is None:
                out = torch.empty(max(n, 1), dtype=torch.int64, device=addr.device)
            _dev(out, "out", _U64, n)
            _check(lib.gleam_remap_translate(self.handle, _ptr(addr), n, _ptr(out), hs))
        return out[:n]

    def export(self, stream=None):
        """(start, length, target, count): the first count intervals, in start order."""
        dev = self.storage.device
        with _on_stream(stream, dev) as hs:
            start = torch.empty(self.capacity, dtype=torch.int64, device=dev)
            length = torch.empty_like(start)
            target = torch.empty_like(start)
            count = torch.empty(1, dtype=torch.int64, device=dev)
            _check(lib.gleam_remap_export(self.handle, _ptr(start), _ptr(length), _ptr(target), _ptr(count), hs))
        return start, length, target, count

    def close(self) -> None:
        if self._h is not None:
            lib.gleam_remap_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def miss_compact(status: torch.Tensor, batch: Batch | None = None, miss_idx: torch.Tensor | None = None,
                 counters: torch.Tensor | None = None, ws: torch.Tensor | None = None, stream=None):
    """(miss_idx[n] int64, counters[2] int64 = [miss_count, miss_bytes]) on the device.

    The first counters[0] entries of miss_idx are valid; counters[1] is filled when
    `batch` is given."""
    n = status.numel()
    _dev(status, "status", _U8)
    dev = status.device
    cb = ctypes.byref(batch.c_struct()) if batch is not None else None
    with _on_stream(stream, dev) as hs:
        if miss_idx is None:
            miss_idx = torch.empty(max(n, 1), dtype=torch.int64, device=dev)
        if counters is None:
            counters = torch.zeros(2, dtype=torch.int64, device=dev)
        if ws is None:
            ws = workspace(n, dev)
        _dev(miss_idx, "miss_idx", _U64, n)
        _dev(counters, "counters", _U64, 2 if batch is not None else 1)
        _dev(ws, "ws", _U8)
        bytes_ptr = ctypes.c_void_p(counters.data_ptr() + 8) if batch is not None else None
        _check(lib.gleam_miss_compact(_ptr(status), n, cb, _ptr(miss_idx), _ptr(counters), bytes_ptr, _ptr(ws),
                                      ws.numel(), hs))
    return miss_idx, counters


class Detect:
    """Outputs of detect calls on one batch (device tensors): digests, status, ref (or
    None), miss_idx and counters = [miss_count, miss_bytes], plus the calls' workspace,
    prepared once here with gleam_detect_ws_init (on `stream`)."""

    def __init__(self, batch: Batch, want_ref: bool = True, device=None, stream=None):
        dev = batch.d_first.device if device is None else device
        n = max(batch.n_blocks, 1)
        with _on_stream(stream, dev) as hs:
            self.digests = torch.empty(n, dtype=torch.int64, device=dev)
            self.status = torch.empty(n, dtype=torch.uint8, device=dev)
            self.ref = torch.empty(n, dtype=torch.int64, device=dev) if want_ref else None
            self.miss_idx = torch.empty(n, dtype=torch.int64, device=dev)
            self.counters = torch.empty(2, dtype=torch.int64, device=dev)
            nb = int(lib.gleam_detect_workspace_bytes(batch.n_blocks))
            if nb == 0:
                raise GleamError(E_UNSUPPORTED, "batch too large for a detect workspace")
            self.ws = torch.empty(nb, dtype=torch.uint8, device=dev)
            _check(lib.gleam_detect_ws_init(_ptr(self.ws), self.ws.numel(), hs))


def detect(batch: Batch, table: Cache, out: Detect | None = None, want_ref: bool = True, stream=None) -> Detect:
    """fp_chunks -> lookup -> miss_compact in one library call (one kernel for a small
    batch). Pass `out` (a Detect made for this batch, or for a larger one) to reuse its
    tensors and workspace; calls that may overlap need separate Detects."""
    dev = batch.d_first.device
    n = batch.n_blocks
    with _on_stream(stream, dev) as hs:
        if out is None:
            out = Detect(batch, want_ref, dev)
        _dev(out.digests, "digests", _U64, n)
        _dev(out.status, "status", _U8, n)
        _dev(out.ref, "ref", _U64, n, optional=True)
        _dev(out.miss_idx, "miss_idx", _U64, n)
        _dev(out.counters, "counters", _U64, 2)
        _dev(out.ws, "ws", _U8)
        _check(lib.gleam_detect(ctypes.byref(batch.c_struct()), table.handle, _ptr(out.digests), _ptr(out.status),
                                _ptr(out.ref), _ptr(out.miss_idx), _ptr(out.counters),
                                ctypes.c_void_p(out.counters.data_ptr() + 8), _ptr(out.ws), out.ws.numel(), hs))
    return out


def identify_weights(batch: Batch, recorded: torch.Tensor, region_first, ws: torch.Tensor | None = None,
                     stream=None):
    """Free-time weight identification: (block_match u8[n_blocks], first_diff int64[n_seg],
    region_weight u8[n_regions]) on the device. `recorded` holds the block digests taken
    when the payloads were written; `region_first` the allocation boundaries over payloads."""
    dev = batch.d_first.device
    _dev(recorded, "recorded", _U64, batch.n_blocks)
    with _on_stream(stream, dev) as hs:
        rf = region_first if isinstance(region_first, torch.Tensor) else _u64_device(np.asarray(region_first), dev)
        n_regions = rf.numel() - 1
        block_match = torch.empty(max(batch.n_blocks, 1), dtype=torch.uint8, device=dev)
        first_diff = torch.empty(max(batch.n_seg, 1), dtype=torch.int64, device=dev)
        region_weight = torch.empty(max(n_regions, 1), dtype=torch.uint8, device=dev)
        if ws is None:
            ws = workspace(batch.n_blocks + batch.n_seg, dev)
        _dev(rf, "region_first", _U64, 1)
        _dev(ws, "ws", _U8)
        _check(lib.gleam_identify_weights(ctypes.byref(batch.c_struct()), _ptr(recorded), _ptr(rf), n_regions,
                                          _ptr(block_match), _ptr(first_diff), _ptr(region_weight), _ptr(ws),
                                          ws.numel(), hs))
    return block_match[:batch.n_blocks], first_diff[:batch.n_seg], region_weight[:n_regions]


def identify_leaves(batch: Batch, recorded_leaves: torch.Tensor, region_first, ws: torch.Tensor | None = None,
                    stream=None):
    """identify_weights at leaf granularity: (leaf_match u8[n_blocks * LPB], first_diff_leaf
    int64[n_seg], region_weight u8[n_regions]) on the device. `recorded_leaves` holds the
    leaf digests fp_chunks(with_leaves=True) gave when the payloads were written."""
    dev = batch.d_first.device
    n_slots = batch.n_blocks * batch.leaves_per_block
    _dev(recorded_leaves, "recorded_leaves", _U64, n_slots)
    with _on_stream(stream, dev) as hs:
        rf = region_first if isinstance(region_first, torch.Tensor) else _u64_device(np.asarray(region_first), dev)
        n_regions = rf.numel() - 1
        leaf_match = torch.empty(max(n_slots, 1), dtype=torch.uint8, device=dev)
        first_diff = torch.empty(max(batch.n_seg, 1), dtype=torch.int64, device=dev)
        region_weight = torch.empty(max(n_regions, 1), dtype=torch.uint8, device=dev)
        if ws is None:
            ws = workspace(n_slots + batch.n_seg, dev)
        _dev(rf, "region_first", _U64, 1)
        _dev(ws, "ws", _U8)
        _check(lib.gleam_identify_leaves(ctypes.byref(batch.c_struct()), _ptr(recorded_leaves), _ptr(rf), n_regions,
                                         _ptr(leaf_match), _ptr(first_diff), _ptr(region_weight), _ptr(ws),
                                         ws.numel(), hs))
    return leaf_match[:n_slots], first_diff[:batch.n_seg], region_weight[:n_regions]


def first_writes_outputs(n_writes: int, n_regions: int, device="cuda"):
    """Output tensors for first_writes over n_writes writes of n_regions allocations:
    (piece_write, piece_offset, piece_len, region_piece_first, region_status)."""
    cap = max(2 * n_writes, 1)
    return (torch.empty(cap, dtype=torch.int64, device=device), torch.empty(cap, dtype=torch.int64, device=device),
            torch.empty(cap, dtype=torch.int64, device=device),
            torch.empty(n_regions + 1, dtype=torch.int64, device=device),
            torch.empty(max(n_regions, 1), dtype=torch.uint8, device=device))


def first_writes_workspace(n_writes: int, n_regions: int, device="cuda") -> torch.Tensor:
    nb = int(lib.gleam_first_writes_ws_bytes(n_writes, n_regions))
    if nb == 0:
        raise GleamError(E_UNSUPPORTED, "too many writes or allocations")
    return torch.empty(nb, dtype=torch.uint8, device=device)


def first_writes(addr, length, region_first, stream=None, device="cuda", out=None, ws=None):
    """The first-write rule over recorded writes (time order, grouped by allocation):
    (piece_write, piece_offset, piece_len, region_piece_first, region_status) device
    tensors; the first region_piece_first[-1] pieces are valid. `out` (from
    first_writes_outputs) and `ws` (from first_writes_workspace) are reused when given."""
    with _on_stream(stream, torch.device(device)) as hs:
        d = [t if isinstance(t, torch.Tensor) else _u64_device(np.asarray(t), device)
             for t in (addr, length, region_first)]
        n, n_regions = d[0].numel(), d[2].numel() - 1
        if d[1].numel() != n:
            raise ValueError("addr and length differ in length")
        for t, name in zip(d, ("addr", "length", "region_first")):
            _dev(t, name, _U64)
        if out is None:
            out = first_writes_outputs(n, n_regions, device)
        pw, po, pl, first, status = out
        cap = max(2 * n, 1)
        for t, name in ((pw, "piece_write"), (po, "piece_offset"), (pl, "piece_len")):
            _dev(t, name, _U64, cap)
        _dev(first, "region_piece_first", _U64, n_regions + 1)
        _dev(status, "region_status", _U8, n_regions)
        if ws is None:
            ws = first_writes_workspace(n, n_regions, device)
        _dev(ws, "ws", _U8)
        _check(lib.gleam_first_writes(_ptr(d[0]), _ptr(d[1]), n, _ptr(d[2]), n_regions, _ptr(pw), _ptr(po), _ptr(pl),
                                      _ptr(first), _ptr(status), _ptr(ws), ws.numel(), hs))
    return pw, po, pl, first, status[:n_regions]


def md5_prefix(batch: Batch, prefix_bytes: int = 128, min_len: int = 1024, stream=None):
    """The paper's identifier per payload: (digest int64[S, 2], key int64[S], eligible u8[S])."""
    dev = batch.d_first.device
    S = max(batch.n_seg, 1)
    with _on_stream(stream, dev) as hs:
        digest = torch.empty(2 * S, dtype=torch.int64, device=dev)
        key = torch.empty(S, dtype=torch.int64, device=dev)
        eligible = torch.empty(S, dtype=torch.uint8, device=dev)
        _check(lib.gleam_md5_prefix(ctypes.byref(batch.c_struct()), prefix_bytes, min_len, _ptr(digest), _ptr(key),
                                    _ptr(eligible), hs))
    n = batch.n_seg
    return digest[:2 * n].view(n, 2), key[:n], eligible[:n]


RECORD_BYTES = 40  # gleam_send_record
RECORD_DTYPE = np.dtype([("block", "<u8"), ("payload", "<u8"), ("offset", "<u8"), ("ident", "<u8"),
                         ("length", "<u4"), ("kind", "<u4")])


def send_plan(batch: Batch, digests: torch.Tensor, status: torch.Tensor, ref: torch.Tensor,
              ws: torch.Tensor | None = None, stream=None):
    """(records as a u8 tensor of n_blocks x 40 bytes, totals int64[4]) on the device."""
    dev = batch.d_first.device
    _dev(digests, "digests", _U64, batch.n_blocks)
    _dev(status, "status", _U8, batch.n_blocks)
    _dev(ref, "ref", _U64, batch.n_blocks)
    with _on_stream(stream, dev) as hs:
        records = torch.empty(max(batch.n_blocks, 1) * RECORD_BYTES, dtype=torch.uint8, device=dev)
        totals = torch.empty(4, dtype=torch.int64, device=dev)
        if ws is None:
            ws = workspace(batch.n_blocks, dev)
        _dev(ws, "ws", _U8)
        _check(lib.gleam_send_plan(ctypes.byref(batch.c_struct()), _ptr(digests), _ptr(status), _ptr(ref),
                                   _ptr(records), _ptr(totals), _ptr(ws), ws.numel(), hs))
    return records[:batch.n_blocks * RECORD_BYTES], totals


def pack_misses(batch: Batch, records: torch.Tensor, out: torch.Tensor, stream=None) -> torch.Tensor:
    _dev(records, "records", _U8, batch.n_blocks * RECORD_BYTES)
    _dev(out, "out", _U8)
    _check(lib.gleam_pack_misses(ctypes.byref(batch.c_struct()), _ptr(records), _ptr(out), out.numel(),
                                 _stream(stream)))
    return out


def restore_blocks(dst: Batch, records: torch.Tensor, packed: torch.Tensor, held: torch.Tensor | None = None,
                   stream=None) -> None:
    _dev(records, "records", _U8, dst.n_blocks * RECORD_BYTES)
    _dev(packed, "packed", _U8)
    _dev(held, "held", _U64, dst.n_blocks, optional=True)
    _check(lib.gleam_restore_blocks(ctypes.byref(dst.c_struct()), _ptr(records), _ptr(packed), packed.numel(),
                                    _ptr(held), _stream(stream)))


def read_stream(src: torch.Tensor, nbytes: int | None = None, sink: torch.Tensor | None = None,
                stream=None) -> torch.Tensor:
    """Calibration read of the first nbytes of a device tensor with the fingerprint
    kernel's load pattern; XORs the fold of its 8-byte words into sink (int64[1])."""
    nbytes = src.numel() * src.element_size() if nbytes is None else int(nbytes)
    _dev(src, "src", None)
    if nbytes > src.numel() * src.element_size():
        raise ValueError("nbytes exceeds the source tensor")
    with _on_stream(stream, src.device) as hs:
        if sink is None:
            sink = torch.zeros(1, dtype=torch.int64, device=src.device)
        _dev(sink, "sink", _U64, 1)
        _check(lib.gleam_read_stream(_ptr(src), nbytes, _ptr(sink), hs))
    return sink


def records_to_numpy(records: torch.Tensor) -> np.ndarray:
    return records.cpu().numpy().view(RECORD_DTYPE)


def as_u64(t: torch.Tensor) -> np.ndarray:
    """Device int64 tensor -> host uint64 array (same bits)."""
    return t.detach().cpu().numpy().view(np.uint64)
