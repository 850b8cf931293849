"""Seeded synthetic inputs for weight-cache hit detection.

This module only produces payload bytes, selections and random digests. It holds
none of the method's arithmetic (no hashing, no lookup, no compaction), so both
the GPU library's callers and the CPU oracle's tests can use it.

Every random draw comes from numpy's PCG64 seeded by
SeedSequence([workload, purpose, index]); purposes: 0 payload bytes, 1 selection,
2 perturbation, 3 random digests. Normal weights are float32 standard normals
times sigma, rounded once to fp16 (numpy's round-to-nearest-even) or bf16
(round-to-nearest-even on the float32 bits), stored little-endian.

The workloads stand in for the weight loads the paper measures (Sec. 2.2.2,
table of memory and weight shares; Appendix, table of per-task weight sizes and
cacheable ratios): real checkpoints are not available, so tensors of the same
shapes are filled with random values.
"""

from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np

PURPOSE_BYTES, PURPOSE_SELECT, PURPOSE_PERTURB, PURPOSE_DIGESTS = 0, 1, 2, 3
LEAF = 4096
KiB, MiB = 1 << 10, 1 << 20


def rng(workload: int, purpose: int, index: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([workload, purpose, index]))


def normal_fp16(gen: np.random.Generator, n: int, sigma: float = 0.02) -> np.ndarray:
    x = gen.standard_normal(n, dtype=np.float32)
    x *= np.float32(sigma)
    return x.astype(np.float16)


def fp32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns the u16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def normal_bf16(gen: np.random.Generator, n: int, sigma: float = 0.02) -> np.ndarray:
    x = gen.standard_normal(n, dtype=np.float32)
    x *= np.float32(sigma)
    return fp32_to_bf16_bits(x)


def as_bytes(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a).view(np.uint8).reshape(-1)


# --------------------------------------------------------------------------- #
# Arena packing: payloads laid out in one buffer
# --------------------------------------------------------------------------- #
def arena_offsets(lengths, align: int = 256, skew: int = 0) -> tuple[np.ndarray, int]:
    """Offsets placing each payload at a multiple of `align` plus `skew`, in order.

    skew != 0 makes every payload start at an unaligned address (parity tests).
    Returns (offsets u64[S], total bytes).
    """
    offs = np.zeros(len(lengths), dtype=np.uint64)
    pos = 0
    for i, n in enumerate(lengths):
        start = ((pos + align - 1) // align) * align + skew
        offs[i] = start
        pos = start + int(n)
    total = ((pos + align - 1) // align) * align + align
    return offs, total


def pack(payloads, align: int = 256, skew: int = 0):
    """Copy payloads into one u8 arena. Returns (arena, offsets, lengths)."""
    lengths = np.array([int(p.size) for p in payloads], dtype=np.uint64)
    offs, total = arena_offsets(lengths.tolist(), align, skew)
    arena = np.zeros(total, dtype=np.uint8)
    for p, o in zip(payloads, offs.tolist()):
        arena[o:o + p.size] = p
    return arena, offs, lengths


def parallel_fill(arena: np.ndarray, offsets, makers, threads: int = 8) -> None:
    """arena[offsets[i]:...] = makers[i]() for every i, over a thread pool."""
    def one(i):
        b = makers[i]()
        o = int(offsets[i])
        arena[o:o + b.size] = b

    if threads <= 1:
        for i in range(len(makers)):
            one(i)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(one, range(len(makers))))


# --------------------------------------------------------------------------- #
# 16 MiB random payload, 64 KiB blocks (workload 1)
# --------------------------------------------------------------------------- #
RANDOM16_BYTES = 16 * MiB
RANDOM16_BLOCK = 64 * KiB


def random16_payload() -> np.ndarray:
    return np.frombuffer(rng(1, PURPOSE_BYTES, 0).bytes(RANDOM16_BYTES), dtype=np.uint8).copy()


def random16_rerandomized(payload: np.ndarray, n_blocks: int = 64):
    """A copy with `n_blocks` distinct 64 KiB blocks overwritten by fresh random bytes.

    Returns (copy, sorted block indices)."""
    nb = payload.size // RANDOM16_BLOCK
    chosen = rng(1, PURPOSE_SELECT, 0).choice(nb, n_blocks, replace=False)
    fresh = rng(1, PURPOSE_BYTES, 1)
    out = payload.copy()
    for b in chosen.tolist():
        out[b * RANDOM16_BLOCK:(b + 1) * RANDOM16_BLOCK] = np.frombuffer(fresh.bytes(RANDOM16_BLOCK), np.uint8)
    return out, np.sort(chosen)


# --------------------------------------------------------------------------- #
# ResNet-50-shaped fp16 weights, 64 KiB blocks (workload 2)
# --------------------------------------------------------------------------- #
RESNET_BLOCK = 64 * KiB


def resnet50_shapes() -> list[tuple[str, tuple[int, ...]]]:
    """The 161 parameter tensors of ResNet-50 (conv weights O,I,kH,kW; BN affine
    weight and bias; fc), in module order; BN running statistics excluded."""
    shapes = [("conv1", (64, 3, 7, 7)), ("bn1.w", (64,)), ("bn1.b", (64,))]
    cin = 64
    for stage, (n, w) in enumerate(zip([3, 4, 6, 3], [64, 128, 256, 512])):
        for b in range(n):
            p = f"layer{stage + 1}.{b}"
            shapes += [(p + ".conv1", (w, cin, 1, 1)), (p + ".bn1.w", (w,)), (p + ".bn1.b", (w,)),
                       (p + ".conv2", (w, w, 3, 3)), (p + ".bn2.w", (w,)), (p + ".bn2.b", (w,)),
                       (p + ".conv3", (4 * w, w, 1, 1)), (p + ".bn3.w", (4 * w,)), (p + ".bn3.b", (4 * w,))]
            if b == 0:
                shapes += [(p + ".down", (4 * w, cin, 1, 1)), (p + ".down_bn.w", (4 * w,)),
                           (p + ".down_bn.b", (4 * w,))]
            cin = 4 * w
    shapes += [("fc.w", (1000, 2048)), ("fc.b", (1000,))]
    return shapes


def resnet50_tensor(i: int) -> np.ndarray:
    n = math.prod(resnet50_shapes()[i][1])
    return as_bytes(normal_fp16(rng(2, PURPOSE_BYTES, i), n))


def resnet50_payloads() -> list[np.ndarray]:
    return [resnet50_tensor(i) for i in range(len(resnet50_shapes()))]


def resnet50_cached_tensors(k: int = 80) -> np.ndarray:
    """The sorted tensor indices whose blocks the cache holds."""
    return np.sort(rng(2, PURPOSE_SELECT, 0).choice(len(resnet50_shapes()), k, replace=False))


# --------------------------------------------------------------------------- #
# 7B decoder-shaped fp16 weights, 1 MiB blocks (workload 3)
# --------------------------------------------------------------------------- #
DECODER_BLOCK = 1 * MiB
PERTURB_RANK = 16
PERTURB_SCALE = 1e-3 / 4.0  # (1e-3/4) * U @ V with N(0,1) U, V of rank 16: entries of std 1e-3
MATRICES = ("q", "k", "v", "o", "gate", "up", "down")


def decoder_shapes(layers: int = 32, d: int = 4096, ffn: int = 11008, vocab: int = 32000):
    """Tensor list of a LLaMA-7B-style decoder: embedding, per layer [attn_norm,
    q, k, v, o, ffn_norm, gate, up, down], final norm, lm head."""
    shapes = [("embed", (vocab, d))]
    for li in range(layers):
        p = f"l{li}."
        shapes += [(p + "attn_norm", (d,)), (p + "q", (d, d)), (p + "k", (d, d)), (p + "v", (d, d)),
                   (p + "o", (d, d)), (p + "ffn_norm", (d,)), (p + "gate", (ffn, d)), (p + "up", (ffn, d)),
                   (p + "down", (d, ffn))]
    shapes += [("final_norm", (d,)), ("lm_head", (vocab, d))]
    return shapes


class Decoder:
    """A decoder weight set and its perturbed copy.

    The base weights are what the cache holds; the payload equals the base except
    in `n_perturbed` = floor(0.1 * layers) layers, whose seven matrices receive a
    rank-16 update: W' = fp16(fp32(W) + (1e-3/4) U V), U, V standard normal.
    """

    def __init__(self, layers: int = 32, d: int = 4096, ffn: int = 11008, vocab: int = 32000, workload: int = 3):
        self.layers, self.d, self.ffn, self.vocab, self.workload = layers, d, ffn, vocab, workload
        self.shapes = decoder_shapes(layers, d, ffn, vocab)
        self.nbytes = [2 * math.prod(s) for _, s in self.shapes]
        n_pert = int(math.floor(0.1 * layers))
        self.perturbed_layers = np.sort(rng(workload, PURPOSE_SELECT, 0).choice(layers, n_pert, replace=False))
        pl = set(self.perturbed_layers.tolist())
        self.perturbed = []
        for i, (name, _) in enumerate(self.shapes):
            layer, _, kind = name.partition(".")
            if kind in MATRICES and int(layer[1:]) in pl:
                self.perturbed.append(i)

    def base(self, i: int) -> np.ndarray:
        n = math.prod(self.shapes[i][1])
        return as_bytes(normal_fp16(rng(self.workload, PURPOSE_BYTES, i), n))

    def payload(self, i: int) -> np.ndarray:
        w = self.base(i)
        if i not in self.perturbed:
            return w
        out_dim, in_dim = self.shapes[i][1]
        g = rng(self.workload, PURPOSE_PERTURB, i)
        u = g.standard_normal((out_dim, PERTURB_RANK), dtype=np.float32)
        v = g.standard_normal((PERTURB_RANK, in_dim), dtype=np.float32)
        delta = (u @ v) * np.float32(PERTURB_SCALE)
        delta += w.view(np.float16).reshape(out_dim, in_dim).astype(np.float32)
        return as_bytes(delta.astype(np.float16))

    def arena(self, perturbed: bool = True, align: int = 256, threads: int = 8):
        """All tensors packed into one u8 arena. Returns (arena, offsets, lengths)."""
        offs, total = arena_offsets(self.nbytes, align)
        arena = np.empty(total, dtype=np.uint8)
        make = self.payload if perturbed else self.base
        parallel_fill(arena, offs, [lambda i=i: make(i) for i in range(len(self.shapes))], threads)
        return arena, offs, np.array(self.nbytes, dtype=np.uint64)


# --------------------------------------------------------------------------- #
# Many small copies, 4 KiB blocks (workload 4)
# --------------------------------------------------------------------------- #
SMALL_BLOCK = 4 * KiB


class SmallCopies:
    """n buffers with sizes floor(exp(U[ln lo, ln hi])) of random bytes; a fraction of
    all full 4 KiB leaves (never the first) are overwritten, in ascending order, with
    a copy of a uniformly chosen earlier full leaf."""

    def __init__(self, n: int = 100_000, lo: int = 256, hi: int = 65536, dup_frac: float = 0.2,
                 workload: int = 4, align: int = 256, skew: int = 0):
        g = rng(workload, PURPOSE_BYTES, 0)
        self.sizes = np.floor(np.exp(g.uniform(math.log(lo), math.log(hi), n))).astype(np.uint64)
        self.offsets, total = arena_offsets(self.sizes.tolist(), align, skew)
        self.arena = np.zeros(total, dtype=np.uint8)
        src = np.frombuffer(rng(workload, PURPOSE_BYTES, 1).bytes(int(self.sizes.sum())), dtype=np.uint8)
        pos = 0
        for o, s in zip(self.offsets.tolist(), self.sizes.tolist()):
            self.arena[o:o + s] = src[pos:pos + s]
            pos += s
        # full leaves in batch order: their arena offsets
        full = []
        for o, s in zip(self.offsets.tolist(), self.sizes.tolist()):
            full.extend(o + LEAF * k for k in range(s // LEAF))
        self.full_leaf_offsets = np.array(full, dtype=np.uint64)
        n_full = len(full)
        k = int(round(dup_frac * n_full))
        sel = rng(workload, PURPOSE_SELECT, 0)
        self.targets = np.sort(sel.choice(np.arange(1, n_full), k, replace=False)) if k else np.zeros(0, np.int64)
        pick = rng(workload, PURPOSE_SELECT, 1)
        self.sources = np.zeros(k, dtype=np.int64)
        for i, t in enumerate(self.targets.tolist()):
            s = int(pick.integers(0, t))
            self.sources[i] = s
            so, to = full[s], full[t]
            self.arena[to:to + LEAF] = self.arena[so:so + LEAF]

    def payloads(self):
        return [self.arena[o:o + s] for o, s in zip(self.offsets.tolist(), self.sizes.tolist())]


# --------------------------------------------------------------------------- #
# Large bf16 weight set, 2 MiB blocks (workload 5)
# --------------------------------------------------------------------------- #
LARGE_BLOCK = 2 * MiB


class LargeSet:
    """n bf16 tensors whose sizes are log-uniform draws in [lo, hi] rescaled so the
    total is exactly `total` bytes (each rounded to an even byte count; the last one
    takes the remainder), values N(0, 0.02)."""

    def __init__(self, n: int = 2000, total: int = 40_000_000_000, lo: int = 1 * MiB, hi: int = 200 * MiB,
                 workload: int = 5):
        self.workload = workload
        x = np.exp(rng(workload, PURPOSE_BYTES, 0).uniform(math.log(lo), math.log(hi), n))
        scaled = x * (total / x.sum())
        sizes = (np.round(scaled / 2.0) * 2).astype(np.int64)
        sizes[-1] = total - int(sizes[:-1].sum())
        if sizes[-1] <= 0 or sizes[-1] % 2:
            raise ValueError("size rescaling failed")
        self.sizes = sizes.astype(np.uint64)

    def tensor(self, i: int) -> np.ndarray:
        return as_bytes(normal_bf16(rng(self.workload, PURPOSE_BYTES, 1 + i), int(self.sizes[i]) // 2))

    def arena(self, align: int = 256, threads: int = 8):
        offs, total = arena_offsets(self.sizes.tolist(), align)
        arena = np.empty(total, dtype=np.uint8)
        parallel_fill(arena, offs, [lambda i=i: self.tensor(i) for i in range(len(self.sizes))], threads)
        return arena, offs, self.sizes.copy()

    def random_digests(self, n: int = 20_000_000) -> np.ndarray:
        return rng(self.workload, PURPOSE_DIGESTS, 0).integers(0, np.iinfo(np.uint64).max, size=n,
                                                               dtype=np.uint64, endpoint=True)

    def cached_blocks(self, n_blocks: int, frac: float = 0.6) -> np.ndarray:
        k = int(math.floor(frac * n_blocks))
        return np.sort(rng(self.workload, PURPOSE_SELECT, 0).choice(n_blocks, k, replace=False))


# --------------------------------------------------------------------------- #
# Address-remap intervals of many tasks (workload 6)
# --------------------------------------------------------------------------- #
TASK_SPACE_BITS = 40          # one 1 TB virtual address space per task
ALLOC_ROUND = 512             # the caching allocator's rounding of tensor sizes
POOL_BASE = 0x7000_0000_0000  # where the server's shareable pool regions start


def model_type_sizes() -> list[np.ndarray]:
    """Tensor byte sizes of the three model types a task can be: the 7B decoder and
    ResNet-50 in fp16, and the 2,000-tensor bf16 set."""
    dec = Decoder()
    res = [2 * math.prod(s) for _, s in resnet50_shapes()]
    return [np.array(dec.nbytes, np.uint64), np.array(res, np.uint64), LargeSet().sizes.copy()]


def _packed(sizes: np.ndarray, base: int) -> np.ndarray:
    rounded = (sizes + np.uint64(ALLOC_ROUND - 1)) // np.uint64(ALLOC_ROUND) * np.uint64(ALLOC_ROUND)
    return np.uint64(base) + np.concatenate([[0], np.cumsum(rounded)[:-1]]).astype(np.uint64)


class RemapTasks:
    """`n_tasks` tasks, each of a model type drawn uniformly, that loaded their tensors
    back to back (sizes rounded up to 512 bytes) from a random 2 MiB-aligned base in the
    lower half of their own 1 TB space [t << 40, (t + 1) << 40). Every tensor maps onto the
    shareable copy of the same tensor of its type: one pool region per type at
    POOL_BASE + type << 40, packed the same way. Homogeneous tasks therefore share
    targets; intervals of different tasks never meet."""

    def __init__(self, n_tasks: int = 256, workload: int = 6, types=None):
        self.workload = workload
        self.type_sizes = model_type_sizes() if types is None else [np.asarray(t, np.uint64) for t in types]
        sel = rng(workload, PURPOSE_SELECT, 0)
        self.task_type = sel.integers(0, len(self.type_sizes), n_tasks)
        self.task_base = sel.integers(0, 1 << (TASK_SPACE_BITS - 1 - 21), n_tasks).astype(np.uint64) << np.uint64(21)
        self.pool = [_packed(s, POOL_BASE + (k << TASK_SPACE_BITS)) for k, s in enumerate(self.type_sizes)]
        self.n_tasks = n_tasks

    def task(self, t: int):
        """(start, length, target) of task t's tensors."""
        k = int(self.task_type[t])
        sizes = self.type_sizes[k]
        base = (t << TASK_SPACE_BITS) + int(self.task_base[t])
        return _packed(sizes, base), sizes.copy(), self.pool[k].copy()

    def intervals(self, tasks=None):
        tasks = range(self.n_tasks) if tasks is None else tasks
        parts = [self.task(int(t)) for t in tasks]
        if not parts:
            z = np.zeros(0, np.uint64)
            return z, z, z
        return tuple(np.concatenate([p[i] for p in parts]) for i in range(3))

    def pointers(self, n: int, hit_frac: float = 0.9, index: int = 0) -> np.ndarray:
        """n pointers: a fraction `hit_frac` at uniform offsets inside uniformly chosen
        tensors, the rest uniform over a random task's whole 1 TB space."""
        start, length, _ = self.intervals()
        g = rng(self.workload, PURPOSE_SELECT, 1 + index)
        inside = g.random(n) < hit_frac
        pick = g.integers(0, start.size, n)
        off = (g.random(n) * length[pick].astype(np.float64)).astype(np.uint64)
        off = np.minimum(off, length[pick] - np.uint64(1))
        task = g.integers(0, self.n_tasks, n).astype(np.uint64)
        anywhere = (task << np.uint64(TASK_SPACE_BITS)) + g.integers(0, 1 << TASK_SPACE_BITS, n).astype(np.uint64)
        return np.where(inside, start[pick] + off, anywhere).astype(np.uint64)


# --------------------------------------------------------------------------- #
# Recorded host-to-device write logs of allocations (workload 7)
# --------------------------------------------------------------------------- #
class WriteLogs:
    """`n_alloc` allocations, allocation r at (r + 1) << 36 with a size drawn log-uniform in
    [4 KiB, 16 MiB], each receiving 1-64 recorded writes in time order: half of them a
    uniformly drawn sub-range of the allocation, three in ten the whole allocation, two in
    ten a repeat of an earlier write of the same allocation (the first write of an
    allocation is never a repeat). Weight-like allocations (one write) and input-like ones
    (the same range written again and again) both occur."""

    def __init__(self, n_alloc: int = 4096, workload: int = 7, max_writes: int = 64):
        g = rng(workload, PURPOSE_SELECT, 0)
        sizes = np.floor(np.exp(g.uniform(math.log(4 * KiB), math.log(16 * MiB), n_alloc))).astype(np.int64)
        counts = g.integers(1, max_writes + 1, n_alloc)
        addr, length = [], []
        first = [0]
        for r in range(n_alloc):
            base, size = (r + 1) << 36, int(sizes[r])
            mine = []
            for j in range(int(counts[r])):
                u = g.random()
                if u < 0.2 and mine:
                    a, n = mine[int(g.integers(0, len(mine)))]
                elif u < 0.5:
                    a, n = base, size
                else:
                    lo, hi = sorted(int(x) for x in g.integers(0, size + 1, 2))
                    a, n = base + lo, hi - lo
                mine.append((a, n))
            addr.extend(a for a, _ in mine)
            length.extend(n for _, n in mine)
            first.append(len(addr))
        self.addr = np.array(addr, dtype=np.uint64)
        self.length = np.array(length, dtype=np.uint64)
        self.region_first = np.array(first, dtype=np.uint64)
        self.n_alloc = n_alloc
