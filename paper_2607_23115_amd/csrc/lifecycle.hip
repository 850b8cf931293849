// Table lifecycle (Gleam Sec. 4.1.3: identified weight chunks stay in a shared cache
// across tasks, and LRU eviction keeps that cache bounded for long-lived multi-task
// serving; Sec. 4.1.2: the server ships the identifiers it holds at connect time).
//
//   touch   stamp present keys with max(stamp, epoch): the "use" of an entry
//   evict   keep the `keep` most recently used entries; order = (stamp, key) ascending
//   erase   remove the given keys
//   export  every entry, sorted by key (the identifier set, or a checkpoint)
//
// Evict and export gather the live entries into the workspace and order them with a
// hand-written radix sort (radix_sort.h): by (stamp, key) for eviction, by key for export.
// Both orders are of distinct keys, so they do not depend on where keys sit in the table.
// Evict then clears the table and re-inserts the survivors. Every maintenance call
// enqueues kernels only (fills are kernels too), so each may be captured in a HIP graph.
//
// Erase costs O(keys erased), not O(capacity), and leaves no tombstones: each erased key's
// cluster (the run of occupied slots around it, bounded by empty slots; linear probing
// never crosses an empty slot) is repaired by one thread. It empties the erased slots, then
// re-inserts the cluster's other entries in cluster order, each at the first empty slot
// from its home, which is never past its old slot, so the cluster stays a valid probe
// sequence and other clusters are not touched. Clusters are found before any is repaired
// (a kernel boundary apart), and each is repaired by exactly one thread (the first to
// claim its start in a workspace set).
//
// The table header keeps the live-entry count (word 3): inserts add their new keys, erase
// subtracts what it removed, evict sets it, so erase can report the count without a scan.

#include "gleam_device.h"
#include "gleam_internal.h"
#include "radix_sort.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;
constexpr uint32_t kMaxGrid = 8192;

struct Entries {  // the live entries, gathered in table-tile order (count in counters[0])
  uint64_t* key;
  uint64_t* val;
  uint64_t* stamp;
  uint64_t* counters;  // [0] live entries; [4..7] the sort's AND/OR words of (key, stamp)
  uint64_t m;          // capacity + 1 (the last slot is the key kEmpty's header side slot)
};

struct MaintLayout {
  uint64_t m;
  size_t counters, key, val, stamp, hi, lo, idx, sort, total;
};

MaintLayout maint_layout(uint64_t capacity) {
  MaintLayout L;
  L.m = capacity + 1;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = (off + bytes + 255) & ~(size_t)255;
    return o;
  };
  L.counters = take(256);
  L.key = take(8 * L.m);
  L.val = take(8 * L.m);
  L.stamp = take(8 * L.m);
  L.hi = take(8 * sort_capacity(L.m));  // the sort's keys and indices (its buffer a)
  L.lo = take(8 * sort_capacity(L.m));
  L.idx = take(4 * sort_capacity(L.m));
  L.sort = take(sort_layout(L.m, 2).total);
  L.total = off;
  return L;
}

Entries entries_at(void* ws, const MaintLayout& L) {
  uint8_t* b = static_cast<uint8_t*>(ws);
  return Entries{reinterpret_cast<uint64_t*>(b + L.key), reinterpret_cast<uint64_t*>(b + L.val),
                 reinterpret_cast<uint64_t*>(b + L.stamp), reinterpret_cast<uint64_t*>(b + L.counters), L.m};
}

SortBuf sort_a(void* ws, const MaintLayout& L, int words) {
  uint8_t* b = static_cast<uint8_t*>(ws);
  return SortBuf{words == 2 ? reinterpret_cast<uint64_t*>(b + L.hi) : nullptr, reinterpret_cast<uint64_t*>(b + L.lo),
                 reinterpret_cast<uint32_t*>(b + L.idx)};
}

SortBuf sort_b(void* ws, const MaintLayout& L, int words) {
  return sort_other(static_cast<uint8_t*>(ws) + L.sort, L.m, words);
}

uint32_t grid_for(uint64_t n) {
  const uint64_t g = (n + kThreads - 1) / kThreads;
  return (uint32_t)(g == 0 ? 1 : (g < kMaxGrid ? g : kMaxGrid));
}

__device__ __forceinline__ unsigned long long* ull(uint64_t* p) { return reinterpret_cast<unsigned long long*>(p); }

// Slot of key k in the table, or -1 (k != kEmpty).
__device__ __forceinline__ int64_t find_slot(const TableRef& t, uint64_t k) {
  uint64_t pos = slot_hash(k, t.shift);
  for (uint64_t probe = 0; probe <= t.mask; ++probe) {
    const uint64_t key = t.slots[2 * pos];
    if (key == k) return (int64_t)pos;
    if (key == kEmpty) return -1;
    pos = (pos + 1) & t.mask;
  }
  return -1;
}

__device__ __forceinline__ uint64_t wave_sum(uint64_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += shfl_xor64(x, o);
  return x;
}

// Touch. Copies of one key in a workgroup are folded first: an LDS table of lane numbers
// finds each key's lowest lane and takes the largest of the copies' epochs, and only that
// lane updates the stamp (at most one atomic per key per workgroup). A batch of one
// repeated key, as a zero-filled tensor gives, would otherwise queue one atomic per copy
// on one word (262,144 copies: 11.6 ms). A stamp only grows, so a lane whose stamp
// already reads at or past its epoch skips the atomic.
constexpr int kTouchSlots = 2 * kThreads;  // power of two, load at most 1/2

__global__ __launch_bounds__(kThreads) void touch_kernel(TableRef t, const uint64_t* keys, uint64_t n,
                                                         const uint64_t* epochs, uint64_t epoch,
                                                         uint64_t* n_touched) {
  __shared__ uint64_t bkeys[kThreads];
  __shared__ uint32_t bslot[kTouchSlots];  // lowest lane + 1 of the key in this slot (0 free)
  __shared__ uint64_t bmax[kTouchSlots];   // the largest epoch of that key's copies
  const uint32_t tid = threadIdx.x;
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + tid;
  const bool valid = i < n;
  const uint64_t k = valid ? keys[i] : 0;
  const uint64_t e = valid ? (epochs ? epochs[i] : epoch) : 0;
  bkeys[tid] = k;
  bslot[tid] = 0;
  bslot[tid + kThreads] = 0;
  bmax[tid] = 0;
  bmax[tid + kThreads] = 0;
  __syncthreads();
  uint32_t at = 0;
  if (valid) {
    static_assert(kTouchSlots == 512, "slot_hash shift");
    at = (uint32_t)slot_hash(k, 64 - 9);
    for (int probe = 0; probe < kTouchSlots; ++probe) {
      const uint32_t prev = atomicCAS(&bslot[at], 0u, tid + 1);
      if (prev == 0) break;
      if (bkeys[prev - 1] == k) {
        atomicMin(&bslot[at], tid + 1);
        break;
      }
      at = (at + 1) & (kTouchSlots - 1);
    }
    atomicMax(reinterpret_cast<unsigned long long*>(&bmax[at]), (unsigned long long)e);
  }
  __syncthreads();
  uint64_t hit = 0;
  if (valid) {
    const bool lead = bslot[at] == tid + 1;
    const uint64_t top = bmax[at];
    uint64_t* stamp = nullptr;
    if (k == kEmpty) {
      if (t.hdr[0]) stamp = &t.hdr[2];
    } else {
      const int64_t pos = find_slot(t, k);
      if (pos >= 0) stamp = &t.stamps[pos];
    }
    if (stamp) {
      hit = 1;
      if (lead && __hip_atomic_load(stamp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < top)
        atomicMax(ull(stamp), (unsigned long long)top);
    }
  }
  hit = wave_sum(hit);
  if (n_touched && (tid & 63) == 0 && hit) atomicAdd(ull(n_touched), (unsigned long long)hit);
}

__global__ void maint_init_kernel(uint64_t* counters) {
  if (threadIdx.x < 8) counters[threadIdx.x] = (threadIdx.x == 4 || threadIdx.x == 6) ? ~0ull : 0ull;
}

// Each workgroup takes tiles of 4096 slots in turn (the last tile also the kEmpty side
// slot), counts a tile's live entries, claims that many positions with one atomic, and
// writes the entries there in slot order: to the entry arrays, and to the sort's buffer
// (key words (stamp, key) or key; index = position). It also folds the AND and OR of
// the keys and stamps into counters[4..7], once per workgroup at the end, from which
// the sort skips the digits every entry shares. The grid is capped so that those folds
// (four atomics on four words per workgroup) stay few.
constexpr uint32_t kGatherItems = 16;
constexpr uint64_t kGatherTile = (uint64_t)kThreads * kGatherItems;
constexpr uint32_t kGatherMaxGrid = 1024;

__global__ __launch_bounds__(kThreads) void gather_kernel(TableRef t, Entries e, SortBuf sb, uint64_t tiles) {
  __shared__ uint32_t wave_live[kThreads / 64];
  __shared__ uint64_t tile_base;
  __shared__ uint64_t fold[kThreads / 64][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
  uint64_t and_k = ~0ull, or_k = 0, and_s = ~0ull, or_s = 0;
  for (uint64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const uint64_t first = tile * kGatherTile + (uint64_t)wave * 64 * kGatherItems + lane;
    uint64_t key[kGatherItems], val[kGatherItems], mask[kGatherItems];
    uint32_t live_n = 0;
#pragma unroll
    for (uint32_t r = 0; r < kGatherItems; ++r) {
      const uint64_t i = first + 64ull * r;
      bool live = false;
      key[r] = kEmpty;
      val[r] = 0;
      if (i + 1 < e.m) {
        const uint4 kv = *reinterpret_cast<const uint4*>(t.slots + 2 * i);
        key[r] = lo64(kv);
        val[r] = hi64(kv);
        live = key[r] != kEmpty;
      } else if (i + 1 == e.m) {
        live = t.hdr[0] != 0;
        val[r] = t.hdr[1];
      }
      mask[r] = __ballot(live);
      live_n += (uint32_t)__popcll(mask[r]);
    }
    if (lane == 0) wave_live[wave] = live_n;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t total = 0;
      for (int w = 0; w < kThreads / 64; ++w) total += wave_live[w];
      tile_base = total ? atomicAdd(ull(&e.counters[0]), (unsigned long long)total) : 0;
    }
    __syncthreads();
    uint64_t at = tile_base;
    for (int w = 0; w < wave; ++w) at += wave_live[w];
#pragma unroll
    for (uint32_t r = 0; r < kGatherItems; ++r) {
      if ((mask[r] >> lane) & 1ull) {
        const uint64_t i = first + 64ull * r;
        const uint64_t s = i + 1 < e.m ? t.stamps[i] : t.hdr[2];
        const uint64_t p = at + (uint64_t)__popcll(mask[r] & lt);
        e.key[p] = key[r];
        e.val[p] = val[r];
        e.stamp[p] = s;
        if (sb.hi) sb.hi[p] = s;
        sb.lo[p] = key[r];
        sb.idx[p] = (uint32_t)p;
        and_k &= key[r];
        or_k |= key[r];
        and_s &= s;
        or_s |= s;
      }
      at += (uint64_t)__popcll(mask[r]);
    }
    __syncthreads();  // wave_live and tile_base read before the next tile rewrites them
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    and_k &= shfl_xor64(and_k, o);
    or_k |= shfl_xor64(or_k, o);
    and_s &= shfl_xor64(and_s, o);
    or_s |= shfl_xor64(or_s, o);
  }
  if (lane == 0) {
    fold[wave][0] = and_k;
    fold[wave][1] = or_k;
    fold[wave][2] = and_s;
    fold[wave][3] = or_s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kThreads / 64; ++w) {
      fold[0][0] &= fold[w][0];
      fold[0][1] |= fold[w][1];
      fold[0][2] &= fold[w][2];
      fold[0][3] |= fold[w][3];
    }
    if (fold[0][0] != ~0ull || fold[0][1] != 0) {  // some live entry was seen (an all-ones key has OR != 0)
      atomicAnd(ull(&e.counters[4]), (unsigned long long)fold[0][0]);
      atomicOr(ull(&e.counters[5]), (unsigned long long)fold[0][1]);
      atomicAnd(ull(&e.counters[6]), (unsigned long long)fold[0][2]);
      atomicOr(ull(&e.counters[7]), (unsigned long long)fold[0][3]);
    }
  }
}

__device__ void insert_entry(const TableRef& t, uint64_t k, uint64_t v, uint64_t s) {
  if (k == kEmpty) {
    t.hdr[0] = 1;
    t.hdr[1] = v;
    t.hdr[2] = s;
    return;
  }
  uint64_t pos = slot_hash(k, t.shift);
  for (uint64_t probe = 0; probe <= t.mask; ++probe) {
    if (atomicCAS(ull(t.slots + 2 * pos), (unsigned long long)kEmpty, (unsigned long long)k) == kEmpty) {
      t.slots[2 * pos + 1] = v;
      t.stamps[pos] = s;
      return;
    }
    pos = (pos + 1) & t.mask;
  }
}

// Eviction: positions [0, E) of the (stamp, key) order go, the rest are re-inserted.
// The evicted keys are read from the sorted keys; the survivors are re-inserted in
// gather order (slot order within each tile, so neighbouring inserts touch neighbouring
// slots), each kept when its (stamp, key) is not below the first survivor's. The pairs
// are distinct, so that is exactly the sorted positions from E on.
__global__ void evict_reinsert_kernel(TableRef t, Entries e, SortBuf a, SortBuf b, uint64_t keep,
                                      uint64_t* evicted, uint64_t* counts) {
  const uint64_t live = e.counters[0];
  const uint64_t drop = live > keep ? live - keep : 0;
  const SortBuf sorted = sort_result(a, b, e.counters + 4, 2);
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t t0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t0 == 0) {
    counts[0] = drop;
    counts[1] = live - drop;
    t.hdr[3] = live - drop;
  }
  if (drop == live) {
    if (evicted)
      for (uint64_t i = t0; i < drop; i += stride) evicted[i] = sorted.lo[i];
    return;
  }
  const uint64_t min_s = sorted.hi[drop], min_k = sorted.lo[drop];
  for (uint64_t i = t0; i < live; i += stride) {
    if (evicted && i < drop) evicted[i] = sorted.lo[i];
    const uint64_t s = e.stamp[i], k = e.key[i];
    if (s > min_s || (s == min_s && k >= min_k)) insert_entry(t, k, e.val[i], s);
  }
}

// ---- erase: O(keys erased) ------------------------------------------------------------
struct EraseWs {          // workspace of an erase of n keys
  uint64_t* hdr;          // [0] entries removed, [1] clusters to repair
  uint64_t* keyset;       // cap slots: index + 1 of an erased key (0 free); keys read back
  uint64_t* starts;       // cap slots: cluster start + 1 (0 free)
  uint64_t* leaders;      // n cluster starts, one per cluster
  uint64_t mask;
  int shift;
};

__device__ __forceinline__ bool in_keyset(const EraseWs& w, const uint64_t* keys, uint64_t k) {
  uint64_t pos = slot_hash(k, w.shift);
  for (uint64_t probe = 0; probe <= w.mask; ++probe) {
    const uint64_t v = w.keyset[pos];
    if (v == 0) return false;
    if (keys[v - 1] == k) return true;
    pos = (pos + 1) & w.mask;
  }
  return false;
}

__global__ void erase_keyset_kernel(const uint64_t* keys, uint64_t n, EraseWs w) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n || keys[i] == kEmpty) return;
  const uint64_t k = keys[i];
  uint64_t pos = slot_hash(k, w.shift);
  for (uint64_t probe = 0; probe <= w.mask; ++probe) {
    const uint64_t prev = atomicCAS(ull(&w.keyset[pos]), 0ull, (unsigned long long)(i + 1));
    if (prev == 0 || keys[prev - 1] == k) return;
    pos = (pos + 1) & w.mask;
  }
}

// Per erased key that is present: the start of its cluster, claimed once.
__global__ void erase_find_kernel(TableRef t, const uint64_t* keys, uint64_t n, EraseWs w) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint64_t k = keys[i];
  if (k == kEmpty) {  // the header's side slot
    if (atomicExch(ull(&t.hdr[0]), 0ull) == 1ull) {
      t.hdr[2] = 0;
      atomicAdd(ull(&w.hdr[0]), 1ull);
    }
    return;
  }
  const int64_t at = find_slot(t, k);
  if (at < 0) return;
  uint64_t c0 = (uint64_t)at;
  for (uint64_t step = 0; step <= t.mask; ++step) {
    const uint64_t before = (c0 - 1) & t.mask;
    if (t.slots[2 * before] == kEmpty) break;
    c0 = before;
  }
  uint64_t pos = slot_hash(c0, w.shift);
  for (uint64_t probe = 0; probe <= w.mask; ++probe) {
    const uint64_t prev = atomicCAS(ull(&w.starts[pos]), 0ull, (unsigned long long)(c0 + 1));
    if (prev == 0) {
      w.leaders[atomicAdd(ull(&w.hdr[1]), 1ull)] = c0;
      return;
    }
    if (prev == c0 + 1) return;  // claimed by another key of this cluster
    pos = (pos + 1) & w.mask;
  }
}

// One thread per cluster: empty the erased slots, then re-insert the rest in cluster order.
__global__ void erase_repair_kernel(TableRef t, const uint64_t* keys, uint64_t n, EraseWs w) {
  const uint64_t clusters = w.hdr[1];
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; c < clusters && c < n; c += stride) {
    const uint64_t c0 = w.leaders[c];
    uint64_t len = 0, removed = 0;
    for (uint64_t p = c0; len <= t.mask; p = (p + 1) & t.mask, ++len) {
      const uint64_t k = t.slots[2 * p];
      if (k == kEmpty) break;  // the cluster's end (slots emptied here lie behind)
      if (in_keyset(w, keys, k)) {
        t.slots[2 * p] = kEmpty;
        t.stamps[p] = 0;
        ++removed;
      }
    }
    if (removed == 0) continue;
    for (uint64_t i = 0; i < len; ++i) {
      const uint64_t p = (c0 + i) & t.mask;
      const uint64_t k = t.slots[2 * p];
      if (k == kEmpty) continue;
      uint64_t q = slot_hash(k, t.shift);
      if (q == p) continue;  // at home: the first empty slot from its home is here
      while (t.slots[2 * q] != kEmpty && q != p) q = (q + 1) & t.mask;
      if (q == p) continue;  // no empty slot before it: stays
      t.slots[2 * q] = k;
      t.slots[2 * q + 1] = t.slots[2 * p + 1];
      t.stamps[q] = t.stamps[p];
      t.slots[2 * p] = kEmpty;
      t.stamps[p] = 0;
    }
    atomicAdd(ull(&w.hdr[0]), (unsigned long long)removed);
  }
}

__global__ void erase_finish_kernel(TableRef t, EraseWs w, uint64_t* counts) {
  const uint64_t removed = w.hdr[0];
  const uint64_t live = t.hdr[3] - removed;
  t.hdr[3] = live;
  counts[0] = removed;
  counts[1] = live;
}

struct EraseLayout {
  uint64_t cap;
  size_t total;
};

EraseLayout erase_layout(uint64_t n) {
  EraseLayout L;
  L.cap = 64;
  while (L.cap < 2 * n) L.cap <<= 1;
  L.total = (kHeaderBytes + 16 * (size_t)L.cap + 8 * (size_t)n + 255) & ~(size_t)255;
  return L;
}

EraseWs erase_ws(void* ws, const EraseLayout& L) {
  uint8_t* b = static_cast<uint8_t*>(ws);
  EraseWs w;
  w.hdr = reinterpret_cast<uint64_t*>(b);
  w.keyset = reinterpret_cast<uint64_t*>(b + kHeaderBytes);
  w.starts = w.keyset + L.cap;
  w.leaders = w.starts + L.cap;
  w.mask = L.cap - 1;
  w.shift = 64 - log2_exact(L.cap);
  return w;
}

__global__ void export_kernel(Entries e, SortBuf a, SortBuf b, uint64_t* keys, uint64_t* vals, uint64_t* stamps,
                              uint64_t* count) {
  const uint64_t live = e.counters[0];
  const SortBuf sorted = sort_result(a, b, e.counters + 4, 1);
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t t0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t0 == 0) *count = live;
  for (uint64_t i = t0; i < live; i += stride) {
    const uint64_t j = sorted.idx[i];
    keys[i] = sorted.lo[i];
    vals[i] = e.val[j];
    if (stamps) stamps[i] = e.stamp[j];
  }
}

gleam_status check_maint(const gleam_cache* c, void* ws, size_t ws_bytes, const char* who, MaintLayout* L) {
  if (!c) {
    set_error("%s: null table", who);
    return GLEAM_E_INVALID;
  }
  if (c->capacity > (1ull << 31)) {
    set_error("%s: tables above 2^31 slots are not supported", who);
    return GLEAM_E_UNSUPPORTED;
  }
  *L = maint_layout(c->capacity);
  if (!ws || !aligned256(ws)) {
    set_error("%s: workspace must be non-null and 256-byte aligned", who);
    return GLEAM_E_INVALID;
  }
  if (ws_bytes < L->total) {
    set_error("%s: workspace of %zu bytes, %zu needed", who, ws_bytes, L->total);
    return GLEAM_E_WORKSPACE;
  }
  return GLEAM_OK;
}

// Reset the live count and the AND/OR words, gather the live entries, and sort them:
// by (stamp, key) for eviction (two key words), by key for export.
gleam_status gather_sorted(const gleam_cache* c, void* ws, const MaintLayout& L, int words, hipStream_t s) {
  uint8_t* b = static_cast<uint8_t*>(ws);
  uint64_t* counters = reinterpret_cast<uint64_t*>(b + L.counters);
  hipLaunchKernelGGL(maint_init_kernel, dim3(1), dim3(64), 0, s, counters);
  gleam_status st = launch_status("maint_init_kernel");
  if (st != GLEAM_OK) return st;
  const SortBuf a = sort_a(ws, L, words);
  const uint64_t tiles = (L.m + kGatherTile - 1) / kGatherTile;
  const uint32_t grid = (uint32_t)(tiles < kGatherMaxGrid ? tiles : kGatherMaxGrid);
  hipLaunchKernelGGL(gather_kernel, dim3(grid), dim3(kThreads), 0, s, table_ref(c), entries_at(ws, L), a, tiles);
  if ((st = launch_status("gather_kernel")) != GLEAM_OK) return st;
  // the key words' bits: (key, stamp) words are counters[4..7]; with one word the sort
  // reads only the key's pair, with two the stamp's as the high word
  return radix_sort_pairs(a, counters, counters + 4, L.m, words, b + L.sort, s);
}

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_lifecycle() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&maint_init_kernel));
}

}  // namespace gleam

extern "C" size_t gleam_cache_maint_bytes(const gleam_cache* c) {
  if (!c || c->capacity > (1ull << 31)) return 0;
  return gleam::maint_layout(c->capacity).total;
}

extern "C" gleam_status gleam_cache_touch(gleam_cache* c, const uint64_t* d_keys, uint64_t n,
                                          const uint64_t* d_epochs, uint64_t epoch, uint64_t* d_n_touched,
                                          void* stream) {
  using namespace gleam;
  clear_error();
  if (!c) {
    set_error("gleam_cache_touch: null table");
    return GLEAM_E_INVALID;
  }
  if (n > 0 && !d_keys) {
    set_error("gleam_cache_touch: null keys");
    return GLEAM_E_INVALID;
  }
  if (n > 0x7fffffffull * kThreads) {
    set_error("gleam_cache_touch: more than 2^31 workgroups of keys");
    return GLEAM_E_UNSUPPORTED;
  }
  hipStream_t s = (hipStream_t)stream;
  gleam_status st = GLEAM_OK;
  if (d_n_touched) st = fill_u64(d_n_touched, 1, 0, s);
  if (st != GLEAM_OK || n == 0) return st;
  hipLaunchKernelGGL(touch_kernel, dim3((uint32_t)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, s,
                     table_ref(c), d_keys, n, d_epochs, epoch, d_n_touched);
  return launch_status("touch_kernel");
}

extern "C" gleam_status gleam_cache_evict(gleam_cache* c, uint64_t keep, uint64_t* d_evicted, uint64_t* d_counts,
                                          void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  MaintLayout L;
  gleam_status st = check_maint(c, d_ws, ws_bytes, "gleam_cache_evict", &L);
  if (st != GLEAM_OK) return st;
  if (!d_counts) {
    set_error("gleam_cache_evict: null counts");
    return GLEAM_E_INVALID;
  }
  hipStream_t s = (hipStream_t)stream;
  if ((st = gather_sorted(c, d_ws, L, 2, s)) != GLEAM_OK) return st;
  if ((st = clear_table(c, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(evict_reinsert_kernel, dim3(grid_for(L.m)), dim3(kThreads), 0, s, table_ref(c),
                     entries_at(d_ws, L), sort_a(d_ws, L, 2), sort_b(d_ws, L, 2), keep, d_evicted, d_counts);
  if ((st = launch_status("evict_reinsert_kernel")) != GLEAM_OK) return st;
  if (keep < c->key_bound) c->key_bound = keep;
  return GLEAM_OK;
}

extern "C" size_t gleam_cache_erase_bytes(uint64_t n) {
  if (n > (1ull << 36)) return 0;
  return gleam::erase_layout(n).total;
}

extern "C" gleam_status gleam_cache_erase(gleam_cache* c, const uint64_t* d_keys, uint64_t n, uint64_t* d_counts,
                                          void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  if (!c || !d_counts || (n > 0 && !d_keys)) {
    set_error("gleam_cache_erase: null table, keys or counts");
    return GLEAM_E_INVALID;
  }
  if (n > (1ull << 36) || n > 0x7fffffffull * kThreads) {
    set_error("gleam_cache_erase: more than 2^36 keys");
    return GLEAM_E_UNSUPPORTED;
  }
  const EraseLayout L = erase_layout(n);
  if (!d_ws || !aligned256(d_ws)) {
    set_error("gleam_cache_erase: workspace must be non-null and 256-byte aligned");
    return GLEAM_E_INVALID;
  }
  if (ws_bytes < L.total) {
    set_error("gleam_cache_erase: workspace of %zu bytes, %zu needed", ws_bytes, L.total);
    return GLEAM_E_WORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  const EraseWs w = erase_ws(d_ws, L);
  const TableRef t = table_ref(c);
  // header and both sets to zero (a fill kernel, so the call can be captured in a graph)
  gleam_status st = fill_u64(w.hdr, (kHeaderBytes + 16 * L.cap) / 8, 0, s);
  if (st != GLEAM_OK) return st;
  if (n > 0) {
    const dim3 grid((uint32_t)((n + kThreads - 1) / kThreads)), block(kThreads);
    hipLaunchKernelGGL(erase_keyset_kernel, grid, block, 0, s, d_keys, n, w);
    if ((st = launch_status("erase_keyset_kernel")) != GLEAM_OK) return st;
    hipLaunchKernelGGL(erase_find_kernel, grid, block, 0, s, t, d_keys, n, w);
    if ((st = launch_status("erase_find_kernel")) != GLEAM_OK) return st;
    hipLaunchKernelGGL(erase_repair_kernel, dim3(grid_for(n)), block, 0, s, t, d_keys, n, w);
    if ((st = launch_status("erase_repair_kernel")) != GLEAM_OK) return st;
  }
  hipLaunchKernelGGL(erase_finish_kernel, dim3(1), dim3(1), 0, s, t, w, d_counts);
  return launch_status("erase_finish_kernel");
}

extern "C" gleam_status gleam_cache_export(const gleam_cache* c, uint64_t* d_keys, uint64_t* d_vals,
                                           uint64_t* d_stamps, uint64_t* d_count, void* d_ws, size_t ws_bytes,
                                           void* stream) {
  using namespace gleam;
  clear_error();
  MaintLayout L;
  gleam_status st = check_maint(c, d_ws, ws_bytes, "gleam_cache_export", &L);
  if (st != GLEAM_OK) return st;
  if (!d_keys || !d_vals || !d_count) {
    set_error("gleam_cache_export: null output");
    return GLEAM_E_INVALID;
  }
  hipStream_t s = (hipStream_t)stream;
  if ((st = gather_sorted(c, d_ws, L, 1, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(export_kernel, dim3(grid_for(L.m)), dim3(kThreads), 0, s, entries_at(d_ws, L),
                     sort_a(d_ws, L, 1), sort_b(d_ws, L, 1), d_keys, d_vals, d_stamps, d_count);
  return launch_status("export_kernel");
}

extern "C" gleam_status gleam_cache_set_key_bound(gleam_cache* c, uint64_t n) {
  gleam::clear_error();
  if (!c || n > c->key_bound) {
    gleam::set_error("gleam_cache_set_key_bound: null table, or the bound would rise");
    return GLEAM_E_INVALID;
  }
  c->key_bound = n;
  return GLEAM_OK;
}
