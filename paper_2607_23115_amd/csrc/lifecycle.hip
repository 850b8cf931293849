// Table lifecycle (Gleam Sec. 4.1.3: identified weight chunks stay in a shared cache
// across tasks, and LRU eviction keeps that cache bounded for long-lived multi-task
// serving; Sec. 4.1.2: the server ships the identifiers it holds at connect time).
//
//   touch   stamp present keys with max(stamp, epoch): the "use" of an entry
//   evict   keep the `keep` most recently used entries; order = (stamp, key) ascending
//   erase   remove the given keys
//   export  every entry, sorted by key (the identifier set, or a checkpoint)
//
// Evict gathers every slot into the workspace, then clears the table and re-inserts the
// survivors; the order for eviction comes from three stable radix passes (key, then
// stamp, then a live/empty bit), so it does not depend on where keys sit in the table.
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

#include <rocprim/device/device_radix_sort.hpp>

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;
constexpr uint32_t kMaxGrid = 8192;

struct Entries {  // gathered entries; m = capacity + 1, the last one is the key kEmpty
  uint64_t* key;
  uint64_t* val;
  uint64_t* stamp;
  uint8_t* live;
  uint8_t* flag;       // erase marks
  uint64_t* counters;  // [0] live entries, [1] live entries marked for removal
  uint64_t m;
};

struct MaintLayout {
  uint64_t m;
  size_t counters, key, val, stamp, live, flag, k_a, k_b, i_a, i_b, sort_tmp, sort_bytes, total;
  bool ok;  // the sort's temporary-storage queries succeeded
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
  L.live = take(L.m);
  L.flag = take(L.m);
  L.k_a = take(8 * L.m);
  L.k_b = take(8 * L.m);
  L.i_a = take(8 * L.m);
  L.i_b = take(8 * L.m);
  size_t full = 0, one_bit = 0;
  const hipError_t e_full = rocprim::radix_sort_pairs(nullptr, full, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                                      (const uint64_t*)nullptr, (uint64_t*)nullptr, (size_t)L.m, 0, 64);
  const hipError_t e_bit = rocprim::radix_sort_pairs(nullptr, one_bit, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                                     (const uint64_t*)nullptr, (uint64_t*)nullptr, (size_t)L.m, 0, 1);
  L.ok = e_full == hipSuccess && e_bit == hipSuccess;
  L.sort_bytes = full > one_bit ? full : one_bit;
  L.sort_tmp = take(L.sort_bytes);
  L.total = off;
  return L;
}

Entries entries_at(void* ws, const MaintLayout& L) {
  uint8_t* b = static_cast<uint8_t*>(ws);
  return Entries{reinterpret_cast<uint64_t*>(b + L.key),   reinterpret_cast<uint64_t*>(b + L.val),
                 reinterpret_cast<uint64_t*>(b + L.stamp), b + L.live,
                 b + L.flag,                               reinterpret_cast<uint64_t*>(b + L.counters),
                 L.m};
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

__global__ void touch_kernel(TableRef t, const uint64_t* keys, uint64_t n, const uint64_t* epochs, uint64_t epoch,
                             uint64_t* n_touched) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint64_t hit = 0;
  if (i < n) {
    const uint64_t k = keys[i];
    const uint64_t e = epochs ? epochs[i] : epoch;
    if (k == kEmpty) {
      if (t.hdr[0]) {
        atomicMax(ull(&t.hdr[2]), (unsigned long long)e);
        hit = 1;
      }
    } else {
      const int64_t pos = find_slot(t, k);
      if (pos >= 0) {
        atomicMax(ull(&t.stamps[pos]), (unsigned long long)e);
        hit = 1;
      }
    }
  }
  hit = wave_sum(hit);
  if (n_touched && (threadIdx.x & 63) == 0 && hit) atomicAdd(ull(n_touched), (unsigned long long)hit);
}

// Copy every slot (and the kEmpty side slot) into the entry arrays; count live and
// live-and-marked entries.
__global__ void gather_kernel(TableRef t, Entries e) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint64_t live = 0, marked = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < e.m; i += stride) {
    uint64_t k, v, s;
    bool is_live;
    if (i + 1 < e.m) {
      const uint4 kv = *reinterpret_cast<const uint4*>(t.slots + 2 * i);
      k = lo64(kv);
      v = hi64(kv);
      s = t.stamps[i];
      is_live = k != kEmpty;
    } else {
      k = kEmpty;
      v = t.hdr[1];
      s = t.hdr[2];
      is_live = t.hdr[0] != 0;
    }
    e.key[i] = k;
    e.val[i] = v;
    e.stamp[i] = s;
    e.live[i] = is_live ? 1 : 0;
    live += is_live ? 1 : 0;
    marked += (is_live && e.flag[i]) ? 1 : 0;
  }
  live = wave_sum(live);
  marked = wave_sum(marked);
  if ((threadIdx.x & 63) == 0) {
    if (live) atomicAdd(ull(&e.counters[0]), (unsigned long long)live);
    if (marked) atomicAdd(ull(&e.counters[1]), (unsigned long long)marked);
  }
}

__global__ void iota_kernel(uint64_t* out, uint64_t m) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) out[i] = i;
}

__global__ void permute_kernel(const uint64_t* src, const uint64_t* perm, uint64_t* dst, uint64_t m) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) dst[i] = src[perm[i]];
}

// 0 for live entries, 1 for empty slots (so a stable 1-bit pass puts live entries first).
__global__ void empty_bit_kernel(const uint8_t* live, const uint64_t* perm, uint64_t* dst, uint64_t m) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride)
    dst[i] = live[perm[i]] ? 0 : 1;
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

// Eviction: positions [0, E) of the (stamp, key) order go, [E, live) are re-inserted.
__global__ void evict_reinsert_kernel(TableRef t, Entries e, const uint64_t* perm, uint64_t keep, uint64_t* evicted,
                                      uint64_t* counts) {
  const uint64_t live = e.counters[0];
  const uint64_t drop = live > keep ? live - keep : 0;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t t0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t0 == 0) {
    counts[0] = drop;
    counts[1] = live - drop;
    t.hdr[3] = live - drop;
  }
  for (uint64_t i = t0; i < live; i += stride) {
    const uint64_t j = perm[i];
    if (i < drop) {
      if (evicted) evicted[i] = e.key[j];
    } else {
      insert_entry(t, e.key[j], e.val[j], e.stamp[j]);
    }
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

__global__ void export_kernel(Entries e, const uint64_t* perm, uint64_t* keys, uint64_t* vals, uint64_t* stamps,
                              uint64_t* count) {
  const uint64_t live = e.counters[0];
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t t0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t0 == 0) *count = live;
  for (uint64_t i = t0; i < live; i += stride) {
    const uint64_t j = perm[i];
    keys[i] = e.key[j];
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
  if (!L->ok) {
    set_error("%s: radix sort storage query failed", who);
    return GLEAM_E_HIP;
  }
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

// Reset counters and erase marks, then gather every entry.
gleam_status gather(const gleam_cache* c, void* ws, const MaintLayout& L, hipStream_t s, bool clear_flags) {
  uint8_t* b = static_cast<uint8_t*>(ws);
  gleam_status st = fill_u64(reinterpret_cast<uint64_t*>(b + L.counters), 4, 0, s);
  if (st == GLEAM_OK && clear_flags) st = fill_u64(reinterpret_cast<uint64_t*>(b + L.flag), (L.m + 7) / 8, 0, s);
  if (st != GLEAM_OK) return st;
  hipLaunchKernelGGL(gather_kernel, dim3(grid_for(L.m)), dim3(kThreads), 0, s, table_ref(c), entries_at(ws, L));
  return launch_status("gather_kernel");
}

gleam_status sort_pass(void* ws, const MaintLayout& L, const uint64_t* kin, uint64_t* kout, const uint64_t* vin,
                       uint64_t* vout, unsigned end_bit, hipStream_t s) {
  size_t bytes = L.sort_bytes;
  const hipError_t e = rocprim::radix_sort_pairs(static_cast<uint8_t*>(ws) + L.sort_tmp, bytes, kin, kout, vin, vout,
                                                 (size_t)L.m, 0, end_bit, s);
  if (e != hipSuccess) {
    set_error("radix sort: %s", hipGetErrorString(e));
    return GLEAM_E_HIP;
  }
  return launch_status("radix sort");
}

}  // namespace
}  // namespace gleam

extern "C" size_t gleam_cache_maint_bytes(const gleam_cache* c) {
  if (!c || c->capacity > (1ull << 31)) return 0;
  const gleam::MaintLayout L = gleam::maint_layout(c->capacity);
  return L.ok ? L.total : 0;
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
  uint8_t* b = static_cast<uint8_t*>(d_ws);
  const Entries e = entries_at(d_ws, L);
  uint64_t* k_a = reinterpret_cast<uint64_t*>(b + L.k_a);
  uint64_t* k_b = reinterpret_cast<uint64_t*>(b + L.k_b);
  uint64_t* i_a = reinterpret_cast<uint64_t*>(b + L.i_a);
  uint64_t* i_b = reinterpret_cast<uint64_t*>(b + L.i_b);
  const dim3 grid(grid_for(L.m)), block(kThreads);
  if ((st = gather(c, d_ws, L, s, true)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(iota_kernel, grid, block, 0, s, i_b, L.m);
  if ((st = launch_status("iota_kernel")) != GLEAM_OK) return st;
  // (stamp, key) order: by key, then stably by stamp, then live entries first
  if ((st = sort_pass(d_ws, L, e.key, k_a, i_b, i_a, 64, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(permute_kernel, grid, block, 0, s, e.stamp, i_a, k_b, L.m);
  if ((st = launch_status("permute_kernel")) != GLEAM_OK) return st;
  if ((st = sort_pass(d_ws, L, k_b, k_a, i_a, i_b, 64, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(empty_bit_kernel, grid, block, 0, s, e.live, i_b, k_b, L.m);
  if ((st = launch_status("empty_bit_kernel")) != GLEAM_OK) return st;
  if ((st = sort_pass(d_ws, L, k_b, k_a, i_b, i_a, 1, s)) != GLEAM_OK) return st;
  if ((st = clear_table(c, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(evict_reinsert_kernel, grid, block, 0, s, table_ref(c), e, i_a, keep, d_evicted, d_counts);
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
  uint8_t* b = static_cast<uint8_t*>(d_ws);
  const Entries e = entries_at(d_ws, L);
  uint64_t* k_a = reinterpret_cast<uint64_t*>(b + L.k_a);
  uint64_t* k_b = reinterpret_cast<uint64_t*>(b + L.k_b);
  uint64_t* i_a = reinterpret_cast<uint64_t*>(b + L.i_a);
  uint64_t* i_b = reinterpret_cast<uint64_t*>(b + L.i_b);
  const dim3 grid(grid_for(L.m)), block(kThreads);
  if ((st = gather(c, d_ws, L, s, true)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(iota_kernel, grid, block, 0, s, i_b, L.m);
  if ((st = launch_status("iota_kernel")) != GLEAM_OK) return st;
  if ((st = sort_pass(d_ws, L, e.key, k_a, i_b, i_a, 64, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(empty_bit_kernel, grid, block, 0, s, e.live, i_a, k_b, L.m);
  if ((st = launch_status("empty_bit_kernel")) != GLEAM_OK) return st;
  if ((st = sort_pass(d_ws, L, k_b, k_a, i_a, i_b, 1, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(export_kernel, grid, block, 0, s, e, i_b, d_keys, d_vals, d_stamps, d_count);
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
