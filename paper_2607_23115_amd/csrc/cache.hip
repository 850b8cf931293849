// The resident identifier table: create, insert, lookup (Gleam Sec. 4.1.2: the
// server's set of identifiers of chunks it holds; a held identifier means only
// metadata travels. Sec. 4.1.3: identified weight chunks are kept for reuse).
//
// Layout: open addressing with linear probing over `capacity` 16-byte slots
// (key u64, value u64), after a 256-byte header. The empty marker is kEmpty; a key
// equal to kEmpty is kept in the header (flag + value), so every u64 is a key.
// The table is never fuller than max_load (enforced on the host), so every probe
// meets an empty slot; probe loops are still bounded by the capacity.
//
// Determinism: results never depend on thread timing. Duplicates inside one call
// are resolved through a workspace scratch table that keeps, per key, the lowest
// index; only that index inserts (insert) or is the MISS (lookup). A scratch slot
// holds just an index: its key is keys[index], the same for every index the slot
// ever holds. So a key's first index takes a slot with one compare-and-swap, and
// only later duplicates need an atomicMin.

#include <mutex>
#include <new>

#include "gleam_device.h"
#include "gleam_internal.h"
#include "gleam_table.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;

struct ScratchRef {
  uint64_t* hdr;    // [0] min index of key kEmpty, [1] new-key counter
  uint64_t* slots;  // cap x lowest index so far of one key (kFree: unused)
  uint64_t mask;
  int shift;
};

constexpr uint64_t kFree = ~0ull;

__device__ __forceinline__ unsigned long long* ull(uint64_t* p) { return reinterpret_cast<unsigned long long*>(p); }

__global__ void fill_kernel(uint64_t* p, uint64_t n, uint64_t value) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = value;
}

// Scratch: record index i of key k = keys[i], keeping the lowest index per key.
__device__ void scratch_mark(const ScratchRef& sc, const uint64_t* keys, uint64_t k, uint64_t i) {
  if (k == kEmpty) {
    atomicMin(ull(&sc.hdr[0]), (unsigned long long)i);
    return;
  }
  uint64_t pos = slot_hash(k, sc.shift);
  for (uint64_t probe = 0; probe <= sc.mask; ++probe) {
    uint64_t* slot = sc.slots + pos;
    const uint64_t prev = atomicCAS(ull(slot), (unsigned long long)kFree, (unsigned long long)i);
    if (prev == kFree) return;
    if (keys[prev] == k) {  // the slot of k; its value only decreases
      if (i < prev) atomicMin(ull(slot), (unsigned long long)i);
      return;
    }
    pos = (pos + 1) & sc.mask;
  }
}

// True for the lowest valid lane of the workgroup holding key k (lanes are in index
// order, so that lane carries the workgroup's lowest index of k). Only those lanes mark
// the device-wide scratch table: a batch of one repeated key (a zero-filled tensor)
// would otherwise queue every thread's compare-and-swap on one word (measured: 262,144
// equal keys took 3.2 ms, 18x their fingerprint). The check is an LDS table of lane
// numbers, so it adds no device memory round trip. Every thread of the workgroup
// (kThreads of them) calls it.
constexpr int kBlockSlots = 2 * kThreads;  // power of two, load at most 1/2
__device__ bool first_in_workgroup(uint64_t k, bool valid, uint64_t* bkeys, uint32_t* bslot) {
  const uint32_t tid = threadIdx.x;
  bkeys[tid] = k;
  bslot[tid] = 0;
  bslot[tid + kThreads] = 0;
  __syncthreads();
  uint32_t pos = 0;
  if (valid) {
    pos = (uint32_t)slot_hash(k, 64 - 9);
    static_assert(kBlockSlots == 512, "slot_hash shift");
    for (int probe = 0; probe < kBlockSlots; ++probe) {
      const uint32_t prev = atomicCAS(&bslot[pos], 0u, tid + 1);
      if (prev == 0) break;
      if (bkeys[prev - 1] == k) {
        atomicMin(&bslot[pos], tid + 1);
        break;
      }
      pos = (pos + 1) & (kBlockSlots - 1);
    }
  }
  __syncthreads();
  return valid && bslot[pos] == tid + 1;
}

// Scratch: the lowest index recorded for key k = keys[g] (g was marked earlier).
__device__ uint64_t scratch_min(const ScratchRef& sc, const uint64_t* keys, uint64_t k, uint64_t g) {
  if (k == kEmpty) return sc.hdr[0];
  uint64_t pos = slot_hash(k, sc.shift);
  for (uint64_t probe = 0; probe <= sc.mask; ++probe) {
    const uint64_t v = sc.slots[pos];
    if (v == kFree) break;
    if (v == g || keys[v] == k) return v;  // v == g: g's own key, so the slot of k
    pos = (pos + 1) & sc.mask;
  }
  return ~0ull;
}

__global__ __launch_bounds__(kThreads) void insert_mark_kernel(ScratchRef sc, const uint64_t* keys, uint64_t n) {
  __shared__ uint64_t bkeys[kThreads];
  __shared__ uint32_t bslot[kBlockSlots];
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool valid = i < n;
  const uint64_t k = valid ? keys[i] : 0;
  if (first_in_workgroup(k, valid, bkeys, bslot)) scratch_mark(sc, keys, k, i);
}

__global__ void insert_commit_kernel(TableRef t, ScratchRef sc, const uint64_t* keys, const uint64_t* vals,
                                     uint64_t n, uint64_t* n_new) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint64_t k = keys[i];
  if (scratch_min(sc, keys, k, i) != i) return;  // a lower index carries this key
  if (k == kEmpty) {
    if (atomicCAS(ull(&t.hdr[0]), 0ull, 1ull) == 0ull) {
      t.hdr[1] = vals[i];
      atomicAdd(ull(n_new), 1ull);
      atomicAdd(ull(&t.hdr[3]), 1ull);
    }
    return;
  }
  uint64_t pos = slot_hash(k, t.shift);
  for (uint64_t probe = 0; probe <= t.mask; ++probe) {
    uint64_t* slot = t.slots + 2 * pos;
    const uint64_t prev = atomicCAS(ull(slot), (unsigned long long)kEmpty, (unsigned long long)k);
    if (prev == kEmpty) {
      slot[1] = vals[i];
      atomicAdd(ull(n_new), 1ull);
      atomicAdd(ull(&t.hdr[3]), 1ull);
      return;
    }
    if (prev == k) return;  // already held: keep the existing value
    pos = (pos + 1) & t.mask;
  }
}

// Lookup pass 1: table probe. Hits are final; the rest are marked in the scratch
// table (by the workgroup's lowest lane of each key) and flagged 0xFF for pass 2.
__global__ __launch_bounds__(kThreads) void lookup_probe_kernel(TableRef t, ScratchRef sc, const uint64_t* keys,
                                                                uint64_t n, uint8_t* status, uint64_t* ref) {
  __shared__ uint64_t bkeys[kThreads];
  __shared__ uint32_t bslot[kBlockSlots];
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool valid = g < n;
  const uint64_t kg = keys[valid ? g : n - 1];  // n >= 1; clamped so the load is unconditional
  const uint64_t k = valid ? kg : 0;
  // the home slot's read is issued before the workgroup's LDS pass, which hides under it
  const uint64_t home = k != kEmpty ? slot_hash(k, t.shift) : 0;
  const uint4 e0 = *reinterpret_cast<const uint4*>(t.slots + 2 * home);
  // a repeat of a lower lane's key has that lane's table result: that lane marks
  const bool marks = first_in_workgroup(k, valid, bkeys, bslot);
  if (!valid) return;
  bool hit = false;
  uint64_t val = 0;
  if (k == kEmpty) {
    hit = t.hdr[0] != 0;
    val = t.hdr[1];
  } else if (lo64(e0) == k) {
    hit = true;
    val = hi64(e0);
  } else if (lo64(e0) != kEmpty) {
    uint64_t pos = (home + 1) & t.mask;
    for (uint64_t probe = 1; probe <= t.mask; ++probe) {
      const uint4 e = *reinterpret_cast<const uint4*>(t.slots + 2 * pos);
      const uint64_t key = lo64(e);
      if (key == k) {
        hit = true;
        val = hi64(e);
        break;
      }
      if (key == kEmpty) break;
      pos = (pos + 1) & t.mask;
    }
  }
  if (hit) {
    status[g] = GLEAM_HIT_CACHE;
    if (ref) ref[g] = val;
  } else {
    status[g] = 0xFF;
    if (marks) scratch_mark(sc, keys, k, g);
  }
}

// Lookups of up to kSmallKeys keys: one 1024-thread workgroup, with the dedup table in
// LDS (kSmallSlots slots of index + 1, 0 = free; the key is read back from `keys`), so
// no clear pass and no device-scope atomics. Pass 1 probes the resident table (each
// thread first issues the reads of all its keys' home slots) and marks non-hits in LDS;
// pass 2 resolves them. At these sizes the cost is launches, not bytes. Measured per
// call on MI355X (three-launch path / this): 256 keys 18.9 / 13.7 us, 4,096 keys 21.7 /
// 16.0 us, 8,192 keys 21.3 / 20.2 us, 12,917 keys 21.3 / 35.5 us: past a few thousand
// keys one CU cannot issue the table's scattered reads fast enough.
constexpr int kSmallThreads = 1024;
constexpr int kSmallPerThread = 4;
constexpr uint64_t kSmallKeys = (uint64_t)kSmallThreads * kSmallPerThread;  // 4,096
constexpr uint32_t kSmallSlots = 2 * kSmallKeys;                              // 32 KiB of LDS
constexpr int kSmallShift = 64 - 13;                                           // log2(kSmallSlots) = 13

__global__ __launch_bounds__(kSmallThreads) void lookup_small_kernel(TableRef t, const uint64_t* keys, uint64_t n,
                                                                     uint8_t* status, uint64_t* ref) {
  __shared__ uint32_t slots[kSmallSlots];
  __shared__ uint32_t empty_min;  // lowest non-hit index of the key kEmpty
  for (uint32_t i = threadIdx.x; i < kSmallSlots; i += kSmallThreads) slots[i] = 0;
  if (threadIdx.x == 0) empty_min = ~0u;
  __syncthreads();
  uint32_t pending = 0;  // bit j: key j is not held by the table
  uint64_t k[kSmallPerThread];
  uint4 home[kSmallPerThread];
  // all loads unconditional (keys at indices clamped to n - 1, n >= 1; slot 0 for a key
  // that is out of range or kEmpty), so that a thread's loads issue together: guarded,
  // they compiled to one round trip each
#pragma unroll
  for (int j = 0; j < kSmallPerThread; ++j) {
    const uint64_t g = threadIdx.x + (uint64_t)j * kSmallThreads;
    const uint64_t kg = keys[g < n ? g : n - 1];
    k[j] = g < n ? kg : kEmpty;
  }
#pragma unroll
  for (int j = 0; j < kSmallPerThread; ++j) {
    const uint64_t pos = k[j] != kEmpty ? slot_hash(k[j], t.shift) : 0;
    home[j] = *reinterpret_cast<const uint4*>(t.slots + 2 * pos);
  }
#pragma unroll
  for (int j = 0; j < kSmallPerThread; ++j) {
    const uint64_t g = threadIdx.x + (uint64_t)j * kSmallThreads;
    if (g >= n) continue;
    uint64_t val = 0;
    bool hit;
    if (k[j] != kEmpty && lo64(home[j]) == k[j]) {
      hit = true;
      val = hi64(home[j]);
    } else if (k[j] != kEmpty && lo64(home[j]) == kEmpty) {
      hit = false;
    } else {
      hit = table_find(t, k[j], &val);
    }
    if (hit) {
      status[g] = GLEAM_HIT_CACHE;
      if (ref) ref[g] = val;
      continue;
    }
    pending |= 1u << j;
    if (k[j] == kEmpty) {
      atomicMin(&empty_min, (uint32_t)g);
      continue;
    }
    uint32_t pos = (uint32_t)slot_hash(k[j], kSmallShift);
    for (uint32_t probe = 0; probe < kSmallSlots; ++probe) {
      const uint32_t prev = atomicCAS(&slots[pos], 0u, (uint32_t)g + 1);
      if (prev == 0) break;
      if (keys[prev - 1] == k[j]) {
        if (g + 1 < prev) atomicMin(&slots[pos], (uint32_t)g + 1);
        break;
      }
      pos = (pos + 1) & (kSmallSlots - 1);
    }
  }
  __syncthreads();
  for (uint32_t m = pending; m; m &= m - 1) {
    const int j = __builtin_ctz(m);
    const uint64_t g = threadIdx.x + (uint64_t)j * kSmallThreads;
    const uint64_t kg = keys[g];
    uint64_t g0 = g;
    if (kg == kEmpty) {
      g0 = empty_min;
    } else {
      uint32_t pos = (uint32_t)slot_hash(kg, kSmallShift);
      for (uint32_t probe = 0; probe < kSmallSlots; ++probe) {
        const uint32_t v = slots[pos];
        if (v == 0) break;
        if (v - 1 == g || keys[v - 1] == kg) {
          g0 = v - 1;
          break;
        }
        pos = (pos + 1) & (kSmallSlots - 1);
      }
    }
    status[g] = g0 == g ? GLEAM_MISS : GLEAM_HIT_BATCH;
    if (ref) ref[g] = g0;
  }
}

// Inserts of up to kSmallInsertKeys keys: one 1024-thread workgroup, the dedup table in
// LDS as in lookup_small_kernel, so one launch and no clear pass. The lowest index of
// each key inserts it; *n_new is written once at the end. GPU time on MI355X (this /
// the three launches): 256 keys 6.4 us, 1,024 keys 10.2 us, 2,048 keys 15.1 us, 4,096
// keys 38 us against about 20 us: past 2,048 keys one CU's chain of table
// compare-and-swaps costs more than the launches it saves.
constexpr uint64_t kSmallInsertKeys = 2048;
__global__ __launch_bounds__(kSmallThreads) void insert_small_kernel(TableRef t, const uint64_t* keys,
                                                                     const uint64_t* vals, uint64_t n,
                                                                     uint64_t* n_new) {
  __shared__ uint32_t slots[kSmallSlots];
  __shared__ uint32_t empty_min;  // lowest index of the key kEmpty
  __shared__ uint32_t wave_new[kSmallThreads / 64];
  for (uint32_t i = threadIdx.x; i < kSmallSlots; i += kSmallThreads) slots[i] = 0;
  if (threadIdx.x == 0) empty_min = ~0u;
  uint64_t k[kSmallPerThread];
#pragma unroll
  for (int j = 0; j < kSmallPerThread; ++j) {  // unconditional (clamped) loads, issued together
    const uint64_t g = threadIdx.x + (uint64_t)j * kSmallThreads;
    k[j] = keys[g < n ? g : n - 1];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kSmallPerThread; ++j) {
    const uint64_t g = threadIdx.x + (uint64_t)j * kSmallThreads;
    if (g >= n) continue;
    if (k[j] == kEmpty) {
      atomicMin(&empty_min, (uint32_t)g);
      continue;
    }
    uint32_t pos = (uint32_t)slot_hash(k[j], kSmallShift);
    for (uint32_t probe = 0; probe < kSmallSlots; ++probe) {
      const uint32_t prev = atomicCAS(&slots[pos], 0u, (uint32_t)g + 1);
      if (prev == 0) break;
      if (keys[prev - 1] == k[j]) {
        if (g + 1 < prev) atomicMin(&slots[pos], (uint32_t)g + 1);
        break;
      }
      pos = (pos + 1) & (kSmallSlots - 1);
    }
  }
  __syncthreads();
  uint32_t added = 0;
#pragma unroll
  for (int j = 0; j < kSmallPerThread; ++j) {
    const uint64_t g = threadIdx.x + (uint64_t)j * kSmallThreads;
    if (g >= n) continue;
    uint64_t g0 = g;
    if (k[j] == kEmpty) {
      g0 = empty_min;
    } else {
      uint32_t pos = (uint32_t)slot_hash(k[j], kSmallShift);
      for (uint32_t probe = 0; probe < kSmallSlots; ++probe) {
        const uint32_t v = slots[pos];
        if (v == 0) break;
        if (v - 1 == g || keys[v - 1] == k[j]) {
          g0 = v - 1;
          break;
        }
        pos = (pos + 1) & (kSmallSlots - 1);
      }
    }
    if (g0 != g) continue;  // a lower index carries this key
    if (k[j] == kEmpty) {
      if (atomicCAS(ull(&t.hdr[0]), 0ull, 1ull) == 0ull) {
        t.hdr[1] = vals[g];
        ++added;
      }
      continue;
    }
    uint64_t pos = slot_hash(k[j], t.shift);
    for (uint64_t probe = 0; probe <= t.mask; ++probe) {
      uint64_t* slot = t.slots + 2 * pos;
      const uint64_t prev = atomicCAS(ull(slot), (unsigned long long)kEmpty, (unsigned long long)k[j]);
      if (prev == kEmpty) {
        slot[1] = vals[g];
        ++added;
        break;
      }
      if (prev == k[j]) break;  // already held: keep the existing value
      pos = (pos + 1) & t.mask;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) added += __shfl_xor(added, o, 64);
  if ((threadIdx.x & 63) == 0) wave_new[threadIdx.x >> 6] = added;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t total = 0;
    for (int w = 0; w < kSmallThreads / 64; ++w) total += wave_new[w];
    if (n_new) *n_new = total;
    if (total) atomicAdd(ull(&t.hdr[3]), (unsigned long long)total);
  }
}

// Lookup pass 2: the earliest block with a digest is the MISS, later ones HIT_BATCH.
__global__ void lookup_resolve_kernel(ScratchRef sc, const uint64_t* keys, uint64_t n, uint8_t* status,
                                      uint64_t* ref) {
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n || status[g] != 0xFF) return;
  const uint64_t g0 = scratch_min(sc, keys, keys[g], g);
  status[g] = g0 == g ? GLEAM_MISS : GLEAM_HIT_BATCH;
  if (ref) ref[g] = g0;
}

ScratchRef scratch_ref(void* ws, const WsLayout& L) {
  ScratchRef s;
  s.hdr = reinterpret_cast<uint64_t*>(ws);
  s.slots = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(ws) + L.scratch_off);
  s.mask = L.scratch_cap - 1;
  s.shift = 64 - log2_exact(L.scratch_cap);
  return s;
}

// One launch resets the scratch table: every slot to kFree, header word 0 (min index of
// key kEmpty) to all-ones, words 1..3 and *also_zero to 0.
__global__ void scratch_clear_kernel(uint64_t* hdr, uint64_t* slots, uint64_t words, uint64_t* also_zero) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < 4) hdr[t] = t == 0 ? ~0ull : 0ull;
  if (t == 4 && also_zero) *also_zero = 0;
  // 16-byte stores (the slot count is a power of two of at least 64, the slots start
  // 256 bytes into a 256-byte aligned workspace)
  uint4* s4 = reinterpret_cast<uint4*>(slots);
  const uint4 ones = make_uint4(~0u, ~0u, ~0u, ~0u);
  for (uint64_t i = t; i < words / 2; i += stride) s4[i] = ones;
}

gleam_status clear_scratch(void* ws, const WsLayout& L, hipStream_t stream, uint64_t* also_zero = nullptr) {
  uint64_t* hdr = reinterpret_cast<uint64_t*>(ws);
  uint64_t* slots = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(ws) + L.scratch_off);
  const uint64_t words = L.scratch_cap;
  const uint64_t want = (words / 2 + kThreads - 1) / kThreads;
  const uint32_t grid = (uint32_t)(want < 2048 ? want : 2048);
  hipLaunchKernelGGL(scratch_clear_kernel, dim3(grid), dim3(kThreads), 0, stream, hdr, slots, words, also_zero);
  return launch_status("scratch_clear_kernel");
}

uint32_t blocks_for(uint64_t n) { return (uint32_t)((n + kThreads - 1) / kThreads); }

}  // namespace

gleam_status fill_u64(uint64_t* p, uint64_t n, uint64_t value, hipStream_t stream) {
  if (n == 0) return GLEAM_OK;
  const uint64_t want = (n + kThreads - 1) / kThreads;
  const uint32_t grid = (uint32_t)(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(fill_kernel, dim3(grid), dim3(kThreads), 0, stream, p, n, value);
  return launch_status("fill_kernel");
}

gleam_status clear_table(const gleam_cache* c, hipStream_t stream) {
  const TableRef t = table_ref(c);
  gleam_status st = fill_u64(t.hdr, kHeaderBytes / 8, 0, stream);
  if (st == GLEAM_OK) st = fill_u64(t.slots, 2 * c->capacity, kEmpty, stream);
  if (st == GLEAM_OK) st = fill_u64(t.stamps, c->capacity, 0, stream);
  return st;
}

}  // namespace gleam

extern "C" size_t gleam_cache_bytes(uint64_t capacity) {
  if (capacity < 16 || gleam::log2_exact(capacity) < 0 || capacity > (1ull << 40)) return 0;
  return gleam::kHeaderBytes + (size_t)capacity * 24;
}

extern "C" gleam_status gleam_cache_create(void* d_storage, size_t bytes, uint64_t capacity, double max_load,
                                           gleam_cache** out, void* stream) {
  using namespace gleam;
  clear_error();
  if (!out) {
    set_error("gleam_cache_create: null output handle");
    return GLEAM_E_INVALID;
  }
  *out = nullptr;
  const size_t need = gleam_cache_bytes(capacity);
  if (need == 0) {
    set_error("gleam_cache_create: capacity must be a power of two in [16, 2^40]");
    return GLEAM_E_INVALID;
  }
  if (!d_storage || !aligned256(d_storage) || bytes < need) {
    set_error("gleam_cache_create: storage must be non-null, 256-byte aligned and >= %zu bytes", need);
    return GLEAM_E_INVALID;
  }
  if (!(max_load > 0.0 && max_load < 1.0)) {
    set_error("gleam_cache_create: max_load must lie in (0, 1)");
    return GLEAM_E_INVALID;
  }
  uint64_t max_keys = (uint64_t)(max_load * (double)capacity);
  if (max_keys > capacity - 1) max_keys = capacity - 1;
  gleam_cache* c = new (std::nothrow) gleam_cache;
  if (!c) {
    set_error("gleam_cache_create: out of host memory");
    return GLEAM_E_INVALID;
  }
  c->storage = static_cast<uint8_t*>(d_storage);
  c->capacity = capacity;
  c->shift = 64 - log2_exact(capacity);
  c->max_keys = max_keys;
  c->key_bound = 0;
  gleam_status st = clear_table(c, (hipStream_t)stream);
  if (st != GLEAM_OK) {
    delete c;
    return st;
  }
  *out = c;
  return GLEAM_OK;
}

extern "C" gleam_status gleam_cache_destroy(gleam_cache* c) {
  delete c;
  return GLEAM_OK;
}

extern "C" uint64_t gleam_cache_key_bound(const gleam_cache* c) { return c ? c->key_bound : UINT64_MAX; }

extern "C" gleam_status gleam_cache_insert(gleam_cache* c, const uint64_t* d_keys, const uint64_t* d_vals, uint64_t n,
                                           uint64_t* d_n_new, void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  if (!c) {
    set_error("gleam_cache_insert: null table");
    return GLEAM_E_INVALID;
  }
  if (n > 0 && (!d_keys || !d_vals)) {
    set_error("gleam_cache_insert: null keys or values");
    return GLEAM_E_INVALID;
  }
  const WsLayout L = ws_layout(n);
  gleam_status st = check_workspace(L, d_ws, ws_bytes, "gleam_cache_insert");
  if (st != GLEAM_OK) return st;
  if (n > 0x7fffffffull * kThreads) {
    set_error("gleam_cache_insert: more than 2^31 workgroups of keys");
    return GLEAM_E_UNSUPPORTED;
  }
  if (n > c->max_keys || c->key_bound > c->max_keys - n) {
    set_error("gleam_cache_insert: %llu more keys could exceed the maximum load (%llu keys, bound %llu)",
              (unsigned long long)n, (unsigned long long)c->max_keys, (unsigned long long)c->key_bound);
    return GLEAM_E_CAPACITY;
  }
  hipStream_t s = (hipStream_t)stream;
  if (n > 0 && n <= kSmallInsertKeys) {
    hipLaunchKernelGGL(insert_small_kernel, dim3(1), dim3(kSmallThreads), 0, s, table_ref(c), d_keys, d_vals, n,
                       d_n_new);
    if ((st = launch_status("insert_small_kernel")) != GLEAM_OK) return st;
    c->key_bound += n;
    return GLEAM_OK;
  }
  st = clear_scratch(d_ws, L, s, d_n_new);
  uint64_t* counter = d_n_new ? d_n_new : reinterpret_cast<uint64_t*>(d_ws) + 1;
  if (st != GLEAM_OK) return st;
  if (n == 0) return GLEAM_OK;
  const ScratchRef sc = scratch_ref(d_ws, L);
  const TableRef t = table_ref(c);
  hipLaunchKernelGGL(insert_mark_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s, sc, d_keys, n);
  if ((st = launch_status("insert_mark_kernel")) != GLEAM_OK) return st;
  hipLaunchKernelGGL(insert_commit_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s, t, sc, d_keys, d_vals, n,
                     counter);
  if ((st = launch_status("insert_commit_kernel")) != GLEAM_OK) return st;
  c->key_bound += n;
  return GLEAM_OK;
}

extern "C" gleam_status gleam_cache_lookup(const gleam_cache* c, const uint64_t* d_keys, uint64_t n,
                                           uint8_t* d_status, uint64_t* d_ref, void* d_ws, size_t ws_bytes,
                                           void* stream) {
  using namespace gleam;
  clear_error();
  if (!c) {
    set_error("gleam_cache_lookup: null table");
    return GLEAM_E_INVALID;
  }
  if (n == 0) return GLEAM_OK;
  if (!d_keys || !d_status) {
    set_error("gleam_cache_lookup: null keys or status");
    return GLEAM_E_INVALID;
  }
  const WsLayout L = ws_layout(n);
  gleam_status st = check_workspace(L, d_ws, ws_bytes, "gleam_cache_lookup");
  if (st != GLEAM_OK) return st;
  if (n > 0x7fffffffull * kThreads) {
    set_error("gleam_cache_lookup: more than 2^31 workgroups of keys");
    return GLEAM_E_UNSUPPORTED;
  }
  hipStream_t s = (hipStream_t)stream;
  if (n <= kSmallKeys) {
    hipLaunchKernelGGL(lookup_small_kernel, dim3(1), dim3(kSmallThreads), 0, s, table_ref(c), d_keys, n, d_status,
                       d_ref);
    return launch_status("lookup_small_kernel");
  }
  st = clear_scratch(d_ws, L, s);
  if (st != GLEAM_OK) return st;
  const ScratchRef sc = scratch_ref(d_ws, L);
  const TableRef t = table_ref(c);
  hipLaunchKernelGGL(lookup_probe_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s, t, sc, d_keys, n, d_status, d_ref);
  if ((st = launch_status("lookup_probe_kernel")) != GLEAM_OK) return st;
  hipLaunchKernelGGL(lookup_resolve_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s, sc, d_keys, n, d_status,
                     d_ref);
  return launch_status("lookup_resolve_kernel");
}

// ---- Lookup without a caller workspace ----------------------------------------------
// For callers that cannot allocate device memory (code under HIP graph capture, tight
// serving loops, hosts that forbid allocation): the dedup scratch table lives in a
// file-scope device array instead of a workspace. Every call on a GPU shares that GPU's
// copy, so overlapping calls on one GPU race. The array's device address is looked up
// once per device with hipGetSymbolAddress; the host-side symbol is not a device address.
namespace gleam {
namespace {

constexpr uint64_t kNoAllocMaxKeys = 1ull << 20;
constexpr uint64_t kNoAllocSlots = 4 * kNoAllocMaxKeys;  // the workspace layout's cap for that n
constexpr size_t kNoAllocBytes = kHeaderBytes + kNoAllocSlots * 8;  // 32 MiB + 256 B

static __device__ __align__(256) uint8_t scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of this device's scratch array (looked up on the first call).
gleam_status noalloc_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    set_error("hipGetDevice: %s", hipGetErrorString(e));
    return GLEAM_E_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    set_error("gleam_cache_lookup_noalloc: device %d beyond the %d this library tracks", dev, kMaxDevices);
    return GLEAM_E_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_error("hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      return GLEAM_E_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GLEAM_OK;
}

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_cache() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&fill_kernel));
}

}  // namespace gleam

extern "C" size_t gleam_cache_lookup_noalloc_max_keys(void) { return (size_t)gleam::kNoAllocMaxKeys; }

extern "C" gleam_status gleam_cache_lookup_noalloc(const gleam_cache* c, const uint64_t* d_keys, uint64_t n,
                                                   uint8_t* d_status, uint64_t* d_ref, void* stream) {
  using namespace gleam;
  clear_error();
  if (!c) {
    set_error("gleam_cache_lookup_noalloc: null table");
    return GLEAM_E_INVALID;
  }
  if (n == 0) return GLEAM_OK;
  if (!d_keys || !d_status) {
    set_error("gleam_cache_lookup_noalloc: null keys or status");
    return GLEAM_E_INVALID;
  }
  if (n > kNoAllocMaxKeys) {
    set_error("gleam_cache_lookup_noalloc: %llu keys, at most %llu without a workspace (use gleam_cache_lookup)",
              (unsigned long long)n, (unsigned long long)kNoAllocMaxKeys);
    return GLEAM_E_UNSUPPORTED;
  }
  hipStream_t s = (hipStream_t)stream;
  if (n <= kSmallKeys) {  // the one-workgroup path dedups in LDS: no scratch at all
    hipLaunchKernelGGL(lookup_small_kernel, dim3(1), dim3(kSmallThreads), 0, s, table_ref(c), d_keys, n, d_status,
                       d_ref);
    return launch_status("lookup_small_kernel");
  }
  void* ws = nullptr;
  gleam_status st = noalloc_scratch(&ws);
  if (st != GLEAM_OK) return st;
  const WsLayout L = ws_layout(n);  // scratch_cap <= kNoAllocSlots for n <= kNoAllocMaxKeys
  st = clear_scratch(ws, L, s);
  if (st != GLEAM_OK) return st;
  const ScratchRef sc = scratch_ref(ws, L);
  const TableRef t = table_ref(c);
  hipLaunchKernelGGL(lookup_probe_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s, t, sc, d_keys, n, d_status, d_ref);
  if ((st = launch_status("lookup_probe_kernel")) != GLEAM_OK) return st;
  hipLaunchKernelGGL(lookup_resolve_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s, sc, d_keys, n, d_status,
                     d_ref);
  return launch_status("lookup_resolve_kernel");
}
