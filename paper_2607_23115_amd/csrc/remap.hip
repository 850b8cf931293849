// Address-remap interval map (Gleam Sec. 4.3: chunks written into one client allocation
// may find their shareable copies in different server allocations, so a virtual memory
// layer maps client device addresses onto those positions; Sec. 6: one 1 TB virtual
// space per task, the mappings kept in a red-black tree).
//
// The map is an array of disjoint intervals sorted by start, in caller-owned device
// storage: [256-byte header: u64 count, fence stride, fence length][start x cap]
// [{end, target} x cap][fence: 4096 x u64], end exclusive. A sorted array answers the
// same ordered queries as the tree; on the GPU a batch of pointers is translated by
// one search per lane, and a batch of changes rebuilds the array in a few passes
// instead of rebalancing node by node.
//
// Translation is bound by dependent, lane-divergent loads (each level of a binary
// search is a different cache line for every lane), not by bytes. So every update also
// writes a fence, every S-th start with S = ceil(count / 4096); a translating workgroup
// keeps the fence in LDS and searches it first, leaving log2(S) levels for global
// memory (6 instead of 18 at 208k intervals), and end and target sit side by side so
// the final step is one 16-byte load. The update:
//
//   1. removal ranges are sorted by start, with a running maximum of their last
//      addresses, so one binary search tells whether an interval meets any of them;
//   2. survivors and valid additions are sorted together by start (rocPRIM radix sort;
//      everything else takes the key kNone and sorts last);
//   3. a running maximum of interval ends: an addition meets an earlier-starting entry
//      iff that maximum, just before it, passes its start, and a later-starting one iff
//      the next start falls before its end;
//   4. an exclusive scan of the kept entries gives their new positions; the scatter
//      writes them only if they fit the capacity, so a refused call changes nothing.

#include <new>

#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/device/device_scan.hpp>

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;
constexpr int kTranslateThreads = 1024;
constexpr uint32_t kMaxGrid = 8192;
constexpr uint64_t kNone = ~0ull;  // sort key of an entry that takes no part; no valid start equals it
constexpr uint64_t kMaxCount = 1ull << 31;

constexpr uint32_t kFence = 4096;  // fence entries (32 KiB of LDS)

struct MapRef {
  uint64_t* hdr;   // [0] number of intervals, [1] fence stride S, [2] fence length
  uint64_t* start;
  ulonglong2* et;  // {end, target} per interval
  uint64_t* fence; // start[k * S] for k < fence length
  uint64_t cap;
};

MapRef map_ref(const gleam_remap* m) {
  uint64_t* hdr = reinterpret_cast<uint64_t*>(m->storage);
  uint64_t* start = reinterpret_cast<uint64_t*>(m->storage + kHeaderBytes);
  ulonglong2* et = reinterpret_cast<ulonglong2*>(start + m->capacity);
  return MapRef{hdr, start, et, reinterpret_cast<uint64_t*>(et + m->capacity), m->capacity};
}

struct UpdLayout {
  uint64_t m;  // capacity + n_add candidates
  uint64_t r;  // removal ranges
  size_t counters, ckey_a, ckey_b, cval_a, cval_b, cend, cmax, ctgt, acc, pos;
  size_t dkey_a, dkey_b, dval_a, dval_b, dmax, tmp, tmp_bytes, total;
  bool ok;  // rocPRIM's storage queries succeeded
};

UpdLayout upd_layout(uint64_t cap, uint64_t n_add, uint64_t n_del) {
  UpdLayout L;
  L.m = cap + n_add;
  L.r = n_del;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = (off + bytes + 255) & ~(size_t)255;
    return o;
  };
  L.counters = take(256);
  L.ckey_a = take(8 * L.m);
  L.ckey_b = take(8 * L.m);
  L.cval_a = take(8 * L.m);
  L.cval_b = take(8 * L.m);
  L.cend = take(8 * L.m);
  L.cmax = take(8 * L.m);
  L.ctgt = take(8 * L.m);
  L.acc = take(8 * L.m);
  L.pos = take(8 * L.m);
  L.dkey_a = take(8 * L.r);
  L.dkey_b = take(8 * L.r);
  L.dval_a = take(8 * L.r);
  L.dval_b = take(8 * L.r);
  L.dmax = take(8 * L.r);
  const uint64_t big = L.m > L.r ? L.m : L.r;
  size_t sort_b = 0, max_b = 0, sum_b = 0;
  const hipError_t e1 = rocprim::radix_sort_pairs(nullptr, sort_b, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                                  (const uint64_t*)nullptr, (uint64_t*)nullptr, (size_t)big, 0, 64);
  const hipError_t e2 = rocprim::inclusive_scan(nullptr, max_b, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                                (size_t)big, rocprim::maximum<uint64_t>());
  const hipError_t e3 = rocprim::exclusive_scan(nullptr, sum_b, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                                (uint64_t)0, (size_t)L.m, rocprim::plus<uint64_t>());
  L.ok = e1 == hipSuccess && e2 == hipSuccess && e3 == hipSuccess;
  L.tmp_bytes = sort_b;
  if (max_b > L.tmp_bytes) L.tmp_bytes = max_b;
  if (sum_b > L.tmp_bytes) L.tmp_bytes = sum_b;
  L.tmp = take(L.tmp_bytes);
  L.total = off;
  return L;
}

uint32_t grid_for(uint64_t n) {
  const uint64_t g = (n + kThreads - 1) / kThreads;
  return (uint32_t)(g == 0 ? 1 : (g < kMaxGrid ? g : kMaxGrid));
}

__device__ __forceinline__ unsigned long long* ull(uint64_t* p) { return reinterpret_cast<unsigned long long*>(p); }

__device__ __forceinline__ void wave_add(uint64_t* counter, uint64_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += shfl_xor64(x, o);
  if ((threadIdx.x & 63) == 0 && x) atomicAdd(ull(counter), (unsigned long long)x);
}

// Number of entries of the ascending keys[0, n) that are <= x.
__device__ __forceinline__ uint64_t count_le(const uint64_t* keys, uint64_t n, uint64_t x) {
  uint64_t lo = 0, hi = n;
  while (lo < hi) {
    const uint64_t mid = lo + ((hi - lo) >> 1);
    if (keys[mid] <= x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Removal ranges as sort key = first address, value = last address (clipped at 2^64 - 1);
// an empty range takes the key kNone and is never found.
__global__ void removal_prep_kernel(const uint64_t* d_start, const uint64_t* d_len, uint64_t r, uint64_t* key,
                                    uint64_t* last) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < r; k += stride) {
    const uint64_t s = d_start[k], n = d_len[k];
    key[k] = n ? s : kNone;
    last[k] = n ? (n - 1 > kNone - s ? kNone : s + n - 1) : 0;
  }
}

// Candidates: slot p < cap is interval p (if it exists and survives the removals),
// p >= cap is addition p - cap (if valid). Key = start or kNone, value = p.
__global__ void candidates_kernel(MapRef map, const uint64_t* rkey, const uint64_t* rmax, uint64_t r,
                                  const uint64_t* a_start, const uint64_t* a_len, const uint64_t* a_target,
                                  uint64_t m, uint8_t* status, uint64_t* ckey, uint64_t* cval, uint64_t* counters) {
  const uint64_t count = map.hdr[0];
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  // every lane of a wave runs the same number of iterations, so wave_add sees them all
  const uint64_t base0 = (uint64_t)blockIdx.x * blockDim.x;
  for (uint64_t base = base0; base < m; base += stride) {
    const uint64_t p = base + threadIdx.x;
    uint64_t removed = 0;
    if (p < m) {
      uint64_t key = kNone;
      if (p < map.cap) {
        if (p < count) {
          const uint64_t s = map.start[p], last = map.et[p].x - 1;
          // the removals starting at or before `last`: does the furthest of them reach s?
          const uint64_t q = r ? count_le(rkey, r, last) : 0;
          if (q && rmax[q - 1] >= s) removed = 1;
          else key = s;
        }
      } else {
        const uint64_t j = p - map.cap;
        const uint64_t s = a_start[j], n = a_len[j], t = a_target[j];
        if (n != 0 && n <= kNone - s && n <= kNone - t) key = s;
        else if (status) status[j] = GLEAM_REMAP_INVALID;
      }
      ckey[p] = key;
      cval[p] = p;
    }
    wave_add(&counters[0], removed);
  }
}

// End and target of each sorted candidate; a non-candidate ends at 0, so the running
// maximum of ends is the furthest end of the real entries before it.
__global__ void gather_kernel(MapRef map, const uint64_t* a_len, const uint64_t* a_target, const uint64_t* ckey,
                              const uint64_t* cval, uint64_t m, uint64_t* cend, uint64_t* ctgt) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p < m; p += stride) {
    const uint64_t key = ckey[p];
    uint64_t e = 0, t = 0;
    if (key != kNone) {
      const uint64_t v = cval[p];
      if (v < map.cap) {
        const ulonglong2 et = map.et[v];
        e = et.x;
        t = et.y;
      } else {
        e = key + a_len[v - map.cap];
        t = a_target[v - map.cap];
      }
    }
    cend[p] = e;
    ctgt[p] = t;
  }
}

// Keep every survivor; keep an addition unless it meets an entry that starts before it
// (the running maximum of earlier ends passes its start) or at/after it (the next
// start comes before its end).
__global__ void classify_kernel(const uint64_t* ckey, const uint64_t* cval, const uint64_t* cend,
                                const uint64_t* cmax, uint64_t cap, uint64_t m, uint8_t* status, uint64_t* acc) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p < m; p += stride) {
    const uint64_t key = ckey[p];
    uint64_t keep = 0;
    if (key != kNone) {
      const uint64_t v = cval[p];
      if (v < cap) {
        keep = 1;
      } else {
        const bool clash = (p > 0 && cmax[p - 1] > key) || (p + 1 < m && ckey[p + 1] < cend[p]);
        keep = clash ? 0 : 1;
        if (status) status[v - cap] = clash ? GLEAM_REMAP_OVERLAP : GLEAM_REMAP_ADDED;
      }
    }
    acc[p] = keep;
  }
}

// Write the kept entries at their scanned positions, and every S-th start into the
// fence, if they all fit; otherwise leave the map as it was and mark the additions that
// would have entered FULL.
__global__ void scatter_kernel(MapRef map, const uint64_t* ckey, const uint64_t* cval, const uint64_t* cend,
                               const uint64_t* ctgt, const uint64_t* acc, const uint64_t* pos, uint64_t m,
                               uint64_t n_add, uint8_t* status, const uint64_t* counters, uint64_t* counts) {
  const uint64_t total = pos[m - 1] + acc[m - 1];
  const bool fits = total <= map.cap;
  const uint64_t S = total > kFence ? (total + kFence - 1) / kFence : 1;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t first = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (first == 0) {
    // kept = the survivors (before - removed) and the accepted additions
    const uint64_t before = map.hdr[0];
    const uint64_t added = fits ? total - (before - counters[0]) : 0;
    counts[0] = fits ? total : before;
    counts[1] = added;
    counts[2] = fits ? counters[0] : 0;
    counts[3] = n_add - added;
    if (fits) {
      map.hdr[0] = total;
      map.hdr[1] = S;
      map.hdr[2] = (total + S - 1) / S;
    }
  }
  for (uint64_t p = first; p < m; p += stride) {
    if (!acc[p]) continue;
    if (fits) {
      const uint64_t q = pos[p];
      map.start[q] = ckey[p];
      map.et[q] = make_ulonglong2(cend[p], ctgt[p]);
      if (q % S == 0) map.fence[q / S] = ckey[p];
    } else if (status && cval[p] >= map.cap) {
      status[cval[p] - map.cap] = GLEAM_REMAP_FULL;
    }
  }
}

// Translation. The interval that can hold address a is the last one starting at or
// before a. The fence (in LDS) narrows it to one run of S starts: if f fence entries
// are <= a, the answer lies in [(f - 1) S, f S), whose first start is known <= a. Both
// searches count the entries <= a by binary lifting, a fixed number of halving steps
// that the lanes of a wave take together. Each global step is a different cache line
// for nearly every lane, so the kernel is bound by the L2's request rate, not by bytes
// or by latency (carrying several addresses per lane measured no faster).
__device__ __forceinline__ uint32_t top_bit(uint32_t x) {  // largest power of two <= x (x >= 1)
  return 1u << (31 - __builtin_clz(x));
}

__global__ void __launch_bounds__(kTranslateThreads)
translate_kernel(MapRef map, const uint64_t* addr, uint64_t n, uint64_t* out) {
  __shared__ uint64_t fence[kFence];
  // count <= 2^31 intervals, so every index and run length fits in 32 bits
  const uint32_t count = (uint32_t)map.hdr[0], S = (uint32_t)map.hdr[1], F = (uint32_t)map.hdr[2];
  for (uint32_t k = threadIdx.x; k < F; k += blockDim.x) fence[k] = map.fence[k];
  __syncthreads();
  const uint32_t f_top = F ? top_bit(F) : 0, s_top = S > 1 ? top_bit(S - 1) : 0;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t a = addr[i];
    uint32_t f = 0;
    for (uint32_t step = f_top; step; step >>= 1)
      if (f + step <= F && fence[f + step - 1] <= a) f += step;
    uint64_t r = GLEAM_UNMAPPED;
    if (f) {
      // the starts in (lo, hi) that are <= a
      const uint32_t lo = (f - 1) * S;
      const uint32_t len = (count - lo > S ? S : count - lo) - 1;
      uint32_t c = 0;
      for (uint32_t step = s_top; step; step >>= 1)
        if (c + step <= len && map.start[lo + c + step] <= a) c += step;
      const uint64_t st = c ? map.start[lo + c] : fence[f - 1];
      const ulonglong2 et = map.et[lo + c];
      if (a < et.x) r = et.y + (a - st);
    }
    out[i] = r;
  }
}

__global__ void export_kernel(MapRef map, uint64_t* d_start, uint64_t* d_len, uint64_t* d_target,
                              uint64_t* d_count) {
  const uint64_t count = map.hdr[0];
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t first = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (first == 0) d_count[0] = count;
  for (uint64_t p = first; p < count; p += stride) {
    const uint64_t s = map.start[p];
    const ulonglong2 et = map.et[p];
    d_start[p] = s;
    d_len[p] = et.x - s;
    d_target[p] = et.y;
  }
}

gleam_status hip_call(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    set_error("%s: %s", what, hipGetErrorString(e));
    return GLEAM_E_HIP;
  }
  return launch_status(what);
}

}  // namespace
}  // namespace gleam

extern "C" size_t gleam_remap_bytes(uint64_t capacity) {
  if (capacity == 0 || capacity > gleam::kMaxCount) return 0;
  return gleam::kHeaderBytes + 24 * (size_t)capacity + 8 * (size_t)gleam::kFence;
}

extern "C" gleam_status gleam_remap_create(void* d_storage, size_t bytes, uint64_t capacity, gleam_remap** out,
                                           void* stream) {
  using namespace gleam;
  clear_error();
  if (!out) {
    set_error("gleam_remap_create: null output handle");
    return GLEAM_E_INVALID;
  }
  *out = nullptr;
  const size_t need = gleam_remap_bytes(capacity);
  if (need == 0) {
    set_error("gleam_remap_create: capacity must be in [1, 2^31]");
    return GLEAM_E_INVALID;
  }
  if (!d_storage || !aligned256(d_storage)) {
    set_error("gleam_remap_create: storage must be non-null and 256-byte aligned");
    return GLEAM_E_INVALID;
  }
  if (bytes < need) {
    set_error("gleam_remap_create: storage of %zu bytes, %zu needed", bytes, need);
    return GLEAM_E_INVALID;
  }
  gleam_remap* m = new (std::nothrow) gleam_remap;
  if (!m) {
    set_error("gleam_remap_create: out of host memory");
    return GLEAM_E_INVALID;
  }
  m->storage = static_cast<uint8_t*>(d_storage);
  m->capacity = capacity;
  const gleam_status st = fill_u64(reinterpret_cast<uint64_t*>(m->storage), kHeaderBytes / 8, 0,
                                   (hipStream_t)stream);
  if (st != GLEAM_OK) {
    delete m;
    return st;
  }
  *out = m;
  return GLEAM_OK;
}

extern "C" gleam_status gleam_remap_destroy(gleam_remap* m) {
  delete m;
  return GLEAM_OK;
}

extern "C" size_t gleam_remap_update_bytes(const gleam_remap* m, uint64_t n_add, uint64_t n_del) {
  if (!m || n_add > gleam::kMaxCount || n_del > gleam::kMaxCount) return 0;
  const gleam::UpdLayout L = gleam::upd_layout(m->capacity, n_add, n_del);
  return L.ok ? L.total : 0;
}

extern "C" gleam_status gleam_remap_update(gleam_remap* m, const uint64_t* d_del_start, const uint64_t* d_del_len,
                                           uint64_t n_del, const uint64_t* d_add_start, const uint64_t* d_add_len,
                                           const uint64_t* d_add_target, uint64_t n_add, uint8_t* d_add_status,
                                           uint64_t* d_counts, void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  if (!m || !d_counts) {
    set_error("gleam_remap_update: null map or counts");
    return GLEAM_E_INVALID;
  }
  if ((n_del > 0 && (!d_del_start || !d_del_len)) || (n_add > 0 && (!d_add_start || !d_add_len || !d_add_target))) {
    set_error("gleam_remap_update: null removal or addition array");
    return GLEAM_E_INVALID;
  }
  if (n_add > kMaxCount || n_del > kMaxCount) {
    set_error("gleam_remap_update: more than 2^31 additions or removals");
    return GLEAM_E_UNSUPPORTED;
  }
  const UpdLayout L = upd_layout(m->capacity, n_add, n_del);
  if (!L.ok) {
    set_error("gleam_remap_update: rocPRIM storage query failed");
    return GLEAM_E_HIP;
  }
  if (!d_ws || !aligned256(d_ws)) {
    set_error("gleam_remap_update: workspace must be non-null and 256-byte aligned");
    return GLEAM_E_INVALID;
  }
  if (ws_bytes < L.total) {
    set_error("gleam_remap_update: workspace of %zu bytes, %zu needed", ws_bytes, L.total);
    return GLEAM_E_WORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  uint8_t* b = static_cast<uint8_t*>(d_ws);
  auto at = [&](size_t off) { return reinterpret_cast<uint64_t*>(b + off); };
  uint64_t* counters = at(L.counters);
  void* tmp = b + L.tmp;
  size_t tmp_bytes = L.tmp_bytes;
  const MapRef map = map_ref(m);
  gleam_status st = fill_u64(counters, 4, 0, s);
  if (st != GLEAM_OK) return st;

  const uint64_t* rkey = nullptr;
  const uint64_t* rmax = nullptr;
  if (n_del > 0) {
    hipLaunchKernelGGL(removal_prep_kernel, dim3(grid_for(n_del)), dim3(kThreads), 0, s, d_del_start, d_del_len,
                       n_del, at(L.dkey_a), at(L.dval_a));
    if ((st = launch_status("removal_prep_kernel")) != GLEAM_OK) return st;
    st = hip_call(rocprim::radix_sort_pairs(tmp, tmp_bytes, at(L.dkey_a), at(L.dkey_b), at(L.dval_a), at(L.dval_b),
                                            (size_t)n_del, 0, 64, s),
                  "radix sort (removals)");
    if (st != GLEAM_OK) return st;
    tmp_bytes = L.tmp_bytes;
    st = hip_call(rocprim::inclusive_scan(tmp, tmp_bytes, at(L.dval_b), at(L.dmax), (size_t)n_del,
                                          rocprim::maximum<uint64_t>(), s),
                  "running maximum (removals)");
    if (st != GLEAM_OK) return st;
    rkey = at(L.dkey_b);
    rmax = at(L.dmax);
  }
  const dim3 grid(grid_for(L.m)), block(kThreads);
  hipLaunchKernelGGL(candidates_kernel, grid, block, 0, s, map, rkey, rmax, n_del, d_add_start, d_add_len,
                     d_add_target, L.m, d_add_status, at(L.ckey_a), at(L.cval_a), counters);
  if ((st = launch_status("candidates_kernel")) != GLEAM_OK) return st;
  tmp_bytes = L.tmp_bytes;
  st = hip_call(rocprim::radix_sort_pairs(tmp, tmp_bytes, at(L.ckey_a), at(L.ckey_b), at(L.cval_a), at(L.cval_b),
                                          (size_t)L.m, 0, 64, s),
                "radix sort (candidates)");
  if (st != GLEAM_OK) return st;
  hipLaunchKernelGGL(gather_kernel, grid, block, 0, s, map, d_add_len, d_add_target, at(L.ckey_b), at(L.cval_b),
                     L.m, at(L.cend), at(L.ctgt));
  if ((st = launch_status("gather_kernel")) != GLEAM_OK) return st;
  tmp_bytes = L.tmp_bytes;
  st = hip_call(rocprim::inclusive_scan(tmp, tmp_bytes, at(L.cend), at(L.cmax), (size_t)L.m,
                                        rocprim::maximum<uint64_t>(), s),
                "running maximum (ends)");
  if (st != GLEAM_OK) return st;
  hipLaunchKernelGGL(classify_kernel, grid, block, 0, s, at(L.ckey_b), at(L.cval_b), at(L.cend), at(L.cmax),
                     m->capacity, L.m, d_add_status, at(L.acc));
  if ((st = launch_status("classify_kernel")) != GLEAM_OK) return st;
  tmp_bytes = L.tmp_bytes;
  st = hip_call(rocprim::exclusive_scan(tmp, tmp_bytes, at(L.acc), at(L.pos), (uint64_t)0, (size_t)L.m,
                                        rocprim::plus<uint64_t>(), s),
                "scan (positions)");
  if (st != GLEAM_OK) return st;
  hipLaunchKernelGGL(scatter_kernel, grid, block, 0, s, map, at(L.ckey_b), at(L.cval_b), at(L.cend), at(L.ctgt),
                     at(L.acc), at(L.pos), L.m, n_add, d_add_status, counters, d_counts);
  return launch_status("scatter_kernel");
}

extern "C" gleam_status gleam_remap_translate(const gleam_remap* m, const uint64_t* d_addr, uint64_t n,
                                              uint64_t* d_out, void* stream) {
  using namespace gleam;
  clear_error();
  if (!m || (n > 0 && (!d_addr || !d_out))) {
    set_error("gleam_remap_translate: null map, addresses or output");
    return GLEAM_E_INVALID;
  }
  if (n == 0) return GLEAM_OK;
  int cus = 0;
  const gleam_status st = device_cu_count(&cus);
  if (st != GLEAM_OK) return st;
  // two 1024-lane workgroups per CU fill it (32 waves); each loads the fence once
  const uint64_t want = (n + kTranslateThreads - 1) / kTranslateThreads;
  const uint64_t grid = want < 2ull * cus ? want : 2ull * cus;
  hipLaunchKernelGGL(translate_kernel, dim3((uint32_t)grid), dim3(kTranslateThreads), 0, (hipStream_t)stream,
                     map_ref(m), d_addr, n, d_out);
  return launch_status("translate_kernel");
}

extern "C" gleam_status gleam_remap_export(const gleam_remap* m, uint64_t* d_start, uint64_t* d_len,
                                           uint64_t* d_target, uint64_t* d_count, void* stream) {
  using namespace gleam;
  clear_error();
  if (!m || !d_start || !d_len || !d_target || !d_count) {
    set_error("gleam_remap_export: null map or output");
    return GLEAM_E_INVALID;
  }
  hipLaunchKernelGGL(export_kernel, dim3(grid_for(m->capacity)), dim3(kThreads), 0, (hipStream_t)stream, map_ref(m),
                     d_start, d_len, d_target, d_count);
  return launch_status("export_kernel");
}
