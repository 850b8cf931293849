// Address-remap interval map (Gleam Sec. 4.1.3, Weight Chunk Sharing: chunks written into
// one client allocation may find their shareable copies in different server allocations,
// so a virtual memory layer maps client device addresses onto those positions; Appendix,
// Implementation Details, Virtual Memory Map: one 1 TB virtual space per task, the
// mappings kept in a red-black tree).
//
// The map is an array of disjoint intervals sorted by start, in caller-owned device
// storage: [256-byte header: u64 count, fence stride, fence length][start x cap]
// [{end, bias} x cap][fence: kFence x u64], end exclusive, bias = target - start (mod
// 2^64, so a translation is one add: p + bias). A sorted array answers the
// same ordered queries as the tree; on the GPU a batch of pointers is translated by
// one search per lane, and a batch of changes is merged in a few passes instead of
// rebalancing node by node.
//
// Translation is bound by lane-divergent loads (each level of a binary search is a
// different cache line for nearly every lane), not by bytes. So every update also
// writes a fence, every S-th start with S = ceil(count / 8192); a translating workgroup
// keeps the fence in LDS and searches it first, leaving log2(S) levels for global
// memory (5 instead of 18 at 208k intervals), and end and bias sit side by side so the
// final step is one 16-byte load and needs no start.
//
// An update never re-sorts the intervals it keeps (they are already in order):
//   1. removal ranges are sorted by start, with a running maximum of their last
//      addresses, so one binary search tells whether an interval meets any of them;
//      the survivors are compacted, in order, into the workspace (one scan);
//   2. only the valid additions are sorted (the library's radix sort, radix_sort.h;
//      invalid ones take the key kNone and sort last);
//   3. an addition meets an earlier-starting addition iff the running maximum of ends
//      just before it passes its start, a later-starting one iff the next start comes
//      before its end, and a survivor iff the last survivor starting at or before its
//      last address ends after its start (survivors are disjoint, so their ends are
//      sorted too); additions that meet nothing are kept (a scan numbers them);
//   4. the two sorted runs are merged by rank: a survivor lands at its own index plus
//      the kept additions that start before it, a kept addition at its own number plus
//      the survivors that start before it. Nothing is written unless everything fits
//      the capacity, so a refused call changes nothing.

#include <new>

#include "device_scan.h"
#include "gleam_device.h"
#include "gleam_internal.h"
#include "radix_sort.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;
constexpr int kTranslateThreads = 1024;
constexpr uint32_t kMaxGrid = 8192;
constexpr uint64_t kNone = ~0ull;  // sort key of an addition that takes no part; no valid start equals it
constexpr uint64_t kMaxCount = 1ull << 31;

constexpr uint32_t kFence = 8192;  // fence entries (64 KiB of LDS: two translating workgroups per CU)

struct MapRef {
  uint64_t* hdr;   // [0] number of intervals, [1] fence stride S, [2] fence length
  uint64_t* start;
  ulonglong2* et;  // {end, target - start} per interval
  uint64_t* fence; // start[k * S] for k < fence length
  uint64_t cap;
};

MapRef map_ref(const gleam_remap* m) {
  uint64_t* hdr = reinterpret_cast<uint64_t*>(m->storage);
  uint64_t* start = reinterpret_cast<uint64_t*>(m->storage + kHeaderBytes);
  ulonglong2* et = reinterpret_cast<ulonglong2*>(start + m->capacity);
  return MapRef{hdr, start, et, reinterpret_cast<uint64_t*>(et + m->capacity), m->capacity};
}

// Workspace of one update (cap = capacity, A = additions, R = removal ranges).
struct UpdLayout {
  size_t hdr;                                // [0] R, [1] A (the sorts' counts); [4..7] R's key bits, [8..11] A's
  size_t keep, kpos, s_start, s_et;         // cap: survivor flag, its scan, compacted survivors
  size_t ka, aidx, kb, vb, aend, amax, acc, apos;  // A: sort keys/indices, sorted keys/indices, ends, running max, kept flag, scan
  size_t rka, ridx, rkb, rvb, rmax;         // R: sort keys/indices, sorted starts, their last addresses, running max
  size_t sort, partial, total;              // the sort's second buffer and counts; the scans' tile totals
};

UpdLayout upd_layout(uint64_t cap, uint64_t n_add, uint64_t n_del) {
  UpdLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = (off + bytes + 255) & ~(size_t)255;
    return o;
  };
  L.hdr = take(256);
  L.keep = take(8 * cap);
  L.kpos = take(8 * cap);
  L.s_start = take(8 * cap);
  L.s_et = take(16 * cap);
  L.ka = take(8 * sort_capacity(n_add));
  L.aidx = take(4 * sort_capacity(n_add));
  L.kb = take(8 * n_add);
  L.vb = take(8 * n_add);
  L.aend = take(8 * n_add);
  L.amax = take(8 * n_add);
  L.acc = take(8 * n_add);
  L.apos = take(8 * n_add);
  L.rka = take(8 * sort_capacity(n_del));
  L.ridx = take(4 * sort_capacity(n_del));
  L.rkb = take(8 * n_del);
  L.rvb = take(8 * n_del);
  L.rmax = take(8 * n_del);
  const uint64_t ar = n_add > n_del ? n_add : n_del;
  const uint64_t most = cap > ar ? cap : ar;
  L.sort = take(sort_layout(ar, 1).total);
  L.partial = take(8 * scan_tiles(most));
  L.total = off;
  return L;
}

uint32_t grid_for(uint64_t n) {
  const uint64_t g = (n + kThreads - 1) / kThreads;
  return (uint32_t)(g == 0 ? 1 : (g < kMaxGrid ? g : kMaxGrid));
}

// Grid of a kernel that folds key bits with one pair of atomics per workgroup: few
// enough workgroups that those atomics on two words do not queue behind each other.
uint32_t fold_grid(uint64_t n) {
  const uint32_t g = grid_for(n);
  return g < 256 ? g : 256;
}

// Number of entries of the ascending keys[0, n) that are <= x (upper bound).
__device__ __forceinline__ uint64_t count_le(const uint64_t* keys, uint64_t n, uint64_t x) {
  uint64_t lo = 0, hi = n;
  while (lo < hi) {
    const uint64_t mid = lo + ((hi - lo) >> 1);
    if (keys[mid] <= x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Number of entries of the ascending keys[0, n) that are < x (lower bound).
__device__ __forceinline__ uint64_t count_lt(const uint64_t* keys, uint64_t n, uint64_t x) {
  uint64_t lo = 0, hi = n;
  while (lo < hi) {
    const uint64_t mid = lo + ((hi - lo) >> 1);
    if (keys[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Removal ranges as sort key = first address, value = last address (clipped at 2^64 - 1);
// an empty range takes the key kNone and is never found.
// Counts of the two sorts and the AND/OR words of their keys (see radix_sort.h).
__global__ void update_init_kernel(uint64_t* hdr, uint64_t r, uint64_t n_add) {
  const int t = threadIdx.x;
  if (t < 12) hdr[t] = t == 0 ? r : t == 1 ? n_add : (t == 4 || t == 8) ? ~0ull : 0ull;
}

// Fold a thread's AND/OR of keys into bits[0] (AND) and bits[1] (OR): one pair of
// atomics per workgroup. Every thread of the workgroup calls it.
__device__ void fold_key_bits(uint64_t and_k, uint64_t or_k, uint64_t* bits) {
  __shared__ uint64_t fold[kThreads / 64][2];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    and_k &= shfl_xor64(and_k, o);
    or_k |= shfl_xor64(or_k, o);
  }
  if (lane == 0) {
    fold[wave][0] = and_k;
    fold[wave][1] = or_k;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kThreads / 64; ++w) {
      and_k &= fold[w][0];
      or_k |= fold[w][1];
    }
    atomicAnd(reinterpret_cast<unsigned long long*>(&bits[0]), (unsigned long long)and_k);
    atomicOr(reinterpret_cast<unsigned long long*>(&bits[1]), (unsigned long long)or_k);
  }
}

// Sort key of removal k: its start, or kNone for an empty range (it sorts last).
__global__ __launch_bounds__(kThreads) void removal_prep_kernel(const uint64_t* d_start, const uint64_t* d_len,
                                                                uint64_t r, uint64_t* key, uint32_t* idx,
                                                                uint64_t* bits) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint64_t and_k = ~0ull, or_k = 0;
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < r; k += stride) {
    const uint64_t s = d_len[k] ? d_start[k] : kNone;
    key[k] = s;
    idx[k] = (uint32_t)k;
    and_k &= s;
    or_k |= s;
  }
  fold_key_bits(and_k, or_k, bits);
}

// Sorted removals: start, and last address (the running maximum of these tells whether
// any removal starting at or before an address reaches it).
__global__ void removal_unpack_kernel(SortBuf a, SortBuf b, const uint64_t* bits, const uint64_t* d_start,
                                      const uint64_t* d_len, uint64_t r, uint64_t* key, uint64_t* last) {
  const SortBuf sorted = sort_result(a, b, bits, 1);
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < r; k += stride) {
    const uint32_t j = sorted.idx[k];
    const uint64_t s = d_start[j], n = d_len[j];
    key[k] = sorted.lo[k];
    last[k] = n ? (n - 1 > kNone - s ? kNone : s + n - 1) : 0;
  }
}

// keep[p] = 1 for an interval that meets no removal range.
__global__ void survive_kernel(MapRef map, const uint64_t* rkey, const uint64_t* rmax, uint64_t r, uint64_t* keep) {
  const uint64_t count = map.hdr[0];
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p < map.cap; p += stride) {
    uint64_t k = 0;
    if (p < count) {
      const uint64_t s = map.start[p], last = map.et[p].x - 1;
      // the removals starting at or before `last`: does the furthest of them reach s?
      const uint64_t q = r ? count_le(rkey, r, last) : 0;
      k = (q && rmax[q - 1] >= s) ? 0 : 1;
    }
    keep[p] = k;
  }
}

__global__ void compact_kernel(MapRef map, const uint64_t* keep, const uint64_t* kpos, uint64_t* s_start,
                               ulonglong2* s_et) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p < map.cap; p += stride) {
    if (!keep[p]) continue;
    s_start[kpos[p]] = map.start[p];
    s_et[kpos[p]] = map.et[p];
  }
}

// Sort key of addition j: its start if valid, else kNone (status INVALID).
__global__ __launch_bounds__(kThreads) void addition_prep_kernel(const uint64_t* a_start, const uint64_t* a_len,
                                                                 const uint64_t* a_target, uint64_t n_add,
                                                                 uint8_t* status, uint64_t* key, uint32_t* idx,
                                                                 uint64_t* bits) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint64_t and_k = ~0ull, or_k = 0;
  for (uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n_add; j += stride) {
    const uint64_t s = a_start[j], n = a_len[j], t = a_target[j];
    const bool valid = n != 0 && n <= kNone - s && n <= kNone - t;
    if (!valid && status) status[j] = GLEAM_REMAP_INVALID;
    const uint64_t k = valid ? s : kNone;
    key[j] = k;
    idx[j] = (uint32_t)j;
    and_k &= k;
    or_k |= k;
  }
  fold_key_bits(and_k, or_k, bits);
}

// Sorted additions: start, original index, and end; an invalid one ends at 0 (it sorts
// last, after every valid one, so the running maximum of ends only ever sees real ends
// before it).
__global__ void addition_unpack_kernel(SortBuf a, SortBuf b, const uint64_t* bits, const uint64_t* a_len,
                                       uint64_t n_add, uint64_t* key, uint64_t* val, uint64_t* aend) {
  const SortBuf sorted = sort_result(a, b, bits, 1);
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n_add; k += stride) {
    const uint64_t s = sorted.lo[k];
    const uint32_t j = sorted.idx[k];
    key[k] = s;
    val[k] = j;
    aend[k] = s == kNone ? 0 : s + a_len[j];
  }
}

// Keep a valid addition that meets no other valid addition and no survivor.
__global__ void addition_classify_kernel(const uint64_t* key, const uint64_t* val, const uint64_t* aend,
                                         const uint64_t* amax, uint64_t n_add, const uint64_t* s_start,
                                         const ulonglong2* s_et, const uint64_t* keep, const uint64_t* kpos,
                                         uint64_t cap, uint8_t* status, uint64_t* acc) {
  const uint64_t n_surv = kpos[cap - 1] + keep[cap - 1];
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n_add; k += stride) {
    const uint64_t s = key[k];
    uint64_t a = 0;
    if (s != kNone) {
      const uint64_t e = aend[k];
      bool clash = (k > 0 && amax[k - 1] > s) || (k + 1 < n_add && key[k + 1] < e);
      if (!clash) {
        const uint64_t q = count_le(s_start, n_surv, e - 1);
        clash = q && s_et[q - 1].x > s;
      }
      a = clash ? 0 : 1;
      if (status) status[val[k]] = clash ? GLEAM_REMAP_OVERLAP : GLEAM_REMAP_ADDED;
    }
    acc[k] = a;
  }
}

// Batches of at most kSmall removals or additions (a task's allocations, its tensors) are
// handled by one 1024-lane workgroup in LDS instead of the several launches of the
// device-wide sort and scans: a bitonic sort of (key, index) pairs and Hillis-Steele
// scans over at most 2048 entries.
constexpr int kSmallThreads = 1024;
constexpr uint32_t kSmall = 2 * kSmallThreads;

__device__ __forceinline__ uint32_t pow2_at_least(uint32_t n) {  // n <= kSmall
  uint32_t p = 1;
  while (p < n) p <<= 1;
  return p;
}

// Sort the pairs (key[i], idx[i]), i < n, ascending by key and then by idx. The indices
// are distinct, so this is a total order and the result is what a stable sort by key
// gives. n is a power of two <= kSmall; every lane of the workgroup calls it.
__device__ void bitonic_sort(uint64_t* key, uint32_t* idx, uint32_t n) {
  for (uint32_t k = 2; k <= n; k <<= 1) {
    for (uint32_t j = k >> 1; j > 0; j >>= 1) {
      const uint32_t t = threadIdx.x;  // pair t of n / 2 <= kSmallThreads
      if (t < n / 2) {
        const uint32_t i = ((t & ~(j - 1)) << 1) | (t & (j - 1));  // bit j of i is clear
        const uint32_t l = i | j;
        const uint64_t ki = key[i], kl = key[l];
        const uint32_t ii = idx[i], il = idx[l];
        const bool greater = ki > kl || (ki == kl && ii > il);
        if (greater == ((i & k) == 0)) {  // out of order for this run's direction
          key[i] = kl;
          key[l] = ki;
          idx[i] = il;
          idx[l] = ii;
        }
      }
      __syncthreads();
    }
  }
}

// In-place inclusive scan of buf[0, n) (n <= kSmall) with `op`; every lane of the
// workgroup calls it; lane t owns entries t and t + kSmallThreads.
template <class Op>
__device__ void block_scan(uint64_t* buf, uint32_t n, Op op) {
  const uint32_t i0 = threadIdx.x, i1 = threadIdx.x + kSmallThreads;
  for (uint32_t off = 1; off < n; off <<= 1) {
    uint64_t v0 = 0, v1 = 0;
    if (i0 < n) v0 = i0 >= off ? op(buf[i0 - off], buf[i0]) : buf[i0];
    if (i1 < n) v1 = i1 >= off ? op(buf[i1 - off], buf[i1]) : buf[i1];
    __syncthreads();
    if (i0 < n) buf[i0] = v0;
    if (i1 < n) buf[i1] = v1;
    __syncthreads();
  }
}

struct MaxOp {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a > b ? a : b; }
};
struct AddOp {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a + b; }
};

// Removal ranges sorted by start, with the running maximum of their last addresses
// (what the radix sort and the scan produce for larger batches).
__global__ void __launch_bounds__(kSmallThreads)
removals_small_kernel(const uint64_t* d_start, const uint64_t* d_len, uint32_t r, uint64_t* rkey, uint64_t* rmax) {
  __shared__ uint64_t key[kSmall], last[kSmall], buf[kSmall];
  __shared__ uint32_t idx[kSmall];
  const uint32_t n = pow2_at_least(r);
  for (uint32_t i = threadIdx.x; i < n; i += kSmallThreads) {
    uint64_t k = kNone, l = 0;  // padding sorts after every range
    if (i < r) {
      const uint64_t s = d_start[i], len = d_len[i];
      k = len ? s : kNone;
      l = len ? (len - 1 > kNone - s ? kNone : s + len - 1) : 0;
    }
    key[i] = k;
    last[i] = l;
    idx[i] = i;
  }
  __syncthreads();
  bitonic_sort(key, idx, n);
  for (uint32_t i = threadIdx.x; i < r; i += kSmallThreads) {
    rkey[i] = key[i];
    buf[i] = last[idx[i]];
  }
  __syncthreads();
  block_scan(buf, r, MaxOp());
  for (uint32_t i = threadIdx.x; i < r; i += kSmallThreads) rmax[i] = buf[i];
}

// Additions sorted, checked against each other and the survivors, and numbered: the
// same outputs (kb, vb, aend, acc, apos) and statuses as the batched path.
__global__ void __launch_bounds__(kSmallThreads)
additions_small_kernel(const uint64_t* a_start, const uint64_t* a_len, const uint64_t* a_target, uint32_t n_add,
                       uint8_t* status, const uint64_t* s_start, const ulonglong2* s_et, const uint64_t* keep,
                       const uint64_t* kpos, uint64_t cap, uint64_t* kb, uint64_t* vb, uint64_t* aend,
                       uint64_t* acc, uint64_t* apos) {
  __shared__ uint64_t key[kSmall], buf[kSmall];
  __shared__ uint32_t idx[kSmall];
  const uint64_t n_surv = kpos[cap - 1] + keep[cap - 1];
  const uint32_t n = pow2_at_least(n_add);
  for (uint32_t j = threadIdx.x; j < n; j += kSmallThreads) {
    uint64_t k = kNone;  // invalid additions and padding sort last (padding after them)
    if (j < n_add) {
      const uint64_t s = a_start[j], len = a_len[j], t = a_target[j];
      const bool valid = len != 0 && len <= kNone - s && len <= kNone - t;
      if (!valid && status) status[j] = GLEAM_REMAP_INVALID;
      if (valid) k = s;
    }
    key[j] = k;
    idx[j] = j;
  }
  __syncthreads();
  bitonic_sort(key, idx, n);
  uint64_t e[2] = {0, 0};
  for (uint32_t h = 0; h < 2; ++h) {
    const uint32_t k = threadIdx.x + h * kSmallThreads;
    if (k >= n_add) continue;
    e[h] = key[k] == kNone ? 0 : key[k] + a_len[idx[k]];
    kb[k] = key[k];
    vb[k] = idx[k];
    aend[k] = e[h];
    buf[k] = e[h];
  }
  __syncthreads();
  block_scan(buf, n_add, MaxOp());  // buf[k] = running maximum of ends through k
  uint64_t a[2] = {0, 0};
  for (uint32_t h = 0; h < 2; ++h) {
    const uint32_t k = threadIdx.x + h * kSmallThreads;
    if (k >= n_add || key[k] == kNone) continue;
    const uint64_t s = key[k];
    bool clash = (k > 0 && buf[k - 1] > s) || (k + 1 < n_add && key[k + 1] < e[h]);
    if (!clash) {
      const uint64_t q = count_le(s_start, n_surv, e[h] - 1);
      clash = q && s_et[q - 1].x > s;
    }
    a[h] = clash ? 0 : 1;
    if (status) status[idx[k]] = clash ? GLEAM_REMAP_OVERLAP : GLEAM_REMAP_ADDED;
  }
  __syncthreads();  // every lane has read buf
  for (uint32_t h = 0; h < 2; ++h) {
    const uint32_t k = threadIdx.x + h * kSmallThreads;
    if (k < n_add) {
      acc[k] = a[h];
      buf[k] = a[h];
    }
  }
  __syncthreads();
  block_scan(buf, n_add, AddOp());  // inclusive count of kept additions
  for (uint32_t h = 0; h < 2; ++h) {
    const uint32_t k = threadIdx.x + h * kSmallThreads;
    if (k < n_add) apos[k] = buf[k] - a[h];
  }
}

struct Totals {
  uint64_t n_surv, n_acc, total, S;
  bool fits;
};

__device__ __forceinline__ Totals totals(const uint64_t* keep, const uint64_t* kpos, uint64_t cap,
                                         const uint64_t* acc, const uint64_t* apos, uint64_t n_add) {
  Totals t;
  t.n_surv = kpos[cap - 1] + keep[cap - 1];
  t.n_acc = n_add ? apos[n_add - 1] + acc[n_add - 1] : 0;
  t.total = t.n_surv + t.n_acc;
  t.fits = t.total <= cap;
  t.S = t.total > kFence ? (t.total + kFence - 1) / kFence : 1;
  return t;
}

__device__ __forceinline__ void place(const MapRef& map, uint64_t q, uint64_t s, ulonglong2 et, uint64_t S) {
  map.start[q] = s;
  map.et[q] = et;
  if (q % S == 0) map.fence[q / S] = s;
}

// Survivor i lands at i + (kept additions that start before it).
__global__ void place_survivors_kernel(MapRef map, const uint64_t* s_start, const ulonglong2* s_et,
                                       const uint64_t* keep, const uint64_t* kpos, const uint64_t* key,
                                       const uint64_t* acc, const uint64_t* apos, uint64_t n_add) {
  const Totals t = totals(keep, kpos, map.cap, acc, apos, n_add);
  if (!t.fits) return;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < t.n_surv; i += stride) {
    const uint64_t s = s_start[i];
    const uint64_t k = count_lt(key, n_add, s);  // additions (any status) starting before s
    const uint64_t before = k < n_add ? apos[k] : t.n_acc;
    place(map, i + before, s, s_et[i], t.S);
  }
}

// Kept addition k lands at its number among kept additions + (survivors that start
// before it); when the result would not fit, it is FULL instead.
__global__ void place_additions_kernel(MapRef map, const uint64_t* s_start, const uint64_t* keep,
                                       const uint64_t* kpos, const uint64_t* key, const uint64_t* val,
                                       const uint64_t* aend, const uint64_t* acc, const uint64_t* apos,
                                       uint64_t n_add, const uint64_t* a_target, uint8_t* status) {
  const Totals t = totals(keep, kpos, map.cap, acc, apos, n_add);
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n_add; k += stride) {
    if (!acc[k]) continue;
    if (t.fits) {
      const uint64_t s = key[k];
      place(map, apos[k] + count_lt(s_start, t.n_surv, s), s, make_ulonglong2(aend[k], a_target[val[k]] - s),
            t.S);
    } else if (status) {
      status[val[k]] = GLEAM_REMAP_FULL;
    }
  }
}

// Header and counts, after both placements.
__global__ void finish_kernel(MapRef map, const uint64_t* keep, const uint64_t* kpos, const uint64_t* acc,
                              const uint64_t* apos, uint64_t n_add, uint64_t* counts) {
  const Totals t = totals(keep, kpos, map.cap, acc, apos, n_add);
  const uint64_t before = map.hdr[0];
  counts[0] = t.fits ? t.total : before;
  counts[1] = t.fits ? t.n_acc : 0;
  counts[2] = t.fits ? before - t.n_surv : 0;
  counts[3] = n_add - (t.fits ? t.n_acc : 0);
  if (t.fits) {
    map.hdr[0] = t.total;
    map.hdr[1] = t.S;
    map.hdr[2] = (t.total + t.S - 1) / t.S;
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
      const ulonglong2 et = map.et[lo + c];  // start[lo + c] <= a: inside iff a < end
      if (a < et.x) r = a + et.y;
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
    d_target[p] = et.y + s;
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
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_remap() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&update_init_kernel));
}

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
  return gleam::upd_layout(m->capacity, n_add, n_del).total;
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
  uint64_t* hdr = at(L.hdr);
  uint64_t* partial = at(L.partial);
  void* sort_ws = b + L.sort;
  const MapRef map = map_ref(m);
  const uint64_t cap = m->capacity;
  gleam_status st;
  hipLaunchKernelGGL(update_init_kernel, dim3(1), dim3(64), 0, s, hdr, n_del, n_add);
  if ((st = launch_status("update_init_kernel")) != GLEAM_OK) return st;

  // 1. removals, survivors
  const uint64_t* rkey = nullptr;
  const uint64_t* rmax = nullptr;
  if (n_del > 0 && n_del <= kSmall) {
    hipLaunchKernelGGL(removals_small_kernel, dim3(1), dim3(kSmallThreads), 0, s, d_del_start, d_del_len,
                       (uint32_t)n_del, at(L.rkb), at(L.rmax));
    if ((st = launch_status("removals_small_kernel")) != GLEAM_OK) return st;
    rkey = at(L.rkb);
    rmax = at(L.rmax);
  } else if (n_del > 0) {
    const SortBuf ra{nullptr, at(L.rka), reinterpret_cast<uint32_t*>(b + L.ridx)};
    const SortBuf rb = sort_other(sort_ws, n_del, 1);
    hipLaunchKernelGGL(removal_prep_kernel, dim3(fold_grid(n_del)), dim3(kThreads), 0, s, d_del_start, d_del_len,
                       n_del, ra.lo, ra.idx, hdr + 4);
    if ((st = launch_status("removal_prep_kernel")) != GLEAM_OK) return st;
    if ((st = radix_sort_pairs(ra, hdr, hdr + 4, n_del, 1, sort_ws, s)) != GLEAM_OK) return st;
    hipLaunchKernelGGL(removal_unpack_kernel, dim3(grid_for(n_del)), dim3(kThreads), 0, s, ra, rb, hdr + 4,
                       d_del_start, d_del_len, n_del, at(L.rkb), at(L.rvb));
    if ((st = launch_status("removal_unpack_kernel")) != GLEAM_OK) return st;
    if ((st = device_scan<ScanMax, false>(at(L.rvb), at(L.rmax), n_del, partial, s)) != GLEAM_OK) return st;
    rkey = at(L.rkb);
    rmax = at(L.rmax);
  }
  const dim3 block(kThreads), gcap(grid_for(cap)), gadd(grid_for(n_add));
  hipLaunchKernelGGL(survive_kernel, gcap, block, 0, s, map, rkey, rmax, n_del, at(L.keep));
  if ((st = launch_status("survive_kernel")) != GLEAM_OK) return st;
  if ((st = device_scan<ScanSum, true>(at(L.keep), at(L.kpos), cap, partial, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(compact_kernel, gcap, block, 0, s, map, at(L.keep), at(L.kpos), at(L.s_start),
                     reinterpret_cast<ulonglong2*>(at(L.s_et)));
  if ((st = launch_status("compact_kernel")) != GLEAM_OK) return st;

  // 2-3. additions: sorted, checked against each other and the survivors, numbered
  if (n_add > 0 && n_add <= kSmall) {
    hipLaunchKernelGGL(additions_small_kernel, dim3(1), dim3(kSmallThreads), 0, s, d_add_start, d_add_len,
                       d_add_target, (uint32_t)n_add, d_add_status, at(L.s_start),
                       reinterpret_cast<const ulonglong2*>(at(L.s_et)), at(L.keep), at(L.kpos), cap, at(L.kb),
                       at(L.vb), at(L.aend), at(L.acc), at(L.apos));
    if ((st = launch_status("additions_small_kernel")) != GLEAM_OK) return st;
  } else if (n_add > 0) {
    const SortBuf aa{nullptr, at(L.ka), reinterpret_cast<uint32_t*>(b + L.aidx)};
    const SortBuf ab = sort_other(sort_ws, n_add, 1);
    hipLaunchKernelGGL(addition_prep_kernel, dim3(fold_grid(n_add)), block, 0, s, d_add_start, d_add_len,
                       d_add_target, n_add, d_add_status, aa.lo, aa.idx, hdr + 8);
    if ((st = launch_status("addition_prep_kernel")) != GLEAM_OK) return st;
    if ((st = radix_sort_pairs(aa, hdr + 1, hdr + 8, n_add, 1, sort_ws, s)) != GLEAM_OK) return st;
    hipLaunchKernelGGL(addition_unpack_kernel, gadd, block, 0, s, aa, ab, hdr + 8, d_add_len, n_add, at(L.kb),
                       at(L.vb), at(L.aend));
    if ((st = launch_status("addition_unpack_kernel")) != GLEAM_OK) return st;
    if ((st = device_scan<ScanMax, false>(at(L.aend), at(L.amax), n_add, partial, s)) != GLEAM_OK) return st;
    hipLaunchKernelGGL(addition_classify_kernel, gadd, block, 0, s, at(L.kb), at(L.vb), at(L.aend), at(L.amax),
                       n_add, at(L.s_start), reinterpret_cast<const ulonglong2*>(at(L.s_et)), at(L.keep),
                       at(L.kpos), cap, d_add_status, at(L.acc));
    if ((st = launch_status("addition_classify_kernel")) != GLEAM_OK) return st;
    if ((st = device_scan<ScanSum, true>(at(L.acc), at(L.apos), n_add, partial, s)) != GLEAM_OK) return st;
  }

  // 4. merge by rank into the storage (only if everything fits), then the header
  hipLaunchKernelGGL(place_survivors_kernel, gcap, block, 0, s, map, at(L.s_start),
                     reinterpret_cast<const ulonglong2*>(at(L.s_et)), at(L.keep), at(L.kpos), at(L.kb), at(L.acc),
                     at(L.apos), n_add);
  if ((st = launch_status("place_survivors_kernel")) != GLEAM_OK) return st;
  if (n_add > 0) {
    hipLaunchKernelGGL(place_additions_kernel, gadd, block, 0, s, map, at(L.s_start), at(L.keep), at(L.kpos),
                       at(L.kb), at(L.vb), at(L.aend), at(L.acc), at(L.apos), n_add, d_add_target, d_add_status);
    if ((st = launch_status("place_additions_kernel")) != GLEAM_OK) return st;
  }
  hipLaunchKernelGGL(finish_kernel, dim3(1), dim3(1), 0, s, map, at(L.keep), at(L.kpos), at(L.acc), at(L.apos),
                     n_add, d_counts);
  return launch_status("finish_kernel");
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
  // as many 1024-lane workgroups per CU as the LDS holds fences (at most two, 32 waves);
  // each loads the fence once
  const uint64_t per_cu = kFence * 8 <= 80 * 1024 ? 2 : 1;
  const uint64_t want = (n + kTranslateThreads - 1) / kTranslateThreads;
  const uint64_t grid = want < per_cu * cus ? want : per_cu * cus;
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
