// gleam_first_writes: the first-write rule of weight identification (Gleam Sec. 4.1.1:
// where an address range of an allocation is written several times, only the first
// host-to-device write counts). Given each allocation's recorded writes in time order,
// it lists, per write, the pieces of its destination range that no earlier write of the
// same allocation covers. Digesting those pieces of each write's payload when it lands,
// and the same pieces of the allocation at free time, compares every written byte with
// its first writer's byte (gleam_identify_weights over the pieces).
//
// One 1024-thread workgroup per allocation, all in LDS (up to kMaxWrites writes):
//   1. the 2n write endpoints are sorted (bitonic) and made unique: boundaries B;
//      consecutive boundaries delimit the elementary intervals;
//   2. the first writer of each elementary interval is the least write index covering
//      it: every write min-updates the O(log) canonical nodes of a segment tree over the
//      elementary intervals that make up its range, and an interval's first writer is
//      the least value on its path to the root (O(n log n) work, whatever the overlap);
//   3. maximal runs of intervals with one first writer are the pieces; they are sorted
//      by (write, address) with a second bitonic sort and written to the workspace.
// A single-workgroup scan then gives each allocation's first piece, and a last pass
// moves the pieces into the caller's dense arrays.

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kFwThreads = 1024;
constexpr uint32_t kMaxWrites = 2048;
constexpr uint32_t kMaxEnds = 2 * kMaxWrites;  // endpoints, boundaries, intervals
constexpr uint32_t kNone = 0xFFFFFFFFu;

struct FwArgs {
  const uint64_t* addr;
  const uint64_t* len;
  uint64_t n_writes;
  const uint64_t* region_first;
  uint64_t n_regions;
  uint64_t* pad_write;   // workspace: u64[2 n_writes] each, allocation r's pieces from 2 region_first[r]
  uint64_t* pad_offset;
  uint64_t* pad_len;
  uint64_t* counts;      // workspace: pieces of each allocation
  uint8_t* status;       // nullable
};

__device__ __forceinline__ uint32_t p2_at_least(uint32_t x) {
  uint32_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Ascending bitonic sort of a[0, n), n a power of two, by the whole workgroup.
template <typename T>
__device__ void bitonic_sort(T* a, uint32_t n) {
  for (uint32_t k = 2; k <= n; k <<= 1) {
    for (uint32_t j = k >> 1; j > 0; j >>= 1) {
      for (uint32_t i = threadIdx.x; i < n; i += kFwThreads) {
        const uint32_t o = i ^ j;
        if (o > i) {
          const T x = a[i], y = a[o];
          const bool up = (i & k) == 0;
          if (up ? (y < x) : (x < y)) {
            a[i] = y;
            a[o] = x;
          }
        }
      }
      __syncthreads();
    }
  }
}

// Exclusive scan of one value per thread over the workgroup; *total gets the sum.
__device__ uint32_t fw_scan(uint32_t x, uint32_t* wave_sums, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = x;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(incl, d, 64);
    if (lane >= d) incl += y;
  }
  if (lane == 63) wave_sums[wave] = incl;
  __syncthreads();
  uint32_t before = 0, sum = 0;
  for (int w = 0; w < kFwThreads / 64; ++w) {
    const uint32_t s = wave_sums[w];
    before += w < wave ? s : 0u;
    sum += s;
  }
  __syncthreads();
  *total = sum;
  return before + incl - x;
}

// First index i in [0, m) with b[i] >= v (m if none).
__device__ __forceinline__ uint32_t lower_bound(const uint64_t* b, uint32_t m, uint64_t v) {
  uint32_t lo = 0, hi = m;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (b[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(kFwThreads) void first_write_region_kernel(FwArgs a) {
  __shared__ uint64_t ends[kMaxEnds];    // sorted endpoints
  __shared__ uint64_t bounds[kMaxEnds];  // unique boundaries
  __shared__ uint32_t tree[2 * kMaxEnds];
  __shared__ uint32_t owner[kMaxEnds];   // first writer of each elementary interval
  __shared__ uint32_t keys[kMaxEnds];    // pieces: (write << 12) | change-point rank
  __shared__ uint16_t cps[kMaxEnds + 1]; // change points (interval index where a run starts)
  __shared__ uint32_t wave_sums[kFwThreads / 64];
  __shared__ uint32_t flag;
  const uint32_t tid = threadIdx.x;
  const uint64_t r = blockIdx.x;
  const uint64_t w0 = a.region_first[r], w1 = a.region_first[r + 1];
  uint8_t st = GLEAM_FW_OK;
  if (w1 < w0 || w1 > a.n_writes) st = GLEAM_FW_INVALID;
  else if (w1 - w0 > kMaxWrites) st = GLEAM_FW_TOO_MANY;
  if (st != GLEAM_FW_OK) {  // uniform across the workgroup
    if (tid == 0) {
      a.counts[r] = 0;
      if (a.status) a.status[r] = st;
    }
    return;
  }
  const uint32_t n = (uint32_t)(w1 - w0);
  const uint32_t P = p2_at_least(n ? 2 * n : 2);
  if (tid == 0) flag = 0;
  __syncthreads();
  for (uint32_t j = tid; j < n; j += kFwThreads) {
    const uint64_t s = a.addr[w0 + j], l = a.len[w0 + j];
    if (l > ~0ull - s) atomicOr(&flag, 1u);  // past the top of the address space
    ends[2 * j] = s;
    ends[2 * j + 1] = s + l;
  }
  for (uint32_t i = 2 * n + tid; i < P; i += kFwThreads) ends[i] = ~0ull;
  __syncthreads();
  if (flag) {
    if (tid == 0) {
      a.counts[r] = 0;
      if (a.status) a.status[r] = GLEAM_FW_INVALID;
    }
    return;
  }
  bitonic_sort(ends, P);

  // unique boundaries: thread t takes ends[4t, 4t + 4)
  uint32_t total;
  {
    uint32_t f[4], c = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t i = 4 * tid + e;
      f[e] = i < P && (i == 0 || ends[i] != ends[i - 1]);
      c += f[e];
    }
    uint32_t at = fw_scan(c, wave_sums, &total);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (f[e]) bounds[at++] = ends[4 * tid + e];
  }
  const uint32_t M = total;        // boundaries
  const uint32_t E = M - 1;        // elementary intervals [bounds[i], bounds[i + 1])
  const uint32_t T2 = p2_at_least(E ? E : 1);
  for (uint32_t i = tid; i < 2 * T2; i += kFwThreads) tree[i] = kNone;
  __syncthreads();

  // every write min-updates the canonical nodes of its interval range
  for (uint32_t j = tid; j < n; j += kFwThreads) {
    const uint64_t s = a.addr[w0 + j], l = a.len[w0 + j];
    if (l == 0) continue;
    uint32_t lo = lower_bound(bounds, M, s) + T2, hi = lower_bound(bounds, M, s + l) + T2;
    while (lo < hi) {
      if (lo & 1) atomicMin(&tree[lo++], j);
      if (hi & 1) atomicMin(&tree[--hi], j);
      lo >>= 1;
      hi >>= 1;
    }
  }
  __syncthreads();
  for (uint32_t i = tid; i < E; i += kFwThreads) {
    uint32_t m = kNone;
    for (uint32_t node = i + T2; node >= 1; node >>= 1) m = min(m, tree[node]);
    owner[i] = m;
  }
  __syncthreads();

  // change points: intervals where a run of one first writer starts (thread t: 4 of them)
  {
    uint32_t f[4], c = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t i = 4 * tid + e;
      f[e] = i < E && (i == 0 || owner[i] != owner[i - 1]);
      c += f[e];
    }
    uint32_t at = fw_scan(c, wave_sums, &total);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (f[e]) cps[at++] = (uint16_t)(4 * tid + e);
  }
  const uint32_t K = total;  // runs
  if (tid == 0) cps[K] = (uint16_t)E;
  __syncthreads();  // every change point written
  const uint32_t KP = p2_at_least(K ? K : 1);
  for (uint32_t k = tid; k < KP; k += kFwThreads) {
    const uint32_t o = k < K ? owner[cps[k]] : kNone;
    keys[k] = o == kNone ? kNone : (o << 12) | k;
  }
  __syncthreads();
  bitonic_sort(keys, KP);

  // keys[0, pieces) are the owned runs, by (write, address)
  uint64_t* pw = a.pad_write + 2 * w0;
  uint64_t* po = a.pad_offset + 2 * w0;
  uint64_t* pl = a.pad_len + 2 * w0;
  uint32_t mine = 0;
  for (uint32_t p = tid; p < KP; p += kFwThreads) {
    const uint32_t key = keys[p];
    if (key == kNone) continue;
    ++mine;
    const uint32_t j = key >> 12, k = key & 0xFFFu;
    const uint64_t lo = bounds[cps[k]], hi = bounds[cps[k + 1]];
    pw[p] = w0 + j;
    po[p] = lo - a.addr[w0 + j];
    pl[p] = hi - lo;
  }
  fw_scan(mine, wave_sums, &total);
  if (tid == 0) {
    a.counts[r] = total;
    if (a.status) a.status[r] = GLEAM_FW_OK;
  }
}

// region_piece_first = exclusive prefix of the counts (and the total at [n_regions]).
__global__ __launch_bounds__(kFwThreads) void first_write_scan_kernel(const uint64_t* counts, uint64_t n_regions,
                                                                      uint64_t* first) {
  __shared__ uint64_t wave_sums[kFwThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t carry = 0;
  for (uint64_t base = 0; base < n_regions; base += kFwThreads) {
    const uint64_t i = base + threadIdx.x;
    const uint64_t x = i < n_regions ? counts[i] : 0;
    uint64_t incl = x;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint64_t y = shfl64(incl, lane >= d ? lane - d : lane);
      if (lane >= d) incl += y;
    }
    if (lane == 63) wave_sums[wave] = incl;
    __syncthreads();
    uint64_t before = 0, sum = 0;
    for (int w = 0; w < kFwThreads / 64; ++w) {
      before += w < wave ? wave_sums[w] : 0;
      sum += wave_sums[w];
    }
    __syncthreads();
    if (i < n_regions) first[i] = carry + before + incl - x;
    carry += sum;
  }
  if (threadIdx.x == 0) first[n_regions] = carry;
}

// One thread per allocation moves its pieces from the workspace to the dense outputs
// (u64[2 n_writes] each: a well-formed region_first yields fewer pieces; an ill-formed one,
// whose regions overlap, is cut at the end of the outputs).
__global__ void first_write_move_kernel(FwArgs a, const uint64_t* first, uint64_t* out_write,
                                        uint64_t* out_offset, uint64_t* out_len) {
  const uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= a.n_regions) return;
  const uint64_t c = a.counts[r], w0 = a.region_first[r], at = first[r];
  const uint64_t cap = 2 * a.n_writes;
  for (uint64_t p = 0; p < c && at + p < cap; ++p) {
    out_write[at + p] = a.pad_write[2 * w0 + p];
    out_offset[at + p] = a.pad_offset[2 * w0 + p];
    out_len[at + p] = a.pad_len[2 * w0 + p];
  }
}

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_first_write() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&first_write_move_kernel));
}

}  // namespace gleam

extern "C" size_t gleam_first_writes_ws_bytes(uint64_t n_writes, uint64_t n_regions) {
  if (n_writes > (1ull << 36) || n_regions > (1ull << 36)) return 0;
  const size_t b = gleam::kHeaderBytes + 8 * (size_t)n_regions + 48 * (size_t)n_writes;
  return (b + 255) & ~(size_t)255;
}

extern "C" gleam_status gleam_first_writes(const uint64_t* d_addr, const uint64_t* d_len, uint64_t n_writes,
                                           const uint64_t* d_region_first, uint64_t n_regions,
                                           uint64_t* d_piece_write, uint64_t* d_piece_offset, uint64_t* d_piece_len,
                                           uint64_t* d_region_piece_first, uint8_t* d_region_status, void* d_ws,
                                           size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  if (!d_region_piece_first || (n_regions > 0 && !d_region_first) ||
      (n_writes > 0 && (!d_addr || !d_len || !d_piece_write || !d_piece_offset || !d_piece_len))) {
    set_error("gleam_first_writes: null write list, region list or output");
    return GLEAM_E_INVALID;
  }
  const size_t need = gleam_first_writes_ws_bytes(n_writes, n_regions);
  if (need == 0 || n_regions > 0x7fffffffull) {
    set_error("gleam_first_writes: more than 2^36 writes or 2^31 allocations");
    return GLEAM_E_UNSUPPORTED;
  }
  if (!d_ws || !aligned256(d_ws)) {
    set_error("gleam_first_writes: workspace must be non-null and 256-byte aligned");
    return GLEAM_E_INVALID;
  }
  if (ws_bytes < need) {
    set_error("gleam_first_writes: workspace of %zu bytes, %zu needed", ws_bytes, need);
    return GLEAM_E_WORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = static_cast<uint8_t*>(d_ws);
  FwArgs a;
  a.addr = d_addr;
  a.len = d_len;
  a.n_writes = n_writes;
  a.region_first = d_region_first;
  a.n_regions = n_regions;
  a.counts = reinterpret_cast<uint64_t*>(ws + kHeaderBytes);
  a.pad_write = a.counts + n_regions;
  a.pad_offset = a.pad_write + 2 * n_writes;
  a.pad_len = a.pad_offset + 2 * n_writes;
  a.status = d_region_status;
  gleam_status st;
  if (n_regions > 0) {
    hipLaunchKernelGGL(first_write_region_kernel, dim3((uint32_t)n_regions), dim3(kFwThreads), 0, s, a);
    if ((st = launch_status("first_write_region_kernel")) != GLEAM_OK) return st;
  }
  hipLaunchKernelGGL(first_write_scan_kernel, dim3(1), dim3(kFwThreads), 0, s, a.counts, n_regions,
                     d_region_piece_first);
  if ((st = launch_status("first_write_scan_kernel")) != GLEAM_OK) return st;
  if (n_regions == 0) return GLEAM_OK;
  hipLaunchKernelGGL(first_write_move_kernel, dim3((uint32_t)((n_regions + 255) / 256)), dim3(256), 0, s, a,
                     d_region_piece_first, d_piece_write, d_piece_offset, d_piece_len);
  return launch_status("first_write_move_kernel");
}
