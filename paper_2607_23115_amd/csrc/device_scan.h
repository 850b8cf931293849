// Device-wide scans of u64 arrays (running sum or running maximum), kernels only (no
// library scan, no memsets), so a call that uses them may be captured in a HIP graph.
// Up to 16384 elements: one workgroup, one launch. Beyond: three launches over
// 4096-element tiles: each tile's total, an exclusive scan of the tile totals in one
// workgroup, and each tile's own scan started from its prefix. A tile's own scan stages
// it through LDS so that each lane scans consecutive elements in registers.
#pragma once

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanWaves = kScanThreads / 64;
constexpr int kScanItems = 16;
constexpr uint64_t kScanTile = (uint64_t)kScanThreads * kScanItems;

struct ScanSum {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a + b; }
};
struct ScanMax {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a > b ? a : b; }
};
// Both operations have identity 0.

__device__ __forceinline__ uint64_t shfl_up64(uint64_t v, int d) {
  const uint32_t lo = __shfl_up((uint32_t)v, d, 64);
  const uint32_t hi = __shfl_up((uint32_t)(v >> 32), d, 64);
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive scan over the workgroup's threads in thread order; *total gets the
// workgroup's total. Every thread calls it; tmp is kScanWaves words of LDS.
template <class Op>
__device__ __forceinline__ uint64_t block_incl_scan(uint64_t x, Op op, uint64_t* tmp, uint64_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t y = shfl_up64(x, d);
    if (lane >= d) x = op(y, x);
  }
  if (lane == 63) tmp[wave] = x;
  __syncthreads();
  uint64_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kScanWaves; ++w) {
    if (w < wave) before = op(before, tmp[w]);
    all = op(all, tmp[w]);
  }
  __syncthreads();  // tmp read by every thread before a later call rewrites it
  *total = all;
  return op(before, x);
}

template <class Op>
__global__ __launch_bounds__(kScanThreads) void scan_tile_total_kernel(const uint64_t* in, uint64_t n,
                                                                       uint64_t* partial) {
  __shared__ uint64_t tmp[kScanWaves];
  const uint64_t tile0 = (uint64_t)blockIdx.x * kScanTile;
  const Op op;
  uint64_t v[kScanItems];
#pragma unroll
  for (int r = 0; r < kScanItems; ++r) {  // unconditional (clamped) loads, issued together
    const uint64_t i = tile0 + (uint64_t)r * kScanThreads + threadIdx.x;
    v[r] = in[i < n ? i : n - 1];
  }
  uint64_t acc = 0;
#pragma unroll
  for (int r = 0; r < kScanItems; ++r) {
    const uint64_t i = tile0 + (uint64_t)r * kScanThreads + threadIdx.x;
    if (i < n) acc = op(acc, v[r]);
  }
  uint64_t total;
  block_incl_scan(acc, op, tmp, &total);
  if (threadIdx.x == 0) partial[blockIdx.x] = total;
}

// One workgroup: partial[0, tiles) becomes its exclusive scan.
template <class Op>
__global__ __launch_bounds__(kScanThreads) void scan_partials_kernel(uint64_t* partial, uint64_t tiles) {
  __shared__ uint64_t tmp[kScanWaves];
  __shared__ uint64_t last_of_wave[kScanWaves];
  const Op op;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t carry = 0;
  for (uint64_t base = 0; base < tiles; base += kScanThreads) {
    const uint64_t t = base + threadIdx.x;
    const uint64_t x = t < tiles ? partial[t] : 0;
    uint64_t total;
    const uint64_t incl = block_incl_scan(x, op, tmp, &total);
    // exclusive = the inclusive value of the thread before (the identity for thread 0)
    const uint64_t prev = shfl_up64(incl, 1);
    if (lane == 63) last_of_wave[wave] = incl;
    __syncthreads();
    const uint64_t excl = lane ? prev : (wave ? last_of_wave[wave - 1] : 0);
    __syncthreads();
    if (t < tiles) partial[t] = op(carry, excl);
    carry = op(carry, total);
  }
}

// Scans `count` elements (at most kThreadsT * kScanItems) of in[] into out[], starting
// from `carry`: loads go through LDS so that each lane then scans 16 consecutive
// elements in registers, and one workgroup scan of the lanes' totals gives each lane its
// start (one chain of shuffles per call instead of one per 16-element round). `buf`
// holds kThreadsT * 17 words (16 per lane plus one of padding, against bank conflicts).
template <class Op, bool kExclusive, int kThreadsT>
__device__ __forceinline__ void scan_span(const uint64_t* in, uint64_t* out, uint32_t count, uint64_t carry,
                                          uint64_t* buf, uint64_t* tmp) {
  static_assert(!kExclusive || sizeof(Op) == sizeof(ScanSum), "exclusive scans are running sums");
  const Op op;
  auto slot = [](uint32_t j) { return j + (j >> 4); };
  uint64_t v[kScanItems];
#pragma unroll
  for (int r = 0; r < kScanItems; ++r) {  // unconditional (clamped) loads, issued together
    const uint32_t j = r * kThreadsT + threadIdx.x;
    v[r] = in[j < count ? j : count - 1];
  }
#pragma unroll
  for (int r = 0; r < kScanItems; ++r) {
    const uint32_t j = r * kThreadsT + threadIdx.x;
    buf[slot(j)] = j < count ? v[r] : 0;
  }
  __syncthreads();
  const uint32_t first = threadIdx.x * kScanItems;
  uint64_t acc = 0;
#pragma unroll
  for (int r = 0; r < kScanItems; ++r) {
    if (first + r < count) acc = op(acc, buf[slot(first + r)]);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t incl = acc;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t y = shfl_up64(incl, d);
    if (lane >= d) incl = op(y, incl);
  }
  if (lane == 63) tmp[wave] = incl;
  __syncthreads();
  uint64_t run = carry;
  for (int w = 0; w < wave; ++w) run = op(run, tmp[w]);
  const uint64_t prev = shfl_up64(incl, 1);
  if (lane) run = op(run, prev);  // the lanes before this one in its wave
#pragma unroll
  for (int r = 0; r < kScanItems; ++r) {
    if (first + r < count) {
      const uint64_t x = buf[slot(first + r)];
      if (kExclusive) {
        buf[slot(first + r)] = run;
        run += x;
      } else {
        run = op(run, x);
        buf[slot(first + r)] = run;
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kScanItems; ++r) {
    const uint32_t j = r * kThreadsT + threadIdx.x;
    if (j < count) out[j] = buf[slot(j)];
  }
}

// out[i] = op over in[0..i] (kExclusive: over in[0..i), a running sum only).
template <class Op, bool kExclusive>
__global__ __launch_bounds__(kScanThreads) void scan_tile_kernel(const uint64_t* in, uint64_t* out, uint64_t n,
                                                                 const uint64_t* partial) {
  __shared__ uint64_t buf[kScanThreads * (kScanItems + 1)];
  __shared__ uint64_t tmp[kScanWaves];
  const uint64_t tile0 = (uint64_t)blockIdx.x * kScanTile;
  if (tile0 >= n) return;
  const uint32_t count = (uint32_t)(n - tile0 < kScanTile ? n - tile0 : kScanTile);
  scan_span<Op, kExclusive, kScanThreads>(in + tile0, out + tile0, count, partial[blockIdx.x], buf, tmp);
}

// Scans of at most kScanSmallMax elements: one 1024-lane workgroup, one launch.
constexpr int kScanSmallThreads = 1024;
constexpr uint64_t kScanSmallMax = (uint64_t)kScanSmallThreads * kScanItems;

template <class Op, bool kExclusive>
__global__ __launch_bounds__(kScanSmallThreads) void scan_small_kernel(const uint64_t* in, uint64_t* out,
                                                                       uint32_t n) {
  __shared__ uint64_t buf[kScanSmallThreads * (kScanItems + 1)];  // 136 KiB
  __shared__ uint64_t tmp[kScanSmallThreads / 64];
  scan_span<Op, kExclusive, kScanSmallThreads>(in, out, n, 0, buf, tmp);
}

inline uint64_t scan_tiles(uint64_t n) { return (n + kScanTile - 1) / kScanTile; }

// Scans in[0, n) into out (not in place); `partial` holds scan_tiles(n) words of device
// scratch. n below 2^31 * kScanTile.
template <class Op, bool kExclusive>
gleam_status device_scan(const uint64_t* in, uint64_t* out, uint64_t n, uint64_t* partial, hipStream_t s) {
  if (n == 0) return GLEAM_OK;
  if (n <= kScanSmallMax) {
    hipLaunchKernelGGL((scan_small_kernel<Op, kExclusive>), dim3(1), dim3(kScanSmallThreads), 0, s, in, out,
                       (uint32_t)n);
    return launch_status("scan_small_kernel");
  }
  const uint64_t tiles = scan_tiles(n);
  hipLaunchKernelGGL(scan_tile_total_kernel<Op>, dim3((uint32_t)tiles), dim3(kScanThreads), 0, s, in, n, partial);
  gleam_status st = launch_status("scan_tile_total_kernel");
  if (st != GLEAM_OK) return st;
  hipLaunchKernelGGL(scan_partials_kernel<Op>, dim3(1), dim3(kScanThreads), 0, s, partial, tiles);
  if ((st = launch_status("scan_partials_kernel")) != GLEAM_OK) return st;
  hipLaunchKernelGGL((scan_tile_kernel<Op, kExclusive>), dim3((uint32_t)tiles), dim3(kScanThreads), 0, s, in, out, n,
                     partial);
  return launch_status("scan_tile_kernel");
}

}  // namespace
}  // namespace gleam
