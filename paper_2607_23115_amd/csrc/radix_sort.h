// Device-wide LSD radix sort of (key, index) pairs for the table's maintenance calls
// (eviction order and export order) and the address map's update (removals and
// additions by start), written for gfx950 so those calls enqueue kernels only (no
// library sort, no memsets): a caller may capture them in a HIP graph.
//
// Keys are 64 or 128 bits (hi:lo), indices u32. Each pass sorts by one 8-bit digit,
// stably, in three launches over 4096-element tiles:
//   1. histogram: each tile counts its digits (LDS atomics) into a digit-major array
//      count[d][tile];
//   2. scan: one workgroup per digit turns its row into exclusive tile offsets, and the
//      digit's total goes to totals[d];
//   3. scatter: each wave of a tile owns 1024 consecutive elements and ranks them
//      stably (the lanes holding one digit find each other with eight ballots, a running
//      per-digit count in LDS carries the rank across the wave's rounds); the tile is
//      then reordered in LDS by digit and written out word by word, so consecutive
//      lanes store consecutive addresses of one digit's run.
// A pass whose digit is the same for every key moves nothing and is skipped on the
// device: the caller supplies the AND and the OR of all key words, the pass kernels
// return at once for such a pass, and the buffers' roles (which holds the input) follow
// from how many passes before it were not skipped. Nothing is decided on the host, so
// the launches are fixed and a graph of them replays correctly for any keys.
// The sort is stable: equal keys keep their input order (the address map's callers
// number their entries in input order, so ties go to the lower index).
#pragma once

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kSortThreads = 256;
constexpr int kSortWaves = kSortThreads / 64;
constexpr int kSortItems = 16;                               // per lane
constexpr uint32_t kSortTile = kSortThreads * kSortItems;    // 4096 elements
constexpr uint32_t kSortWaveSpan = 64 * kSortItems;          // 1024 elements per wave
constexpr int kDigits = 256;

struct SortBuf {
  uint64_t* hi;  // null for 64-bit keys
  uint64_t* lo;
  uint32_t* idx;
};

// bits = {AND of lo words, OR of lo words, AND of hi words, OR of hi words} over the
// keys being sorted. Pass p's digit is bits 8p..8p+7 of the 128-bit key.
__device__ __forceinline__ bool pass_trivial(const uint64_t* bits, uint32_t p) {
  const uint32_t w = p >= 8 ? 2u : 0u;
  const uint64_t differ = bits[w] ^ bits[w + 1];
  return ((differ >> ((8 * p) & 63)) & 0xFFu) == 0;
}

// Whether pass p reads the workspace buffer (b) rather than the caller's (a).
__device__ __forceinline__ bool reads_b(const uint64_t* bits, uint32_t p) {
  uint32_t moved = 0;
  for (uint32_t q = 0; q < p; ++q) moved += pass_trivial(bits, q) ? 0u : 1u;
  return (moved & 1u) != 0;
}

// Where the sorted pairs are after all 8 * words passes.
__device__ __forceinline__ SortBuf sort_result(const SortBuf& a, const SortBuf& b, const uint64_t* bits, int words) {
  return reads_b(bits, 8u * (uint32_t)words) ? b : a;
}

__global__ __launch_bounds__(kSortThreads) void sort_hist_kernel(SortBuf a, SortBuf b, const uint64_t* n_dev,
                                                                 const uint64_t* bits, uint32_t pass,
                                                                 uint32_t* count, uint64_t tiles) {
  if (pass_trivial(bits, pass)) return;
  __shared__ uint32_t h[kDigits];
  const SortBuf in = reads_b(bits, pass) ? b : a;
  const uint64_t* word = pass >= 8 ? in.hi : in.lo;
  const uint32_t sh = (8 * pass) & 63;
  const uint64_t n = *n_dev;
  h[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t base = (uint64_t)blockIdx.x * kSortTile;
  const uint64_t last = n ? n - 1 : 0;  // element 0 exists: the buffers hold n_max >= 1
  uint64_t w[kSortItems];
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {  // unconditional (clamped) loads, issued together
    const uint64_t i = base + (uint64_t)r * kSortThreads + threadIdx.x;
    w[r] = word[i < last ? i : last];
  }
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const uint64_t i = base + (uint64_t)r * kSortThreads + threadIdx.x;
    if (i < n) atomicAdd(&h[(uint32_t)(w[r] >> sh) & 0xFFu], 1u);
  }
  __syncthreads();
  count[(uint64_t)threadIdx.x * tiles + blockIdx.x] = h[threadIdx.x];
}

// One workgroup per digit: exclusive prefix of count[d][0..tiles) in place, total to totals[d].
__global__ __launch_bounds__(kSortThreads) void sort_scan_kernel(const uint64_t* bits, uint32_t pass,
                                                                 uint32_t* count, uint64_t tiles, uint32_t* totals) {
  if (pass_trivial(bits, pass)) return;
  __shared__ uint32_t wave_sums[kSortWaves];
  uint32_t* row = count + (uint64_t)blockIdx.x * tiles;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t carry = 0;
  for (uint64_t base = 0; base < tiles; base += kSortThreads) {
    const uint64_t t = base + threadIdx.x;
    const uint32_t x = t < tiles ? row[t] : 0u;
    uint32_t incl = x;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(incl, d, 64);
      if (lane >= d) incl += y;
    }
    if (lane == 63) wave_sums[wave] = incl;
    __syncthreads();
    uint32_t before = 0, sum = 0;
#pragma unroll
    for (int w = 0; w < kSortWaves; ++w) {
      before += w < wave ? wave_sums[w] : 0u;
      sum += wave_sums[w];
    }
    __syncthreads();
    if (t < tiles) row[t] = carry + before + incl - x;
    carry += sum;
  }
  if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

// Exclusive prefix over the workgroup's 256 threads of two values at once.
__device__ __forceinline__ void block_excl_scan2(uint32_t& x, uint32_t& y, uint32_t (*tmp)[2]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t ix = x, iy = y;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t px = __shfl_up(ix, d, 64), py = __shfl_up(iy, d, 64);
    if (lane >= d) {
      ix += px;
      iy += py;
    }
  }
  if (lane == 63) {
    tmp[wave][0] = ix;
    tmp[wave][1] = iy;
  }
  __syncthreads();
  uint32_t bx = 0, by = 0;
#pragma unroll
  for (int w = 0; w < kSortWaves; ++w) {
    if (w < wave) {
      bx += tmp[w][0];
      by += tmp[w][1];
    }
  }
  x = bx + ix - x;
  y = by + iy - y;
}

template <int kWords>
__global__ __launch_bounds__(kSortThreads) void sort_scatter_kernel(SortBuf a, SortBuf b, const uint64_t* n_dev,
                                                                    const uint64_t* bits, uint32_t pass,
                                                                    const uint32_t* offset, const uint32_t* totals,
                                                                    uint64_t tiles) {
  __shared__ uint32_t run[kSortWaves][kDigits];  // per wave: running digit counts, then first local positions
  __shared__ uint32_t gdelta[kDigits];           // global position = gdelta[d] + local sorted position
  __shared__ uint32_t scan_tmp[kSortWaves][2];
  __shared__ uint64_t xch[kSortTile];            // the tile in local sorted order, one word at a time
  __shared__ uint8_t xdig[kSortTile];            // digit of each local sorted position
  const uint64_t n = *n_dev;
  const uint64_t tile0 = (uint64_t)blockIdx.x * kSortTile;
  if (tile0 >= n || pass_trivial(bits, pass)) return;  // uniform over the workgroup
  const bool from_b = reads_b(bits, pass);
  const SortBuf in = from_b ? b : a, out = from_b ? a : b;
  const uint32_t in_tile = (uint32_t)(n - tile0 < kSortTile ? n - tile0 : kSortTile);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t lt_mask = lane ? (~0ull >> (64 - lane)) : 0ull;
  const uint32_t sh = (8 * pass) & 63;
  const bool digit_in_hi = kWords == 2 && pass >= 8;

  for (int k = threadIdx.x; k < kSortWaves * kDigits; k += kSortThreads) (&run[0][0])[k] = 0;

  uint64_t lo[kSortItems], hi[kSortItems];
  uint32_t ix[kSortItems], dg[kSortItems], pos[kSortItems];
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {  // unconditional (clamped) loads, issued together
    const uint32_t li = wave * kSortWaveSpan + r * 64 + lane;
    const uint64_t at = tile0 + (li < in_tile ? li : in_tile - 1);
    lo[r] = in.lo[at];
    hi[r] = kWords == 2 ? in.hi[at] : 0;
    ix[r] = in.idx[at];
  }
  __syncthreads();  // run[] cleared

  // rank inside the wave, in element order: earlier rounds through run[wave][d], this
  // round through the peers below this lane
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const uint32_t li = wave * kSortWaveSpan + r * 64 + lane;
    const bool valid = li < in_tile;
    const uint32_t d = (uint32_t)((digit_in_hi ? hi[r] : lo[r]) >> sh) & 0xFFu;
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t ones = __ballot(valid && ((d >> bit) & 1u));
      peers &= ((d >> bit) & 1u) ? ones : ~ones;
    }
    const uint32_t below = (uint32_t)__popcll(peers & lt_mask);
    const uint32_t prior = run[wave][d];
    dg[r] = d;
    pos[r] = prior + below;
    if (valid && below == 0) run[wave][d] = prior + (uint32_t)__popcll(peers);
    wave_lds_sync();  // this round's counts before the next round's reads
  }
  __syncthreads();  // every wave's digit counts complete

  {
    const int d = threadIdx.x;
    const uint32_t c0 = run[0][d], c1 = run[1][d], c2 = run[2][d], c3 = run[3][d];
    uint32_t local = c0 + c1 + c2 + c3;  // becomes the digit's first local position
    uint32_t global = totals[d];         // becomes the digit's first global position
    block_excl_scan2(local, global, scan_tmp);
    __syncthreads();  // run[] read by every thread before it is overwritten
    run[0][d] = local;
    run[1][d] = local + c0;
    run[2][d] = local + c0 + c1;
    run[3][d] = local + c0 + c1 + c2;
    gdelta[d] = global + offset[(uint64_t)d * tiles + blockIdx.x] - local;
  }
  __syncthreads();

#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const uint32_t li = wave * kSortWaveSpan + r * 64 + lane;
    if (li < in_tile) {
      pos[r] += run[wave][dg[r]];
      xdig[pos[r]] = (uint8_t)dg[r];
      xch[pos[r]] = lo[r];
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kSortItems; ++k) {
    const uint32_t j = k * kSortThreads + threadIdx.x;
    if (j < in_tile) out.lo[gdelta[xdig[j]] + j] = xch[j];
  }
  if (kWords == 2) {
    __syncthreads();  // xch read out before it is refilled
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      const uint32_t li = wave * kSortWaveSpan + r * 64 + lane;
      if (li < in_tile) xch[pos[r]] = hi[r];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
      const uint32_t j = k * kSortThreads + threadIdx.x;
      if (j < in_tile) out.hi[gdelta[xdig[j]] + j] = xch[j];
    }
  }
  __syncthreads();
  uint32_t* xidx = reinterpret_cast<uint32_t*>(xch);
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const uint32_t li = wave * kSortWaveSpan + r * 64 + lane;
    if (li < in_tile) xidx[pos[r]] = ix[r];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kSortItems; ++k) {
    const uint32_t j = k * kSortThreads + threadIdx.x;
    if (j < in_tile) out.idx[gdelta[xdig[j]] + j] = xidx[j];
  }
}

// Sorts of at most kSortSmallMax elements run whole in one 1024-lane workgroup: every
// pass in one launch instead of three launches per pass. Wave w owns elements
// [w * 1024, (w + 1) * 1024), 16 per lane (element w * 1024 + 64 r + lane in round r).
// A pass loads the digit word of the wave's share, ranks it stably with the same
// ballots and a running per-digit count in the wave's own LDS row (so no barrier
// between rounds), and turns the row totals into each wave's offset within each digit
// and a scan over digits into each digit's first position. It then moves the elements
// one word at a time through LDS: each lane reads its elements' word again (coalesced;
// the share does not fit in registers beside the ranks) and places it at its sorted
// position in LDS, and the workgroup writes LDS out in order, so the global stores
// are coalesced (a single CU scattering 8-byte stores is slow). Passes alternate
// between the two buffers through global memory, a workgroup barrier apart, and skip
// exactly the passes the large sort skips, so the result is where sort_result() says.
constexpr int kSortSmallThreads = 1024;
constexpr int kSortSmallWaves = kSortSmallThreads / 64;
constexpr uint32_t kSortSmallMax = (uint32_t)kSortSmallThreads * kSortItems;  // 16384

// A lane's 16 elements first + 64 r of src, loaded without a guard (the buffers hold
// sort_capacity(n_max) elements, a whole number of wave spans, so a wave that holds any
// element may read its whole span), so that the loads issue together rather than as one
// guarded round trip each. Elements past n are read but never used.
template <typename T>
__device__ __forceinline__ void small_share(const T* src, uint32_t first, T (&x)[kSortItems]) {
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) x[r] = src[first + r * 64];
}

template <int kWords>
__global__ __launch_bounds__(kSortSmallThreads) void sort_small_kernel(SortBuf a, SortBuf b, const uint64_t* n_dev,
                                                                       const uint64_t* bits, uint64_t n_max) {
  __shared__ uint32_t run[kSortSmallWaves][kDigits];  // per wave: digit counts, then offsets within each digit
  __shared__ uint32_t dstart[kDigits];                 // each digit's first position
  __shared__ uint32_t wsum[kDigits / 64];
  __shared__ uint64_t xch[kSortSmallMax];              // one word of every element, in sorted order
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t lt_mask = lane ? (~0ull >> (64 - lane)) : 0ull;
  const uint32_t span0 = (uint32_t)wave * kSortWaveSpan;
  const uint64_t n_all = *n_dev;
  const uint32_t n = (uint32_t)(n_all < n_max ? n_all : n_max);
  if (n == 0) return;
  const bool has = span0 < n;  // this wave's span holds elements (uniform over the wave)
  SortBuf in = a, out = b;
  for (uint32_t pass = 0; pass < 8u * kWords; ++pass) {
    if (pass_trivial(bits, pass)) continue;  // uniform: every lane reads the same words

    const uint32_t sh = (8 * pass) & 63;
    const uint64_t* word = (kWords == 2 && pass >= 8) ? in.hi : in.lo;
    for (int k = threadIdx.x; k < kSortSmallWaves * kDigits; k += kSortSmallThreads) (&run[0][0])[k] = 0;
    uint32_t rank[kSortItems];  // (position within the wave's share of the digit) << 8 | digit
    {
      uint64_t w[kSortItems] = {};
      if (has) small_share(word, span0 + lane, w);
#pragma unroll
      for (int r = 0; r < kSortItems; ++r) rank[r] = (uint32_t)(w[r] >> sh) & 0xFFu;
    }
    __syncthreads();  // run[] cleared
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
      const bool valid = span0 + r * 64 + lane < n;
      const uint32_t d = rank[r];
      uint64_t peers = __ballot(valid);
#pragma unroll
      for (int bit = 0; bit < 8; ++bit) {
        const uint64_t ones = __ballot(valid && ((d >> bit) & 1u));
        peers &= ((d >> bit) & 1u) ? ones : ~ones;
      }
      const uint32_t below = (uint32_t)__popcll(peers & lt_mask);
      const uint32_t prior = run[wave][d];
      rank[r] = (prior + below) << 8 | d;
      if (valid && below == 0) run[wave][d] = prior + (uint32_t)__popcll(peers);
      wave_lds_sync();  // this round's counts before the next round's reads
    }
    __syncthreads();  // every wave's digit counts complete
    uint32_t tot = 0, incl = 0;
    if (threadIdx.x < kDigits) {  // digit d = threadIdx.x: each wave's offset within d
      const int d = threadIdx.x;
      for (int w = 0; w < kSortSmallWaves; ++w) {
        const uint32_t c = run[w][d];
        run[w][d] = tot;
        tot += c;
      }
      incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      if (lane == 63) wsum[wave] = incl;
    }
    __syncthreads();
    if (threadIdx.x < kDigits) {
      uint32_t before = 0;
      for (int w = 0; w < wave; ++w) before += wsum[w];
      dstart[threadIdx.x] = before + incl - tot;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {  // rank becomes the sorted position
      const uint32_t d = rank[r] & 0xFFu;
      rank[r] = dstart[d] + run[wave][d] + (rank[r] >> 8);
    }
    // move every element's words and index to its position through LDS, one array at a
    // time, so that the global stores are in order
    uint64_t x[kSortItems] = {};
    uint32_t xi[kSortItems] = {};
    if (has) {
      small_share(in.lo, span0 + lane, x);
      small_share(in.idx, span0 + lane, xi);
    }
#pragma unroll
    for (int r = 0; r < kSortItems; ++r)
      if (span0 + r * 64 + lane < n) xch[rank[r]] = x[r];
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < n; j += kSortSmallThreads) out.lo[j] = xch[j];
    if (kWords == 2) {
      if (has) small_share(in.hi, span0 + lane, x);
      __syncthreads();  // xch read out before it is refilled
#pragma unroll
      for (int r = 0; r < kSortItems; ++r)
        if (span0 + r * 64 + lane < n) xch[rank[r]] = x[r];
      __syncthreads();
      for (uint32_t j = threadIdx.x; j < n; j += kSortSmallThreads) out.hi[j] = xch[j];
    }
    __syncthreads();
    uint32_t* xidx = reinterpret_cast<uint32_t*>(xch);
#pragma unroll
    for (int r = 0; r < kSortItems; ++r)
      if (span0 + r * 64 + lane < n) xidx[rank[r]] = xi[r];
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < n; j += kSortSmallThreads) out.idx[j] = xidx[j];
    __syncthreads();  // this pass's stores visible to the workgroup before the next pass loads
    const SortBuf t = in;
    in = out;
    out = t;
  }
}

// Workspace of a sort of n elements with `words` 64-bit key words: the second key/index
// buffer (b), the digit-major tile counts and the digit totals.
struct SortLayout {
  uint64_t tiles;
  size_t hi, lo, idx, count, totals, total;
};

// Elements to allocate in each key/index buffer of a sort of at most n elements (the
// caller's buffer a too): a one-workgroup sort reads whole wave spans.
inline uint64_t sort_capacity(uint64_t n) {
  return n <= kSortSmallMax ? (n + kSortWaveSpan - 1) / kSortWaveSpan * kSortWaveSpan : n;
}

inline SortLayout sort_layout(uint64_t n_max, int words) {
  SortLayout L;
  const uint64_t n = sort_capacity(n_max);
  L.tiles = (n_max + kSortTile - 1) / kSortTile;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = (off + bytes + 255) & ~(size_t)255;
    return o;
  };
  L.hi = take(words == 2 ? 8 * n : 0);
  L.lo = take(8 * n);
  L.idx = take(4 * n);
  L.count = take(4 * (size_t)kDigits * L.tiles);
  L.totals = take(4 * kDigits);
  L.total = off;
  return L;
}

inline SortBuf sort_other(void* ws, uint64_t n_max, int words) {
  const SortLayout L = sort_layout(n_max, words);
  uint8_t* p = static_cast<uint8_t*>(ws);
  return SortBuf{words == 2 ? reinterpret_cast<uint64_t*>(p + L.hi) : nullptr, reinterpret_cast<uint64_t*>(p + L.lo),
                 reinterpret_cast<uint32_t*>(p + L.idx)};
}

// Sorts the first *n_dev (at most n_max, a device count the host does not read) pairs of
// `a` (keys of `words` 64-bit words, 1 or 2; n_max below 2^32) by key, ascending. Each
// of a's arrays holds sort_capacity(n_max) elements.
// `bits` (device u64[4], see pass_trivial) must describe those keys. The result is in `a`
// or in the workspace's buffer (sort_other), as sort_result() tells on the device. Grids
// are sized for n_max; tiles past *n_dev do nothing.
inline gleam_status radix_sort_pairs(SortBuf a, const uint64_t* n_dev, const uint64_t* bits, uint64_t n_max,
                                     int words, void* ws, hipStream_t s) {
  if (n_max == 0) return GLEAM_OK;
  if (n_max <= kSortSmallMax) {
    const SortBuf b = sort_other(ws, n_max, words);
    if (words == 2)
      hipLaunchKernelGGL(sort_small_kernel<2>, dim3(1), dim3(kSortSmallThreads), 0, s, a, b, n_dev, bits, n_max);
    else
      hipLaunchKernelGGL(sort_small_kernel<1>, dim3(1), dim3(kSortSmallThreads), 0, s, a, b, n_dev, bits, n_max);
    return launch_status("sort_small_kernel");
  }
  const SortLayout L = sort_layout(n_max, words);
  uint8_t* p = static_cast<uint8_t*>(ws);
  const SortBuf b = sort_other(ws, n_max, words);
  uint32_t* count = reinterpret_cast<uint32_t*>(p + L.count);
  uint32_t* totals = reinterpret_cast<uint32_t*>(p + L.totals);
  const uint32_t passes = 8u * (uint32_t)words;
  for (uint32_t q = 0; q < passes; ++q) {
    hipLaunchKernelGGL(sort_hist_kernel, dim3((uint32_t)L.tiles), dim3(kSortThreads), 0, s, a, b, n_dev, bits, q,
                       count, L.tiles);
    gleam_status st = launch_status("sort_hist_kernel");
    if (st != GLEAM_OK) return st;
    hipLaunchKernelGGL(sort_scan_kernel, dim3(kDigits), dim3(kSortThreads), 0, s, bits, q, count, L.tiles, totals);
    if ((st = launch_status("sort_scan_kernel")) != GLEAM_OK) return st;
    if (words == 2)
      hipLaunchKernelGGL(sort_scatter_kernel<2>, dim3((uint32_t)L.tiles), dim3(kSortThreads), 0, s, a, b, n_dev, bits,
                         q, count, totals, L.tiles);
    else
      hipLaunchKernelGGL(sort_scatter_kernel<1>, dim3((uint32_t)L.tiles), dim3(kSortThreads), 0, s, a, b, n_dev, bits,
                         q, count, totals, L.tiles);
    if ((st = launch_status("sort_scatter_kernel")) != GLEAM_OK) return st;
  }
  return GLEAM_OK;
}

}  // namespace
}  // namespace gleam
