// gleam_miss_compact: the blocks whose bytes must still travel (Gleam Sec. 4.1.2:
// on a miss the full chunk is transmitted), as an ascending index list, its length
// and its byte total.
//
// Order-preserving stream compaction. Up to kSmallItems statuses (and payloads), one
// 1024-thread workgroup does it all in one launch: rounds of 16 statuses per thread,
// a workgroup scan per round, and a workgroup sum for the short-block bytes. Larger
// inputs are cut into tiles of 2048 statuses. Up to kPrefixTiles tiles take two passes:
// a tally (count per tile, and the short-block bytes summed per workgroup over a grid
// wide enough for one payload per thread), then each tile sums the counts before it and
// writes its MISS indices at that offset using a workgroup scan of per-thread counts.
// More tiles take three passes: count per tile, one-workgroup exclusive scan of the
// tile counts, then the same per-tile writes.
// Byte total = count * block_bytes minus, for every payload whose short last block is
// a MISS, the part of that block that does not exist.
// All sums are integer, so the results do not depend on thread timing.

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = (int)(kTileItems / kThreads);  // 8 statuses per thread
constexpr int kScanThreads = 1024;
constexpr int kSmallPerThread = 16;
constexpr uint64_t kSmallItems = 1u << 16;  // single-workgroup path up to this many statuses

// Bit e set: status first + e is a MISS (first + e < n). The loads are unconditional,
// at indices clamped to the last status (n >= 1), so a thread's loads issue together: a
// guarded load per status compiles to one round trip each.
template <int kCount>
__device__ __forceinline__ uint32_t miss_bits(const uint8_t* status, uint64_t n, uint64_t first) {
  uint8_t v[kCount];
#pragma unroll
  for (int e = 0; e < kCount; ++e) {
    const uint64_t g = first + e;
    v[e] = status[g < n ? g : n - 1];
  }
  uint32_t bits = 0;
#pragma unroll
  for (int e = 0; e < kCount; ++e) bits |= (first + e < n && v[e] == GLEAM_MISS) ? (1u << e) : 0u;
  return bits;
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  return x;
}

// Exclusive scan of one value per thread over a workgroup of `waves` waves.
// Returns the exclusive prefix; *total receives the workgroup sum.
template <int kWaves>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* wave_sums, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t incl = wave_inclusive_scan(x, lane);
  if (lane == 63) wave_sums[wave] = incl;
  __syncthreads();
  uint32_t before = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t s = wave_sums[w];
    before += w < wave ? s : 0u;
    sum += s;
  }
  __syncthreads();
  *total = sum;
  return before + incl - x;
}

__global__ __launch_bounds__(kThreads) void compact_count_kernel(const uint8_t* status, uint64_t n,
                                                                 uint64_t* tile_counts) {
  __shared__ uint32_t wave_sums[kThreads / 64];
  const uint64_t first = (uint64_t)blockIdx.x * kTileItems + (uint64_t)threadIdx.x * kPerThread;
  const uint32_t c = (uint32_t)__builtin_popcount(miss_bits<kPerThread>(status, n, first));
  uint32_t total;
  block_exclusive_scan<kThreads / 64>(c, wave_sums, &total);
  if (threadIdx.x == 0) tile_counts[blockIdx.x] = total;
}

__global__ __launch_bounds__(kScanThreads) void compact_scan_kernel(const uint64_t* tile_counts, uint64_t tiles,
                                                                    uint64_t* tile_offsets, uint64_t* miss_count,
                                                                    uint64_t* miss_bytes, uint64_t block_bytes) {
  __shared__ uint32_t wave_sums[kScanThreads / 64];
  uint64_t carry = 0;
  for (uint64_t base = 0; base < tiles; base += kScanThreads) {
    const uint64_t t = base + threadIdx.x;
    const uint32_t c = t < tiles ? (uint32_t)tile_counts[t] : 0u;
    uint32_t total;
    const uint32_t excl = block_exclusive_scan<kScanThreads / 64>(c, wave_sums, &total);
    if (t < tiles) tile_offsets[t] = carry + excl;
    carry += total;
  }
  if (threadIdx.x == 0) {
    *miss_count = carry;
    if (miss_bytes) *miss_bytes = carry * block_bytes;
  }
}

struct ShortBlocks {  // payload geometry for the byte total; seg_len == nullptr: not wanted
  const uint64_t* seg_len;
  const uint64_t* blk_first;
  uint64_t n_seg;
  uint64_t block_bytes;
  uint64_t* miss_bytes;
};

// Writes the tile's MISS indices at its offset; also subtracts, for every payload of its
// grid-stride share whose last block is short and a MISS, the bytes that block lacks.
__global__ __launch_bounds__(kThreads) void compact_scatter_kernel(const uint8_t* status, uint64_t n,
                                                                   const uint64_t* tile_offsets,
                                                                   uint64_t* miss_idx, ShortBlocks sb) {
  __shared__ uint32_t wave_sums[kThreads / 64];
  const uint64_t first = (uint64_t)blockIdx.x * kTileItems + (uint64_t)threadIdx.x * kPerThread;
  const uint32_t bits = miss_bits<kPerThread>(status, n, first);
  uint32_t total;
  const uint32_t excl = block_exclusive_scan<kThreads / 64>((uint32_t)__builtin_popcount(bits), wave_sums, &total);
  uint64_t out = tile_offsets[blockIdx.x] + excl;
  for (uint32_t m = bits; m; m &= m - 1) miss_idx[out++] = first + (uint64_t)__builtin_ctz(m);
  if (!sb.seg_len) return;
  // the grid strides over all payloads (a per-tile range would need a binary search of
  // blk_first: a chain of dependent reads)
  uint64_t deficit = 0;
  const uint64_t stride = (uint64_t)gridDim.x * kThreads;
  for (uint64_t s = (uint64_t)blockIdx.x * kThreads + threadIdx.x; s < sb.n_seg; s += stride) {
    const uint64_t b0 = sb.blk_first[s], b1 = sb.blk_first[s + 1];
    if (b1 <= b0 || b1 - 1 >= n || status[b1 - 1] != GLEAM_MISS) continue;
    const uint64_t last_len = sb.seg_len[s] - (b1 - b0 - 1) * sb.block_bytes;
    if (last_len < sb.block_bytes) deficit += sb.block_bytes - last_len;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint32_t lo32 = __shfl_xor((uint32_t)deficit, o, 64);
    const uint32_t hi32 = __shfl_xor((uint32_t)(deficit >> 32), o, 64);
    deficit += ((uint64_t)hi32 << 32) | lo32;
  }
  if ((threadIdx.x & 63) == 0 && deficit)
    atomicAdd(reinterpret_cast<unsigned long long*>(sb.miss_bytes), (unsigned long long)(0 - deficit));
}

// ---- Two launches for up to kPrefixTiles tiles -------------------------------------
// Pass 1 (tally): workgroups below `tiles` count their tile's MISS statuses; every
// workgroup also sums, over its grid-stride share of payloads, the bytes that a short
// last block which is a MISS lacks, into deficits[blockIdx.x] (the grid is made wide
// enough that most threads take one payload). Pass 2 (place): each tile sums the counts
// of the tiles before it for its offset and writes its MISS indices; the last tile
// writes the count and the byte total.
constexpr uint64_t kPrefixTiles = 1024;
constexpr uint64_t kMaxDeficitGroups = 1024;

__device__ __forceinline__ uint64_t block_sum64(uint64_t x, uint64_t* wave_parts) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += shfl_xor64(x, o);
  if ((threadIdx.x & 63) == 0) wave_parts[threadIdx.x >> 6] = x;
  __syncthreads();
  uint64_t s = 0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) s += wave_parts[w];
  __syncthreads();
  return s;
}

__global__ __launch_bounds__(kThreads) void compact_tally_kernel(const uint8_t* status, uint64_t n, uint64_t tiles,
                                                                 uint64_t* tile_counts, uint64_t* deficits,
                                                                 ShortBlocks sb) {
  __shared__ uint32_t wave_sums[kThreads / 64];
  __shared__ uint64_t wave_parts[kThreads / 64];
  if (blockIdx.x < tiles) {
    const uint64_t first = (uint64_t)blockIdx.x * kTileItems + (uint64_t)threadIdx.x * kPerThread;
    uint32_t total;
    block_exclusive_scan<kThreads / 64>((uint32_t)__builtin_popcount(miss_bits<kPerThread>(status, n, first)),
                                        wave_sums, &total);
    if (threadIdx.x == 0) tile_counts[blockIdx.x] = total;
  }
  if (!sb.seg_len) return;
  uint64_t deficit = 0;
  const uint64_t stride = (uint64_t)gridDim.x * kThreads;
  for (uint64_t s = (uint64_t)blockIdx.x * kThreads + threadIdx.x; s < sb.n_seg; s += stride) {
    const uint64_t b0 = sb.blk_first[s], b1 = sb.blk_first[s + 1], len = sb.seg_len[s];
    if (b1 <= b0 || b1 - 1 >= n || status[b1 - 1] != GLEAM_MISS) continue;
    const uint64_t last_len = len - (b1 - b0 - 1) * sb.block_bytes;
    if (last_len < sb.block_bytes) deficit += sb.block_bytes - last_len;
  }
  deficit = block_sum64(deficit, wave_parts);
  if (threadIdx.x == 0) deficits[blockIdx.x] = deficit;
}

__global__ __launch_bounds__(kThreads) void compact_place_kernel(const uint8_t* status, uint64_t n, uint64_t tiles,
                                                                 const uint64_t* tile_counts, const uint64_t* deficits,
                                                                 uint64_t n_parts, uint64_t* miss_idx,
                                                                 uint64_t* miss_count, uint64_t* miss_bytes,
                                                                 uint64_t block_bytes) {
  __shared__ uint32_t wave_sums[kThreads / 64];
  __shared__ uint64_t wave_parts[kThreads / 64];
  uint64_t before = 0;
  for (uint64_t t = threadIdx.x; t < blockIdx.x; t += kThreads) before += tile_counts[t];
  before = block_sum64(before, wave_parts);
  const uint64_t first = (uint64_t)blockIdx.x * kTileItems + (uint64_t)threadIdx.x * kPerThread;
  const uint32_t bits = miss_bits<kPerThread>(status, n, first);
  uint32_t total;
  const uint32_t excl = block_exclusive_scan<kThreads / 64>((uint32_t)__builtin_popcount(bits), wave_sums, &total);
  uint64_t out = before + excl;
  for (uint32_t m = bits; m; m &= m - 1) miss_idx[out++] = first + (uint64_t)__builtin_ctz(m);
  if (blockIdx.x + 1 != tiles) return;
  uint64_t d = 0;
  if (miss_bytes)
    for (uint64_t w = threadIdx.x; w < n_parts; w += kThreads) d += deficits[w];
  d = block_sum64(d, wave_parts);
  if (threadIdx.x == 0) {
    const uint64_t count = before + total;
    *miss_count = count;
    if (miss_bytes) *miss_bytes = count * block_bytes - d;
  }
}

// Inputs of up to kSmallItems statuses and payloads: count, scan, scatter and byte total
// in one workgroup (launch count is what such sizes pay for, not bytes). `sb` is used
// only when n > 0; *miss_bytes (nullable) gets the byte total.
__global__ __launch_bounds__(kScanThreads) void compact_small_kernel(const uint8_t* status, uint64_t n,
                                                                     uint64_t* miss_idx, uint64_t* miss_count,
                                                                     uint64_t* miss_bytes, uint64_t block_bytes,
                                                                     ShortBlocks sb) {
  __shared__ uint32_t wave_sums[kScanThreads / 64];
  __shared__ uint64_t deficits[kScanThreads / 64];
  const bool vec = (reinterpret_cast<uintptr_t>(status) & 15) == 0;
  uint64_t carry = 0;
  for (uint64_t base = 0; base < n; base += (uint64_t)kScanThreads * kSmallPerThread) {
    const uint64_t first = base + (uint64_t)threadIdx.x * kSmallPerThread;
    uint32_t bits = 0;
    if (vec && first + kSmallPerThread <= n) {
      const uint4 v = *reinterpret_cast<const uint4*>(status + first);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < kSmallPerThread; ++e)
        bits |= ((w[e >> 2] >> (8 * (e & 3))) & 0xFFu) == GLEAM_MISS ? (1u << e) : 0u;
    } else if (first < n) {
      bits = miss_bits<kSmallPerThread>(status, n, first);
    }
    uint32_t total;
    const uint32_t excl = block_exclusive_scan<kScanThreads / 64>((uint32_t)__builtin_popcount(bits), wave_sums,
                                                                   &total);
    uint64_t out = carry + excl;
    for (uint32_t m = bits; m; m &= m - 1) miss_idx[out++] = first + (uint64_t)__builtin_ctz(m);
    carry += total;
  }
  const bool short_blocks = miss_bytes && n > 0;
  if (short_blocks) {
    uint64_t deficit = 0;
    for (uint64_t s = threadIdx.x; s < sb.n_seg; s += kScanThreads) {
      const uint64_t b0 = sb.blk_first[s], b1 = sb.blk_first[s + 1];
      if (b1 <= b0 || b1 - 1 >= n || status[b1 - 1] != GLEAM_MISS) continue;
      const uint64_t last_len = sb.seg_len[s] - (b1 - b0 - 1) * block_bytes;
      if (last_len < block_bytes) deficit += block_bytes - last_len;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) deficit += shfl_xor64(deficit, o);
    if ((threadIdx.x & 63) == 0) deficits[threadIdx.x >> 6] = deficit;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    *miss_count = carry;
    if (miss_bytes) {
      uint64_t d = 0;
      if (short_blocks)
        for (int w = 0; w < kScanThreads / 64; ++w) d += deficits[w];
      *miss_bytes = carry * block_bytes - d;
    }
  }
}

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_compact() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&compact_scan_kernel));
}

}  // namespace gleam

extern "C" gleam_status gleam_miss_compact(const uint8_t* d_status, uint64_t n, const gleam_batch* b,
                                           uint64_t* d_miss_idx, uint64_t* d_miss_count, uint64_t* d_miss_bytes,
                                           void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  if (!d_miss_count || (n > 0 && (!d_status || !d_miss_idx))) {
    set_error("gleam_miss_compact: null status, index list or count");
    return GLEAM_E_INVALID;
  }
  if (d_miss_bytes) {
    if (!b || b->n_blocks != n || !valid_block_bytes(b->block_bytes)) {
      set_error("gleam_miss_compact: miss_bytes needs the batch of these n statuses");
      return GLEAM_E_INVALID;
    }
    if (n > 0 && (b->n_seg == 0 || !b->seg_len || !b->blk_first)) {
      set_error("gleam_miss_compact: null batch descriptor");
      return GLEAM_E_INVALID;
    }
  }
  const WsLayout L = ws_layout(n);
  gleam_status st = check_workspace(L, d_ws, ws_bytes, "gleam_miss_compact");
  if (st != GLEAM_OK) return st;
  if (L.tiles > 0x7fffffffull) {
    set_error("gleam_miss_compact: more than 2^31 tiles");
    return GLEAM_E_UNSUPPORTED;
  }
  hipStream_t s = (hipStream_t)stream;
  // (n == 0 always goes here: the tiled paths need at least one tile, and a batch of
  // only empty payloads may be longer than kSmallItems)
  if (n == 0 || (n <= kSmallItems && (!d_miss_bytes || b->n_seg <= kSmallItems))) {
    ShortBlocks sb{nullptr, nullptr, 0, 0, nullptr};
    if (d_miss_bytes) sb = ShortBlocks{b->seg_len, b->blk_first, b->n_seg, b->block_bytes, d_miss_bytes};
    hipLaunchKernelGGL(compact_small_kernel, dim3(1), dim3(kScanThreads), 0, s, d_status, n,
                       d_miss_idx, d_miss_count, d_miss_bytes, (uint64_t)(d_miss_bytes ? b->block_bytes : 0), sb);
    return launch_status("compact_small_kernel");
  }
  uint64_t* counts = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(d_ws) + L.tiles_off);
  uint64_t* offsets = counts + L.tiles;
  const uint64_t block_bytes = d_miss_bytes ? b->block_bytes : 0;
  if (L.tiles <= kPrefixTiles) {
    // deficit partials go to the scratch table's words, which compaction does not use
    uint64_t n_def = 0;
    if (d_miss_bytes) {
      n_def = (b->n_seg + kThreads - 1) / kThreads;
      if (n_def > kMaxDeficitGroups) n_def = kMaxDeficitGroups;
      if (n_def > L.scratch_cap) n_def = L.scratch_cap;
    }
    uint64_t* deficits = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(d_ws) + L.scratch_off);
    ShortBlocks sb{nullptr, nullptr, 0, 0, nullptr};
    if (d_miss_bytes) sb = ShortBlocks{b->seg_len, b->blk_first, b->n_seg, block_bytes, d_miss_bytes};
    const uint64_t grid = L.tiles > n_def ? L.tiles : n_def;
    hipLaunchKernelGGL(compact_tally_kernel, dim3((uint32_t)grid), dim3(kThreads), 0, s, d_status, n, L.tiles,
                       counts, deficits, sb);
    if ((st = launch_status("compact_tally_kernel")) != GLEAM_OK) return st;
    // every tally workgroup writes a partial (grid <= max(kPrefixTiles, kMaxDeficitGroups),
    // and tiles <= n <= scratch_cap / 2, so the partials fit in the scratch words)
    hipLaunchKernelGGL(compact_place_kernel, dim3((uint32_t)L.tiles), dim3(kThreads), 0, s, d_status, n, L.tiles,
                       counts, deficits, d_miss_bytes ? grid : 0, d_miss_idx, d_miss_count, d_miss_bytes,
                       block_bytes);
    return launch_status("compact_place_kernel");
  }
  hipLaunchKernelGGL(compact_count_kernel, dim3((uint32_t)L.tiles), dim3(kThreads), 0, s, d_status, n, counts);
  if ((st = launch_status("compact_count_kernel")) != GLEAM_OK) return st;
  hipLaunchKernelGGL(compact_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, counts, L.tiles, offsets, d_miss_count,
                     d_miss_bytes, block_bytes);
  if ((st = launch_status("compact_scan_kernel")) != GLEAM_OK) return st;
  ShortBlocks sb{nullptr, nullptr, 0, 0, nullptr};
  if (d_miss_bytes) sb = ShortBlocks{b->seg_len, b->blk_first, b->n_seg, block_bytes, d_miss_bytes};
  hipLaunchKernelGGL(compact_scatter_kernel, dim3((uint32_t)L.tiles), dim3(kThreads), 0, s, d_status, n, offsets,
                     d_miss_idx, sb);
  return launch_status("compact_scatter_kernel");
}
