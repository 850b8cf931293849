// The data path around the decision (Gleam Sec. 4.1.2): the sender turns each block's
// status into a record, packs the bytes that must travel into one buffer, and the
// receiver rebuilds every payload from the records, that buffer and the bytes it
// already holds.
//
//   gleam_send_plan       one record per block; MISS blocks get 16-byte-aligned offsets
//                         in the packed buffer (an order-preserving scan of lengths)
//   gleam_pack_misses     copy every MISS block's bytes to its offset
//   gleam_restore_blocks  write every block of the destination payloads: MISS from the
//                         packed buffer, HIT_CACHE from the holder's copy, HIT_BATCH from
//                         the packed bytes of the earlier block it repeats
//
// The copies are HBM-bound: one read and one write per byte moved.

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = (int)(kTileItems / kThreads);  // 8 blocks per thread
constexpr int kScanThreads = 1024;
// Copy grid: one workgroup per 64 KiB item up to 2^24 items (1 TiB), a grid-stride loop
// beyond. Measured on a 4 GiB copy (read + write traffic): one workgroup per item 5.48 TB/s;
// a persistent grid of 1-16 workgroups per CU 4.9-5.3 TB/s; hipMemcpyAsync 4.68 TB/s.
constexpr uint32_t kMaxCopyGrid = 1u << 24;
constexpr uint64_t kChunk = 64 << 10;  // copy work item: up to 64 KiB of one block

__device__ __forceinline__ uint64_t round16(uint64_t n) { return (n + 15) & ~15ull; }

__device__ __forceinline__ uint64_t wave_inclusive_scan64(uint64_t x, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t lo = __shfl_up((uint32_t)x, d, 64);
    const uint32_t hi = __shfl_up((uint32_t)(x >> 32), d, 64);
    if (lane >= d) x += ((uint64_t)hi << 32) | lo;
  }
  return x;
}

// Exclusive scan of one u64 per thread over a workgroup of kWaves waves.
template <int kWaves>
__device__ __forceinline__ uint64_t block_exclusive_scan64(uint64_t x, uint64_t* wave_sums, uint64_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t incl = wave_inclusive_scan64(x, lane);
  if (lane == 63) wave_sums[wave] = incl;
  __syncthreads();
  uint64_t before = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint64_t s = wave_sums[w];
    before += w < wave ? s : 0;
    sum += s;
  }
  __syncthreads();
  *total = sum;
  return before + incl - x;
}

struct Geo {
  const uint64_t* seg_len;
  const uint64_t* blk_first;
  uint64_t n_seg;
  uint64_t n_blocks;
  uint64_t block_bytes;
};

// Walks consecutive blocks from `g`, tracking their payload.
struct BlockWalker {
  const Geo& geo;
  uint64_t s;
  __device__ BlockWalker(const Geo& gg, uint64_t g) : geo(gg), s(find_segment(gg.blk_first, gg.n_seg, g)) {}
  __device__ void at(uint64_t g, uint64_t* payload, uint64_t* offset, uint64_t* length) {
    while (s + 1 < geo.n_seg && geo.blk_first[s + 1] <= g) ++s;
    const uint64_t j = g - geo.blk_first[s];
    const uint64_t start = j * geo.block_bytes;
    const uint64_t len_s = geo.seg_len[s];
    *payload = s;
    *offset = start;
    *length = start < len_s ? min(len_s - start, geo.block_bytes) : 0;
  }
};

// Per tile: MISS/HIT_CACHE/HIT_BATCH counts and the packed bytes of its MISS blocks.
__global__ __launch_bounds__(kThreads) void plan_tile_kernel(Geo geo, const uint8_t* status, uint64_t* tiles) {
  __shared__ uint64_t sums[kThreads / 64];
  const uint64_t first = (uint64_t)blockIdx.x * kTileItems + (uint64_t)threadIdx.x * kPerThread;
  uint64_t miss = 0, hit = 0, dup = 0, bytes = 0;
  if (first < geo.n_blocks) {
    BlockWalker w(geo, first);
    for (int e = 0; e < kPerThread; ++e) {
      const uint64_t g = first + e;
      if (g >= geo.n_blocks) break;
      uint64_t s, off, len;
      w.at(g, &s, &off, &len);
      const uint8_t st = status[g];
      if (st == GLEAM_MISS) {
        ++miss;
        bytes += round16(len);
      } else if (st == GLEAM_HIT_CACHE) {
        ++hit;
      } else {
        ++dup;
      }
    }
  }
  uint64_t total;
  block_exclusive_scan64<kThreads / 64>(bytes, sums, &total);
  const uint64_t counts = miss | (hit << 21) | (dup << 42);  // <= 2048 each per tile
  uint64_t packed_counts;
  block_exclusive_scan64<kThreads / 64>(counts, sums, &packed_counts);
  if (threadIdx.x == 0) {
    tiles[2 * blockIdx.x] = total;
    tiles[2 * blockIdx.x + 1] = packed_counts;
  }
}

// One workgroup: tile byte offsets (exclusive) and the totals.
__global__ __launch_bounds__(kScanThreads) void plan_scan_kernel(uint64_t* tiles, uint64_t n_tiles, uint64_t* offs,
                                                                 uint64_t* totals) {
  __shared__ uint64_t sums[kScanThreads / 64];
  uint64_t carry = 0, miss = 0, hit = 0, dup = 0;
  for (uint64_t base = 0; base < n_tiles; base += kScanThreads) {
    const uint64_t t = base + threadIdx.x;
    const uint64_t b = t < n_tiles ? tiles[2 * t] : 0;
    const uint64_t c = t < n_tiles ? tiles[2 * t + 1] : 0;
    uint64_t total;
    const uint64_t excl = block_exclusive_scan64<kScanThreads / 64>(b, sums, &total);
    if (t < n_tiles) offs[t] = carry + excl;
    carry += total;
    uint64_t m = c & ((1ull << 21) - 1), h = (c >> 21) & ((1ull << 21) - 1), d = c >> 42, sum;
    block_exclusive_scan64<kScanThreads / 64>(m, sums, &sum);
    miss += sum;
    block_exclusive_scan64<kScanThreads / 64>(h, sums, &sum);
    hit += sum;
    block_exclusive_scan64<kScanThreads / 64>(d, sums, &sum);
    dup += sum;
  }
  if (threadIdx.x == 0) {
    totals[0] = miss;
    totals[1] = hit;
    totals[2] = dup;
    totals[3] = carry;
  }
}

__global__ __launch_bounds__(kThreads) void plan_write_kernel(Geo geo, const uint64_t* digest, const uint8_t* status,
                                                              const uint64_t* ref, const uint64_t* tile_offs,
                                                              gleam_send_record* rec) {
  __shared__ uint64_t sums[kThreads / 64];
  const uint64_t first = (uint64_t)blockIdx.x * kTileItems + (uint64_t)threadIdx.x * kPerThread;
  uint64_t mine = 0;
  if (first < geo.n_blocks) {
    BlockWalker w(geo, first);
    for (int e = 0; e < kPerThread; ++e) {
      const uint64_t g = first + e;
      if (g >= geo.n_blocks) break;
      uint64_t s, off, len;
      w.at(g, &s, &off, &len);
      if (status[g] == GLEAM_MISS) mine += round16(len);
    }
  }
  uint64_t total;
  uint64_t pos = tile_offs[blockIdx.x] + block_exclusive_scan64<kThreads / 64>(mine, sums, &total);
  if (first >= geo.n_blocks) return;
  BlockWalker w(geo, first);
  for (int e = 0; e < kPerThread; ++e) {
    const uint64_t g = first + e;
    if (g >= geo.n_blocks) break;
    uint64_t s, off, len;
    w.at(g, &s, &off, &len);
    const uint8_t st = status[g];
    gleam_send_record r;
    r.block = g;
    r.payload = s;
    r.offset = off;
    r.length = (uint32_t)len;
    r.kind = st;
    if (st == GLEAM_MISS) {
      r.ident = pos;
      pos += round16(len);
    } else if (st == GLEAM_HIT_CACHE) {
      r.ident = digest[g];
    } else {
      r.ident = ref[g];
    }
    rec[g] = r;
  }
}

// Copy len bytes with the whole workgroup: 16-byte non-temporal words from either end's
// start at any alignment (gfx950 under HSA runs with unaligned access enabled; each word
// covers 16 bytes of the range, so every byte is touched once and none outside it), then
// the last len mod 16 bytes one by one.
typedef u32x4 u32x4_any __attribute__((aligned(1)));
__device__ __forceinline__ void wg_copy(uint8_t* dst, const uint8_t* src, uint64_t len) {
  const uint64_t words = len >> 4;
  u32x4_any* d = reinterpret_cast<u32x4_any*>(dst);
  const u32x4_any* s = reinterpret_cast<const u32x4_any*>(src);
  uint64_t i = threadIdx.x;
  for (; i + 3 * kThreads < words; i += 4 * kThreads) {
    const u32x4 a = __builtin_nontemporal_load(s + i);
    const u32x4 b = __builtin_nontemporal_load(s + i + kThreads);
    const u32x4 c = __builtin_nontemporal_load(s + i + 2 * kThreads);
    const u32x4 e = __builtin_nontemporal_load(s + i + 3 * kThreads);
    __builtin_nontemporal_store(a, d + i);
    __builtin_nontemporal_store(b, d + i + kThreads);
    __builtin_nontemporal_store(c, d + i + 2 * kThreads);
    __builtin_nontemporal_store(e, d + i + 3 * kThreads);
  }
  for (; i < words; i += kThreads) __builtin_nontemporal_store(__builtin_nontemporal_load(s + i), d + i);
  for (uint64_t k = (words << 4) + threadIdx.x; k < len; k += kThreads) dst[k] = src[k];
}

// [at, at + len) lies inside [0, size), without overflow.
__device__ __forceinline__ bool inside(uint64_t at, uint64_t len, uint64_t size) {
  return at <= size && len <= size - at;
}

// The record's block lies inside its payload of the batch.
__device__ __forceinline__ bool block_in_batch(const gleam_send_record& r, const uint64_t* seg_len, uint64_t n_seg) {
  return r.payload < n_seg && inside(r.offset, r.length, seg_len[r.payload]);
}

// Work items: (block, 64 KiB chunk of it); `per_block` chunks per block. Records whose
// block is not inside its payload, or whose bytes are not inside the packed buffer, are
// skipped.
__global__ __launch_bounds__(kThreads) void pack_kernel(const uint64_t* seg_addr, const uint64_t* seg_len,
                                                        uint64_t n_seg, const gleam_send_record* rec, uint64_t n,
                                                        uint64_t per_block, uint8_t* out, uint64_t out_bytes) {
  for (uint64_t item = blockIdx.x; item < n * per_block; item += gridDim.x) {
    const uint64_t g = item / per_block, c0 = (item % per_block) * kChunk;
    const gleam_send_record r = rec[g];
    if (r.kind != GLEAM_MISS || c0 >= r.length || !inside(r.ident, r.length, out_bytes) ||
        !block_in_batch(r, seg_len, n_seg))
      continue;
    const uint64_t len = min((uint64_t)r.length - c0, kChunk);
    wg_copy(out + r.ident + c0, reinterpret_cast<const uint8_t*>(seg_addr[r.payload]) + r.offset + c0, len);
  }
}

__global__ __launch_bounds__(kThreads) void restore_kernel(const uint64_t* dst_addr, const uint64_t* dst_len,
                                                           uint64_t n_seg, const gleam_send_record* rec, uint64_t n,
                                                           uint64_t per_block, const uint8_t* packed,
                                                           uint64_t packed_bytes, const uint64_t* held) {
  for (uint64_t item = blockIdx.x; item < n * per_block; item += gridDim.x) {
    const uint64_t g = item / per_block, c0 = (item % per_block) * kChunk;
    // the held address does not depend on the record: read both at once, so the range
    // check of the record is the only dependent read before the copy
    const uint64_t held_addr = held ? held[g] : 0;
    const gleam_send_record r = rec[g];
    if (c0 >= r.length || !block_in_batch(r, dst_len, n_seg)) continue;
    const uint8_t* src = nullptr;
    if (r.kind == GLEAM_MISS) {
      if (inside(r.ident, r.length, packed_bytes)) src = packed + r.ident;
    } else if (r.kind == GLEAM_HIT_CACHE) {
      src = reinterpret_cast<const uint8_t*>(held_addr);
    } else if (r.kind == GLEAM_HIT_BATCH && r.ident < n) {
      const gleam_send_record first = rec[r.ident];
      if (first.kind == GLEAM_MISS && first.length == r.length && inside(first.ident, r.length, packed_bytes))
        src = packed + first.ident;
    }
    if (!src) continue;
    const uint64_t len = min((uint64_t)r.length - c0, kChunk);
    wg_copy(reinterpret_cast<uint8_t*>(dst_addr[r.payload]) + r.offset + c0, src + c0, len);
  }
}

uint32_t copy_grid(uint64_t n) { return (uint32_t)(n < kMaxCopyGrid ? (n ? n : 1) : kMaxCopyGrid); }
uint64_t chunks_per_block(uint32_t block_bytes) { return block_bytes > kChunk ? block_bytes / kChunk : 1; }

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_transfer() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&plan_scan_kernel));
}

}  // namespace gleam

extern "C" gleam_status gleam_send_plan(const gleam_batch* b, const uint64_t* d_digest, const uint8_t* d_status,
                                        const uint64_t* d_ref, gleam_send_record* d_records, uint64_t* d_totals,
                                        void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  gleam_status st = validate_batch(b, "gleam_send_plan");
  if (st != GLEAM_OK) return st;
  if (!d_totals || (b->n_blocks > 0 && (!d_digest || !d_status || !d_ref || !d_records))) {
    set_error("gleam_send_plan: null input or output");
    return GLEAM_E_INVALID;
  }
  const WsLayout L = ws_layout(b->n_blocks);
  st = check_workspace(L, d_ws, ws_bytes, "gleam_send_plan");
  if (st != GLEAM_OK) return st;
  if (L.tiles > 0x7fffffffull) {
    set_error("gleam_send_plan: more than 2^31 tiles");
    return GLEAM_E_UNSUPPORTED;
  }
  hipStream_t s = (hipStream_t)stream;
  uint64_t* tiles = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(d_ws) + L.scratch_off);
  uint64_t* offs = tiles + 2 * L.tiles;
  const Geo geo{b->seg_len, b->blk_first, b->n_seg, b->n_blocks, b->block_bytes};
  if (b->n_blocks > 0) {
    hipLaunchKernelGGL(plan_tile_kernel, dim3((uint32_t)L.tiles), dim3(kThreads), 0, s, geo, d_status, tiles);
    if ((st = launch_status("plan_tile_kernel")) != GLEAM_OK) return st;
  }
  hipLaunchKernelGGL(plan_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, tiles, L.tiles, offs, d_totals);
  if ((st = launch_status("plan_scan_kernel")) != GLEAM_OK) return st;
  if (b->n_blocks == 0) return GLEAM_OK;
  hipLaunchKernelGGL(plan_write_kernel, dim3((uint32_t)L.tiles), dim3(kThreads), 0, s, geo, d_digest, d_status, d_ref,
                     offs, d_records);
  return launch_status("plan_write_kernel");
}

extern "C" gleam_status gleam_pack_misses(const gleam_batch* b, const gleam_send_record* d_records, uint8_t* d_out,
                                          uint64_t out_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  gleam_status st = validate_batch(b, "gleam_pack_misses");
  if (st != GLEAM_OK) return st;
  if (b->n_blocks == 0) return GLEAM_OK;
  if (!d_records || (!d_out && out_bytes > 0)) {
    set_error("gleam_pack_misses: null records or output");
    return GLEAM_E_INVALID;
  }
  const uint64_t per = chunks_per_block(b->block_bytes);
  hipLaunchKernelGGL(pack_kernel, dim3(copy_grid(b->n_blocks * per)), dim3(kThreads), 0, (hipStream_t)stream,
                     b->seg_addr, b->seg_len, b->n_seg, d_records, b->n_blocks, per, d_out, out_bytes);
  return launch_status("pack_kernel");
}

extern "C" gleam_status gleam_restore_blocks(const gleam_batch* dst, const gleam_send_record* d_records,
                                             const uint8_t* d_packed, uint64_t packed_bytes, const uint64_t* d_held,
                                             void* stream) {
  using namespace gleam;
  clear_error();
  gleam_status st = validate_batch(dst, "gleam_restore_blocks");
  if (st != GLEAM_OK) return st;
  if (dst->n_blocks == 0) return GLEAM_OK;
  if (!d_records || (!d_packed && packed_bytes > 0)) {
    set_error("gleam_restore_blocks: null records or packed buffer");
    return GLEAM_E_INVALID;
  }
  const uint64_t per = chunks_per_block(dst->block_bytes);
  hipLaunchKernelGGL(restore_kernel, dim3(copy_grid(dst->n_blocks * per)), dim3(kThreads), 0, (hipStream_t)stream,
                     dst->seg_addr, dst->seg_len, dst->n_seg, d_records, dst->n_blocks, per, d_packed, packed_bytes,
                     d_held);
  return launch_status("restore_kernel");
}
