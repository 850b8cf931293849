// Leaf hashing shared by the gfx950 fingerprint kernels (gleam_fp_chunks and the
// one-launch gleam_detect): XXH64 (seed 0) of 4 KiB leaves streamed through per-wave
// LDS tiles, two lanes per leaf (fp_kernel) or four (the small-batch kernels), and the
// tree steps inside a wave. The kernels and their launch choices are in fp_chunks.hip
// and detect.hip; this header holds only device code (an anonymous namespace, so each
// translation unit has its own copy).
#pragma once

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

// Streaming 16-byte load at any byte address. Under HSA, gfx950 runs with unaligned
// access enabled (the compiler itself turns a byte-aligned 16-byte copy into one
// global_load_dwordx4), so a leaf that does not start 16-byte aligned streams through
// the same tile as an aligned one, each load covering 16 of its own bytes. Measured on
// MI355X: a 4-byte aligned start streams at about 85% of the aligned rate, other starts
// at 65-70%, both faster than reading aligned chunks and shifting them in registers.
// The payload pointers are built from integer addresses, so the compiler cannot tell
// their address space and would emit flat loads, which on gfx950 also count against the
// LDS wait counter: a wait for the stage tile's LDS accesses would then wait for the
// loads in flight too. The loads name the global address space instead.
typedef u32x4 u32x4_any __attribute__((aligned(1)));
typedef const __attribute__((address_space(1))) u32x4_any global_u32x4_any;
typedef const __attribute__((address_space(1))) uint64_t global_u64;
__device__ __forceinline__ uint4 load_stream16_any(const uint8_t* p) {
  const u32x4 v = __builtin_nontemporal_load((global_u32x4_any*)(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

constexpr int kLeavesPerWave = 32;
constexpr int kRunLanes = 32;                     // lanes reading one contiguous run
constexpr int kRun = kRunLanes * 16;              // 512 B of one leaf per load
constexpr int kLoads = kLeavesPerWave / (64 / kRunLanes);  // 16 loads per stage
constexpr int kStages = 4096 / kRun;              // 8 stages per leaf
constexpr int kWaveLds = kLeavesPerWave * kRun;   // 16 KiB tile per wave
constexpr int kMaxRoots = 128;                    // 32-leaf group roots of a 16 MiB block

struct FpArgs {
  const uint64_t* seg_addr;
  const uint64_t* seg_len;
  const uint64_t* blk_first;
  uint64_t n_seg;
  uint64_t n_blocks;
  uint64_t* block_out;
  uint64_t* leaf_out;
  uint32_t lpb_log2;
  uint64_t items;  // work items: groups of GROUP slots (LPB <= GROUP) or blocks
};

struct Leaf {
  const uint8_t* addr;
  uint32_t len;        // 0: no leaf in this slot
  uint32_t blk_leaves; // leaves of the slot's block (0 past the batch)
};

__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// x as held by lane `src` (a constant after unrolling): a register read, no memory trip.
__device__ __forceinline__ uint64_t lane64(uint64_t x, int src) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, src);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(x >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

// Leaf k of block g, which lies in segment s.
__device__ __forceinline__ Leaf locate_at(const FpArgs& a, uint64_t g, uint32_t k, uint64_t s) {
  Leaf lf{nullptr, 0, 0};
  if (g >= a.n_blocks) return lf;
  const uint32_t shift = 12 + a.lpb_log2;
  const uint64_t j = g - a.blk_first[s];
  const uint64_t start = j << shift;
  const uint64_t len_s = a.seg_len[s];
  if (start >= len_s) return lf;
  const uint64_t blen = min(len_s - start, (uint64_t)1 << shift);
  lf.blk_leaves = (uint32_t)((blen + 4095) >> 12);
  const uint64_t off = start + ((uint64_t)k << 12);
  if (off < len_s) {
    lf.addr = reinterpret_cast<const uint8_t*>(a.seg_addr[s] + off);
    lf.len = (uint32_t)min(len_s - off, (uint64_t)4096);
  }
  return lf;
}

// Leaf k of block g. `s` is a segment with blk_first[s] <= g (a lower start for the walk).
__device__ __forceinline__ Leaf locate(const FpArgs& a, uint64_t g, uint32_t k, uint64_t s) {
  if (g >= a.n_blocks) return Leaf{nullptr, 0, 0};
  while (s + 1 < a.n_seg && a.blk_first[s + 1] <= g) ++s;
  return locate_at(a, g, k, s);
}

// Leaf k of block g for every lane of a wave whose blocks start at block g_first (the same
// in every lane): the wave finds g_first's segment, then each lane its own (a wave of
// small payloads spans many segments). Every lane must call this.
__device__ __forceinline__ Leaf locate_wave(const FpArgs& a, uint64_t g_first, uint64_t g, uint32_t k, int lane) {
  if (g_first >= a.n_blocks) return Leaf{nullptr, 0, 0};
  const uint64_t s0 = uniform64(wave_find_segment(a.blk_first, a.n_seg, g_first, lane));
  const uint64_t s = lane_segment(a.blk_first, a.n_seg, s0, g < a.n_blocks ? g : a.n_blocks - 1, lane);
  return locate_at(a, g, k, s);
}

// XXH64 after the stripe loop: fold (or the short-input start), length, tail, avalanche.
// The tail (the < 32 bytes after the last full stripe, at any address) lies in at most
// five aligned 8-byte words, each holding tail bytes. load_tail reads them together (one
// round trip, no byte loads; the gathered paths issue it before their stage loop, so it
// overlaps the first stage's loads); finish_leaf_words shifts the tail's own 8-byte
// words out of adjacent pairs and runs the XXH64 tail steps in registers: whole words,
// then a 4-byte step, then single bytes.

// The aligned 8-byte words holding the tail of a leaf of `len` bytes at p; W[i] = 0 past
// them (len 0: no read).
__device__ __forceinline__ void load_tail(const uint8_t* p, uint32_t len, uint64_t W[5]) {
  const uint32_t stripes = len >> 5;
  const uint32_t tail = len - (stripes << 5);
  const uint64_t at = reinterpret_cast<uint64_t>(p) + (stripes << 5);
  const uint32_t lead = (uint32_t)(at & 7);
  const uint32_t words = tail ? (lead + tail + 7) >> 3 : 0;
  global_u64* w = (global_u64*)(at - lead);
#pragma unroll
  for (int i = 0; i < 5; ++i) W[i] = (uint32_t)i < words ? w[i] : 0;
}

__device__ __forceinline__ uint64_t finish_leaf_words(uint64_t v1, uint64_t v2, uint64_t v3, uint64_t v4,
                                                      const uint8_t* p, uint32_t len, const uint64_t W[5]) {
  const uint32_t stripes = len >> 5;
  uint64_t h = stripes ? xxh_converge(v1, v2, v3, v4) : kP5;
  h += len;
  const uint32_t tail = len - (stripes << 5);  // 0..31
  const uint64_t at = reinterpret_cast<uint64_t>(p) + (stripes << 5);
  const uint32_t lead = (uint32_t)(at & 7);    // tail bytes start this far into a word
  const uint32_t sh = lead * 8;
  uint64_t t[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) t[j] = sh ? (W[j] >> sh) | (W[j + 1] << (64 - sh)) : W[j];
  const uint32_t whole = tail >> 3;
#pragma unroll
  for (int j = 0; j < 3; ++j)
    if ((uint32_t)j < whole) h = xxh_tail8(h, t[j]);
  uint64_t rest = whole == 0 ? t[0] : whole == 1 ? t[1] : whole == 2 ? t[2] : t[3];
  if (tail & 4) {
    h = xxh_tail4(h, (uint32_t)rest);
    rest >>= 32;
  }
  for (uint32_t i = 0; i < (tail & 3); ++i) {
    h = xxh_tail1(h, (uint8_t)rest);
    rest >>= 8;
  }
  return xxh_avalanche(h);
}

// Lane roles shared by the streamed paths.
struct Roles {
  int lm, lc;            // loader: leaf within the load instruction (0/1), 16-byte chunk (0..31)
  int rl, rp;            // reader: leaf of the wave (0..31), half of each stripe (0/1)
  const uint8_t* rbase;  // reader's half-stripe 0 in the tile (before the swizzle)
  int rf;                // reader's swizzle key
};

__device__ __forceinline__ Roles roles(const uint8_t* tile, int lane) {
  Roles r;
  r.lm = lane / kRunLanes;
  r.lc = lane % kRunLanes;
  r.rl = lane >> 1;
  r.rp = lane & 1;
  r.rbase = tile + r.rl * kRun + r.rp * 16;
  r.rf = r.rl & 7;
  return r;
}

// Tile position of the chunk loaded by this lane for load instruction k:
// leaf l = 2k + lm, stripe lc / 2 swizzled by (l mod 8), half lc % 2.
__device__ __forceinline__ int tile_slot(const Roles& r, int k) {
  const int l = 2 * k + r.lm;
  return l * kRun + (((r.lc >> 1) ^ (l & 7)) * 32) + (r.lc & 1) * 16;
}

// 32 full, contiguous leaves from `base` (any alignment); lane pair l hashes leaf l.
// Returns the leaf digest in the even lane.
__device__ uint64_t hash_wave_contiguous(const uint8_t* base, uint8_t* tile, int lane) {
  const Roles r = roles(tile, lane);
  const uint8_t* lp = base + r.lm * 4096 + r.lc * 16;
  uint64_t va = r.rp ? 0 : kP1 + kP2, vb = r.rp ? 0 - kP1 : kP2;
  uint4 R[kLoads];
#pragma unroll
  for (int k = 0; k < kLoads; ++k) R[k] = load_stream16_any(lp + k * 2 * 4096);
  for (int s = 0; s < kStages; ++s) {
#pragma unroll
    for (int k = 0; k < kLoads; ++k) *reinterpret_cast<uint4*>(tile + tile_slot(r, k)) = R[k];
    wave_lds_sync();
    if (s + 1 < kStages) {
#pragma unroll
      for (int k = 0; k < kLoads; ++k) R[k] = load_stream16_any(lp + k * 2 * 4096 + (s + 1) * kRun);
    }
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      uint4 D[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) D[j] = *reinterpret_cast<const uint4*>(r.rbase + (((half * 8 + j) ^ r.rf) * 32));
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        va = xxh_round(va, lo64(D[j]));
        vb = xxh_round(vb, hi64(D[j]));
      }
    }
    wave_lds_sync();
  }
  const uint64_t pa = shfl_xor64(va, 1), pb = shfl_xor64(vb, 1);
  return r.rp ? 0 : xxh_avalanche(xxh_converge(va, vb, pa, pb) + 4096);
}

// Any 32 leaves (lengths 0..4096, at any alignment, anywhere in
// memory). Full stripes stream through the tile as above; for each load instruction the
// loader lanes take their leaf's address and full-stripe chunk count from the lane pair
// that hashes that leaf, by register reads (a table in LDS cost two dependent LDS round
// trips per load); the wave runs as many stages as its longest leaf needs; the even lane
// then finishes its leaf's tail directly.
__device__ uint64_t hash_wave_gathered(const Leaf& lf, uint8_t* tile, int lane) {
  const Roles r = roles(tile, lane);
  const uint32_t stripes = lf.len >> 5;
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  const uint32_t chunks = 2 * stripes;  // 16-byte chunks in the leaf's whole stripes
  uint32_t longest = stripes;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) longest = max(longest, (uint32_t)__shfl_xor((int)longest, o, 64));
  const uint32_t stages = __builtin_amdgcn_readfirstlane((longest + 15) / 16);
  uint64_t W[5];
  load_tail(lf.addr, r.rp ? 0u : lf.len, W);

  // load instruction k: lanes 0-31 read leaf 2k (held by lanes 4k, 4k + 1), lanes 32-63
  // leaf 2k + 1 (lanes 4k + 2, 4k + 3)
  auto stage_loads = [&](uint4* R, uint64_t chunk) {
#pragma unroll
    for (int k = 0; k < kLoads; ++k) {
      const uint64_t a0 = lane64(addr, 4 * k), a1 = lane64(addr, 4 * k + 2);
      const uint32_t n0 = __builtin_amdgcn_readlane(chunks, 4 * k), n1 = __builtin_amdgcn_readlane(chunks, 4 * k + 2);
      const uint64_t a = r.lm ? a1 : a0;
      const uint32_t n = r.lm ? n1 : n0;
      R[k] = chunk < n ? load_stream16_any(reinterpret_cast<const uint8_t*>(a) + chunk * 16) : make_uint4(0, 0, 0, 0);
    }
  };
  uint64_t va = r.rp ? 0 : kP1 + kP2, vb = r.rp ? 0 - kP1 : kP2;
  uint4 R[kLoads];
  stage_loads(R, (uint64_t)r.lc);
  for (uint32_t s = 0; s < stages; ++s) {
#pragma unroll
    for (int k = 0; k < kLoads; ++k) *reinterpret_cast<uint4*>(tile + tile_slot(r, k)) = R[k];
    wave_lds_sync();
    if (s + 1 < stages) stage_loads(R, (uint64_t)(s + 1) * kRunLanes + r.lc);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      uint4 D[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) D[j] = *reinterpret_cast<const uint4*>(r.rbase + (((half * 8 + j) ^ r.rf) * 32));
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (s * 16 + half * 8 + j < stripes) {
          va = xxh_round(va, lo64(D[j]));
          vb = xxh_round(vb, hi64(D[j]));
        }
      }
    }
    wave_lds_sync();
  }
  const uint64_t pa = shfl_xor64(va, 1), pb = shfl_xor64(vb, 1);
  if (r.rp || lf.len == 0) return 0;
  return finish_leaf_words(va, vb, pa, pb, lf.addr, lf.len, W);
}

// Digest of this lane pair's leaf, in the even lane.
__device__ __forceinline__ uint64_t hash_slot(const Leaf& lf, uint8_t* tile, int lane) {
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  const uint64_t a0 = shfl64(addr, 0);
  const bool contiguous = lf.len == 4096 && addr == a0 + (uint64_t)(lane >> 1) * 4096;
  if (__all(contiguous)) return hash_wave_contiguous(reinterpret_cast<const uint8_t*>(uniform64(a0)), tile, lane);
  if (!__any(lf.len != 0)) return 0;
  return hash_wave_gathered(lf, tile, lane);
}

// Bottom-up tree over `count` roots in LDS (double-buffered), by one wave.
__device__ uint64_t tree_reduce_lds(uint64_t* a, uint64_t* b, uint32_t count, int lane) {
  while (count > 1) {
    const uint32_t pairs = count / 2;
    for (uint32_t i = lane; i < pairs; i += 64) b[i] = tree_node(a[2 * i], a[2 * i + 1]);
    if ((count & 1) && lane == 0) b[pairs] = a[count - 1];
    wave_lds_sync();
    uint64_t* t = a;
    a = b;
    b = t;
    count = pairs + (count & 1);
  }
  return a[0];
}


// ---- Small batches: four lanes per leaf ---------------------------------------------
// A batch too small to fill the GPU (at most kQuadMaxSlots leaf slots, where the kernel
// above would launch at most two workgroups per CU) is latency-bound: a wave's time is
// its chain of load round trips. Here four lanes own one leaf (lane 4l + a keeps XXH64
// accumulator a + 1 of the wave's leaf l), so a wave covers 16 leaves in 4 stages of
// 1 KiB per leaf instead of 32 leaves in 8 stages, and the batch gets twice the waves.
// Loads keep the pattern above (two 512-byte runs of two leaves per instruction); the
// stage tile holds 1 KiB per leaf with 32-byte stripes XOR-swizzled by the leaf index,
// and each lane reads the 8-byte word of its accumulator from every stripe. Blocks of
// up to 16 leaves (64 KiB) only, so a wave holds whole blocks.
// Larger batches take this kernel too when their payloads average at least
// kQuadLargePayloadSlots leaf slots (mostly full, contiguous waves). Measured on MI355X:
// 1 GiB in one payload, 4 KiB and 64 KiB blocks, 6.5 against 6.2 TB/s; the 7B decoder in
// 4 KiB blocks 6.99 against 6.83 TB/s; 20 ResNet-50 weight sets (89 slots per payload)
// and the decoder in 64 KiB blocks the same either way. Many small payloads stay with the
// two-lanes kernel: 100k small copies, 4.5 against 4.9 TB/s (3.5 slots per payload).

constexpr int kQuadLeaves = 16;                  // leaves per wave
constexpr int kQuadStage = 1024;                 // bytes of each leaf per stage
constexpr int kQuadStages = 4096 / kQuadStage;   // 4 stages per leaf
constexpr int kQuadLoads = 16;                   // load instructions per stage
constexpr int kQuadWaveLds = kQuadLeaves * kQuadStage;
constexpr uint64_t kQuadMaxSlots = 1u << 16;
constexpr uint64_t kQuadLargePayloadSlots = 64;

// Load instruction k (0..15) of a stage: lanes 0-31 (lm = 0) and 32-63 (lm = 1) read
// leaf 2 (k mod 8) + lm, run k / 8 (the first or second 512 bytes of the stage's 1 KiB),
// 16-byte chunk lc = lane mod 32 of the run.
__device__ __forceinline__ int quad_leaf(int lm, int k) { return 2 * (k & 7) + lm; }
__device__ __forceinline__ int quad_chunk(int lc, int k) { return (k >> 3) * 32 + lc; }  // in the stage
// Tile position of that chunk: stripe j = chunk / 2 of leaf l at slot j ^ l, half chunk mod 2.
__device__ __forceinline__ int quad_tile_slot(int lm, int lc, int k) {
  const int l = quad_leaf(lm, k), c = quad_chunk(lc, k);
  return l * kQuadStage + (((c >> 1) ^ l) * 32) + (c & 1) * 16;
}

__device__ __forceinline__ uint64_t quad_acc_init(int a) {
  return a == 0 ? kP1 + kP2 : a == 1 ? kP2 : a == 2 ? 0ull : 0ull - kP1;
}

// XXH64 rounds of accumulator `a` over the tile's `count` stripes of leaf l (count <= 32).
__device__ __forceinline__ uint64_t quad_rounds(uint64_t v, const uint8_t* tile, int l, int a, int count) {
  const uint8_t* rb = tile + l * kQuadStage + a * 8;
#pragma unroll
  for (int j0 = 0; j0 < 32; j0 += 8) {
    uint64_t w[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = *reinterpret_cast<const uint64_t*>(rb + (((j0 + j) ^ l) * 32));
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j0 + j < count) v = xxh_round(v, w[j]);
  }
  return v;
}

// 16 full, contiguous leaves from `base` (any alignment); digest in lane 4l of leaf l.
__device__ uint64_t hash_quad_contiguous(const uint8_t* base, uint8_t* tile, int lane) {
  const int lm = lane / 32, lc = lane % 32, rl = lane >> 2, ra = lane & 3;
  uint64_t v = quad_acc_init(ra);
  uint4 R[kQuadLoads];
#pragma unroll
  for (int k = 0; k < kQuadLoads; ++k) R[k] = load_stream16_any(base + quad_leaf(lm, k) * 4096 + quad_chunk(lc, k) * 16);
  for (int s = 0; s < kQuadStages; ++s) {
#pragma unroll
    for (int k = 0; k < kQuadLoads; ++k) *reinterpret_cast<uint4*>(tile + quad_tile_slot(lm, lc, k)) = R[k];
    wave_lds_sync();
    if (s + 1 < kQuadStages) {
#pragma unroll
      for (int k = 0; k < kQuadLoads; ++k)
        R[k] = load_stream16_any(base + quad_leaf(lm, k) * 4096 + (s + 1) * kQuadStage + quad_chunk(lc, k) * 16);
    }
    v = quad_rounds(v, tile, rl, ra, 32);
    wave_lds_sync();
  }
  const int q = lane & ~3;
  const uint64_t v1 = shfl64(v, q), v2 = shfl64(v, q + 1), v3 = shfl64(v, q + 2), v4 = shfl64(v, q + 3);
  return ra ? 0 : xxh_avalanche(xxh_converge(v1, v2, v3, v4) + 4096);
}

// Any 16 leaves at any alignment: full stripes through the tile, each load instruction's
// leaf address and full-stripe chunk count read from the quad that hashes the leaf (as in
// hash_wave_gathered), as many stages as the longest leaf needs; lane 4l finishes leaf
// l's tail.
__device__ uint64_t hash_quad_gathered(const Leaf& lf, uint8_t* tile, int lane) {
  const int lm = lane / 32, lc = lane % 32, rl = lane >> 2, ra = lane & 3;
  const uint32_t stripes = lf.len >> 5;
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  const uint32_t chunks = 2 * stripes;
  uint32_t longest = stripes;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) longest = max(longest, (uint32_t)__shfl_xor((int)longest, o, 64));
  const uint32_t stages = __builtin_amdgcn_readfirstlane((longest + 31) / 32);
  uint64_t W[5];
  load_tail(lf.addr, ra ? 0u : lf.len, W);
  // load instruction k: lanes 0-31 read leaf 2 (k mod 8) (held by lane 8 (k mod 8)),
  // lanes 32-63 leaf 2 (k mod 8) + 1 (held by lane 8 (k mod 8) + 4)
  auto stage_loads = [&](uint4* R, uint64_t stage_chunk) {
#pragma unroll
    for (int k = 0; k < kQuadLoads; ++k) {
      const int h0 = 8 * (k & 7);
      const uint64_t a0 = lane64(addr, h0), a1 = lane64(addr, h0 + 4);
      const uint32_t n0 = __builtin_amdgcn_readlane(chunks, h0), n1 = __builtin_amdgcn_readlane(chunks, h0 + 4);
      const uint64_t la = lm ? a1 : a0;
      const uint32_t n = lm ? n1 : n0;
      const uint64_t c = stage_chunk + (uint64_t)quad_chunk(lc, k);
      R[k] = c < n ? load_stream16_any(reinterpret_cast<const uint8_t*>(la) + c * 16) : make_uint4(0, 0, 0, 0);
    }
  };
  uint64_t v = quad_acc_init(ra);
  uint4 R[kQuadLoads];
  stage_loads(R, 0);
  for (uint32_t s = 0; s < stages; ++s) {
#pragma unroll
    for (int k = 0; k < kQuadLoads; ++k) *reinterpret_cast<uint4*>(tile + quad_tile_slot(lm, lc, k)) = R[k];
    wave_lds_sync();
    if (s + 1 < stages) stage_loads(R, (uint64_t)(s + 1) * 64);
    const int left = (int)stripes - (int)(s * 32);
    v = quad_rounds(v, tile, rl, ra, left < 0 ? 0 : (left > 32 ? 32 : left));
    wave_lds_sync();
  }
  const int q = lane & ~3;
  const uint64_t v1 = shfl64(v, q), v2 = shfl64(v, q + 1), v3 = shfl64(v, q + 2), v4 = shfl64(v, q + 3);
  if (ra || lf.len == 0) return 0;
  return finish_leaf_words(v1, v2, v3, v4, lf.addr, lf.len, W);
}

// Digest of this lane quad's leaf, in lane 4l.
__device__ __forceinline__ uint64_t hash_slot_quad(const Leaf& lf, uint8_t* tile, int lane) {
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  const uint64_t a0 = shfl64(addr, 0);
  const bool contiguous = lf.len == 4096 && addr == a0 + (uint64_t)(lane >> 2) * 4096;
  if (__all(contiguous)) return hash_quad_contiguous(reinterpret_cast<const uint8_t*>(uniform64(a0)), tile, lane);
  if (!__any(lf.len != 0)) return 0;
  return hash_quad_gathered(lf, tile, lane);
}

// ---- One round trip per wave: every stage straight into LDS --------------------------
// With one wave per workgroup and at most two per CU (the smallest batches), a wave can
// keep all four 1 KiB stages of its 16 leaves in LDS (64 KiB) and issue them together with
// gfx950's direct-to-LDS loads (global_load_lds_dwordx4: lane i of an instruction writes
// bytes [16 i, 16 i + 16) of the instruction's 1 KiB LDS window), so the wave waits for
// memory once instead of once per stage. One instruction carries one leaf's stage; lane i
// loads the 16-byte chunk that the swizzled tile puts at position 16 i (stripe (i / 2) xor
// leaf, half i mod 2), so each stage's tile is laid out as in the staged path and the
// rounds read it unchanged. These loads take 16-byte aligned leaves only: a wave with any
// other leaf runs the staged path.
constexpr int kQuadDirectLds = kQuadStages * kQuadWaveLds;  // 64 KiB per wave
constexpr int kWaitLoads = 0x0F70;                          // s_waitcnt vmcnt(0)
constexpr int kNonTemporal = 2;                             // cache policy: nt

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void load_lds16(const uint8_t* src, uint8_t* window) {
  __builtin_amdgcn_global_load_lds(src, (lds_void*)window, 16, 0, kNonTemporal);
}

// 16 full, contiguous, 16-byte aligned leaves from `base`; digest in lane 4l of leaf l.
__device__ uint64_t hash_quad_contiguous_direct(const uint8_t* base, uint8_t* tile, int lane) {
  const int rl = lane >> 2, ra = lane & 3, t = lane >> 1, h = lane & 1;
#pragma unroll
  for (int s = 0; s < kQuadStages; ++s) {
#pragma unroll
    for (int l = 0; l < kQuadLeaves; ++l)
      load_lds16(base + l * 4096 + s * kQuadStage + ((t ^ l) * 32) + h * 16,
                 tile + s * kQuadWaveLds + l * kQuadStage);
  }
  __builtin_amdgcn_s_waitcnt(kWaitLoads);
  wave_lds_sync();
  uint64_t v = quad_acc_init(ra);
#pragma unroll
  for (int s = 0; s < kQuadStages; ++s) v = quad_rounds(v, tile + s * kQuadWaveLds, rl, ra, 32);
  const int q = lane & ~3;
  const uint64_t v1 = shfl64(v, q), v2 = shfl64(v, q + 1), v3 = shfl64(v, q + 2), v4 = shfl64(v, q + 3);
  return ra ? 0 : xxh_avalanche(xxh_converge(v1, v2, v3, v4) + 4096);
}

// Any 16 leaves at 16-byte aligned addresses: every stage the longest leaf needs, issued
// together (a lane loads a chunk only if it lies in its leaf's whole stripes); lane 4l
// finishes leaf l's tail.
__device__ uint64_t hash_quad_gathered_direct(const Leaf& lf, uint8_t* tile, int lane) {
  const int rl = lane >> 2, ra = lane & 3, t = lane >> 1, h = lane & 1;
  const uint32_t stripes = lf.len >> 5;
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  const uint32_t chunks = 2 * stripes;
  uint32_t longest = stripes;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) longest = max(longest, (uint32_t)__shfl_xor((int)longest, o, 64));
  const uint32_t stages = __builtin_amdgcn_readfirstlane((longest + 31) / 32);
  uint64_t W[5];
  load_tail(lf.addr, ra ? 0u : lf.len, W);
  for (uint32_t s = 0; s < stages; ++s) {
#pragma unroll
    for (int l = 0; l < kQuadLeaves; ++l) {
      // leaf l's address and chunk count, from lane 4l that hashes it (the same in every lane)
      const uint64_t la = lane64(addr, 4 * l);
      const uint32_t n = __builtin_amdgcn_readlane(chunks, 4 * l);
      const uint64_t c = (uint64_t)s * 64 + ((t ^ l) * 2) + h;  // chunk of leaf l for this lane
      if (c < n) load_lds16(reinterpret_cast<const uint8_t*>(la) + c * 16, tile + s * kQuadWaveLds + l * kQuadStage);
    }
  }
  __builtin_amdgcn_s_waitcnt(kWaitLoads);
  wave_lds_sync();
  uint64_t v = quad_acc_init(ra);
  for (uint32_t s = 0; s < stages; ++s) {
    const int left = (int)stripes - (int)(s * 32);
    v = quad_rounds(v, tile + s * kQuadWaveLds, rl, ra, left < 0 ? 0 : (left > 32 ? 32 : left));
  }
  const int q = lane & ~3;
  const uint64_t v1 = shfl64(v, q), v2 = shfl64(v, q + 1), v3 = shfl64(v, q + 2), v4 = shfl64(v, q + 3);
  if (ra || lf.len == 0) return 0;
  return finish_leaf_words(v1, v2, v3, v4, lf.addr, lf.len, W);
}

// hash_slot_quad with a 64 KiB tile: the direct loads when every leaf of the wave is
// 16-byte aligned, else the staged path.
__device__ __forceinline__ uint64_t hash_slot_quad_direct(const Leaf& lf, uint8_t* tile, int lane) {
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  if (!__all((addr & 15) == 0 || lf.len == 0)) return hash_slot_quad(lf, tile, lane);
  const uint64_t a0 = shfl64(addr, 0);
  const bool contiguous = lf.len == 4096 && addr == a0 + (uint64_t)(lane >> 2) * 4096;
  if (__all(contiguous))
    return hash_quad_contiguous_direct(reinterpret_cast<const uint8_t*>(uniform64(a0)), tile, lane);
  if (!__any(lf.len != 0)) return 0;
  return hash_quad_gathered_direct(lf, tile, lane);
}

// The four-lanes-per-leaf pass of one workgroup of W waves over the W * kQuadLeaves slots
// of group `group` (LPB <= kQuadLeaves, so every wave holds whole blocks): leaf digests
// (optional) and
// block digests. With kLen, the lane holding a block's last leaf also writes the
// block's byte length to blen[g]. With kDirect (W = 1), `lds` holds kQuadDirectLds bytes
// and aligned waves load every stage at once; otherwise kQuadWaveLds per wave.
//
// With a Probe (the one-launch detect path), the lane holding a block's digest also probes
// the resident table for it right away (its latency overlapping other waves' streaming):
// a held digest gets status HIT_CACHE and its value as ref; any other gets kProbePending.
constexpr uint8_t kProbePending = 0xFF;

struct NoProbe {
  __device__ __forceinline__ void operator()(uint64_t, uint64_t) const {}
};

template <int W, bool kLen, bool kDirect = false, typename Probe = NoProbe>
__device__ __forceinline__ void quad_pass(const FpArgs& a, uint64_t group, uint8_t* lds, uint32_t* blen,
                                          const Probe& probe = Probe()) {
  static_assert(!kDirect || W == 1, "the direct loads hold one wave's stages");
  constexpr uint64_t kQuadGroup = (uint64_t)W * kQuadLeaves;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const uint32_t L2 = a.lpb_log2;
  const uint32_t lpb = 1u << L2;
  const uint64_t wave_slot0 = uniform64(group * kQuadGroup + (uint64_t)wave * kQuadLeaves);
  const uint64_t slot = wave_slot0 + (lane >> 2);
  const uint64_t g = slot >> L2;
  const uint32_t k = (uint32_t)(slot & (lpb - 1));
  const Leaf lf = locate_wave(a, wave_slot0 >> L2, g, k, lane);
  const uint64_t d = kDirect ? hash_slot_quad_direct(lf, lds, lane) : hash_slot_quad(lf, lds + wave * kQuadWaveLds, lane);
  const bool head = (lane & 3) == 0;
  if (a.leaf_out && head && g < a.n_blocks) a.leaf_out[slot] = lf.len ? d : 0;
  if (kLen && head && g < a.n_blocks && lf.len && k + 1 == lf.blk_leaves) blen[g] = (k << 12) + lf.len;
  const uint64_t v = tree_reduce_lanes(d, k, lf.blk_leaves, lpb, 4);
  if (head && k == 0 && g < a.n_blocks) {
    a.block_out[g] = v;
    probe(g, v);
  }
}

}  // namespace
}  // namespace gleam
