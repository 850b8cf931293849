// gleam_fp_chunks: block digests of a batch of payloads on gfx950.
//
// Identifier of a block (Gleam Sec. 4.1.2, hash of the source bytes): XXH64 with
// seed 0 of each 4 KiB leaf over its actual bytes, folded by a bottom-up pairwise
// tree (node = XXH64 of LE64(left) || LE64(right); an odd last element moves up).
//
// Work decomposition. Leaf slot = g * LPB + k (block g, leaf k, LPB = leaves per
// block). Two lanes own one slot: the even lane keeps XXH64 accumulators 1 and 2, the
// odd lane 3 and 4, so each lane runs two independent chains of 128 rounds and a
// wave covers 32 leaves. A workgroup of 4 waves owns GROUP = 128 consecutive slots
// (LPB <= GROUP), or one whole block walked GROUP slots at a time (LPB > GROUP).
//
// Occupancy. HBM read rate on MI355X rises as fewer waves stream at once: one 4-wave
// workgroup per CU reads faster than two or more (measured with plain read kernels and
// with this one). For blocks of 1 MiB and up the workgroup's LDS is padded past half
// of the CU's 160 KiB, so each CU holds exactly one, and a grid of 4 per CU walks the
// blocks. Smaller blocks keep one workgroup per item at normal occupancy: their
// gathered waves need the extra waves to hide latency.
//
// Memory path (the kernel is HBM-bound; XXH64 itself runs far above HBM rate).
// A wave whose 32 leaves are full and contiguous streams them with non-temporal
// 16-byte loads in which 32 consecutive lanes read one 512-byte run of one leaf (2
// leaves per load instruction, 16 loads = 32 leaves x 512 B per stage). Each stage goes
// through a per-wave LDS tile, 512 B per leaf, whose 32-byte stripes are XOR-swizzled by
// the leaf index, so both the stores and each lane's 16-byte reads of its own
// half-stripes are free of bank conflicts; the next stage's loads are in flight while
// the current one is hashed. Waves that are not one contiguous full run (payload ends,
// small payloads) use the same tile with per-instruction leaf addresses from a small
// LDS table. Every load covers 16 bytes of its own leaf from the leaf's start, at any
// alignment (see load_stream16_any), so a leaf's bytes reach the tile in order and no
// path shifts them.
//
// Tree: levels inside a wave's 32 leaves use cross-lane shuffles; the roots of
// 32-leaf groups meet in LDS. Pairing by aligned position level by level is the same
// computation as the plain bottom-up definition.

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
typedef u32x4 u32x4_any __attribute__((aligned(1)));
__device__ __forceinline__ uint4 load_stream16_any(const uint8_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_any*>(p));
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
  const uint64_t* w = reinterpret_cast<const uint64_t*>(at - lead);
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
// memory). Full stripes stream through the tile as above; the loader lanes find each
// leaf's address and full-stripe chunk count in a small per-wave LDS table (kept out of
// registers, which the streamed stage already fills); the wave runs as many stages as
// its longest leaf needs; the even lane then finishes its leaf's tail directly.
__device__ uint64_t hash_wave_gathered(const Leaf& lf, uint8_t* tile, uint64_t* table, int lane) {
  const Roles r = roles(tile, lane);
  const uint32_t stripes = lf.len >> 5;
  if ((lane & 1) == 0) {
    table[lane] = reinterpret_cast<uint64_t>(lf.addr);  // entry of leaf lane / 2: {address, chunks}
    table[lane + 1] = 2ull * stripes;
  }
  uint32_t longest = stripes;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) longest = max(longest, (uint32_t)__shfl_xor((int)longest, o, 64));
  const uint32_t stages = __builtin_amdgcn_readfirstlane((longest + 15) / 16);
  uint64_t W[5];
  load_tail(lf.addr, r.rp ? 0u : lf.len, W);
  wave_lds_sync();

  uint64_t va = r.rp ? 0 : kP1 + kP2, vb = r.rp ? 0 - kP1 : kP2;
  uint4 R[kLoads];
#pragma unroll
  for (int k = 0; k < kLoads; ++k) {
    const uint64_t* e = table + 2 * (2 * k + r.lm);
    R[k] = (uint64_t)r.lc < e[1] ? load_stream16_any(reinterpret_cast<const uint8_t*>(e[0]) + r.lc * 16)
                                 : make_uint4(0, 0, 0, 0);
  }
  for (uint32_t s = 0; s < stages; ++s) {
#pragma unroll
    for (int k = 0; k < kLoads; ++k) *reinterpret_cast<uint4*>(tile + tile_slot(r, k)) = R[k];
    wave_lds_sync();
    if (s + 1 < stages) {
      const uint64_t chunk = (uint64_t)(s + 1) * kRunLanes + r.lc;
#pragma unroll
      for (int k = 0; k < kLoads; ++k) {
        const uint64_t* e = table + 2 * (2 * k + r.lm);
        R[k] = chunk < e[1] ? load_stream16_any(reinterpret_cast<const uint8_t*>(e[0]) + chunk * 16)
                            : make_uint4(0, 0, 0, 0);
      }
    }
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
__device__ __forceinline__ uint64_t hash_slot(const Leaf& lf, uint8_t* tile, uint64_t* table, int lane) {
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  const uint64_t a0 = shfl64(addr, 0);
  const bool contiguous = lf.len == 4096 && addr == a0 + (uint64_t)(lane >> 1) * 4096;
  if (__all(contiguous)) return hash_wave_contiguous(reinterpret_cast<const uint8_t*>(uniform64(a0)), tile, lane);
  if (!__any(lf.len != 0)) return 0;
  return hash_wave_gathered(lf, tile, table, lane);
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

constexpr int kThreads = 256;
constexpr int kSoloPad = 24 << 10;  // takes the workgroup's LDS past 80 KiB: one per CU

template <bool kSolo>
__global__ __launch_bounds__(kThreads) void fp_kernel(FpArgs a) {
  constexpr int W = kThreads / 64;
  constexpr uint32_t GROUP = W * kLeavesPerWave;
  __shared__ __attribute__((aligned(16))) uint8_t lds[W * kWaveLds + (kSolo ? kSoloPad : 0)];
  __shared__ uint64_t roots[2][kMaxRoots];
  __shared__ uint64_t tables[W][2 * kLeavesPerWave];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  uint8_t* tile = lds + wave * kWaveLds;
  uint64_t* table = tables[wave];
  const uint32_t L2 = a.lpb_log2;
  const uint32_t lpb = 1u << L2;
  const bool even = (lane & 1) == 0;

  // Persistent workgroups: a grid of a few workgroups per CU walks the work items.
  for (uint64_t item = blockIdx.x; item < a.items; item += gridDim.x) {
    __syncthreads();  // the previous item's roots have been consumed
    if (lpb <= GROUP) {
      // GROUP consecutive slots: GROUP / LPB whole blocks.
      const uint64_t wave_slot0 = uniform64(item * GROUP + (uint64_t)wave * kLeavesPerWave);
      const uint64_t slot = wave_slot0 + (lane >> 1);
      const uint64_t g = slot >> L2;
      const uint32_t k = (uint32_t)(slot & (lpb - 1));
      const Leaf lf = locate_wave(a, wave_slot0 >> L2, g, k, lane);
      const uint64_t d = hash_slot(lf, tile, table, lane);
      if (a.leaf_out && even && g < a.n_blocks) a.leaf_out[slot] = lf.len ? d : 0;
      const uint32_t G = lpb <= kLeavesPerWave ? lpb : (uint32_t)kLeavesPerWave;
      const uint32_t p = k & (G - 1);
      uint32_t n = lf.blk_leaves;
      if (lpb > kLeavesPerWave) {
        const uint32_t before = k & ~(uint32_t)(kLeavesPerWave - 1);
        n = n > before ? min(n - before, (uint32_t)kLeavesPerWave) : 0u;
      }
      const uint64_t v = tree_reduce_lanes(d, p, n, G, 2);
      if (lpb <= kLeavesPerWave) {
        if (even && p == 0 && g < a.n_blocks) a.block_out[g] = v;
      } else {
        if (lane == 0) roots[0][wave] = v;
        __syncthreads();
        if (wave == 0) {
          // W wave roots = GROUP / LPB blocks of G2 = LPB / 32 roots each
          const uint32_t G2 = lpb / kLeavesPerWave;
          const uint64_t g2 = ((item * GROUP) >> L2) + (uint64_t)(lane / G2);
          uint32_t n2 = 0;
          uint64_t v2 = 0;
          const Leaf head = locate_wave(a, (item * GROUP) >> L2, g2, 0, lane);
          if (lane < W && g2 < a.n_blocks) {
            n2 = (head.blk_leaves + kLeavesPerWave - 1) / kLeavesPerWave;
            v2 = roots[0][lane];
          }
          v2 = tree_reduce_lanes(v2, lane & (G2 - 1), n2, G2);
          if (lane < W && (lane & (G2 - 1)) == 0 && g2 < a.n_blocks) a.block_out[g2] = v2;
        }
      }
    } else {
      // One block of LPB > GROUP leaves, GROUP slots at a time.
      const uint64_t g = item;
      const uint64_t s0 = uniform64(find_segment(a.blk_first, a.n_seg, g));
      const uint32_t nleaf = locate(a, g, 0, s0).blk_leaves;
      const uint32_t groups = a.leaf_out ? lpb / GROUP : (nleaf + GROUP - 1) / GROUP;
      for (uint32_t grp = 0; grp < groups; ++grp) {
        const uint32_t k = grp * GROUP + (uint32_t)wave * kLeavesPerWave + (lane >> 1);
        const Leaf lf = locate(a, g, k, s0);
        const uint64_t d = hash_slot(lf, tile, table, lane);
        if (a.leaf_out && even) a.leaf_out[((uint64_t)g << L2) + k] = lf.len ? d : 0;
        const uint32_t before = k & ~(uint32_t)(kLeavesPerWave - 1);
        const uint32_t n = nleaf > before ? min(nleaf - before, (uint32_t)kLeavesPerWave) : 0u;
        const uint64_t v = tree_reduce_lanes(d, (uint32_t)(lane >> 1), n, kLeavesPerWave, 2);
        if (lane == 0) roots[0][grp * W + wave] = v;
      }
      __syncthreads();
      if (wave == 0) {
        const uint32_t n2 = (nleaf + kLeavesPerWave - 1) / kLeavesPerWave;  // <= kMaxRoots
        const uint64_t r = tree_reduce_lds(roots[0], roots[1], n2, lane);
        if (lane == 0) a.block_out[g] = r;
      }
    }
  }
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

// Any 16 leaves at any alignment: full stripes through the tile
// (leaf addresses and full-stripe chunk counts in a per-wave LDS table), as many stages
// as the longest leaf needs; lane 4l finishes leaf l's tail.
__device__ uint64_t hash_quad_gathered(const Leaf& lf, uint8_t* tile, uint64_t* table, int lane) {
  const int lm = lane / 32, lc = lane % 32, rl = lane >> 2, ra = lane & 3;
  const uint32_t stripes = lf.len >> 5;
  if (ra == 0) {
    table[2 * rl] = reinterpret_cast<uint64_t>(lf.addr);
    table[2 * rl + 1] = 2ull * stripes;
  }
  uint32_t longest = stripes;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) longest = max(longest, (uint32_t)__shfl_xor((int)longest, o, 64));
  const uint32_t stages = __builtin_amdgcn_readfirstlane((longest + 31) / 32);
  uint64_t W[5];
  load_tail(lf.addr, ra ? 0u : lf.len, W);
  wave_lds_sync();
  uint64_t v = quad_acc_init(ra);
  uint4 R[kQuadLoads];
#pragma unroll
  for (int k = 0; k < kQuadLoads; ++k) {
    const uint64_t* e = table + 2 * quad_leaf(lm, k);
    const uint64_t c = (uint64_t)quad_chunk(lc, k);
    R[k] = c < e[1] ? load_stream16_any(reinterpret_cast<const uint8_t*>(e[0]) + c * 16) : make_uint4(0, 0, 0, 0);
  }
  for (uint32_t s = 0; s < stages; ++s) {
#pragma unroll
    for (int k = 0; k < kQuadLoads; ++k) *reinterpret_cast<uint4*>(tile + quad_tile_slot(lm, lc, k)) = R[k];
    wave_lds_sync();
    if (s + 1 < stages) {
#pragma unroll
      for (int k = 0; k < kQuadLoads; ++k) {
        const uint64_t* e = table + 2 * quad_leaf(lm, k);
        const uint64_t c = (uint64_t)(s + 1) * 64 + quad_chunk(lc, k);
        R[k] = c < e[1] ? load_stream16_any(reinterpret_cast<const uint8_t*>(e[0]) + c * 16) : make_uint4(0, 0, 0, 0);
      }
    }
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
__device__ __forceinline__ uint64_t hash_slot_quad(const Leaf& lf, uint8_t* tile, uint64_t* table, int lane) {
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  const uint64_t a0 = shfl64(addr, 0);
  const bool contiguous = lf.len == 4096 && addr == a0 + (uint64_t)(lane >> 2) * 4096;
  if (__all(contiguous)) return hash_quad_contiguous(reinterpret_cast<const uint8_t*>(uniform64(a0)), tile, lane);
  if (!__any(lf.len != 0)) return 0;
  return hash_quad_gathered(lf, tile, table, lane);
}

// One workgroup of W waves per W * kQuadLeaves slots; LPB <= kQuadLeaves, so every wave
// holds whole blocks. W = 1 for the smallest batches (more CUs then share the loads), 4
// otherwise.
template <int W>
__global__ __launch_bounds__(64 * W) void fp_quad_kernel(FpArgs a) {
  constexpr uint64_t kQuadGroup = (uint64_t)W * kQuadLeaves;
  __shared__ __attribute__((aligned(16))) uint8_t lds[W * kQuadWaveLds];
  __shared__ uint64_t tables[W][2 * kQuadLeaves];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const uint32_t L2 = a.lpb_log2;
  const uint32_t lpb = 1u << L2;
  const uint64_t wave_slot0 = uniform64((uint64_t)blockIdx.x * kQuadGroup + (uint64_t)wave * kQuadLeaves);
  const uint64_t slot = wave_slot0 + (lane >> 2);
  const uint64_t g = slot >> L2;
  const uint32_t k = (uint32_t)(slot & (lpb - 1));
  const Leaf lf = locate_wave(a, wave_slot0 >> L2, g, k, lane);
  const uint64_t d = hash_slot_quad(lf, lds + wave * kQuadWaveLds, tables[wave], lane);
  const bool head = (lane & 3) == 0;
  if (a.leaf_out && head && g < a.n_blocks) a.leaf_out[slot] = lf.len ? d : 0;
  const uint64_t v = tree_reduce_lanes(d, k, lf.blk_leaves, lpb, 4);
  if (head && k == 0 && g < a.n_blocks) a.block_out[g] = v;
}

}  // namespace

gleam_status validate_batch(const gleam_batch* b, const char* who) {
  if (!b) {
    set_error("%s: null batch", who);
    return GLEAM_E_INVALID;
  }
  if (b->leaf_bytes != GLEAM_LEAF_BYTES || !valid_block_bytes(b->block_bytes)) {
    set_error("%s: leaf_bytes must be 4096 and block_bytes 4096 << k (k <= 12)", who);
    return GLEAM_E_INVALID;
  }
  if (b->n_blocks > 0 && (b->n_seg == 0 || !b->seg_addr || !b->seg_len || !b->blk_first)) {
    set_error("%s: null descriptor for a non-empty batch", who);
    return GLEAM_E_INVALID;
  }
  if (b->n_blocks > (UINT64_MAX >> 13)) {
    set_error("%s: batch too large", who);
    return GLEAM_E_UNSUPPORTED;
  }
  return GLEAM_OK;
}

gleam_status launch_fp(const gleam_batch* b, uint64_t* d_block_digest, uint64_t* d_leaf_digest, hipStream_t stream) {
  if (b->n_blocks == 0) return GLEAM_OK;
  const int lpb_log2 = log2_exact(b->block_bytes) - 12;
  const uint64_t lpb = 1ull << lpb_log2;
  const uint64_t slots = b->n_blocks * lpb;  // n_blocks < 2^51: no overflow
  // (a large batch takes the four-lanes kernel only while its grid of one 4-wave
  // workgroup per 64 slots stays below 2^31)
  if (lpb <= (uint64_t)kQuadLeaves &&
      (slots <= kQuadMaxSlots ||
       (slots / kQuadLargePayloadSlots >= b->n_seg && slots / (4 * kQuadLeaves) < 0x7fffffffull))) {
    int cus = 0;
    gleam_status st = device_cu_count(&cus);
    if (st != GLEAM_OK) return st;
    const uint64_t waves = (b->n_blocks * lpb + kQuadLeaves - 1) / kQuadLeaves;
    FpArgs a{b->seg_addr, b->seg_len, b->blk_first, b->n_seg, b->n_blocks, d_block_digest, d_leaf_digest,
             (uint32_t)lpb_log2, waves};
    // one-wave workgroups while they spread the batch over more CUs (16 MiB, 256 waves:
    // 10.1 vs 11.2 us), 4-wave ones above two waves per CU (ResNet-50, 895 waves: 16.6 vs
    // 17.9 us with one-wave workgroups)
    if (waves <= 2ull * (uint64_t)cus) {
      hipLaunchKernelGGL(fp_quad_kernel<1>, dim3((uint32_t)waves), dim3(64), 0, stream, a);
    } else {
      hipLaunchKernelGGL(fp_quad_kernel<4>, dim3((uint32_t)((waves + 3) / 4)), dim3(256), 0, stream, a);
    }
    return launch_status("fp_quad_kernel");
  }
  constexpr uint64_t group = (kThreads / 64) * kLeavesPerWave;
  const uint64_t items = lpb <= group ? (b->n_blocks * lpb + group - 1) / group : b->n_blocks;
  // 1 MiB blocks and up: one workgroup resident per CU, a grid of 4 per CU walking the
  // blocks. Smaller blocks: one workgroup per item (both measured best on MI355X).
  const bool solo = lpb >= 256;
  uint64_t grid = items;
  if (solo) {
    int cus = 0;
    gleam_status st = device_cu_count(&cus);
    if (st != GLEAM_OK) return st;
    grid = items < 4ull * (uint64_t)cus ? items : 4ull * (uint64_t)cus;
  }
  if (grid > 0x7fffffffull) {
    set_error("fingerprint: batch needs more than 2^31 workgroups");
    return GLEAM_E_UNSUPPORTED;
  }
  FpArgs a{b->seg_addr, b->seg_len, b->blk_first, b->n_seg, b->n_blocks, d_block_digest, d_leaf_digest,
           (uint32_t)lpb_log2, items};
  if (solo)
    hipLaunchKernelGGL(fp_kernel<true>, dim3((uint32_t)grid), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(fp_kernel<false>, dim3((uint32_t)grid), dim3(kThreads), 0, stream, a);
  return launch_status("fp_kernel");
}

}  // namespace gleam

extern "C" gleam_status gleam_fp_chunks(const gleam_batch* b, uint64_t* d_block_digest, uint64_t* d_leaf_digest,
                                        void* stream) {
  using namespace gleam;
  clear_error();
  gleam_status st = validate_batch(b, "gleam_fp_chunks");
  if (st != GLEAM_OK) return st;
  if (b->n_blocks == 0) return GLEAM_OK;
  if (!d_block_digest) {
    set_error("gleam_fp_chunks: null output for a non-empty batch");
    return GLEAM_E_INVALID;
  }
  return launch_fp(b, d_block_digest, d_leaf_digest, (hipStream_t)stream);
}
