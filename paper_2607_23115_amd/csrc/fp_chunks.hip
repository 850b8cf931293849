// gleam_fp_chunks: block digests of a batch of payloads on gfx950.
//
// Identifier of a block (Gleam Sec. 4.1.2, hash of the source bytes): XXH64 with
// seed 0 of each 4 KiB leaf over its actual bytes, folded by a bottom-up pairwise
// tree (node = XXH64 of LE64(left) || LE64(right); an odd last element moves up).
//
// Work decomposition. Leaf slot = g * LPB + k (block g, leaf k, LPB = leaves per
// block). One thread owns one slot: it keeps the four XXH64 accumulators of its
// leaf in registers, so a 4 KiB leaf is four independent chains of 128 rounds in
// one lane. A workgroup of 256 threads owns 256 consecutive slots (LPB <= 256), or
// one whole block walked 256 slots at a time (LPB > 256).
//
// Memory path (the kernel is HBM-bound; XXH64 itself runs far above HBM rate).
// A wave whose 64 leaves are full, contiguous and 16-byte aligned streams them
// with non-temporal 16-byte loads in which 16 consecutive lanes read one 256-byte
// run of one leaf (4 leaves per load instruction, 16 loads = 64 leaves x 256 B per
// stage). The stage goes through a per-wave LDS tile with an XOR swizzle so that
// each lane then reads its own leaf's 256 bytes conflict-free; the next stage's
// loads are in flight while the current one is hashed. Other waves (short leaves,
// unaligned payloads, payload boundaries) hash lane by lane with direct loads.
//
// Tree: levels inside a 64-lane group use cross-lane shuffles; groups of 64 leaves
// are combined by wave 0 from LDS. Pairing by aligned position level by level is
// the same computation as the plain bottom-up definition.

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kWG = 256;
constexpr int kRunLanes = 16;                       // lanes reading one contiguous run
constexpr int kRun = kRunLanes * 16;                // 256 B of one leaf per load
constexpr int kLeavesPerLoad = 64 / kRunLanes;      // 4
constexpr int kLoads = kRunLanes;                   // 16 loads per stage
constexpr int kStages = 4096 / kRun;                // 16
constexpr int kSlotStride = 1024 + 16;              // LDS stride between load slots
constexpr int kWaveLds = kLoads * kSlotStride;      // 16,640 B per wave

struct FpArgs {
  const uint64_t* seg_addr;
  const uint64_t* seg_len;
  const uint64_t* blk_first;
  uint64_t n_seg;
  uint64_t n_blocks;
  uint64_t* block_out;
  uint64_t* leaf_out;
  uint32_t lpb_log2;
  uint64_t items;  // work items: groups of 256 slots (LPB <= 256) or blocks (LPB > 256)
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

// Leaf k of block g. `s` is a segment with blk_first[s] <= g (a lower start for the walk).
__device__ __forceinline__ Leaf locate(const FpArgs& a, uint64_t g, uint32_t k, uint64_t s) {
  Leaf lf{nullptr, 0, 0};
  if (g >= a.n_blocks) return lf;
  while (s + 1 < a.n_seg && a.blk_first[s + 1] <= g) ++s;
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

__device__ __forceinline__ uint64_t read_le64_bytes(const uint8_t* p) {
  uint64_t v = 0;
#pragma unroll
  for (int i = 7; i >= 0; --i) v = (v << 8) | p[i];
  return v;
}
__device__ __forceinline__ uint32_t read_le32_bytes(const uint8_t* p) {
  uint32_t v = 0;
#pragma unroll
  for (int i = 3; i >= 0; --i) v = (v << 8) | p[i];
  return v;
}

// One leaf of 1..4096 bytes at any alignment, by one lane.
__device__ uint64_t hash_leaf_lane(const uint8_t* p, uint32_t len) {
  const bool a16 = (reinterpret_cast<uintptr_t>(p) & 15) == 0;
  uint32_t pos = 0;
  uint64_t h;
  if (len >= 32) {
    uint64_t v1 = kP1 + kP2, v2 = kP2, v3 = 0, v4 = 0 - kP1;
    const uint32_t stripes = len >> 5;
    if (a16) {
#pragma unroll 4
      for (uint32_t i = 0; i < stripes; ++i) {
        const uint4 x = load_stream16(p + 32 * i);
        const uint4 y = load_stream16(p + 32 * i + 16);
        v1 = xxh_round(v1, lo64(x));
        v2 = xxh_round(v2, hi64(x));
        v3 = xxh_round(v3, lo64(y));
        v4 = xxh_round(v4, hi64(y));
      }
    } else {
      for (uint32_t i = 0; i < stripes; ++i) {
        const uint8_t* q = p + 32 * i;
        v1 = xxh_round(v1, read_le64_bytes(q));
        v2 = xxh_round(v2, read_le64_bytes(q + 8));
        v3 = xxh_round(v3, read_le64_bytes(q + 16));
        v4 = xxh_round(v4, read_le64_bytes(q + 24));
      }
    }
    pos = stripes << 5;
    h = xxh_converge(v1, v2, v3, v4);
  } else {
    h = kP5;
  }
  h += len;
  for (; pos + 8 <= len; pos += 8)
    h = xxh_tail8(h, a16 ? *reinterpret_cast<const uint64_t*>(p + pos) : read_le64_bytes(p + pos));
  if (pos + 4 <= len) {
    h = xxh_tail4(h, a16 ? *reinterpret_cast<const uint32_t*>(p + pos) : read_le32_bytes(p + pos));
    pos += 4;
  }
  for (; pos < len; ++pos) h = xxh_tail1(h, p[pos]);
  return xxh_avalanche(h);
}

// 64 full, contiguous, 16-byte aligned leaves starting at `base`; lane l hashes leaf l.
__device__ uint64_t hash_wave_streamed(const uint8_t* base, uint8_t* tile, int lane) {
  // loader role: 16 lanes per 256-byte run, 4 leaves per load instruction
  const int wm = lane / kRunLanes, wc = lane % kRunLanes;
  const uint8_t* lp = base + wm * 4096 + wc * 16;
  const int wslot = (wm * kRunLanes + (wc ^ (wm * 4))) * 16;
  // reader role: leaf `lane` lives in load slot lane / 4, position lane % 4
  const int rk = lane / kLeavesPerLoad, rm = lane % kLeavesPerLoad;
  const uint8_t* rp = tile + rk * kSlotStride + rm * kRun;
  const int rsw = rm * 4;

  uint64_t v1 = kP1 + kP2, v2 = kP2, v3 = 0, v4 = 0 - kP1;
  uint4 R[kLoads];
#pragma unroll
  for (int k = 0; k < kLoads; ++k) R[k] = load_stream16(lp + k * kLeavesPerLoad * 4096);
  for (int s = 0; s < kStages; ++s) {
#pragma unroll
    for (int k = 0; k < kLoads; ++k) *reinterpret_cast<uint4*>(tile + k * kSlotStride + wslot) = R[k];
    wave_lds_sync();
    if (s + 1 < kStages) {
#pragma unroll
      for (int k = 0; k < kLoads; ++k) R[k] = load_stream16(lp + k * kLeavesPerLoad * 4096 + (s + 1) * kRun);
    }
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      uint4 D[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) D[j] = *reinterpret_cast<const uint4*>(rp + (((half * 8 + j) ^ rsw) * 16));
#pragma unroll
      for (int j = 0; j < 8; j += 2) {
        v1 = xxh_round(v1, lo64(D[j]));
        v2 = xxh_round(v2, hi64(D[j]));
        v3 = xxh_round(v3, lo64(D[j + 1]));
        v4 = xxh_round(v4, hi64(D[j + 1]));
      }
    }
    wave_lds_sync();
  }
  return xxh_avalanche(xxh_converge(v1, v2, v3, v4) + 4096);
}

// Any 64 leaves whose present ones start 16-byte aligned (lengths 0..4096, anywhere in
// memory): the full 32-byte stripes stream through the LDS tile as above, with each loader
// lane holding the addresses of the 16 leaves it loads for; the wave runs as many stages as
// its longest leaf needs. Each lane then finishes its own tail (< 32 bytes) directly.
__device__ uint64_t hash_wave_gathered(const Leaf& lf, uint8_t* tile, int lane) {
  const int wm = lane / kRunLanes, wc = lane % kRunLanes;
  const int wslot = (wm * kRunLanes + (wc ^ (wm * 4))) * 16;
  const int rk = lane / kLeavesPerLoad, rm = lane % kLeavesPerLoad;
  const uint8_t* rp = tile + rk * kSlotStride + rm * kRun;
  const int rsw = rm * 4;
  const uint32_t stripes = lf.len >> 5;
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);

  const uint8_t* la[kLoads];  // this loader lane's 16-byte chunk of leaf 4k + wm, stage 0
  uint32_t lim[kLoads];       // that leaf's number of 16-byte chunks in full stripes
  uint32_t longest = stripes;
#pragma unroll
  for (int k = 0; k < kLoads; ++k) {
    const int src = k * kLeavesPerLoad + wm;
    la[k] = reinterpret_cast<const uint8_t*>(shfl64(addr, src)) + wc * 16;
    lim[k] = 2 * (uint32_t)__shfl((int)stripes, src, 64);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) longest = max(longest, (uint32_t)__shfl_xor((int)longest, o, 64));
  const uint32_t stages = __builtin_amdgcn_readfirstlane((longest + 7) / 8);

  uint64_t v1 = kP1 + kP2, v2 = kP2, v3 = 0, v4 = 0 - kP1;
  uint4 R[kLoads];
#pragma unroll
  for (int k = 0; k < kLoads; ++k) R[k] = (uint32_t)wc < lim[k] ? load_stream16(la[k]) : make_uint4(0, 0, 0, 0);
  for (uint32_t s = 0; s < stages; ++s) {
#pragma unroll
    for (int k = 0; k < kLoads; ++k) *reinterpret_cast<uint4*>(tile + k * kSlotStride + wslot) = R[k];
    wave_lds_sync();
    if (s + 1 < stages) {
      const uint32_t chunk = (s + 1) * kRunLanes + wc;
#pragma unroll
      for (int k = 0; k < kLoads; ++k)
        R[k] = chunk < lim[k] ? load_stream16(la[k] + (s + 1) * kRun) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      uint4 D[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) D[j] = *reinterpret_cast<const uint4*>(rp + (((half * 8 + j) ^ rsw) * 16));
#pragma unroll
      for (int j = 0; j < 8; j += 2) {
        if (s * 8 + half * 4 + j / 2 < stripes) {
          v1 = xxh_round(v1, lo64(D[j]));
          v2 = xxh_round(v2, hi64(D[j]));
          v3 = xxh_round(v3, lo64(D[j + 1]));
          v4 = xxh_round(v4, hi64(D[j + 1]));
        }
      }
    }
    wave_lds_sync();
  }
  if (lf.len == 0) return 0;
  uint64_t h = stripes ? xxh_converge(v1, v2, v3, v4) : kP5;
  h += lf.len;
  uint32_t pos = stripes << 5;
  for (; pos + 8 <= lf.len; pos += 8) h = xxh_tail8(h, *reinterpret_cast<const uint64_t*>(lf.addr + pos));
  if (pos + 4 <= lf.len) {
    h = xxh_tail4(h, *reinterpret_cast<const uint32_t*>(lf.addr + pos));
    pos += 4;
  }
  for (; pos < lf.len; ++pos) h = xxh_tail1(h, lf.addr[pos]);
  return xxh_avalanche(h);
}

__device__ __forceinline__ uint64_t hash_slot(const Leaf& lf, uint8_t* tile, int lane) {
  const uint64_t addr = reinterpret_cast<uint64_t>(lf.addr);
  const uint64_t a0 = shfl64(addr, 0);
  const bool contiguous = lf.len == 4096 && addr == a0 + (uint64_t)lane * 4096 && (a0 & 15) == 0;
  if (__all(contiguous)) return hash_wave_streamed(reinterpret_cast<const uint8_t*>(uniform64(a0)), tile, lane);
  if (!__any(lf.len != 0)) return 0;
  if (__all(lf.len == 0 || (addr & 15) == 0)) return hash_wave_gathered(lf, tile, lane);
  return lf.len ? hash_leaf_lane(lf.addr, lf.len) : 0;
}

__global__ __launch_bounds__(kWG) void fp_kernel(FpArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[4 * kWaveLds];
  __shared__ uint64_t roots[64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  uint8_t* tile = lds + wave * kWaveLds;
  const uint32_t L2 = a.lpb_log2;
  const uint64_t lpb = 1ull << L2;

  // Persistent workgroups: a grid of a few workgroups per CU walks the work items.
  for (uint64_t item = blockIdx.x; item < a.items; item += gridDim.x) {
  __syncthreads();  // the previous item's roots have been consumed
  if (L2 <= 8) {
    // 256 consecutive slots: 256 / LPB whole blocks.
    const uint64_t wave_slot0 = uniform64(item * kWG + (uint64_t)wave * 64);
    const uint64_t slot = wave_slot0 + lane;
    const uint64_t g = slot >> L2;
    const uint32_t k = (uint32_t)(slot & (lpb - 1));
    const uint64_t g_first = wave_slot0 >> L2;
    const uint64_t s0 = g_first < a.n_blocks ? uniform64(find_segment(a.blk_first, a.n_seg, g_first)) : 0;
    const Leaf lf = locate(a, g, k, s0);
    const uint64_t d = hash_slot(lf, tile, lane);
    if (a.leaf_out && g < a.n_blocks) a.leaf_out[slot] = lf.len ? d : 0;
    const uint32_t G = L2 <= 6 ? (uint32_t)lpb : 64u;
    const uint32_t p = k & (G - 1);
    uint32_t n = lf.blk_leaves;
    if (L2 > 6) {
      const uint32_t before = k & ~63u;
      n = n > before ? min(n - before, 64u) : 0u;
    }
    const uint64_t v = tree_reduce_lanes(d, p, n, G);
    if (L2 <= 6) {
      if (p == 0 && g < a.n_blocks) a.block_out[g] = v;
    } else {
      if (lane == 0) roots[wave] = v;
      __syncthreads();
      if (wave == 0) {
        // 4 group roots = 256 / LPB blocks of G2 = LPB / 64 roots each
        const uint32_t G2 = (uint32_t)(lpb >> 6);
        const uint64_t g2 = ((item * kWG) >> L2) + (uint64_t)(lane / G2);
        uint32_t n2 = 0;
        uint64_t v2 = 0;
        if (lane < 4 && g2 < a.n_blocks) {
          const Leaf head = locate(a, g2, 0, find_segment(a.blk_first, a.n_seg, g2));
          n2 = (head.blk_leaves + 63) / 64;
          v2 = roots[lane];
        }
        v2 = tree_reduce_lanes(v2, lane & (G2 - 1), n2, G2);
        if (lane < 4 && (lane & (G2 - 1)) == 0 && g2 < a.n_blocks) a.block_out[g2] = v2;
      }
    }
  } else {
    // One block of LPB > 256 leaves, 256 slots at a time.
    const uint64_t g = item;
    const uint64_t s0 = uniform64(find_segment(a.blk_first, a.n_seg, g));
    const uint32_t nleaf = locate(a, g, 0, s0).blk_leaves;
    const uint32_t groups = a.leaf_out ? (uint32_t)(lpb >> 8) : (nleaf + 255) / 256;
    for (uint32_t grp = 0; grp < groups; ++grp) {
      const uint32_t k = grp * kWG + threadIdx.x;
      const Leaf lf = locate(a, g, k, s0);
      const uint64_t d = hash_slot(lf, tile, lane);
      if (a.leaf_out) a.leaf_out[(g << L2) + k] = lf.len ? d : 0;
      const uint32_t before = k & ~63u;
      const uint32_t n = nleaf > before ? min(nleaf - before, 64u) : 0u;
      const uint64_t v = tree_reduce_lanes(d, (uint32_t)lane, n, 64);
      if (lane == 0) roots[grp * 4 + wave] = v;
    }
    __syncthreads();
    if (wave == 0) {
      const uint32_t G2 = (uint32_t)(lpb >> 6);  // 8 .. 64 group roots
      const uint32_t n2 = (nleaf + 63) / 64;
      const uint64_t v2 = (uint32_t)lane < n2 ? roots[lane] : 0;
      const uint64_t r = tree_reduce_lanes(v2, lane & (G2 - 1), (uint32_t)lane < G2 ? n2 : 0, G2);
      if (lane == 0) a.block_out[g] = r;
    }
  }
  }
}

}  // namespace
}  // namespace gleam

namespace gleam {

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
  const uint64_t items = lpb_log2 <= 8 ? (b->n_blocks * lpb + kWG - 1) / kWG : b->n_blocks;
  int cus = 0;
  gleam_status st = device_cu_count(&cus);
  if (st != GLEAM_OK) return st;
  // Items of <= 1 MiB: four workgroups per CU (two resident at a time, by LDS) walk
  // them, which trims the launch tail (measured best on MI355X). Larger blocks
  // already amortise per-item setup and balance better with one workgroup per item.
  const uint64_t cap = lpb_log2 <= 8 ? 4ull * (uint64_t)cus : items;
  const uint64_t grid = items < cap ? items : cap;
  if (grid > 0x7fffffffull) {
    set_error("fingerprint: batch needs more than 2^31 workgroups");
    return GLEAM_E_UNSUPPORTED;
  }
  FpArgs a{b->seg_addr, b->seg_len, b->blk_first, b->n_seg, b->n_blocks, d_block_digest, d_leaf_digest,
           (uint32_t)lpb_log2, items};
  hipLaunchKernelGGL(fp_kernel, dim3((uint32_t)grid), dim3(kWG), 0, stream, a);
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
