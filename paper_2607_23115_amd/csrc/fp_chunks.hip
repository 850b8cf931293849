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
// (LPB <= GROUP), or one whole block walked GROUP slots at a time (LPB > GROUP). In a
// large batch of blocks of up to 64 KiB, the last kQuadTailSlots slots go to workgroups
// of four lanes per leaf (64 slots each, half the stages): the batch's last round of
// workgroups, during which part of the GPU already idles, then ends sooner.
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
// small payloads) use the same tile with per-instruction leaf addresses read from the
// registers of the lanes that hash each leaf. Every load covers 16 bytes of its own leaf
// from the leaf's start, at any
// alignment (see load_stream16_any), so a leaf's bytes reach the tile in order and no
// path shifts them.
//
// Tree: levels inside a wave's 32 leaves use cross-lane shuffles; the roots of
// 32-leaf groups meet in LDS. Pairing by aligned position level by level is the same
// computation as the plain bottom-up definition.

#include "fp_core.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;
constexpr int kSoloPad = 24 << 10;  // takes the workgroup's LDS past 80 KiB: one per CU
constexpr uint64_t kQuadTailSlots = 16384;

template <bool kSolo>
__global__ __launch_bounds__(kThreads) void fp_kernel(FpArgs a) {
  constexpr int W = kThreads / 64;
  constexpr uint32_t GROUP = W * kLeavesPerWave;
  __shared__ __attribute__((aligned(16))) uint8_t lds[W * kWaveLds + (kSolo ? kSoloPad : 0)];
  __shared__ uint64_t roots[2][kMaxRoots];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  uint8_t* tile = lds + wave * kWaveLds;
  const uint32_t L2 = a.lpb_log2;
  const uint32_t lpb = 1u << L2;
  const bool even = (lane & 1) == 0;

  // The last slots of a batch of small blocks, past a.items groups: four lanes per leaf,
  // W * kQuadLeaves slots per workgroup (see launch_fp).
  if (!kSolo && blockIdx.x >= a.items) {
    constexpr uint64_t kPerGroup = GROUP / (W * kQuadLeaves);
    quad_pass<W, false>(a, a.items * kPerGroup + (blockIdx.x - a.items), lds, nullptr);
    return;
  }

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
      const uint64_t d = hash_slot(lf, tile, lane);
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
        const uint64_t d = hash_slot(lf, tile, lane);
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


// One workgroup of W waves per W * kQuadLeaves slots; LPB <= kQuadLeaves, so every wave
// holds whole blocks. W = 1 for the smallest batches (more CUs then share the loads; each
// wave loads all its stages into LDS at once), 4 otherwise.
template <int W>
__global__ __launch_bounds__(64 * W) void fp_quad_kernel(FpArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[W == 1 ? kQuadDirectLds : W * kQuadWaveLds];
  quad_pass<W, false, W == 1>(a, blockIdx.x, lds, nullptr);
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
  uint64_t items = lpb <= group ? (b->n_blocks * lpb + group - 1) / group : b->n_blocks;
  // 1 MiB blocks and up: one workgroup resident per CU, a grid of 4 per CU walking the
  // blocks. Smaller blocks: one workgroup per item (both measured best on MI355X).
  const bool solo = lpb >= 256;
  uint64_t grid = items;
  // Blocks of up to 64 KiB in a batch of several rounds of workgroups: the last
  // kQuadTailSlots slots (rounded to whole groups) run as workgroups of four lanes per
  // leaf, which finish in half the time, so the GPU drains faster at the end.
  if (lpb <= (uint64_t)kQuadLeaves && slots > 4 * kQuadTailSlots) {
    items = (slots - kQuadTailSlots) / group;
    const uint64_t quad_group = (kThreads / 64) * kQuadLeaves;
    grid = items + (slots - items * group + quad_group - 1) / quad_group;
  }
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


// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_fp_chunks() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&fp_kernel<true>));
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
