// gleam_identify_weights: weight identification at free time (Gleam Sec. 4.1.1,
// "Weight Block Identification"). An allocation holds weights only if every payload
// recorded at its first host-to-device write still has the same bytes when the
// allocation is freed; in-place activations or inputs make it non-weights (Appendix,
// discussion of corner cases). Instead of the recorded bytes, the digests recorded
// at write time are compared with digests of the current device bytes: the same
// fingerprint kernel, then a compare pass and two small reductions.

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr int kThreads = 256;

__global__ void identify_init_kernel(uint64_t* first_diff, uint64_t n_seg, const uint64_t* region_first,
                                     uint64_t n_regions, uint8_t* region_weight) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (uint64_t s = t; s < n_seg; s += stride) first_diff[s] = ~0ull;
  for (uint64_t r = t; r < n_regions; r += stride) region_weight[r] = region_first[r + 1] > region_first[r] ? 1 : 0;
}

// first_diff[s] = min(first_diff[s], x) for the lanes with `differs`. When every such lane
// of the wave lies in one payload (all but the waves at payload boundaries), the wave
// takes the minimum itself and one lane issues the atomic: a payload whose blocks all changed
// (a layer updated in place) would otherwise queue one atomic per block on its word
// (262,144 leaves of one payload: 3.2 ms, 15x the comparison of unchanged leaves). Every
// lane of the wave calls it.
__device__ __forceinline__ void lower_first_diff(uint64_t* first_diff, uint64_t s, bool differs, uint64_t x) {
  const int lane = threadIdx.x & 63;
  const uint64_t active = __ballot(differs);
  const int leader = active ? __ffsll((unsigned long long)active) - 1 : 0;
  const uint64_t s0 = shfl64(s, leader);
  if (__ballot(differs && s != s0) == 0) {  // one payload for every differing lane
    uint64_t m = differs ? x : ~0ull;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const uint64_t y = shfl_xor64(m, o);
      m = y < m ? y : m;
    }
    if (lane == leader && m != ~0ull) atomicMin(reinterpret_cast<unsigned long long*>(&first_diff[s0]), m);
  } else if (differs) {
    atomicMin(reinterpret_cast<unsigned long long*>(&first_diff[s]), (unsigned long long)x);
  }
}

// Per block: equal digests? The first differing block of each payload by atomicMin.
__global__ void identify_compare_kernel(const uint64_t* current, const uint64_t* recorded, uint64_t n_blocks,
                                        const uint64_t* blk_first, uint64_t n_seg, uint8_t* block_match,
                                        uint64_t* first_diff) {
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool valid = g < n_blocks;
  const bool same = !valid || current[g] == recorded[g];
  if (valid && block_match) block_match[g] = same ? 1 : 0;
  uint64_t s = 0, x = 0;
  if (!same) {
    s = find_segment(blk_first, n_seg, g);
    x = g - blk_first[s];
  }
  lower_first_diff(first_diff, s, !same, x);
}

// Per leaf slot (slot = g * LPB + k): equal digests? Slots past a short block's last leaf
// hold 0 on both sides, so they always agree. The first differing leaf of each payload by
// atomicMin of its index within the payload, (g - blk_first[s]) * LPB + k.
__global__ void identify_leaf_compare_kernel(const uint64_t* current, const uint64_t* recorded, uint64_t n_slots,
                                             uint32_t lpb_log2, const uint64_t* blk_first, uint64_t n_seg,
                                             uint8_t* leaf_match, uint64_t* first_diff) {
  const uint64_t slot = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool valid = slot < n_slots;
  const bool same = !valid || current[slot] == recorded[slot];
  if (valid && leaf_match) leaf_match[slot] = same ? 1 : 0;
  uint64_t s = 0, leaf = 0;
  if (!same) {
    const uint64_t g = slot >> lpb_log2;
    s = find_segment(blk_first, n_seg, g);
    leaf = ((g - blk_first[s]) << lpb_log2) + (slot & ((1ull << lpb_log2) - 1));
  }
  lower_first_diff(first_diff, s, !same, leaf);
}

// Per payload: a difference clears its allocation's weight flag.
__global__ void identify_region_kernel(const uint64_t* first_diff, uint64_t n_seg, const uint64_t* region_first,
                                       uint64_t n_regions, uint8_t* region_weight) {
  const uint64_t s = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_seg || first_diff[s] == ~0ull) return;
  if (s < region_first[0] || s >= region_first[n_regions]) return;
  const uint64_t r = find_segment(region_first, n_regions, s);
  region_weight[r] = 0;
}

uint32_t grid_for(uint64_t n, uint64_t cap = 0x7fffffffull) {
  const uint64_t g = (n + kThreads - 1) / kThreads;
  return (uint32_t)(g < cap ? (g ? g : 1) : cap);
}

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_identify() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&identify_init_kernel));
}

}  // namespace gleam

extern "C" gleam_status gleam_identify_weights(const gleam_batch* b, const uint64_t* d_recorded,
                                               const uint64_t* d_region_first, uint64_t n_regions,
                                               uint8_t* d_block_match, uint64_t* d_seg_first_diff,
                                               uint8_t* d_region_weight, void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  gleam_status st = validate_batch(b, "gleam_identify_weights");
  if (st != GLEAM_OK) return st;
  if ((b->n_blocks > 0 && !d_recorded) || (n_regions > 0 && (!d_region_first || !d_region_weight))) {
    set_error("gleam_identify_weights: null recorded digests, region list or output");
    return GLEAM_E_INVALID;
  }
  if (b->n_seg > 0x7fffffffull * kThreads || n_regions > 0x7fffffffull * kThreads ||
      b->n_blocks > 0x7fffffffull * kThreads) {
    set_error("gleam_identify_weights: more than 2^31 workgroups of blocks, payloads or regions");
    return GLEAM_E_UNSUPPORTED;
  }
  const WsLayout L = ws_layout(b->n_blocks + b->n_seg);
  st = check_workspace(L, d_ws, ws_bytes, "gleam_identify_weights");
  if (st != GLEAM_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  uint64_t* current = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(d_ws) + L.scratch_off);
  uint64_t* first_diff = d_seg_first_diff ? d_seg_first_diff : current + b->n_blocks;
  const uint64_t init_n = b->n_seg > n_regions ? b->n_seg : n_regions;
  hipLaunchKernelGGL(identify_init_kernel, dim3(grid_for(init_n, 4096)), dim3(kThreads), 0, s, first_diff, b->n_seg,
                     d_region_first, n_regions, d_region_weight);
  if ((st = launch_status("identify_init_kernel")) != GLEAM_OK) return st;
  if (b->n_blocks == 0) return GLEAM_OK;
  if ((st = launch_fp(b, current, nullptr, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(identify_compare_kernel, dim3(grid_for(b->n_blocks)), dim3(kThreads), 0, s, current,
                     d_recorded, b->n_blocks, b->blk_first, b->n_seg, d_block_match, first_diff);
  if ((st = launch_status("identify_compare_kernel")) != GLEAM_OK) return st;
  if (n_regions == 0) return GLEAM_OK;
  hipLaunchKernelGGL(identify_region_kernel, dim3(grid_for(b->n_seg)), dim3(kThreads), 0, s, first_diff, b->n_seg,
                     d_region_first, n_regions, d_region_weight);
  return launch_status("identify_region_kernel");
}

extern "C" gleam_status gleam_identify_leaves(const gleam_batch* b, const uint64_t* d_recorded_leaf,
                                              const uint64_t* d_region_first, uint64_t n_regions,
                                              uint8_t* d_leaf_match, uint64_t* d_seg_first_diff,
                                              uint8_t* d_region_weight, void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  gleam_status st = validate_batch(b, "gleam_identify_leaves");
  if (st != GLEAM_OK) return st;
  if ((b->n_blocks > 0 && !d_recorded_leaf) || (n_regions > 0 && (!d_region_first || !d_region_weight))) {
    set_error("gleam_identify_leaves: null recorded leaf digests, region list or output");
    return GLEAM_E_INVALID;
  }
  const uint32_t lpb_log2 = (uint32_t)(log2_exact(b->block_bytes) - 12);
  const uint64_t n_slots = b->n_blocks << lpb_log2;  // n_blocks < 2^51 (validate_batch)
  if (b->n_seg > 0x7fffffffull * kThreads || n_regions > 0x7fffffffull * kThreads ||
      n_slots > 0x7fffffffull * kThreads) {
    set_error("gleam_identify_leaves: more than 2^31 workgroups of leaf slots, payloads or regions");
    return GLEAM_E_UNSUPPORTED;
  }
  const WsLayout L = ws_layout(n_slots + b->n_seg);
  st = check_workspace(L, d_ws, ws_bytes, "gleam_identify_leaves");
  if (st != GLEAM_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  // workspace: current leaf digests [n_slots], block digests [n_blocks], first_diff [n_seg]
  // (16 * (n_slots + n_seg) bytes of scratch hold them)
  uint64_t* cur_leaf = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(d_ws) + L.scratch_off);
  uint64_t* cur_block = cur_leaf + n_slots;
  uint64_t* first_diff = d_seg_first_diff ? d_seg_first_diff : cur_block + b->n_blocks;
  const uint64_t init_n = b->n_seg > n_regions ? b->n_seg : n_regions;
  hipLaunchKernelGGL(identify_init_kernel, dim3(grid_for(init_n, 4096)), dim3(kThreads), 0, s, first_diff, b->n_seg,
                     d_region_first, n_regions, d_region_weight);
  if ((st = launch_status("identify_init_kernel")) != GLEAM_OK) return st;
  if (b->n_blocks == 0) return GLEAM_OK;
  if ((st = launch_fp(b, cur_block, cur_leaf, s)) != GLEAM_OK) return st;
  hipLaunchKernelGGL(identify_leaf_compare_kernel, dim3(grid_for(n_slots)), dim3(kThreads), 0, s, cur_leaf,
                     d_recorded_leaf, n_slots, lpb_log2, b->blk_first, b->n_seg, d_leaf_match, first_diff);
  if ((st = launch_status("identify_leaf_compare_kernel")) != GLEAM_OK) return st;
  if (n_regions == 0) return GLEAM_OK;
  hipLaunchKernelGGL(identify_region_kernel, dim3(grid_for(b->n_seg)), dim3(kThreads), 0, s, first_diff, b->n_seg,
                     d_region_first, n_regions, d_region_weight);
  return launch_status("identify_region_kernel");
}
