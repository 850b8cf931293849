// Device helpers shared by the gfx950 kernels of libgleam.
//
// XXH64 is the 64-bit xxHash algorithm as published by its author (the xxHash
// specification): four 64-bit accumulators over 32-byte stripes, a byte-granular
// tail, and a final avalanche. Everything here is integer arithmetic mod 2^64.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gleam {

// XXH64 primes.
constexpr uint64_t kP1 = 0x9E3779B185EBCA87ull;
constexpr uint64_t kP2 = 0xC2B2AE3D27D4EB4Full;
constexpr uint64_t kP3 = 0x165667B19E3779F9ull;
constexpr uint64_t kP4 = 0x85EBCA77C2B2AE63ull;
constexpr uint64_t kP5 = 0x27D4EB2F165667C5ull;

// The table's empty-slot marker. Any u64 is a valid key: a key equal to kEmpty
// lives in a side slot of the table header instead.
constexpr uint64_t kEmpty = ~0ull;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint64_t rotl64(uint64_t x, int r) { return (x << r) | (x >> (64 - r)); }

__device__ __forceinline__ uint64_t xxh_round(uint64_t acc, uint64_t w) {
  return rotl64(acc + w * kP2, 31) * kP1;
}

__device__ __forceinline__ uint64_t xxh_merge(uint64_t h, uint64_t acc) {
  h ^= xxh_round(0, acc);
  return h * kP1 + kP4;
}

__device__ __forceinline__ uint64_t xxh_avalanche(uint64_t h) {
  h ^= h >> 33;
  h *= kP2;
  h ^= h >> 29;
  h *= kP3;
  h ^= h >> 32;
  return h;
}

// Fold the four stripe accumulators (input of >= 32 bytes).
__device__ __forceinline__ uint64_t xxh_converge(uint64_t v1, uint64_t v2, uint64_t v3, uint64_t v4) {
  uint64_t h = rotl64(v1, 1) + rotl64(v2, 7) + rotl64(v3, 12) + rotl64(v4, 18);
  h = xxh_merge(h, v1);
  h = xxh_merge(h, v2);
  h = xxh_merge(h, v3);
  h = xxh_merge(h, v4);
  return h;
}

// Tail steps.
__device__ __forceinline__ uint64_t xxh_tail8(uint64_t h, uint64_t w) {
  h ^= xxh_round(0, w);
  return rotl64(h, 27) * kP1 + kP4;
}
__device__ __forceinline__ uint64_t xxh_tail4(uint64_t h, uint32_t w) {
  h ^= (uint64_t)w * kP1;
  return rotl64(h, 23) * kP2 + kP3;
}
__device__ __forceinline__ uint64_t xxh_tail1(uint64_t h, uint8_t c) {
  h ^= (uint64_t)c * kP5;
  return rotl64(h, 11) * kP1;
}

// Tree node: XXH64 (seed 0) of the 16-byte string LE64(left) || LE64(right).
__device__ __forceinline__ uint64_t tree_node(uint64_t left, uint64_t right) {
  uint64_t h = kP5 + 16;
  h = xxh_tail8(h, left);
  h = xxh_tail8(h, right);
  return xxh_avalanche(h);
}

__device__ __forceinline__ uint64_t lo64(uint4 v) { return ((uint64_t)v.y << 32) | v.x; }
__device__ __forceinline__ uint64_t hi64(uint4 v) { return ((uint64_t)v.w << 32) | v.z; }

// Streaming 16-byte load that bypasses cache retention (each payload byte is read once).
__device__ __forceinline__ uint4 load_stream16(const uint8_t* p) {
  u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int mask) {
  uint32_t lo = __shfl_xor((uint32_t)v, mask, 64);
  uint32_t hi = __shfl_xor((uint32_t)(v >> 32), mask, 64);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
  uint32_t lo = __shfl((uint32_t)v, src, 64);
  uint32_t hi = __shfl((uint32_t)(v >> 32), src, 64);
  return ((uint64_t)hi << 32) | lo;
}

// Orders this wave's LDS writes before its later LDS reads (LDS executes one
// wave's instructions in order; this keeps the compiler from reordering them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Bottom-up pairwise tree over aligned groups of G positions (G a power of two), one
// position per `stride` lanes (stride * G <= 64). Position p in [0, G) holds element p
// of level 0; n elements are present (positions >= n absent). At the level with step
// s, element e = p / s pairs with e + 1 when e is even and e + 1 < ceil(n / s); an odd
// last element moves up unchanged. Position 0 ends with the group's root. Every lane
// must call this.
__device__ __forceinline__ uint64_t tree_reduce_lanes(uint64_t v, uint32_t p, uint32_t n, uint32_t G,
                                                      uint32_t stride = 1) {
  for (uint32_t s = 1; s < G; s <<= 1) {
    const uint64_t o = shfl_xor64(v, (int)(s * stride));
    const uint32_t count = (n + s - 1) / s;
    if ((p & (2 * s - 1)) == 0 && p / s + 1 < count) v = tree_node(v, o);
  }
  return v;
}

// Largest s in [0, n_seg) with blk_first[s] <= g (the payload holding block g).
__device__ __forceinline__ uint64_t find_segment(const uint64_t* blk_first, uint64_t n_seg, uint64_t g) {
  uint64_t lo = 0, hi = n_seg - 1;
  while (lo < hi) {
    const uint64_t mid = (lo + hi + 1) >> 1;
    if (blk_first[mid] <= g) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// find_segment for a g that is the same in every lane, by the whole wave: each round
// reads 64 evenly spaced pivots at once and keeps the interval the ballot points to, so
// n_seg payloads cost about log64(n_seg) dependent reads instead of log2(n_seg). Every
// lane must call this with the same arguments; blk_first[0] <= g < blk_first[n_seg].
__device__ __forceinline__ uint64_t wave_find_segment(const uint64_t* blk_first, uint64_t n_seg, uint64_t g,
                                                      int lane) {
  uint64_t lo = 0, hi = n_seg;  // the answer lies in [lo, hi) and blk_first[lo] <= g
  while (hi - lo > 64) {
    const uint64_t step = (hi - lo + 63) / 64;
    const uint64_t idx = lo + (uint64_t)lane * step;
    const bool le = idx < hi && blk_first[idx] <= g;
    // pivots 0..c-1 are <= g; c >= 1 for a well-formed blk_first (the max keeps every
    // read inside [0, n_seg) even for a malformed one)
    const uint32_t c = max((uint32_t)__popcll(__ballot(le)), 1u);
    lo += (uint64_t)(c - 1) * step;
    hi = min(lo + step, hi);
  }
  const uint64_t idx = lo + (uint64_t)lane;
  const bool le = idx < hi && blk_first[idx] <= g;
  return lo + (uint64_t)max((uint32_t)__popcll(__ballot(le)), 1u) - 1;
}

// Per-lane find_segment for blocks at or after the start of segment s0 (same in every
// lane): one read of the 64 segment starts after s0, a binary search over them through
// lane shuffles, and a forward walk only for a block beyond that window. Every lane must
// call this; g need only be meaningful in lanes whose result is used (g < n_blocks).
__device__ __forceinline__ uint64_t lane_segment(const uint64_t* blk_first, uint64_t n_seg, uint64_t s0,
                                                 uint64_t g, int lane) {
  const uint64_t e = s0 + 1 + (uint64_t)lane;
  const uint64_t w = e < n_seg ? blk_first[e] : ~0ull;  // start of the lane-th segment after s0
  const uint64_t last = shfl64(w, 63);
  uint32_t c = 0;  // number of window starts <= g
#pragma unroll
  for (uint32_t step = 32; step >= 1; step >>= 1) {
    const uint64_t v = shfl64(w, (int)(c + step - 1));
    if (v <= g) c += step;
  }
  uint64_t s = s0 + c;
  if (last <= g) {  // beyond the window
    s = s0 + 64;
    while (s + 1 < n_seg && blk_first[s + 1] <= g) ++s;
  }
  return s;
}

// Table hashing: Fibonacci multiplicative hash, top bits.
__device__ __forceinline__ uint64_t slot_hash(uint64_t key, int shift) {
  return (key * 0x9E3779B97F4A7C15ull) >> shift;
}

}  // namespace gleam
