// Device-side probe of the resident identifier table (layout in gleam_internal.h:
// open addressing with linear probing over 16-byte {key, value} slots; the key kEmpty
// lives in the header). Shared by the lookup kernels and the one-launch detect kernel.
#pragma once

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

// (hit, value) of key k. The table is never full (the host caps its load), so the walk
// meets an empty slot; it is still bounded by the capacity.
__device__ __forceinline__ bool table_find(const TableRef& t, uint64_t k, uint64_t* val) {
  if (k == kEmpty) {
    *val = t.hdr[1];
    return t.hdr[0] != 0;
  }
  uint64_t pos = slot_hash(k, t.shift);
  for (uint64_t probe = 0; probe <= t.mask; ++probe) {
    const uint4 e = *reinterpret_cast<const uint4*>(t.slots + 2 * pos);
    const uint64_t key = lo64(e);
    if (key == k) {
      *val = hi64(e);
      return true;
    }
    if (key == kEmpty) return false;
    pos = (pos + 1) & t.mask;
  }
  return false;
}

// The home slot of key k (k != kEmpty), read ahead of table_find: most probes end there.
__device__ __forceinline__ uint4 table_home(const TableRef& t, uint64_t k) {
  return *reinterpret_cast<const uint4*>(t.slots + 2 * slot_hash(k, t.shift));
}

// table_find given the home slot already read: a hit or an empty home decides at once.
__device__ __forceinline__ bool table_find_from(const TableRef& t, uint64_t k, uint4 home, uint64_t* val) {
  if (k != kEmpty && lo64(home) == k) {
    *val = hi64(home);
    return true;
  }
  if (k != kEmpty && lo64(home) == kEmpty) return false;
  return table_find(t, k, val);
}

}  // namespace
}  // namespace gleam
