// Host-side helpers shared by the libgleam translation units (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "gleam.h"

// Host view of a table: storage = [256-byte header][capacity x (key u64, value u64)]
// [capacity x last-use stamp u64]. Header u64 words: 0 flag "the key kEmpty is
// present", 1 its value, 2 its stamp.
struct gleam_cache {
  uint8_t* storage;
  uint64_t capacity;
  int shift;           // 64 - log2(capacity)
  uint64_t max_keys;   // floor(max_load * capacity), at most capacity - 1
  uint64_t key_bound;  // upper bound on keys present
};

// Host view of an address-remap map: storage = [256-byte header][capacity x start]
// [capacity x {end, target}][fence], sorted by start (layout in remap.hip).
struct gleam_remap {
  uint8_t* storage;
  uint64_t capacity;
};

namespace gleam {

constexpr size_t kHeaderBytes = 256;

// Device view of a table (kernel argument).
struct TableRef {
  uint64_t* hdr;     // [0] flag: key kEmpty present, [1] its value, [2] its stamp
  uint64_t* slots;   // capacity x {key, value}
  uint64_t* stamps;  // capacity last-use stamps
  uint64_t mask;
  int shift;
};

inline TableRef table_ref(const gleam_cache* c) {
  TableRef t;
  t.hdr = reinterpret_cast<uint64_t*>(c->storage);
  t.slots = reinterpret_cast<uint64_t*>(c->storage + kHeaderBytes);
  t.stamps = t.slots + 2 * c->capacity;
  t.mask = c->capacity - 1;
  t.shift = c->shift;
  return t;
}

// Enqueue the clear of a table: header zero, keys kEmpty, values and stamps zero.
gleam_status clear_table(const gleam_cache* c, hipStream_t stream);
constexpr uint64_t kTileItems = 2048;  // statuses per compaction workgroup

// Workspace layout for n items: [header 256 B][scratch table][tile counts][tile offsets].
// Header u64 words: 0 = scratch min-index of the key kEmpty, 1 = new-key counter,
// 2 = short-block byte deficit.
struct WsLayout {
  uint64_t scratch_cap;   // power of two >= max(64, 4n)
  size_t scratch_off;
  uint64_t tiles;
  size_t tiles_off;
  size_t total;
};
constexpr uint64_t kMaxWsItems = 1ull << 40;  // larger n: total = SIZE_MAX, refused
WsLayout ws_layout(uint64_t n);
// The workspace checks every call makes, in one order: an n beyond any layout
// (GLEAM_E_UNSUPPORTED), a null or unaligned pointer (GLEAM_E_INVALID), too few bytes
// (GLEAM_E_WORKSPACE). Sets the error text with `who`.
gleam_status check_workspace(const WsLayout& L, const void* ws, size_t ws_bytes, const char* who);

void set_error(const char* fmt, ...);
void clear_error();
gleam_status launch_status(const char* what);  // GLEAM_OK, or GLEAM_E_HIP after a failed launch
bool valid_block_bytes(uint32_t block_bytes);
int log2_exact(uint64_t x);                    // -1 unless x is a power of two
bool aligned256(const void* p);
gleam_status device_cu_count(int* cus);        // compute units of the current device (cached)

// Batch checks shared by the entry points that take a batch (nothing enqueued on error).
gleam_status validate_batch(const gleam_batch* b, const char* who);
// Block digests of a validated batch (the fingerprint kernel launch).
gleam_status launch_fp(const gleam_batch* b, uint64_t* d_block_digest, uint64_t* d_leaf_digest, hipStream_t stream);

// Fill n u64 words with value on stream (a kernel, so it can live in a captured graph).
gleam_status fill_u64(uint64_t* p, uint64_t n, uint64_t value, hipStream_t stream);


// Each source file's code-object preload (gleam_preload calls them all).
hipError_t preload_cache();
hipError_t preload_calib();
hipError_t preload_compact();
hipError_t preload_detect();
hipError_t preload_first_write();
hipError_t preload_fp_chunks();
hipError_t preload_identify();
hipError_t preload_lifecycle();
hipError_t preload_md5();
hipError_t preload_remap();
hipError_t preload_transfer();

}  // namespace gleam
