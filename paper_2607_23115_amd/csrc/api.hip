// Host-side parts of the libgleam C ABI: status text, error detail, batch geometry
// and workspace sizing.

#include <stdarg.h>
#include <atomic>
#include <stdio.h>

#include "gleam_internal.h"

namespace gleam {
namespace {
thread_local char g_last_error[512] = "";
}

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
}

void clear_error() { g_last_error[0] = '\0'; }

gleam_status launch_status(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return GLEAM_OK;
  set_error("%s: %s", what, hipGetErrorString(e));
  return GLEAM_E_HIP;
}

int log2_exact(uint64_t x) {
  if (x == 0 || (x & (x - 1)) != 0) return -1;
  int r = 0;
  while ((1ull << r) != x) ++r;
  return r;
}

bool valid_block_bytes(uint32_t block_bytes) {
  const int l = log2_exact(block_bytes);
  return l >= 12 && l <= 24;
}

bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255) == 0; }

gleam_status device_cu_count(int* cus) {
  static std::atomic<int> cached[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    set_error("hipGetDevice: %s", hipGetErrorString(e));
    return GLEAM_E_HIP;
  }
  if (dev >= 0 && dev < 64) {
    const int c = cached[dev].load(std::memory_order_relaxed);
    if (c > 0) {
      *cus = c;
      return GLEAM_OK;
    }
  }
  int n = 0;
  e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess || n <= 0) {
    set_error("hipDeviceGetAttribute(multiprocessor count): %s", hipGetErrorString(e));
    return GLEAM_E_HIP;
  }
  if (dev >= 0 && dev < 64) cached[dev].store(n, std::memory_order_relaxed);
  *cus = n;
  return GLEAM_OK;
}

WsLayout ws_layout(uint64_t n) {
  WsLayout L{};
  if (n > kMaxWsItems) {  // no workspace is that large; the calls refuse such an n
    L.total = SIZE_MAX;
    return L;
  }
  uint64_t cap = 64;
  while (cap < 4 * n) cap <<= 1;
  L.scratch_cap = cap;
  L.scratch_off = kHeaderBytes;
  L.tiles = (n + kTileItems - 1) / kTileItems;
  L.tiles_off = L.scratch_off + (size_t)cap * 8;
  L.total = L.tiles_off + (size_t)(L.tiles + 1) * 16;
  L.total = (L.total + 255) & ~(size_t)255;
  return L;
}

gleam_status check_workspace(const WsLayout& L, const void* ws, size_t ws_bytes, const char* who) {
  if (L.total == SIZE_MAX) {
    set_error("%s: more than 2^40 items", who);
    return GLEAM_E_UNSUPPORTED;
  }
  if (!ws || !aligned256(ws)) {
    set_error("%s: workspace must be non-null and 256-byte aligned", who);
    return GLEAM_E_INVALID;
  }
  if (ws_bytes < L.total) {
    set_error("%s: workspace of %zu bytes, %zu needed", who, ws_bytes, L.total);
    return GLEAM_E_WORKSPACE;
  }
  return GLEAM_OK;
}

}  // namespace gleam

extern "C" gleam_status gleam_preload(void) {
  using namespace gleam;
  clear_error();
  hipError_t (*const loads[])() = {preload_fp_chunks, preload_cache,    preload_compact, preload_detect,
                                   preload_identify,  preload_first_write, preload_md5,  preload_lifecycle,
                                   preload_transfer,  preload_remap,    preload_calib};
  for (auto load : loads) {
    const hipError_t e = load();
    if (e != hipSuccess) {
      set_error("gleam_preload: %s", hipGetErrorString(e));
      return GLEAM_E_HIP;
    }
  }
  return GLEAM_OK;
}

extern "C" const char* gleam_status_string(gleam_status s) {
  switch (s) {
    case GLEAM_OK: return "ok";
    case GLEAM_E_INVALID: return "invalid argument";
    case GLEAM_E_CAPACITY: return "table capacity exceeded";
    case GLEAM_E_WORKSPACE: return "workspace too small";
    case GLEAM_E_HIP: return "HIP error";
    case GLEAM_E_UNSUPPORTED: return "unsupported";
    default: return "unknown status";
  }
}

extern "C" const char* gleam_last_error(void) { return gleam::g_last_error; }

extern "C" size_t gleam_workspace_bytes(uint64_t n) {
  if (n > gleam::kMaxWsItems) return 0;
  return gleam::ws_layout(n).total;
}

extern "C" gleam_status gleam_batch_geometry(const uint64_t* host_seg_len, uint64_t n_seg, uint32_t block_bytes,
                                             uint64_t* host_blk_first, uint64_t* n_blocks) {
  gleam::clear_error();
  if (!gleam::valid_block_bytes(block_bytes)) {
    gleam::set_error("gleam_batch_geometry: block_bytes must be 4096 << k, k <= 12");
    return GLEAM_E_INVALID;
  }
  if (!host_blk_first || (n_seg > 0 && !host_seg_len)) {
    gleam::set_error("gleam_batch_geometry: null array");
    return GLEAM_E_INVALID;
  }
  uint64_t total = 0;
  for (uint64_t s = 0; s < n_seg; ++s) {
    host_blk_first[s] = total;
    total += host_seg_len[s] / block_bytes + (host_seg_len[s] % block_bytes != 0);
  }
  host_blk_first[n_seg] = total;
  if (n_blocks) *n_blocks = total;
  return GLEAM_OK;
}
