// gleam_read_stream: a read-only pass over device bytes, the measured HBM read ceiling
// that the fingerprint kernel's roofline fraction is set against. It is a measurement
// aid beside the path, not a step of it.
//
// The pattern is the fastest plain read found on MI355X: each wave streams whole
// 128 KiB regions (region w, w + waves, ...), one contiguous 1 KiB per load
// instruction, 16 non-temporal 16-byte loads in flight per lane, with one 4-wave
// workgroup per CU (more waves in flight read slower). Bytes past the last whole
// region are read 16 bytes per lane. Every loaded word is XOR-folded, so no load is
// dead; one atomic XOR per wave publishes the fold.

#include "gleam_device.h"
#include "gleam_internal.h"

namespace gleam {
namespace {

constexpr uint64_t kRegion = 128u << 10;
constexpr int kThreads = 256;
constexpr int kDepth = 16;

__global__ __launch_bounds__(kThreads) void read_stream_kernel(const uint8_t* src, uint64_t regions,
                                                               uint64_t tail_chunks, unsigned long long* sink) {
  const int lane = threadIdx.x & 63;
  constexpr int W = kThreads / 64;
  uint64_t acc = 0;
  const uint64_t waves = (uint64_t)gridDim.x * W;
  for (uint64_t r = (uint64_t)blockIdx.x * W + (threadIdx.x >> 6); r < regions; r += waves) {
    const uint8_t* lp = src + r * kRegion + lane * 16;
    // kept rolled: unrolled, the compiler interleaves the XORs with the loads and keeps
    // only one or two loads in flight
#pragma unroll 1
    for (int t0 = 0; t0 < (int)(kRegion / 1024); t0 += kDepth) {
      uint4 R[kDepth];
#pragma unroll
      for (int k = 0; k < kDepth; ++k) R[k] = load_stream16(lp + (uint64_t)(t0 + k) * 1024);
#pragma unroll
      for (int k = 0; k < kDepth; ++k) acc ^= lo64(R[k]) ^ hi64(R[k]);
    }
  }
  const uint8_t* tail = src + regions * kRegion;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; c < tail_chunks; c += stride) {
    const uint4 v = load_stream16(tail + 16 * c);
    acc ^= lo64(v) ^ hi64(v);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc ^= shfl_xor64(acc, o);
  if (lane == 0) atomicXor(sink, (unsigned long long)acc);
}

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_calib() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&read_stream_kernel));
}

}  // namespace gleam

extern "C" gleam_status gleam_read_stream(const void* d_src, uint64_t bytes, uint64_t* d_sink, void* stream) {
  using namespace gleam;
  clear_error();
  if (!d_sink || (bytes > 0 && !d_src)) {
    set_error("gleam_read_stream: null source or sink");
    return GLEAM_E_INVALID;
  }
  if ((reinterpret_cast<uintptr_t>(d_src) & 15) || (bytes & 15)) {
    set_error("gleam_read_stream: source and length must be multiples of 16 bytes");
    return GLEAM_E_INVALID;
  }
  if (bytes == 0) return GLEAM_OK;
  int cus = 0;
  gleam_status st = device_cu_count(&cus);
  if (st != GLEAM_OK) return st;
  const uint64_t regions = bytes / kRegion;
  const uint64_t tail_chunks = (bytes % kRegion) / 16;
  // one workgroup per CU; fewer when there are fewer regions than waves
  const uint64_t want = regions > 0 ? (regions + 3) / 4 : 1;
  const uint32_t grid = (uint32_t)(want < (uint64_t)cus ? want : (uint64_t)cus);
  hipLaunchKernelGGL(read_stream_kernel, dim3(grid), dim3(kThreads), 0, (hipStream_t)stream,
                     static_cast<const uint8_t*>(d_src), regions, tail_chunks,
                     reinterpret_cast<unsigned long long*>(d_sink));
  return launch_status("read_stream_kernel");
}
