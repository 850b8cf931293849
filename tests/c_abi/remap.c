/*
 * A plain C11 caller of the address-remap calls: hipMalloc'd storage, a HIP stream, no
 * C++ and no torch. Task 3's client allocation at (3 << 40) + 0x4000 holds two chunks
 * whose shareable copies sit in two different server allocations (the weight-sharing
 * case) and task 4 holds one more mapping; a later addition that overlaps task 3's first
 * chunk is refused. The translations of fixed probes are printed, then task 3's
 * allocation is freed and the probes are translated again, for the test that compares
 * everything printed with the CPU oracle.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "gleam.h"

#define HIP_OK(x)                                                                   \
  do {                                                                              \
    hipError_t e_ = (x);                                                            \
    if (e_ != hipSuccess) {                                                         \
      fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, hipGetErrorString(e_));    \
      return 1;                                                                     \
    }                                                                               \
  } while (0)
#define GLEAM_OK_(x)                                                                \
  do {                                                                              \
    gleam_status s_ = (x);                                                          \
    if (s_ != GLEAM_OK) {                                                           \
      fprintf(stderr, "%s:%d: %s (%s)\n", __FILE__, __LINE__, gleam_status_string(s_), \
              gleam_last_error());                                                  \
      return 1;                                                                     \
    }                                                                               \
  } while (0)

enum { N_ADD = 3, N_PROBE = 9, CAP = 64 };

static int print_translation(const gleam_remap* m, const uint64_t* d_probe, uint64_t* d_out, uint64_t* out,
                             hipStream_t stream, const char* tag) {
  GLEAM_OK_(gleam_remap_translate(m, d_probe, N_PROBE, d_out, stream));
  HIP_OK(hipStreamSynchronize(stream));
  HIP_OK(hipMemcpy(out, d_out, N_PROBE * sizeof(uint64_t), hipMemcpyDeviceToHost));
  for (int i = 0; i < N_PROBE; ++i) printf("%s %d %016llx\n", tag, i, (unsigned long long)out[i]);
  return 0;
}

int main(void) {
  const uint64_t va = (3ull << 40) + 0x4000;
  const uint64_t add_start[N_ADD] = {va, va + 0x3000, 4ull << 40};
  const uint64_t add_len[N_ADD] = {0x3000, 0x500, 16};
  const uint64_t add_target[N_ADD] = {0x7F0000000000ull, 0x7F8000001000ull, 1ull << 20};
  const uint64_t clash[3] = {va + 0x100, 8, 5};  /* start, length, target */
  const uint64_t probe[N_PROBE] = {va, va + 0x2FFF, va + 0x3000, va + 0x3004, va + 0x3500, va - 1,
                                   (4ull << 40) + 15, (4ull << 40) + 16, UINT64_MAX};
  const uint64_t del_start[1] = {va}, del_len[1] = {0x4000};

  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  const size_t bytes = gleam_remap_bytes(CAP);
  if (bytes == 0) return 1;
  void* d_storage;
  HIP_OK(hipMalloc(&d_storage, bytes));
  gleam_remap* m = NULL;
  GLEAM_OK_(gleam_remap_create(d_storage, bytes, CAP, &m, stream));

  uint64_t *d_add, *d_clash, *d_del, *d_probe, *d_out, *d_counts;
  uint8_t* d_status;
  HIP_OK(hipMalloc((void**)&d_add, 3 * N_ADD * sizeof(uint64_t)));
  HIP_OK(hipMalloc((void**)&d_clash, 3 * sizeof(uint64_t)));
  HIP_OK(hipMalloc((void**)&d_del, 2 * sizeof(uint64_t)));
  HIP_OK(hipMalloc((void**)&d_probe, N_PROBE * sizeof(uint64_t)));
  HIP_OK(hipMalloc((void**)&d_out, N_PROBE * sizeof(uint64_t)));
  HIP_OK(hipMalloc((void**)&d_counts, 4 * sizeof(uint64_t)));
  HIP_OK(hipMalloc((void**)&d_status, N_ADD));
  HIP_OK(hipMemcpy(d_add, add_start, sizeof add_start, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_add + N_ADD, add_len, sizeof add_len, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_add + 2 * N_ADD, add_target, sizeof add_target, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_clash, clash, sizeof clash, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_del, del_start, sizeof del_start, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_del + 1, del_len, sizeof del_len, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_probe, probe, sizeof probe, hipMemcpyHostToDevice));

  size_t ws_bytes = gleam_remap_update_bytes(m, N_ADD, 1);
  if (ws_bytes == 0) return 1;
  void* d_ws;
  HIP_OK(hipMalloc(&d_ws, ws_bytes));

  uint64_t counts[4], out[N_PROBE];
  uint8_t status[N_ADD];
  GLEAM_OK_(gleam_remap_update(m, NULL, NULL, 0, d_add, d_add + N_ADD, d_add + 2 * N_ADD, N_ADD, d_status,
                               d_counts, d_ws, ws_bytes, stream));
  HIP_OK(hipStreamSynchronize(stream));
  HIP_OK(hipMemcpy(counts, d_counts, sizeof counts, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(status, d_status, sizeof status, hipMemcpyDeviceToHost));
  printf("add %llu %llu %llu %llu\n", (unsigned long long)counts[0], (unsigned long long)counts[1],
         (unsigned long long)counts[2], (unsigned long long)counts[3]);
  for (int i = 0; i < N_ADD; ++i) printf("status %d %d\n", i, status[i]);

  GLEAM_OK_(gleam_remap_update(m, NULL, NULL, 0, d_clash, d_clash + 1, d_clash + 2, 1, d_status, d_counts, d_ws,
                               ws_bytes, stream));
  HIP_OK(hipStreamSynchronize(stream));
  HIP_OK(hipMemcpy(counts, d_counts, sizeof counts, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(status, d_status, 1, hipMemcpyDeviceToHost));
  printf("clash %llu %llu %llu %llu %d\n", (unsigned long long)counts[0], (unsigned long long)counts[1],
         (unsigned long long)counts[2], (unsigned long long)counts[3], status[0]);
  if (print_translation(m, d_probe, d_out, out, stream, "before")) return 1;

  GLEAM_OK_(gleam_remap_update(m, d_del, d_del + 1, 1, NULL, NULL, NULL, 0, NULL, d_counts, d_ws, ws_bytes,
                               stream));
  HIP_OK(hipStreamSynchronize(stream));
  HIP_OK(hipMemcpy(counts, d_counts, sizeof counts, hipMemcpyDeviceToHost));
  printf("free %llu %llu %llu %llu\n", (unsigned long long)counts[0], (unsigned long long)counts[1],
         (unsigned long long)counts[2], (unsigned long long)counts[3]);
  if (print_translation(m, d_probe, d_out, out, stream, "after")) return 1;

  GLEAM_OK_(gleam_remap_destroy(m));
  HIP_OK(hipFree(d_ws));
  HIP_OK(hipFree(d_status));
  HIP_OK(hipFree(d_counts));
  HIP_OK(hipFree(d_out));
  HIP_OK(hipFree(d_probe));
  HIP_OK(hipFree(d_del));
  HIP_OK(hipFree(d_clash));
  HIP_OK(hipFree(d_add));
  HIP_OK(hipFree(d_storage));
  HIP_OK(hipStreamDestroy(stream));
  return 0;
}
