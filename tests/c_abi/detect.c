/*
 * A plain C11 caller of libgleam: hipMalloc'd buffers, a HIP stream, no C++ and no torch.
 * Three payloads of a deterministic byte pattern go through fingerprint -> insert of the
 * first payload's blocks -> lookup of all blocks -> miss compaction, and the outputs are
 * printed as text for the test that compares them with the CPU oracle.
 *
 * Pattern: byte i of payload p is (uint8_t)((i * 2654435761u + p * 40503u) >> 11), then
 * payload 2 starts with a copy of payload 0's first 64 KiB block (held by the table after
 * the insert) and payload 3 repeats payload 1 (a duplicate inside the batch).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

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

enum { N_SEG = 4, BLOCK = 65536 };

int main(void) {
  const uint64_t lens[N_SEG] = {(1u << 20) + 17, 4096, 100000, 4096};
  uint64_t offs[N_SEG], total = 0;
  for (int p = 0; p < N_SEG; ++p) {
    offs[p] = total;
    total += (lens[p] + 255) / 256 * 256;
  }
  uint8_t* host = (uint8_t*)calloc(total, 1);
  if (!host) return 1;
  for (int p = 0; p < N_SEG; ++p)
    for (uint64_t i = 0; i < lens[p]; ++i)
      host[offs[p] + i] = (uint8_t)((((uint32_t)i * 2654435761u) + (uint32_t)p * 40503u) >> 11);
  memcpy(host + offs[2], host + offs[0], BLOCK);
  memcpy(host + offs[3], host + offs[1], 4096);

  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  uint8_t* d_arena;
  HIP_OK(hipMalloc((void**)&d_arena, total));
  HIP_OK(hipMemcpy(d_arena, host, total, hipMemcpyHostToDevice));

  uint64_t blk_first[N_SEG + 1], n_blocks = 0, addr[N_SEG];
  GLEAM_OK_(gleam_batch_geometry(lens, N_SEG, BLOCK, blk_first, &n_blocks));
  for (int p = 0; p < N_SEG; ++p) addr[p] = (uint64_t)(uintptr_t)(d_arena + offs[p]);
  uint64_t *d_addr, *d_len, *d_first;
  HIP_OK(hipMalloc((void**)&d_addr, sizeof addr));
  HIP_OK(hipMalloc((void**)&d_len, sizeof lens));
  HIP_OK(hipMalloc((void**)&d_first, sizeof blk_first));
  HIP_OK(hipMemcpy(d_addr, addr, sizeof addr, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_len, lens, sizeof lens, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_first, blk_first, sizeof blk_first, hipMemcpyHostToDevice));
  const gleam_batch batch = {d_addr, d_len, d_first, N_SEG, n_blocks, GLEAM_LEAF_BYTES, BLOCK};

  uint64_t *d_digest, *d_ref, *d_miss, *d_counters, *d_vals;
  uint8_t* d_status;
  void* d_ws;
  const size_t ws_bytes = gleam_workspace_bytes(n_blocks);
  HIP_OK(hipMalloc((void**)&d_digest, n_blocks * 8));
  HIP_OK(hipMalloc((void**)&d_ref, n_blocks * 8));
  HIP_OK(hipMalloc((void**)&d_miss, n_blocks * 8));
  HIP_OK(hipMalloc((void**)&d_counters, 16));
  HIP_OK(hipMalloc((void**)&d_vals, n_blocks * 8));
  HIP_OK(hipMalloc((void**)&d_status, n_blocks));
  HIP_OK(hipMalloc(&d_ws, ws_bytes));

  const uint64_t capacity = 1024;
  void* d_table;
  HIP_OK(hipMalloc(&d_table, gleam_cache_bytes(capacity)));
  gleam_cache* table = NULL;
  GLEAM_OK_(gleam_cache_create(d_table, gleam_cache_bytes(capacity), capacity, 0.7, &table, stream));

  GLEAM_OK_(gleam_fp_chunks(&batch, d_digest, NULL, stream));
  uint64_t vals[64];
  for (uint64_t g = 0; g < 64; ++g) vals[g] = 1000 + g;
  HIP_OK(hipMemcpyAsync(d_vals, vals, blk_first[1] * 8, hipMemcpyHostToDevice, stream));
  GLEAM_OK_(gleam_cache_insert(table, d_digest, d_vals, blk_first[1], NULL, d_ws, ws_bytes, stream));
  GLEAM_OK_(gleam_cache_lookup(table, d_digest, n_blocks, d_status, d_ref, d_ws, ws_bytes, stream));
  GLEAM_OK_(gleam_miss_compact(d_status, n_blocks, &batch, d_miss, d_counters, d_counters + 1, d_ws, ws_bytes,
                               stream));
  HIP_OK(hipStreamSynchronize(stream));

  uint64_t* digest = (uint64_t*)malloc(n_blocks * 8);
  uint64_t* ref = (uint64_t*)malloc(n_blocks * 8);
  uint64_t* miss = (uint64_t*)malloc(n_blocks * 8);
  uint8_t* status = (uint8_t*)malloc(n_blocks);
  uint64_t counters[2];
  if (!digest || !ref || !miss || !status) return 1;
  HIP_OK(hipMemcpy(digest, d_digest, n_blocks * 8, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(ref, d_ref, n_blocks * 8, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(miss, d_miss, n_blocks * 8, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(status, d_status, n_blocks, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(counters, d_counters, 16, hipMemcpyDeviceToHost));
  printf("blocks %llu\n", (unsigned long long)n_blocks);
  for (uint64_t g = 0; g < n_blocks; ++g)
    printf("block %llu %016llx %u %llu\n", (unsigned long long)g, (unsigned long long)digest[g], status[g],
           (unsigned long long)ref[g]);
  printf("misses %llu bytes %llu\n", (unsigned long long)counters[0], (unsigned long long)counters[1]);
  for (uint64_t i = 0; i < counters[0]; ++i) printf("miss %llu\n", (unsigned long long)miss[i]);

  gleam_cache_destroy(table);
  hipFree(d_table);
  hipFree(d_ws);
  hipFree(d_status);
  hipFree(d_vals);
  hipFree(d_counters);
  hipFree(d_miss);
  hipFree(d_ref);
  hipFree(d_digest);
  hipFree(d_first);
  hipFree(d_len);
  hipFree(d_addr);
  hipFree(d_arena);
  hipStreamDestroy(stream);
  free(host);
  free(digest);
  free(ref);
  free(miss);
  free(status);
  return 0;
}
