// gleam_detect: the whole decision for one batch in one call (Gleam Sec. 4.1.2: a chunk
// whose identifier the server holds sends only its hash and size, any other chunk its
// bytes): block digests, the table probe with dedup inside the batch, and the ascending
// list of blocks whose bytes must travel, with its count and byte total. The outputs are
// those of gleam_fp_chunks, gleam_cache_lookup and gleam_miss_compact called in order.
//
// Small batches are latency-bound: their three launches cost more than their bytes. Up
// to kDetectMaxSlots leaf slots, in blocks of at most 64 KiB and at most kDetectMaxBlocks
// blocks, one kernel does it all. Every workgroup fingerprints its leaves with four lanes
// per leaf (the small-batch scheme of gleam_fp_chunks), stores each block's byte length
// in the workspace, probes the resident table for each of its blocks (a hit's status is
// final; the probe's latency overlaps other workgroups' streaming), makes its writes
// visible to the whole device and arrives at a counter. The last workgroup to arrive
// resolves the blocks that the table does not hold and that repeat inside the batch in an
// LDS table (the lowest index is the MISS), and compacts the misses with one workgroup
// scan, then re-arms the counter for the next call. The
// counter is armed once per workspace (gleam_detect_ws_init), so a call is one launch.
// Larger batches run the kernels of the three calls in order.

#include "fp_core.h"
#include "gleam_table.h"

namespace gleam {
namespace {

constexpr uint64_t kDetectMaxSlots = kQuadMaxSlots;  // 65,536 leaf slots
constexpr uint64_t kDetectMaxBlocks = 4096;
constexpr uint64_t kDetectSoloBlocks = 512;  // one-wave workgroups: at most 8 blocks per lane
constexpr size_t kArriveWord = 16;           // workspace header word holding the counter
// Arrival counter: kArmed in the upper 32 bits, arrivals in the lower. gleam_detect_ws_init
// arms it; the last workgroup of every call re-arms it, so no call needs a clear launch.
constexpr uint64_t kArmed = 0x676C6561ull;
// s_waitcnt vmcnt(0) (expcnt and lgkmcnt left at their maxima): this wave's stores done
constexpr int kWaitStores = 0x0F70;

struct DetectArgs {
  FpArgs fp;  // block_out: the digests
  TableRef t;
  uint8_t* status;
  uint64_t* ref;         // nullable
  uint64_t* miss_idx;
  uint64_t* miss_count;
  uint64_t* miss_bytes;  // nullable
  uint32_t* blen;        // workspace: byte length of each block
  uint64_t* arrive;      // workspace: the armed arrival counter
};

// Workspace of gleam_detect: [256-byte header, word 16 the arrival counter][u32 per block:
// its byte length (one-kernel path)]; larger batches use it as the three calls' workspace,
// which leaves header word 16 alone. gleam_detect_ws_init arms the counter.
size_t detect_own_bytes(uint64_t n) { return (kHeaderBytes + 4 * (size_t)n + 255) & ~(size_t)255; }

// Exclusive scan of one value per thread over a workgroup of W waves; *total gets the sum.
template <int W>
__device__ __forceinline__ uint32_t wg_exclusive_scan(uint32_t x, uint32_t* wave_sums, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = x;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(incl, d, 64);
    if (lane >= d) incl += y;
  }
  if (lane == 63) wave_sums[wave] = incl;
  __syncthreads();
  uint32_t before = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < W; ++w) {
    const uint32_t s = wave_sums[w];
    before += w < wave ? s : 0u;
    sum += s;
  }
  *total = sum;
  return before + incl - x;
}

// Phase-1 probe of one block's digest (in the lane that computed it).
struct TableProbe {
  TableRef t;
  uint8_t* status;
  uint64_t* ref;
  __device__ __forceinline__ void operator()(uint64_t g, uint64_t key) const {
    uint64_t val = 0;
    if (table_find(t, key, &val)) {
      status[g] = GLEAM_HIT_CACHE;
      if (ref) ref[g] = val;
    } else {
      status[g] = kProbePending;
    }
  }
};

template <int W>
__global__ __launch_bounds__(64 * W) void detect_small_kernel(DetectArgs a) {
  constexpr int T = 64 * W;
  constexpr uint32_t kMax = W == 1 ? (uint32_t)kDetectSoloBlocks : (uint32_t)kDetectMaxBlocks;
  constexpr int K = (int)(kMax / T);                 // blocks per thread in the tail
  constexpr uint32_t kSlots = W * kQuadWaveLds / 8;  // dedup slots over (part of) the stage tiles
  constexpr int kShift = 64 - (W == 1 ? 11 : 13);    // log2(kSlots)
  static_assert(kSlots == (1u << (64 - kShift)), "dedup table size");
  static_assert(kSlots >= 2 * kMax, "dedup table load at most 1/2");
  static_assert(16 * T >= (int)kMax, "one compaction round");
  __shared__ __attribute__((aligned(16))) uint8_t lds[W == 1 ? kQuadDirectLds : W * kQuadWaveLds];
  __shared__ __attribute__((aligned(16))) uint8_t st[kMax];
  __shared__ uint32_t last;
  __shared__ uint32_t wave_sums[W];
  __shared__ uint64_t wave_bytes[W];

  // digests, block lengths, and each block's table probe
  quad_pass<W, true, W == 1>(a.fp, blockIdx.x, lds, a.blen, TableProbe{a.t, a.status, a.ref});
  // Arrive. Each thread waits for its own stores (digests, lengths, statuses) to
  // complete; after the barrier one release at device scope per workgroup writes them
  // back from this XCD's L2, and the arrival counts. (A device-scope fence in every wave
  // costs a cache write-back per wave: measured 2x slower on a 224-workgroup batch.)
  __builtin_amdgcn_s_waitcnt(kWaitStores);
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    const uint64_t old = atomicAdd(reinterpret_cast<unsigned long long*>(a.arrive), 1ull);
    const bool armed = (old >> 32) == kArmed;
    last = !armed ? 2u : ((uint32_t)old + 1 == gridDim.x ? 1u : 0u);
  }
  __syncthreads();
  if (last == 2) {  // the workspace was not prepared: say so in the count
    if (threadIdx.x == 0) *a.miss_count = ~0ull;
    return;
  }
  if (!last) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");

  // ---- the last workgroup: dedup of the blocks the table does not hold, then compaction
  // (thread t owns blocks g = j * T + t)
  const uint32_t n = (uint32_t)a.fp.n_blocks;
  const uint64_t* keys = a.fp.block_out;
  // dedup slots: (low 32 bits of the key) << 32 | (lowest index + 1); 0 = free
  uint64_t* slots = reinterpret_cast<uint64_t*>(lds);
  const uint32_t tid = threadIdx.x;
  if (tid == 0) *a.arrive = kArmed << 32;  // every workgroup has arrived: ready for the next call
  // statuses, keys and lengths of this thread's blocks, all loaded together (the keys and
  // lengths of held blocks are not needed, but waiting for the statuses first would cost
  // a round trip)
  uint8_t s0[K];
  uint64_t k[K];
  uint32_t len[K];
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const uint32_t g = (uint32_t)j * T + tid;
    s0[j] = g < n ? a.status[g] : (uint8_t)GLEAM_HIT_CACHE;
    k[j] = g < n ? keys[g] : 0;
    len[j] = g < n ? a.blen[g] : 0;
  }
  for (uint32_t i = tid; i < kSlots; i += T) slots[i] = 0;
  __syncthreads();  // dedup table cleared
  uint32_t at[K];   // a pending block's dedup slot
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const uint32_t g = (uint32_t)j * T + tid;
    at[j] = 0;
    if (g >= n) continue;
    st[g] = s0[j];
    if (s0[j] != kProbePending) continue;
    const uint64_t tag = (uint64_t)(uint32_t)k[j] << 32;
    const uint64_t mine = tag | (g + 1);
    uint32_t pos = (uint32_t)slot_hash(k[j], kShift);
    for (uint32_t probe = 0; probe < kSlots; ++probe) {
      const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long*>(&slots[pos]), 0ull, mine);
      // the slot of this key: same tag, and (read only then) the same whole key; every
      // value it ever holds has this tag, so the minimum keeps the lowest index
      if (prev == 0 || ((prev & ~0xFFFFFFFFull) == tag && keys[(uint32_t)prev - 1] == k[j])) {
        if (prev != 0) atomicMin(reinterpret_cast<unsigned long long*>(&slots[pos]), mine);
        break;
      }
      pos = (pos + 1) & (kSlots - 1);
    }
    at[j] = pos;
  }
  __syncthreads();
  uint64_t bytes = 0;  // bytes of this thread's MISS blocks
#pragma unroll
  for (int j = 0; j < K; ++j) {
    if (s0[j] != kProbePending) continue;
    const uint32_t g = (uint32_t)j * T + tid;
    const uint32_t g0 = (uint32_t)slots[at[j]] - 1;
    const uint8_t s = g0 == g ? (uint8_t)GLEAM_MISS : (uint8_t)GLEAM_HIT_BATCH;
    a.status[g] = s;
    if (a.ref) a.ref[g] = g0;
    st[g] = s;
    if (s == GLEAM_MISS) bytes += len[j];
  }
  __syncthreads();

  // ---- compaction: thread t takes statuses [16 t, 16 t + 16), one workgroup scan
  const uint32_t first = tid * 16;
  uint32_t bits = 0;
  if (first < n) {
    const uint4 v = *reinterpret_cast<const uint4*>(st + first);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (first + e < n && ((w[e >> 2] >> (8 * (e & 3))) & 0xFFu) == GLEAM_MISS) bits |= 1u << e;
  }
  uint32_t total;
  const uint32_t excl = wg_exclusive_scan<W>((uint32_t)__builtin_popcount(bits), wave_sums, &total);
  uint64_t out = excl;
  for (uint32_t m = bits; m; m &= m - 1) a.miss_idx[out++] = first + (uint32_t)__builtin_ctz(m);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) bytes += shfl_xor64(bytes, o);
  if ((tid & 63) == 0) wave_bytes[tid >> 6] = bytes;
  __syncthreads();
  if (tid == 0) {
    uint64_t sum = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) sum += wave_bytes[w];
    *a.miss_count = total;
    if (a.miss_bytes) *a.miss_bytes = sum;
  }
}

__global__ void detect_arm_kernel(uint64_t* arrive) { *arrive = kArmed << 32; }

}  // namespace
// Loads this file's GPU code object on the current device (gleam_preload).
hipError_t preload_detect() {
  hipFuncAttributes attr;
  return hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(&detect_arm_kernel));
}

}  // namespace gleam

extern "C" size_t gleam_detect_workspace_bytes(uint64_t n_blocks) {
  using namespace gleam;
  if (n_blocks > kMaxWsItems) return 0;
  const size_t own = detect_own_bytes(n_blocks), three = ws_layout(n_blocks).total;
  return own > three ? own : three;
}

extern "C" gleam_status gleam_detect_ws_init(void* d_ws, size_t ws_bytes, void* stream) {
  using namespace gleam;
  clear_error();
  if (!d_ws || !aligned256(d_ws) || ws_bytes < kHeaderBytes) {
    set_error("gleam_detect_ws_init: workspace must be non-null, 256-byte aligned and at least %zu bytes",
              kHeaderBytes);
    return GLEAM_E_INVALID;
  }
  hipLaunchKernelGGL(detect_arm_kernel, dim3(1), dim3(1), 0, (hipStream_t)stream,
                     static_cast<uint64_t*>(d_ws) + kArriveWord);
  return launch_status("detect_arm_kernel");
}

extern "C" gleam_status gleam_detect(const gleam_batch* b, const gleam_cache* c, uint64_t* d_digest,
                                     uint8_t* d_status, uint64_t* d_ref, uint64_t* d_miss_idx,
                                     uint64_t* d_miss_count, uint64_t* d_miss_bytes, void* d_ws, size_t ws_bytes,
                                     void* stream) {
  using namespace gleam;
  clear_error();
  gleam_status st = validate_batch(b, "gleam_detect");
  if (st != GLEAM_OK) return st;
  if (!c || !d_miss_count) {
    set_error("gleam_detect: null table or miss count");
    return GLEAM_E_INVALID;
  }
  const uint64_t n = b->n_blocks;
  if (n > 0 && (!d_digest || !d_status || !d_miss_idx)) {
    set_error("gleam_detect: null digest, status or miss list for a non-empty batch");
    return GLEAM_E_INVALID;
  }
  const size_t need = gleam_detect_workspace_bytes(n);
  if (need == 0) {
    set_error("gleam_detect: more than 2^40 blocks");
    return GLEAM_E_UNSUPPORTED;
  }
  if (!d_ws || !aligned256(d_ws)) {
    set_error("gleam_detect: workspace must be non-null and 256-byte aligned");
    return GLEAM_E_INVALID;
  }
  if (ws_bytes < need) {
    set_error("gleam_detect: workspace of %zu bytes, %zu needed", ws_bytes, need);
    return GLEAM_E_WORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  if (n == 0) return gleam_miss_compact(nullptr, 0, b, nullptr, d_miss_count, d_miss_bytes, d_ws, ws_bytes, stream);

  uint8_t* ws = static_cast<uint8_t*>(d_ws);
  uint64_t* hdr = reinterpret_cast<uint64_t*>(d_ws);
  const int lpb_log2 = log2_exact(b->block_bytes) - 12;
  const uint64_t lpb = 1ull << lpb_log2;
  const uint64_t slots = n * lpb;
  if (lpb <= (uint64_t)kQuadLeaves && slots <= kDetectMaxSlots && n <= kDetectMaxBlocks) {
    int cus = 0;
    st = device_cu_count(&cus);
    if (st != GLEAM_OK) return st;
    const uint64_t waves = (slots + kQuadLeaves - 1) / kQuadLeaves;
    DetectArgs a;
    a.fp = FpArgs{b->seg_addr, b->seg_len, b->blk_first, b->n_seg, n, d_digest, nullptr, (uint32_t)lpb_log2, waves};
    a.t = table_ref(c);
    a.status = d_status;
    a.ref = d_ref;
    a.miss_idx = d_miss_idx;
    a.miss_count = d_miss_count;
    a.miss_bytes = d_miss_bytes;
    a.blen = reinterpret_cast<uint32_t*>(ws + kHeaderBytes);
    a.arrive = hdr + kArriveWord;
    // one-wave workgroups while they spread the batch over more CUs (as in gleam_fp_chunks)
    // and the last one's 64 lanes hold at most 8 blocks each
    if (waves <= 2ull * (uint64_t)cus && n <= kDetectSoloBlocks) {
      hipLaunchKernelGGL(detect_small_kernel<1>, dim3((uint32_t)waves), dim3(64), 0, s, a);
    } else {
      hipLaunchKernelGGL(detect_small_kernel<4>, dim3((uint32_t)((waves + 3) / 4)), dim3(256), 0, s, a);
    }
    return launch_status("detect_small_kernel");
  }
  // larger batches: the three calls' kernels (measured faster than a fused pipeline, in
  // which the fingerprint kernel's lanes probed the table and recorded their digests
  // in the workspace: that kernel's workgroups waited for the atomics' round trips)
  st = launch_fp(b, d_digest, nullptr, s);
  if (st != GLEAM_OK) return st;
  st = gleam_cache_lookup(c, d_digest, n, d_status, d_ref, d_ws, ws_bytes, stream);
  if (st != GLEAM_OK) return st;
  return gleam_miss_compact(d_status, n, d_miss_bytes ? b : nullptr, d_miss_idx, d_miss_count, d_miss_bytes, d_ws,
                            ws_bytes, stream);
}
