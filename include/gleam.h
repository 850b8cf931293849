/*
 * gleam.h -- GPU cache-hit detection for host-to-device weight payloads (gfx950).
 *
 * The operation (Gleam, Sec. 4.1.2 "Hash-based Weight Chunk Retrieval"): the
 * server keeps the hash identifiers of the weight chunks it already holds; every
 * host-to-device copy payload is hashed from its bytes, and only payloads whose
 * identifier is not held must send their bytes over the network (a hit sends the
 * identifier and size, and the server restores the bytes locally). Sec. 4.1.1
 * defines the payload ("chunk") as the bytes of one host-to-device copy, and
 * Sec. 4.1.3 keeps identified chunks for later reuse.
 *
 * This library decides it per fixed-size block of each payload, on the GPU:
 *   gleam_fp_chunks     -- digest every block (XXH64 per 4 KiB leaf, seed 0,
 *                          folded by a bottom-up pairwise tree)
 *   gleam_cache_lookup  -- probe the resident identifier table; detect blocks
 *                          repeated inside the batch
 *   gleam_miss_compact  -- list the blocks whose bytes must still travel
 *   gleam_detect        -- the three above in one call (one launch for a small batch)
 *   gleam_cache_insert  -- add identifiers to the table
 *   gleam_cache_touch / _evict / _erase / _export -- the table's lifecycle: last-use
 *                          stamps, LRU eviction, removal, the identifier set (4.1.3)
 *   gleam_identify_weights -- at free time, decide which allocations still hold
 *                          exactly what was written to them (Sec. 4.1.1)
 *   gleam_identify_leaves  -- the same, located to the first changed 4 KiB leaf
 *   gleam_first_writes  -- the first-write rule: the bytes each recorded write owns
 *   gleam_md5_prefix    -- the paper's own identifier (MD5 of a payload's first
 *                          1024 bits), as an ablation
 *   gleam_send_plan / gleam_pack_misses / gleam_restore_blocks -- the transfer
 *                          around the decision: what travels, packed, and rebuilt
 *   gleam_remap_*       -- the address-remap map of the weight-sharing layer: ranges
 *                          of client device addresses onto shareable positions (4.1.3)
 *   gleam_read_stream   -- calibration only: the measured HBM read ceiling
 *
 * Conventions for every entry point:
 *   - C ABI; no exception crosses it; functions are thread-compatible (distinct
 *     handles and buffers may be used from distinct threads).
 *   - "device" pointers point to GPU memory (hipMalloc'd or a torch tensor);
 *     "host" pointers to CPU memory. The CALLER owns all device memory:
 *     payloads, descriptors, outputs, workspace and table storage. The library
 *     allocates no device memory; it owns only the small host-side
 *     gleam_cache handle.
 *   - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued
 *     asynchronously on it; outputs are valid once the stream has synchronised.
 *     The library never synchronises.
 *   - A workspace (d_ws) is scratch for the one call it is passed to: its contents on
 *     entry do not matter and are undefined on return. Calls that may run at the same
 *     time (on different streams) need separate workspaces.
 *   - Arguments are validated on the host before anything is enqueued; on any
 *     error a negative status is returned and nothing has been enqueued. A HIP
 *     launch failure returns GLEAM_E_HIP; gleam_last_error() then holds the HIP
 *     message (thread-local).
 *   - HIP graph capture: every call enqueues kernel launches only (clears are fill
 *     kernels, not memsets; sorts and scans are the library's own kernels), so a caller
 *     may capture it in a graph and replay it. gleam_cache_insert's and
 *     gleam_cache_evict's host-side key bound changes once, when the call is captured,
 *     not on each replay.
 *   - Device descriptor contents (seg_addr, seg_len, blk_first) are not read on
 *     the host. The caller guarantees they describe the batch. Whatever they hold,
 *     a kernel reads a payload P = [seg_addr[s], seg_addr[s] + seg_len[s]) only
 *     with loads that lie inside P, or with aligned 8-byte loads that hold at least
 *     one byte of P, so it never touches a page that holds no byte of P:
 *       fingerprint (and identify): 16-byte loads at a leaf's own start + 16 i,
 *         covering the leaf's whole 32-byte stripes; the tail (< 32 bytes) in the
 *         aligned 8-byte words that hold it;
 *       MD5 prefix: 4-byte loads at the payload start + 4 i over whole 64-byte
 *         blocks of the prefix, then single bytes;
 *       pack / restore: 16-byte loads and stores at a block's own start + 16 i,
 *         then single bytes.
 *     These loads keep the payload's alignment, so they are unaligned whenever the
 *     payload is: the library relies on the unaligned global access that gfx950
 *     runs with under ROCm (the HSA default). 16-byte aligned payloads stream
 *     fastest, 4-byte aligned ones at about 85% of that rate, others at 65-70%.
 */
#ifndef GLEAM_H
#define GLEAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t gleam_status;
enum {
  GLEAM_OK = 0,
  GLEAM_E_INVALID = -1,     /* a null required pointer, a bad size or alignment */
  GLEAM_E_CAPACITY = -2,    /* an insert could push the table past its maximum load */
  GLEAM_E_WORKSPACE = -3,   /* workspace smaller than gleam_workspace_bytes(n) */
  GLEAM_E_HIP = -4,         /* a HIP call or kernel launch failed */
  GLEAM_E_UNSUPPORTED = -5  /* valid, but beyond what this library handles */
};

/* Per-block status byte written by gleam_cache_lookup. */
enum {
  GLEAM_MISS = 0,       /* bytes must travel; ref = the block's own index */
  GLEAM_HIT_CACHE = 1,  /* digest held by the table; ref = the table's value */
  GLEAM_HIT_BATCH = 2   /* an earlier block of this batch has the same digest;
                           ref = the earliest such block (which is a MISS) */
};

#define GLEAM_LEAF_BYTES 4096u
#define GLEAM_MIN_BLOCK_BYTES 4096u
#define GLEAM_MAX_BLOCK_BYTES (4096u << 12) /* 16 MiB */

/*
 * A batch of host-to-device payloads (Sec. 4.1.1: one payload = the bytes of one
 * host-to-device copy). Each payload is cut, from its first byte, into 4 KiB
 * leaves and blocks of block_bytes; a payload's last leaf and last block may be
 * short. Global block index g = blk_first[s] + j for block j of payload s.
 *   seg_addr  device u64[n_seg]    device address of payload s (any alignment; 16-byte
 *                                  aligned payloads stream fastest, then 4-byte aligned)
 *   seg_len   device u64[n_seg]    bytes of payload s (0 allowed)
 *   blk_first device u64[n_seg+1]  exclusive prefix of ceil(seg_len[s]/block_bytes);
 *                                  gleam_batch_geometry computes it
 *   n_seg, n_blocks                host copies; n_blocks == blk_first[n_seg]
 *   leaf_bytes                     must be GLEAM_LEAF_BYTES
 *   block_bytes                    4096 << k for 0 <= k <= 12
 */
typedef struct {
  const uint64_t* seg_addr;
  const uint64_t* seg_len;
  const uint64_t* blk_first;
  uint64_t n_seg;
  uint64_t n_blocks;
  uint32_t leaf_bytes;
  uint32_t block_bytes;
} gleam_batch;

/* Opaque host handle of a device-resident identifier table (the server's set of
 * identifiers of resident chunks, Sec. 4.1.2). Table storage is caller-owned
 * device memory that must outlive the handle. */
typedef struct gleam_cache gleam_cache;

/*
 * Batch geometry (Sec. 4.1.1: decisions are made per payload, restarting at its
 * first byte). host_seg_len: host u64[n_seg]; host_blk_first: host u64[n_seg+1]
 * receives the exclusive prefix of ceil(len/block_bytes); *n_blocks (nullable)
 * receives the total. Errors: GLEAM_E_INVALID for null arrays with n_seg > 0 or a
 * bad block_bytes.
 */
gleam_status gleam_batch_geometry(const uint64_t* host_seg_len, uint64_t n_seg, uint32_t block_bytes,
                                  uint64_t* host_blk_first, uint64_t* n_blocks);

/*
 * Digest every block of a batch (Sec. 4.1.2: the identifier is a hash of the
 * source bytes). Leaf digest = XXH64(leaf bytes, seed 0) over the actual bytes
 * (no padding); block digest = bottom-up pairwise tree over the block's leaf
 * digests, node = XXH64(LE64(left) || LE64(right), seed 0), an odd last element
 * moving up unchanged; a one-leaf block's digest is its leaf digest.
 *   b               host pointer to the batch descriptor (device arrays inside)
 *   d_block_digest  device u64[n_blocks] output
 *   d_leaf_digest   nullable device u64[n_blocks * block_bytes/4096] output,
 *                   block-major; slots past a short block's last leaf get 0
 * Errors: GLEAM_E_INVALID (null b, null descriptor or output with n_blocks > 0,
 * leaf_bytes != 4096, bad block_bytes, n_blocks > 0 with n_seg == 0),
 * GLEAM_E_UNSUPPORTED (a grid beyond 2^31 workgroups), GLEAM_E_HIP.
 * n_blocks == 0 is a no-op.
 */
gleam_status gleam_fp_chunks(const gleam_batch* b, uint64_t* d_block_digest, uint64_t* d_leaf_digest,
                             void* stream);

/* Device bytes of table storage for `capacity` slots (a power of two >= 16):
 * 256 + 24 * capacity (key, value and last-use stamp per slot); 0 for an invalid
 * capacity. */
size_t gleam_cache_bytes(uint64_t capacity);

/*
 * Create a handle over caller-owned storage and enqueue the table clear.
 *   d_storage  device memory, 256-byte aligned, >= gleam_cache_bytes(capacity)
 *   capacity   power of two >= 16
 *   max_load   in (0, 1): inserts are refused once the number of keys could
 *              exceed floor(max_load * capacity) (at most capacity - 1)
 *   out        receives the handle (host memory, freed by gleam_cache_destroy)
 * Errors: GLEAM_E_INVALID, GLEAM_E_HIP.
 */
gleam_status gleam_cache_create(void* d_storage, size_t bytes, uint64_t capacity, double max_load,
                                gleam_cache** out, void* stream);

/* Free the host handle; the storage is not touched. NULL is allowed. */
gleam_status gleam_cache_destroy(gleam_cache* c);

/* Host-side upper bound on the keys the table may hold (exact unless inserts
 * carried keys already present). UINT64_MAX for a NULL handle. */
uint64_t gleam_cache_key_bound(const gleam_cache* c);

/* Device workspace bytes needed by lookup, insert and compaction of n items; 0 for n
 * above 2^40, which those calls refuse with GLEAM_E_UNSUPPORTED. */
size_t gleam_workspace_bytes(uint64_t n);

/*
 * Insert identifiers (Sec. 4.1.2 and 4.1.3: a chunk identified as a weight is kept
 * and its identifier reused by later connections). Set semantics: a key already
 * present keeps its value; among equal keys of this call the lowest index's value
 * is stored. Every u64 is a valid key.
 *   d_keys, d_vals  device u64[n]
 *   d_n_new         nullable device u64[1]: number of keys that were new
 *   d_ws, ws_bytes  device workspace, 256-byte aligned, >= gleam_workspace_bytes(n)
 * Capacity is enforced on the host without a device sync: if key_bound + n could
 * exceed the maximum load, GLEAM_E_CAPACITY is returned and nothing is inserted.
 * Errors: GLEAM_E_INVALID, GLEAM_E_CAPACITY, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED (n
 * above 2^31 workgroups of 256 keys, or 2^40), GLEAM_E_HIP.
 */
gleam_status gleam_cache_insert(gleam_cache* c, const uint64_t* d_keys, const uint64_t* d_vals, uint64_t n,
                                uint64_t* d_n_new, void* d_ws, size_t ws_bytes, void* stream);

/*
 * Decide each block's fate (Sec. 4.1.2: identifier held -> only metadata travels).
 *   d_keys    device u64[n] block digests in batch order
 *   d_status  device u8[n] output: GLEAM_MISS / GLEAM_HIT_CACHE / GLEAM_HIT_BATCH
 *   d_ref     nullable device u64[n] output (see the status enum)
 *   d_ws      device workspace, 256-byte aligned, >= gleam_workspace_bytes(n)
 * The table is only read.
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED (n above 2^31
 * workgroups of 256 keys, or 2^40), GLEAM_E_HIP. n == 0 is a no-op.
 */
gleam_status gleam_cache_lookup(const gleam_cache* c, const uint64_t* d_keys, uint64_t n, uint8_t* d_status,
                                uint64_t* d_ref, void* d_ws, size_t ws_bytes, void* stream);

/*
 * gleam_cache_lookup without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, hosts that forbid allocation). The
 * same outputs as gleam_cache_lookup; the batch-dedup scratch table lives in a
 * library-owned device array of 32 MiB + 256 B per GPU (held until the process ends),
 * so n is at most gleam_cache_lookup_noalloc_max_keys() = 2^20. The call allocates
 * nothing (its first call on a device looks up that device's array address).
 * Every call on one GPU shares that GPU's array: calls that overlap on one GPU (on
 * different streams, or from different threads) race and their outputs are undefined;
 * order them on one stream. Each call clears what it uses (a fill kernel).
 *   d_keys, d_status, d_ref   as for gleam_cache_lookup
 * Errors: GLEAM_E_INVALID (null table, keys or status), GLEAM_E_UNSUPPORTED (n above
 * 2^20), GLEAM_E_HIP. n == 0 is a no-op.
 */
size_t gleam_cache_lookup_noalloc_max_keys(void);
gleam_status gleam_cache_lookup_noalloc(const gleam_cache* c, const uint64_t* d_keys, uint64_t n, uint8_t* d_status,
                                        uint64_t* d_ref, void* stream);

/*
 * The blocks whose bytes must still cross the network (Sec. 4.1.2: on a miss the
 * full chunk is sent).
 *   d_status      device u8[n] (as written by gleam_cache_lookup)
 *   b             nullable host pointer to the batch the statuses belong to;
 *                 needed only for d_miss_bytes (b->n_blocks must equal n)
 *   d_miss_idx    device u64[n] output: ascending indices g with status MISS,
 *                 in its first *d_miss_count entries
 *   d_miss_count  device u64[1] output
 *   d_miss_bytes  nullable device u64[1] output: total bytes of those blocks
 *   d_ws          device workspace, 256-byte aligned, >= gleam_workspace_bytes(n)
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED (n above 2^40),
 * GLEAM_E_HIP. With n == 0 the counters are still set to 0.
 */
gleam_status gleam_miss_compact(const uint8_t* d_status, uint64_t n, const gleam_batch* b, uint64_t* d_miss_idx,
                                uint64_t* d_miss_count, uint64_t* d_miss_bytes, void* d_ws, size_t ws_bytes,
                                void* stream);

/*
 * The whole decision for one batch in one call (Sec. 4.1.2: a chunk whose identifier the
 * server holds sends only its hash and size; any other chunk sends its bytes). Writes
 * exactly what gleam_fp_chunks, then gleam_cache_lookup, then gleam_miss_compact (with
 * the batch, when d_miss_bytes is given) write, in one call:
 *   b, c                  the batch and the table (only read)
 *   d_digest              device u64[n_blocks]: block digests
 *   d_status, d_ref       device u8[n_blocks] and nullable u64[n_blocks]: as for
 *                         gleam_cache_lookup
 *   d_miss_idx, d_miss_count, d_miss_bytes   as for gleam_miss_compact (d_miss_bytes
 *                         nullable)
 *   d_ws, ws_bytes        device workspace, 256-byte aligned,
 *                         >= gleam_detect_workspace_bytes(n_blocks), PREPARED: unlike the
 *                         other calls' workspaces it carries one word from call to call (an
 *                         arrival counter at byte 128), which gleam_detect_ws_init arms and
 *                         every gleam_detect call leaves armed. Prepare a workspace once
 *                         after allocating it, and again after any other use of its memory;
 *                         a workspace sized for n blocks serves any smaller batch; calls
 *                         that may overlap need separate workspaces.
 * A small batch (blocks of at most 64 KiB, at most 65,536 leaf slots and 4,096 blocks:
 * the latency-bound case, e.g. one copy of a few MB) runs as ONE kernel: every workgroup
 * digests its leaves and probes the table for them, then arrives at the counter, and the
 * last to arrive resolves repeats inside the batch and compacts. A larger batch runs the
 * three calls' kernels in order. Enqueues kernel launches only (graph-capturable). If the
 * one-kernel path finds the workspace unprepared, it writes UINT64_MAX to *d_miss_count
 * (statuses undefined).
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED, GLEAM_E_HIP. An empty
 * batch still sets the miss count (and bytes) to 0.
 *
 * gleam_detect_ws_init: prepare d_ws (device, 256-byte aligned, >= 256 bytes) for
 * gleam_detect (one small kernel on `stream`).
 * gleam_detect_workspace_bytes: the workspace for batches of up to n_blocks blocks (0 for
 * n_blocks above 2^40). Errors: GLEAM_E_INVALID, GLEAM_E_HIP.
 */
gleam_status gleam_detect(const gleam_batch* b, const gleam_cache* c, uint64_t* d_digest, uint8_t* d_status,
                          uint64_t* d_ref, uint64_t* d_miss_idx, uint64_t* d_miss_count, uint64_t* d_miss_bytes,
                          void* d_ws, size_t ws_bytes, void* stream);
gleam_status gleam_detect_ws_init(void* d_ws, size_t ws_bytes, void* stream);
size_t gleam_detect_workspace_bytes(uint64_t n_blocks);

/*
 * Table lifecycle (Sec. 4.1.3: identified weight chunks stay in a shared cache across
 * tasks and LRU eviction keeps it bounded; Sec. 4.1.2: at connect time the server sends
 * the identifiers it holds). Every entry has a last-use stamp (0 when inserted). These
 * calls must not overlap, on any stream, with other calls on the same table.
 *
 * gleam_cache_maint_bytes: device workspace bytes for evict and export of this
 * table, about 64 bytes per slot (0 for NULL or a table above 2^31 slots).
 *
 * gleam_cache_touch: for every key present, stamp = max(stamp, epoch), the epoch being
 * d_epochs[i] (device u64[n]) or, when d_epochs is NULL, the scalar `epoch`.
 * d_n_touched (nullable device u64[1]) receives how many of the n keys were present.
 *
 * gleam_cache_evict: keep the `keep` most recently used entries. Entries are ordered by
 * (stamp, key) ascending and the first live - keep of them are removed; d_evicted
 * (nullable device u64[capacity + 1]) receives their keys in that order; d_counts
 * (device u64[2]) receives {removed, live after}. The host key bound drops to `keep`.
 *
 * gleam_cache_erase: remove the given keys (device u64[n]) that are present; d_counts
 * (device u64[2]) receives {removed, live after}. The cost follows the keys erased, not
 * the capacity: each erased key's cluster (the run of occupied slots around it) is
 * repaired in place, no tombstones remain, and the call enqueues kernels only (it may be
 * captured in a graph). Its workspace: device, 256-byte aligned,
 * >= gleam_cache_erase_bytes(n) (O(n); 0 for n above 2^36). The host bound is
 * unchanged; lower it with gleam_cache_set_key_bound once the live count has been read
 * back.
 *
 * gleam_cache_export: every entry sorted by key into device u64[capacity + 1] arrays
 * d_keys, d_vals and (nullable) d_stamps; *d_count (device u64[1]) = entries written.
 * Evict and export gather the live entries and order them with a radix sort of their
 * own (kernels only), so both may be captured in a graph; their cost follows the
 * capacity.
 * Re-inserting the exported pairs (and touching them with their stamps) rebuilds the
 * table: the export is also its checkpoint.
 *
 * gleam_cache_set_key_bound: lower the host key bound to n (a live count read back
 * from d_counts); raising it is refused.
 *
 * Workspace (evict, export): device, 256-byte aligned, >= gleam_cache_maint_bytes(c).
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED, GLEAM_E_HIP.
 */
size_t gleam_cache_maint_bytes(const gleam_cache* c);
gleam_status gleam_cache_touch(gleam_cache* c, const uint64_t* d_keys, uint64_t n, const uint64_t* d_epochs,
                               uint64_t epoch, uint64_t* d_n_touched, void* stream);
gleam_status gleam_cache_evict(gleam_cache* c, uint64_t keep, uint64_t* d_evicted, uint64_t* d_counts, void* d_ws,
                               size_t ws_bytes, void* stream);
size_t gleam_cache_erase_bytes(uint64_t n);
gleam_status gleam_cache_erase(gleam_cache* c, const uint64_t* d_keys, uint64_t n, uint64_t* d_counts, void* d_ws,
                               size_t ws_bytes, void* stream);
gleam_status gleam_cache_export(const gleam_cache* c, uint64_t* d_keys, uint64_t* d_vals, uint64_t* d_stamps,
                                uint64_t* d_count, void* d_ws, size_t ws_bytes, void* stream);
gleam_status gleam_cache_set_key_bound(gleam_cache* c, uint64_t n);

/*
 * Weight identification at free time (Sec. 4.1.1 "Weight Block Identification"): an
 * allocation holds weights only if every payload recorded at its first host-to-device
 * write still has the same bytes when the allocation is freed (in-place activations or
 * inputs disqualify it; Appendix, corner cases of weight identification). The digests
 * recorded at write time (gleam_fp_chunks on the payloads as written) are compared with
 * digests of the current device bytes.
 *   b                  the recorded payloads at their device addresses, lengths as recorded
 *   d_recorded         device u64[b->n_blocks]: block digests recorded at write time
 *   d_region_first     device u64[n_regions+1]: payloads of allocation r are
 *                      [region_first[r], region_first[r+1]); non-decreasing, starting at 0
 *                      and ending at b->n_seg (payloads outside it are ignored)
 *   d_block_match      nullable device u8[n_blocks]: 1 where the block is unchanged
 *   d_seg_first_diff   nullable device u64[n_seg]: index, within its payload, of the first
 *                      changed block; UINT64_MAX if none
 *   d_region_weight    device u8[n_regions]: 1 iff the allocation has at least one recorded
 *                      payload and none of them changed
 *   d_ws, ws_bytes     device workspace, 256-byte aligned,
 *                      >= gleam_workspace_bytes(n_blocks + n_seg)
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED, GLEAM_E_HIP.
 */
gleam_status gleam_identify_weights(const gleam_batch* b, const uint64_t* d_recorded,
                                    const uint64_t* d_region_first, uint64_t n_regions,
                                    uint8_t* d_block_match, uint64_t* d_seg_first_diff,
                                    uint8_t* d_region_weight, void* d_ws, size_t ws_bytes, void* stream);

/*
 * gleam_identify_weights located to the leaf: the first changed 4 KiB leaf of each
 * payload (Sec. 4.1.1's consistency check compares every recorded chunk byte with the
 * current data; a leaf digest narrows a mismatch to 4 KiB).
 *   b                  as for gleam_identify_weights
 *   d_recorded_leaf    device u64[n_blocks * block_bytes/4096]: the leaf digests recorded
 *                      at write time, as gleam_fp_chunks writes them (block-major, 0 in
 *                      the slots past a short block's last leaf)
 *   d_region_first     as for gleam_identify_weights
 *   d_leaf_match       nullable device u8[n_blocks * block_bytes/4096]: 1 where the slot's
 *                      recorded and current digests agree (slots without a leaf read 1)
 *   d_seg_first_diff   nullable device u64[n_seg]: index, within its payload, of the first
 *                      changed leaf (leaf k of block j is j * block_bytes/4096 + k);
 *                      UINT64_MAX if none
 *   d_region_weight    device u8[n_regions]: as for gleam_identify_weights (the verdicts
 *                      agree: a block changed iff one of its leaves did)
 *   d_ws, ws_bytes     device workspace, 256-byte aligned,
 *                      >= gleam_workspace_bytes(n_blocks * block_bytes/4096 + n_seg)
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED, GLEAM_E_HIP.
 */
gleam_status gleam_identify_leaves(const gleam_batch* b, const uint64_t* d_recorded_leaf,
                                   const uint64_t* d_region_first, uint64_t n_regions, uint8_t* d_leaf_match,
                                   uint64_t* d_seg_first_diff, uint8_t* d_region_weight, void* d_ws,
                                   size_t ws_bytes, void* stream);

/*
 * The first-write rule of weight identification (Sec. 4.1.1: where an address range is
 * overwritten, only the first host-to-device write counts). The recorded writes are
 * listed in time order, grouped by allocation: the writes of allocation r are
 * [region_first[r], region_first[r+1]). A write owns the bytes of [addr, addr + len)
 * that no earlier write of its allocation covers; a piece is a maximal run of bytes one
 * write owns. Digesting each write's pieces from its payload when it lands (gleam_fp_chunks
 * over a batch of the pieces at the payload: payload + offset) and the same pieces of the
 * allocation at free time (the pieces at addr + offset), then gleam_identify_weights over
 * the pieces with region_first = region_piece_first, checks every written byte against
 * its first writer's byte.
 *   d_addr, d_len        device u64[n_writes]: destination address and bytes of each write
 *   d_region_first       device u64[n_regions+1]: non-decreasing, from 0 to n_writes
 *   d_piece_write        device u64[2 * n_writes] output: the write owning piece p
 *   d_piece_offset       device u64[2 * n_writes] output: its start minus the write's addr
 *   d_piece_len          device u64[2 * n_writes] output: its bytes
 *                        (pieces in order of allocation, write, then address; at most
 *                        2 * n_writes - 1 of them)
 *   d_region_piece_first device u64[n_regions+1] output: allocation r's pieces are
 *                        [region_piece_first[r], region_piece_first[r+1]); the last entry
 *                        is the piece count
 *   d_region_status      nullable device u8[n_regions] output: GLEAM_FW_OK;
 *                        GLEAM_FW_TOO_MANY (more than 2048 writes: no pieces);
 *                        GLEAM_FW_INVALID (a write past the top of the address space, or
 *                        a malformed region_first: no pieces)
 *   d_ws, ws_bytes       device workspace, 256-byte aligned, >=
 *                        gleam_first_writes_ws_bytes(n_writes, n_regions)
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED (more than 2^36 writes or
 * 2^31 allocations), GLEAM_E_HIP. gleam_first_writes_ws_bytes returns 0 beyond those.
 */
enum { GLEAM_FW_OK = 0, GLEAM_FW_TOO_MANY = 1, GLEAM_FW_INVALID = 2 };
size_t gleam_first_writes_ws_bytes(uint64_t n_writes, uint64_t n_regions);
gleam_status gleam_first_writes(const uint64_t* d_addr, const uint64_t* d_len, uint64_t n_writes,
                                const uint64_t* d_region_first, uint64_t n_regions, uint64_t* d_piece_write,
                                uint64_t* d_piece_offset, uint64_t* d_piece_len, uint64_t* d_region_piece_first,
                                uint8_t* d_region_status, void* d_ws, size_t ws_bytes, void* stream);

/*
 * The paper's own identifier (Appendix, discussion of hash cost and collisions): an MD5
 * (RFC 1321) of the first 1024 bits of each host-to-device chunk; chunks of at most 1024
 * bytes get no cache entry. Kept as an ablation of the full-content block digests.
 *   b             the payloads (only seg_addr, seg_len and n_seg are used; block_bytes
 *                 must still be valid)
 *   prefix_bytes  bytes hashed per payload: min(len, prefix_bytes); 128 in the paper;
 *                 at most 1 MiB
 *   min_len       payloads longer than this are eligible for a cache entry (1024)
 *   d_digest      device u64[2 * n_seg]: the 16-byte MD5 of payload s at [2s, 2s+1]
 *                 (byte order of the digest, little-endian words)
 *   d_key         nullable device u64[n_seg]: the digest's first 8 bytes, usable as a
 *                 gleam_cache key
 *   d_eligible    nullable device u8[n_seg]: 1 iff seg_len[s] > min_len
 * Errors: GLEAM_E_INVALID, GLEAM_E_UNSUPPORTED, GLEAM_E_HIP. n_seg == 0 is a no-op.
 */
gleam_status gleam_md5_prefix(const gleam_batch* b, uint32_t prefix_bytes, uint64_t min_len, uint64_t* d_digest,
                              uint64_t* d_key, uint8_t* d_eligible, void* stream);

/*
 * One block of a send plan (Sec. 4.1.2: a chunk whose identifier the server holds sends
 * only reuse metadata -- its hash and size -- any other chunk sends its bytes).
 *   block, payload, offset, length  the block's global index, payload, byte offset in
 *                                   that payload, and bytes
 *   kind   GLEAM_MISS: the bytes travel; ident = their offset in the packed buffer
 *          GLEAM_HIT_CACHE: (digest, length) travels; ident = the digest
 *          GLEAM_HIT_BATCH: (earlier block, length) travels; ident = that block's index
 */
typedef struct {
  uint64_t block;
  uint64_t payload;
  uint64_t offset;
  uint64_t ident;
  uint32_t length;
  uint32_t kind;
} gleam_send_record;

/*
 * Sender side (Sec. 4.1.2): one record per block from the lookup's results. MISS blocks
 * are laid out in block order in a packed buffer, each at a multiple of 16 bytes.
 *   b                     the batch the statuses belong to
 *   d_digest, d_status, d_ref   device arrays of n_blocks (gleam_fp_chunks and
 *                         gleam_cache_lookup outputs)
 *   d_records             device gleam_send_record[n_blocks] output
 *   d_totals              device u64[4] output: MISS blocks, HIT_CACHE blocks,
 *                         HIT_BATCH blocks, packed buffer bytes
 *   d_ws                  device workspace, 256-byte aligned, >= gleam_workspace_bytes(n_blocks)
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED, GLEAM_E_HIP.
 */
gleam_status gleam_send_plan(const gleam_batch* b, const uint64_t* d_digest, const uint8_t* d_status,
                             const uint64_t* d_ref, gleam_send_record* d_records, uint64_t* d_totals, void* d_ws,
                             size_t ws_bytes, void* stream);

/*
 * Copy every MISS block's bytes to its planned offset in d_out (device, out_bytes long,
 * at least the plan's packed total). A record whose block is not inside its payload of
 * `b`, or whose bytes would not fit d_out, is skipped. Padding bytes between blocks are
 * not written.
 * Errors: GLEAM_E_INVALID, GLEAM_E_HIP.
 */
gleam_status gleam_pack_misses(const gleam_batch* b, const gleam_send_record* d_records, uint8_t* d_out,
                               uint64_t out_bytes, void* stream);

/*
 * Receiver side (Sec. 4.1.2: on a hit the server restores the bytes locally): write
 * every block of the destination payloads `dst` (same geometry as the plan's batch).
 * MISS blocks come from d_packed (packed_bytes long); HIT_CACHE blocks from the
 * receiver's own copy at device address d_held[g] (device u64[n_blocks], e.g. the
 * lookup's ref output when table values are addresses of held blocks; nullable: then
 * HIT_CACHE blocks are left untouched); HIT_BATCH blocks from the packed bytes of the
 * block they repeat. A record whose block is not inside its payload of `dst`, whose
 * packed bytes lie outside d_packed, or whose kind is unknown is skipped; d_held
 * addresses are the caller's and are read as given.
 * Errors: GLEAM_E_INVALID, GLEAM_E_HIP.
 */
gleam_status gleam_restore_blocks(const gleam_batch* dst, const gleam_send_record* d_records,
                                  const uint8_t* d_packed, uint64_t packed_bytes, const uint64_t* d_held,
                                  void* stream);

/*
 * Address-remap map (Sec. 4.1.3, Weight Chunk Sharing: two chunks written into one client
 * allocation may find their shareable copies in two different server allocations, so
 * a virtual memory layer maps client device addresses onto the actual shareable
 * positions; Appendix, Implementation Details, Virtual Memory Map: each task gets a
 * 1 TB virtual address space and the mappings are kept in a red-black tree). Device
 * pointers carried by remoted calls are translated through it.
 *
 * The map holds disjoint, non-empty intervals [start, start + length) of the 64-bit
 * address space, each with a target: address p inside one translates to
 * target + (p - start), any other address to GLEAM_UNMAPPED. One map may serve many
 * tasks when each task's addresses live in a range of its own (e.g. task t at
 * [t << 40, (t + 1) << 40), the paper's 1 TB per task). Storage is caller-owned device
 * memory that must outlive the handle: a 256-byte header (u64 interval count, fence
 * stride, fence length), u64 start[capacity] sorted ascending, {end (exclusive),
 * target - start}[capacity] pairs in the same order, and an 8192-entry fence (every
 * stride-th start) that translation searches in LDS first. Calls on one map must not overlap, on
 * any stream, with an update of it.
 *
 * gleam_remap_bytes: storage bytes for `capacity` intervals (1 <= capacity <= 2^31):
 * 256 + 24 * capacity + 65536; 0 for an invalid capacity.
 *
 * gleam_remap_create: a handle over d_storage (device, 256-byte aligned, >=
 * gleam_remap_bytes(capacity) bytes) and the clear of its header (an empty map).
 * *out (host) receives the handle, freed by gleam_remap_destroy (storage untouched;
 * NULL allowed). Errors: GLEAM_E_INVALID, GLEAM_E_HIP.
 *
 * gleam_remap_update: one batch of changes, removals first, then additions:
 *   d_del_start, d_del_len   device u64[n_del]: every interval sharing an address with
 *                            a range [start, start + len) (clipped at 2^64; len 0 is an
 *                            empty range) is removed whole
 *   d_add_start, d_add_len, d_add_target   device u64[n_add]: intervals to add
 *   d_add_status  nullable device u8[n_add]: GLEAM_REMAP_ADDED; GLEAM_REMAP_INVALID
 *                 (length 0, or start + length or target + length above 2^64 - 1);
 *                 GLEAM_REMAP_OVERLAP (shares an address with a surviving interval or
 *                 with another valid addition of this call: both of two clashing
 *                 additions are refused, whatever their order); GLEAM_REMAP_FULL
 *   d_counts      device u64[4]: {intervals after, added, removed, additions refused}
 *   d_ws          device workspace, 256-byte aligned,
 *                 >= gleam_remap_update_bytes(m, n_add, n_del)
 * If the survivors and the accepted additions exceed the capacity, the map is left
 * exactly as it was (the removals included) and those additions get GLEAM_REMAP_FULL.
 * Every update passes over the whole capacity (survivors are marked and compacted)
 * whatever the count, plus a sort of the additions: size the capacity to the map.
 * Errors: GLEAM_E_INVALID, GLEAM_E_WORKSPACE, GLEAM_E_UNSUPPORTED (n_add or n_del
 * above 2^31), GLEAM_E_HIP. gleam_remap_update_bytes returns 0 for a NULL map or counts
 * above 2^31.
 *
 * gleam_remap_translate: d_out[i] (device u64[n]) = the translation of d_addr[i]
 * (device u64[n]). The map is only read. Errors: GLEAM_E_INVALID, GLEAM_E_HIP.
 *
 * gleam_remap_export: the intervals in start order into device u64[capacity] arrays
 * d_start, d_len, d_target; *d_count (device u64[1]) = their number. Adding the
 * exported intervals to an empty map rebuilds it. Errors: GLEAM_E_INVALID, GLEAM_E_HIP.
 */
typedef struct gleam_remap gleam_remap;
enum {
  GLEAM_REMAP_ADDED = 0,
  GLEAM_REMAP_INVALID = 1,
  GLEAM_REMAP_OVERLAP = 2,
  GLEAM_REMAP_FULL = 3
};
#define GLEAM_UNMAPPED UINT64_MAX

size_t gleam_remap_bytes(uint64_t capacity);
gleam_status gleam_remap_create(void* d_storage, size_t bytes, uint64_t capacity, gleam_remap** out,
                                void* stream);
gleam_status gleam_remap_destroy(gleam_remap* m);
size_t gleam_remap_update_bytes(const gleam_remap* m, uint64_t n_add, uint64_t n_del);
gleam_status gleam_remap_update(gleam_remap* m, const uint64_t* d_del_start, const uint64_t* d_del_len,
                                uint64_t n_del, const uint64_t* d_add_start, const uint64_t* d_add_len,
                                const uint64_t* d_add_target, uint64_t n_add, uint8_t* d_add_status,
                                uint64_t* d_counts, void* d_ws, size_t ws_bytes, void* stream);
gleam_status gleam_remap_translate(const gleam_remap* m, const uint64_t* d_addr, uint64_t n, uint64_t* d_out,
                                   void* stream);
gleam_status gleam_remap_export(const gleam_remap* m, uint64_t* d_start, uint64_t* d_len, uint64_t* d_target,
                                uint64_t* d_count, void* stream);

/*
 * Calibration (a measurement aid, not a step of the path): read `bytes` bytes at d_src
 * (device, 16-byte aligned, bytes a multiple of 16) once, with the fastest plain read
 * pattern measured on MI355X, and XOR into *d_sink (device u64, caller-initialised) the
 * XOR of every 8-byte little-endian word read. Its duration gives the measured HBM read
 * ceiling against which the fingerprint kernel's roofline fraction is also reported.
 * Errors: GLEAM_E_INVALID (null pointers, misaligned source or length), GLEAM_E_HIP.
 */
gleam_status gleam_read_stream(const void* d_src, uint64_t bytes, uint64_t* d_sink, void* stream);

/* Static text for a status code. */
/*
 * gleam_preload: load the library's GPU code on the current device now rather than at
 * each source file's first kernel launch, where the HIP runtime loads it lazily (about
 * 0.8 ms of host time before the fingerprint's first launch on MI355X). For callers
 * that want the first model load of a process to pay only for its own work: call once
 * per device at start-up. Optional; without it the same loading happens on first use.
 * Enqueues nothing. Errors: GLEAM_E_HIP (no usable device).
 */
gleam_status gleam_preload(void);

const char* gleam_status_string(gleam_status s);

/* Thread-local detail of the last error on this thread ("" if none). */
const char* gleam_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GLEAM_H */
