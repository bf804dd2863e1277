/*
 * kvr_verify.h -- block commit digests for flush-free recovery.
 *
 * The paper flushes and refills the whole KV pool at handover because after a
 * failure the pool may hold a mix of old and new entries, and it leaves
 * fine-grained consistency tracking to future work (Sec. 4.2, flush
 * paragraph; Sec. 2.3 Finding 2; Sec. 8 future work).  These calls are that
 * tracking at block granularity: the engine records a digest for each block
 * when its contents are committed (kv_block_digests), and the replacement
 * worker recomputes them over the retained arena (kv_verify) to find the
 * requests whose KV survived intact; only the others need kv_rebuild.
 *
 * The digest of a block covering n slots: the bytes of slots 0 .. n-1 in every
 * layer and both planes, read as little-endian 32-bit words u_0 .. u_{N-1} in
 * the order (layer, K then V, slot, byte within the slot row), give
 *     digest = sum over i of (u_i XOR (i * 0x9E3779B9 mod 2^32))^2  mod 2^64.
 * A change of any single covered word always changes it; bytes outside the
 * covered slots never enter it.
 *
 * Request r of a set occupies blocks tables[r][0 .. ceil(lens[r]/B)-1]; block j
 * covers min(B, lens[r] - j*B) slots.  Entries are numbered request by request,
 * block by block: entry count E = sum over r of ceil(lens[r]/B).
 * Same conventions as kvr.h (host arrays, device outputs, void* streams,
 * validation before any device work, thread-compatible per arena).
 */
#ifndef KVR_VERIFY_H
#define KVR_VERIFY_H

#include <stdint.h>

#include "kvr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Workspace bytes for a call over num_requests requests occupying num_entries
 * blocks in total; 0 for negative sizes. */
uint64_t kv_verify_workspace_bytes(int32_t num_requests, int64_t num_entries);

/* Commit records: digests (device uint64 [E]) of every block the request set
 * occupies.  Host arrays lens [num_requests] and block_tables
 * [num_requests][max_blocks_per_req] may be reused when the call returns.
 *   KV_EINVAL    null arrays or outputs, num_requests < 0, a length < 0, a slot
 *                row that is not a multiple of 16 bytes
 *   KV_ECAPACITY ceil(lens[r]/B) > max_blocks_per_req
 *   KV_ERANGE    a used table entry outside [0, num_blocks)
 *   KV_ENOMEM    workspace smaller than kv_verify_workspace_bytes
 *   KV_ESTATE    unknown arena handle
 * Blocks may be listed more than once (the scan only reads the arena). */
kv_status kv_block_digests(kv_arena_t arena, const int32_t* lens, int32_t num_requests,
                           const int32_t* block_tables, int32_t max_blocks_per_req,
                           void* workspace, uint64_t workspace_bytes, void* stream,
                           uint64_t* digests);

/* Verification against commit records: committed (device uint64 [E]) in the
 * entry order above.  Writes each entry's current digest to digests (device
 * uint64 [E], may be NULL) and, per request, the number of its leading blocks
 * whose digest equals the committed one to intact (device int32
 * [num_requests]); request r survived intact when intact[r] equals its block
 * count.  Same status codes as kv_block_digests. */
kv_status kv_verify(kv_arena_t arena, const int32_t* lens, int32_t num_requests,
                    const int32_t* block_tables, int32_t max_blocks_per_req,
                    const uint64_t* committed, void* workspace, uint64_t workspace_bytes,
                    void* stream, uint64_t* digests, int32_t* intact);

/* Verification that allocates nothing: kv_verify without a workspace, for
 * callers that cannot allocate device memory (code being captured into a HIP
 * graph, tight recovery or serving loops, harnesses that forbid hipMalloc).
 * Its scratch memory (the uploaded lens and tables, the entry list, request
 * offsets, match flags and, when `digests` is NULL, the digests) lives in a
 * device array of KV_VERIFY_NOALLOC_SCRATCH_BYTES that the library holds on
 * every device it runs on until the process ends; the call never allocates
 * device or pinned host memory.  Arguments, outputs and status codes are
 * those of kv_verify, plus
 *   KV_ENOMEM    the call needs more than KV_VERIFY_NOALLOC_SCRATCH_BYTES of
 *                scratch: 4R + 4*R*max_blocks_per_req + 17E bytes (+ 8E
 *                without `digests`), each part rounded up to 256 bytes
 *   KV_EDEVICE   the scratch array's device address cannot be obtained
 * lens and block_tables are copied with hipMemcpyAsync on `stream`: from
 * ordinary (pageable) host memory the copy has consumed them when the call
 * returns; arrays in page-locked host memory must stay unchanged until the
 * stream has passed this call.  Every call on one device shares that device's
 * scratch array, so calls that overlap on one device (other streams, other
 * threads) race; calls ordered on one stream do not.  Nothing in the scratch
 * needs to start at zero: each call writes every element it later reads. */
#define KV_VERIFY_NOALLOC_SCRATCH_BYTES (16u << 20)
kv_status kv_verify_noalloc(kv_arena_t arena, const int32_t* lens, int32_t num_requests,
                            const int32_t* block_tables, int32_t max_blocks_per_req,
                            const uint64_t* committed, void* stream, uint64_t* digests,
                            int32_t* intact);

#ifdef __cplusplus
}
#endif
#endif
