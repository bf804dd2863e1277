/*
 * kvr_reuse.h -- rebuild from a retained prefix.
 *
 * The paper rebuilds every interrupted request from position 0 because it
 * flushes the whole pool (Sec. 4.2 flush paragraph; Sec. 4.3), and names
 * recovery without a full refill as future work (Sec. 8).  When part of a
 * request's K/V is known to be intact -- its blocks passed verification
 * (kvr_verify.h), or a prefix shared with another request is already in the
 * arena -- only the positions after it need computing.  kv_rebuild_from
 * recomputes positions starts[r] .. lens[r]-1 of each request: they attend
 * to all positions 0 .. p, reading the K/V of positions < starts[r] from the
 * arena, and are written through the block tables exactly as kv_rebuild
 * writes them.  With every start 0 it is kv_rebuild.
 *
 * Shared prefixes need no copy: requests may list the same blocks for a
 * common prefix, read-only, and an earlier request in the same call may be
 * the one that computes them (waves run in request order, and each layer's
 * K/V reach the arena before that layer's prefix reads).
 *
 * Same conventions as kvr.h.
 */
#ifndef KVR_REUSE_H
#define KVR_REUSE_H

#include <stdint.h>

#include "kvr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Workspace bytes for up to num_requests requests with total_rows positions
 * to compute (sum of lens - starts) and total_keys positions in all (sum of
 * lens), in waves of about wave_rows computed positions.  0 for an invalid
 * description or sizes (total_keys < total_rows included). */
uint64_t kv_rebuild_from_workspace_bytes(const kv_model_desc* desc, int32_t num_requests,
                                         int64_t total_rows, int64_t total_keys,
                                         int64_t wave_rows);

/* Host-only argument check (no device access); the status kv_rebuild_from
 * would return, workspace aside.  Beyond kv_rebuild_check's rules:
 *   KV_EINVAL  null starts; a start outside [0, len]; a start that is not a
 *              multiple of 8 (unless it equals len)
 *   KV_EALIAS  a block holding a position >= start listed twice for writing,
 *              or read as prefix by a request that comes before its writer
 * tokens holds the tokens of the computed positions only, request after
 * request: sum over r of (lens[r] - starts[r]). */
kv_status kv_rebuild_from_check(const kv_model_desc* desc, int32_t block_size, int64_t num_blocks,
                                const int32_t* tokens, const int32_t* lens, const int32_t* starts,
                                int32_t num_requests, const int32_t* block_tables,
                                int32_t max_blocks_per_req);

/* Rebuild from retained prefixes (arguments as kv_rebuild, plus starts,
 * host int32 [num_requests]).  Writes the slots of positions
 * starts[r] .. lens[r]-1 in every layer; reads, never writes, the slots of
 * positions < starts[r].  Deterministic; results match kv_rebuild's for the
 * same arena contents within the rebuild's tolerance, and bit for bit when
 * every start is a multiple of 256. */
kv_status kv_rebuild_from(const kv_weights* w, const int32_t* tokens, const int32_t* lens,
                          const int32_t* starts, int32_t num_requests, const int32_t* block_tables,
                          int32_t max_blocks_per_req, kv_arena_t arena, void* workspace,
                          uint64_t workspace_bytes, void* stream);

/* kv_rebuild_from split as kv_rebuild_stage / kv_rebuild_execute: the plan
 * is executed with kv_rebuild_execute and released with kv_plan_release. */
kv_status kv_rebuild_stage_from(kv_arena_t arena, const int32_t* tokens, const int32_t* lens,
                                const int32_t* starts, int32_t num_requests,
                                const int32_t* block_tables, int32_t max_blocks_per_req,
                                void* workspace, uint64_t workspace_bytes, void* stream,
                                kv_plan_t* out);

#ifdef __cplusplus
}
#endif
#endif
