/*
 * kvr_decode.h -- resumed generation over a rebuilt arena.
 *
 * The paper judges recovery by whether generation continues from the rebuilt
 * state as it would have from the original one (Sec. 7.3.1 Recoverability;
 * Sec. 4.2 step 5 resumes the interrupted requests; Sec. 6 resumes them on the
 * same engine).  kv_decode_step is that continuation: one greedy decode step
 * per request, reading the K/V that kv_rebuild (or earlier decode steps) left
 * in the arena through the same block tables, and appending the new token's
 * K/V.  Same conventions as kvr.h (status codes, host/device pointers, void*
 * streams, host-side validation before any device work, thread-compatible).
 */
#ifndef KVR_DECODE_H
#define KVR_DECODE_H

#include <stdint.h>

#include "kvr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Workspace bytes for decode steps of up to `num_requests` requests whose
 * positions are all < max_position.  Returns 0 for an invalid description or
 * non-positive sizes. */
uint64_t kv_decode_workspace_bytes(const kv_model_desc* desc, int32_t num_requests,
                                   int64_t max_position);

/* Host-only argument check of a decode step (no device access): the status
 * kv_decode_step would return on an arena of this geometry, workspace aside.
 *   KV_EINVAL    null arrays, num_requests < 0, a position < 0
 *   KV_ERANGE    a token outside [0, vocab), a block entry outside [0, num_blocks)
 *   KV_ECAPACITY position / block_size >= max_blocks_per_req
 *   KV_EALIAS    the block holding a request's position (the one the step
 *                writes) listed anywhere else among the used entries of any
 *                request; blocks the step only reads may be shared */
kv_status kv_decode_check(const kv_model_desc* desc, int32_t block_size, int64_t num_blocks,
                          const int32_t* tokens, const int32_t* positions, int32_t num_requests,
                          const int32_t* block_tables, int32_t max_blocks_per_req);

/* One greedy decode step.
 *   w              the decoder weights (as for kv_rebuild)
 *   final_norm     device [hidden], the final RMSNorm gain (model dtype)
 *   lm_head        device [vocab, hidden], model dtype (may equal w->embed)
 *   tokens         host int32 [num_requests]: the token at positions[r]
 *   positions      host int32 [num_requests], >= 0: its position; the K/V of
 *                  positions 0 .. positions[r]-1 of request r must already be
 *                  in the arena at their slots
 *   block_tables   host int32 [num_requests][max_blocks_per_req]; entries
 *                  0 .. positions[r]/block_size are used
 *   workspace      device scratch, kv_decode_workspace_bytes(desc, R, max p + 1)
 *   next_tokens    device int32 [num_requests]: greedy argmax of the logits
 *                  (the lowest index among equal maxima)
 *   logits         optional device float [num_requests][vocab] (NULL = none)
 * Writes, in every layer, exactly the K row (rotated) and V row of position
 * positions[r] at slot (table[r][p/B], p%B); nothing else in the arena.
 * Attention for that token covers positions 0 .. positions[r].  Host arrays
 * may be reused when the call returns; the step runs asynchronously on
 * `stream`, and next_tokens / logits are complete when it is. */
kv_status kv_decode_step(const kv_weights* w, const void* final_norm, const void* lm_head,
                         const int32_t* tokens, const int32_t* positions, int32_t num_requests,
                         const int32_t* block_tables, int32_t max_blocks_per_req,
                         kv_arena_t arena, void* workspace, uint64_t workspace_bytes,
                         void* stream, int32_t* next_tokens, float* logits);

#ifdef __cplusplus
}
#endif
#endif
