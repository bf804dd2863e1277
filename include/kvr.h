/*
 * kvr.h -- KV rebuild into a retained paged KV arena on one MI355X (gfx950).
 *
 * After a rollout-worker failure, the replacement worker keeps the weights and
 * the raw KV arena that independent owner processes hold (Sec. 4.1 Selective
 * State Reuse and Shadow Worker, state-isolation paragraph), checks GPU health
 * with a lightweight GPU operation and refuses reuse when it fails (Sec. 4.2
 * Handover, steps 2 and the unhealthy-GPU sentence), flushes the KV pool and
 * rebuilds every interrupted request's KV contents from its logged token
 * prefix (Sec. 4.2 step 5; Sec. 4.3 LLM Context Recovery).  Request-specific
 * KV contents and worker-local metadata are never reused (Sec. 7.3.1
 * Recoverability; Sec. 2.3 Finding 2).  The worker obtains the arena as
 * "pointers and metadata" (Sec. 6 Implementation, shadow-worker integration):
 * kv_arena_bind takes exactly that.
 *
 * The rebuild is a batched variable-length causal prefill of a Llama-style
 * pre-norm decoder (RMSNorm, Q/K/V projections, NeoX RoPE, causal grouped-
 * query attention, output projection, SwiGLU FFN, fp32 residual) whose rotated
 * K and V rows are written into arena slots through per-request block tables.
 * Every kernel is hand-written HIP for gfx950.
 *
 * Conventions for every entry point
 *   - Return value: kv_status, 0 on success, negative on error.  On error,
 *     kv_last_error() returns a message for the calling thread.
 *   - "device" pointers are HIP device allocations on the arena's device;
 *     "host" pointers are ordinary CPU memory.  The library never frees or
 *     takes ownership of caller memory.
 *   - Streams are hipStream_t values passed as void* (NULL = default stream).
 *   - All argument errors are detected on the host before any device work is
 *     enqueued, so a rejected call leaves the arena untouched.
 *   - Thread-compatible: calls on different arenas may run concurrently;
 *     calls on one arena must not overlap.
 */
#ifndef KVR_H
#define KVR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KV_OK = 0,
  KV_EINVAL = -1,    /* null pointer, negative size, unsupported shape          */
  KV_ERANGE = -2,    /* token outside [0, vocab) or block outside [0, num_blocks) */
  KV_EALIAS = -3,    /* a block listed twice in one call                         */
  KV_ECAPACITY = -4, /* ceil(len / block_size) > max_blocks_per_req              */
  KV_EDEVICE = -5,   /* failed health probe, pointer not on the device, HIP error */
  KV_ENOMEM = -6,    /* workspace too small, host allocation failure             */
  KV_ESTATE = -7     /* weights/arena/plan mismatch or use of a released handle  */
} kv_status;

typedef enum { KV_F32 = 0, KV_BF16 = 1 } kv_dtype;

/* Decoder shape.  Weights, activations and arena share `dtype`.
 * Supported: num_q_heads % num_kv_heads == 0; for KV_BF16 head_dim == 128,
 * hidden % 256 == 0, num_kv_heads even, ffn_dim % 128 == 0; for KV_F32
 * 128 % head_dim == 0 and (num_kv_heads * head_dim) % 128 == 0.
 * Two attention variants of the model families the paper evaluates (Qwen3
 * in Sec. 7.1, Qwen2.5 in Fig. 3): qk_norm = 1 applies an RMSNorm with a
 * [head_dim] gain (and rms_eps) to every q and k head before RoPE (head_dim
 * >= 32); qkv_bias = 1 adds biases to the q, k and v projections. */
typedef struct {
  int32_t num_layers, hidden, num_q_heads, num_kv_heads, head_dim, ffn_dim, vocab;
  double rms_eps;    /* RMSNorm epsilon                                   */
  double rope_theta; /* RoPE base; angle of pair i at position p is p * theta^(-2i/d) */
  int32_t dtype;     /* kv_dtype                                          */
  int32_t qk_norm;   /* 0 or 1: per-head q/k RMSNorm before RoPE          */
  int32_t qkv_bias;  /* 0 or 1: biases on the q, k, v projections         */
} kv_model_desc;

/* One layer, device pointers, nn.Linear layout [out, in] row-major:
 * attn_norm, ffn_norm [hidden]; wq [nq*d, hidden]; wk, wv [nkv*d, hidden]
 * (row h*d + e is head h, dim e); wo [hidden, nq*d]; w_gate, w_up
 * [ffn, hidden]; w_down [hidden, ffn].  Variant weights: q_norm, k_norm
 * [head_dim] (required when qk_norm), bq [nq*d], bk, bv [nkv*d] (required
 * when qkv_bias); NULL otherwise.  Read in place, never copied. */
typedef struct {
  const void *attn_norm, *wq, *wk, *wv, *wo, *ffn_norm, *w_gate, *w_up, *w_down;
  const void *q_norm, *k_norm, *bq, *bk, *bv;
} kv_layer_weights;

typedef struct {
  kv_model_desc desc;
  const void* embed;               /* device [vocab, hidden]                  */
  const kv_layer_weights* layers;  /* host array of num_layers entries        */
} kv_weights;

typedef struct kv_arena* kv_arena_t;
typedef struct kv_plan* kv_plan_t;

/* Bind a retained arena (Sec. 4.1 state isolation; Sec. 6 "KV-cache pointers
 * and metadata").  `base` is a device allocation of `bytes` bytes on `device`
 * laid out as, in elements of desc->dtype,
 *   off(l, kv, b, s, h, e) = ((((l*2 + kv)*num_blocks + b)*block_size + s)*nkv + h)*d + e
 * with kv = 0 for K and 1 for V, i.e. each (layer, K|V) plane is
 * [num_blocks*block_size token slots][nkv][d].  Requires
 * bytes >= L*2*num_blocks*block_size*nkv*d*elem.  Runs the health probe of
 * Sec. 4.2 step 2 (a kernel round trip on `device` plus a pointer-attribute
 * check); on failure returns KV_EDEVICE and creates no handle.  Never writes
 * the arena.  *out receives the handle. */
kv_status kv_arena_bind(void* base, uint64_t bytes, const kv_model_desc* desc,
                        int32_t block_size, int64_t num_blocks, int32_t device,
                        kv_arena_t* out);

/* Drop a handle.  Never frees or writes `base`.  Waits for nothing. */
kv_status kv_arena_release(kv_arena_t arena);

/* Workspace bytes for rebuilding `num_requests` requests totalling
 * `total_tokens` tokens in waves of at most `wave_tokens` tokens (a request
 * is never split, so wave_tokens must be >= the longest request).  Returns 0
 * for an invalid description. */
uint64_t kv_rebuild_workspace_bytes(const kv_model_desc* desc, int32_t num_requests,
                                    int64_t total_tokens, int64_t wave_tokens);

/* Host-only argument check of a rebuild (no device access), returning the
 * status kv_rebuild would return for these arguments on an arena of this
 * geometry, workspace aside. */
kv_status kv_rebuild_check(const kv_model_desc* desc, int32_t block_size, int64_t num_blocks,
                           const int32_t* token_prefixes, const int32_t* prefix_lens,
                           int32_t num_requests, const int32_t* block_tables,
                           int32_t max_blocks_per_req);

/* Rebuild (Sec. 4.2 step 5, Sec. 4.3).
 *   token_prefixes  host int32, sum(prefix_lens) entries packed in request order
 *   prefix_lens     host int32 [num_requests], each >= 0 (0 = no-op request)
 *   block_tables    host int32 [num_requests][max_blocks_per_req]; entry b of
 *                   request r is the arena block holding positions
 *                   [b*block_size, (b+1)*block_size); entries past
 *                   ceil(len/block_size) are ignored
 *   workspace       device scratch of workspace_bytes bytes (see
 *                   kv_rebuild_workspace_bytes); the largest wave that fits is used
 * Write contract: for every request r, position p < len_r and layer l, exactly
 * the K row (rotated) and V row at slot (table[r][p/B], p%B) are written;
 * nothing else in the arena is written (other blocks, tail slots of the last
 * block, table entries past the used ones).  Positions restart at 0 for each
 * request.  Results do not depend on prior slot contents, and a repeat of the
 * same call rewrites bit-identical values (deterministic kernels).
 * Host arrays may be reused when the call returns (they are staged into the
 * workspace); the rebuild itself runs asynchronously on `stream`. */
kv_status kv_rebuild(const kv_weights* w, const int32_t* token_prefixes,
                     const int32_t* prefix_lens, int32_t num_requests,
                     const int32_t* block_tables, int32_t max_blocks_per_req,
                     kv_arena_t arena, void* workspace, uint64_t workspace_bytes, void* stream);

/* kv_rebuild split in two: kv_rebuild_stage validates, plans the waves and
 * uploads all metadata into `workspace` on `stream`; kv_rebuild_execute runs
 * the device work of a staged plan (any number of times, each a full rebuild
 * with identical results) on a stream ordered after the staging.  The
 * workspace must not be reused while the plan is alive. */
kv_status kv_rebuild_stage(kv_arena_t arena, const int32_t* token_prefixes,
                           const int32_t* prefix_lens, int32_t num_requests,
                           const int32_t* block_tables, int32_t max_blocks_per_req,
                           void* workspace, uint64_t workspace_bytes, void* stream,
                           kv_plan_t* out);
kv_status kv_rebuild_execute(const kv_weights* w, kv_plan_t plan, void* stream);
kv_status kv_plan_release(kv_plan_t plan);

/* Planned wave count and the token count of the largest wave of a plan. */
kv_status kv_plan_info(kv_plan_t plan, int32_t* num_waves, int64_t* max_wave_tokens);

/* Message for the calling thread's last non-OK status ("" if none). */
const char* kv_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
