/*
 * kvr_profile.h -- optional per-kernel-class timing of kv_rebuild_execute.
 *
 * When enabled on an arena, every kernel launch of a rebuild is bracketed by
 * two HIP events on the caller's stream.  kv_profile_read waits for the
 * recorded events and returns, per kernel class, the accumulated device time
 * (ms), the number of launches and the algorithmic flops of those launches
 * (GEMMs: 2*T*N*K over the real, unpadded tokens T; attention: 4*nq*d per
 * visible causal (query, key) pair).
 * Used for roofline accounting; adds two event records per launch.
 */
#ifndef KVR_PROFILE_H
#define KVR_PROFILE_H
#include <stdint.h>
#include "kvr.h"

#ifdef __cplusplus
extern "C" {
#endif

enum {
  KV_PROF_ROPE = 0,        /* RoPE cos/sin table                               */
  KV_PROF_NORM = 1,        /* embedding gather + RMSNorm, RMSNorm              */
  KV_PROF_GEMM_QKV = 2,    /* QKV GEMM + RoPE + arena scatter                  */
  KV_PROF_ATTN = 3,        /* causal GQA attention                             */
  KV_PROF_GEMM_O = 4,      /* output projection + residual                     */
  KV_PROF_GEMM_GATEUP = 5, /* gate/up GEMM + SwiGLU                            */
  KV_PROF_GEMM_DOWN = 6,   /* down projection + residual                       */
  KV_PROF_CLASSES = 7
};

kv_status kv_profile_enable(kv_arena_t arena, int32_t enable);
/* Accumulated totals since the last reset; arrays of n_classes entries (any may be NULL). */
kv_status kv_profile_read(kv_arena_t arena, double* ms, int64_t* launches, double* flops,
                          int32_t n_classes);
kv_status kv_profile_reset(kv_arena_t arena);

#ifdef __cplusplus
}
#endif
#endif
