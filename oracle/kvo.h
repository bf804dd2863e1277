/*
 * kvo.h -- CPU oracle for the KV rebuild.  TEST INFRASTRUCTURE ONLY.
 *
 * This is the plain, slow reference that the HIP rebuild is checked against.
 * Only the test suite, the package smoke check and the benchmark's CPU
 * baseline may load it; the product library never calls into it, and the two
 * share no code, headers or tables.
 *
 * What it computes: the re-prefill that rebuilds request-specific KV contents
 * from logged token prefixes into a retained raw KV arena after a worker
 * failure (Sec. 4.2 Handover, step 5; Sec. 4.3 LLM Context Recovery), with the
 * whole pool flushed and refilled because complete KV contents are not
 * trusted across the failure (Sec. 4.2, flush-and-refill paragraph; Sec. 2.3
 * Finding 2).  The paper does not write out the model forward; the oracle
 * takes a Llama-style pre-norm decoder (RMSNorm, Q/K/V projections, NeoX
 * half-split RoPE, causal GQA softmax attention, output projection, SwiGLU
 * FFN, fp32 residual stream), optionally with the two variants of the Qwen
 * models the paper evaluates (Sec. 7.1; Fig. 3 uses Qwen2.5): biases on the
 * q/k/v projections, and a per-head RMSNorm of q and k before RoPE and writes the rotated K and the V of every
 * position of every layer into a paged arena through per-request block tables.
 *
 * Precision contract: every reduction is accumulated in fp64; every op output
 * is rounded to fp32 (the working precision) and, for bf16 models, the
 * normed activations, rotated Q/K, V, the attention output and the SwiGLU
 * output are rounded to bf16 (round-to-nearest-even).  dtype KVO_F64 is a pin
 * mode in which nothing is rounded at all.
 */
#ifndef KVO_ORACLE_H
#define KVO_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { KVO_F32 = 0, KVO_BF16 = 1, KVO_F64 = 2 };

typedef struct {
  int32_t num_layers, hidden, num_q_heads, num_kv_heads, head_dim, ffn_dim, vocab;
  double rms_eps, rope_theta;
  int32_t dtype;         /* element type of weights and arena: KVO_F32/BF16/F64 */
  int32_t qk_norm;       /* 1: per-head RMSNorm of q and k before RoPE (Qwen3)   */
  int32_t qkv_bias;      /* 1: q, k, v projections carry a bias (Qwen2.5)        */
  int32_t round_p;       /* 1: attention weights rounded to the model dtype
                            before the P.V sum and the denominator, each weight
                            exp(z - max z) scaled by a power of two first:
                            P_j = rnd(2^(z_j log2 e - c)), c = ceil(max z log2 e)
                            (the GPU's declared freedom; 0 = the definition)   */
} kvo_model;

/* One layer's weights, host pointers, nn.Linear layout [out, in] row-major.
 * q_norm, k_norm [head_dim] (qk_norm models); bq [nq*d], bk, bv [nkv*d]
 * (qkv_bias models); otherwise NULL. */
typedef struct {
  const void *attn_norm, *wq, *wk, *wv, *wo, *ffn_norm, *w_gate, *w_up, *w_down;
  const void *q_norm, *k_norm, *bq, *bk, *bv;
} kvo_layer;

/* Paged arena (host memory): element offset of (layer l, plane kv, block b,
 * slot s, kv head h, dim e) is ((((l*2+kv)*num_blocks+b)*block_size+s)*nkv+h)*d+e. */
typedef struct {
  void* base;
  int32_t block_size;
  int64_t num_blocks;
} kvo_arena;

/* Prefill mode: all positions of each request per layer.
 * tokens: packed [sum(lens)]; block_tables: [R][max_blocks].
 * final_hidden (optional, may be NULL): [sum(lens)][hidden] fp64 residual
 * after the last layer's FFN (computed only when non-NULL).
 * Returns 0 on success, -1 on an invalid argument. */
int kvo_rebuild(const kvo_model* m, const void* embed, const kvo_layer* layers,
                const int32_t* tokens, const int32_t* lens, int32_t num_requests,
                const int32_t* block_tables, int32_t max_blocks,
                kvo_arena* arena, double* final_hidden);

/* Decode mode: the same requests fed one token at a time through all layers,
 * attention reading past K/V back from the arena through the block table. */
int kvo_decode(const kvo_model* m, const void* embed, const kvo_layer* layers,
               const int32_t* tokens, const int32_t* lens, int32_t num_requests,
               const int32_t* block_tables, int32_t max_blocks,
               kvo_arena* arena, double* final_hidden);

/* One decode step of the resumed generation: token tokens[r] of request r at
 * position positions[r], whose K/V for positions < positions[r] are already in
 * the arena.  Writes its K/V at slot (table[p/B], p%B) in every layer and, if
 * final_hidden is non-NULL ([R][hidden] fp64), the residual after the last
 * layer (the paper's recoverability criterion: generation continues from the
 * rebuilt state as from the original one, Sec. 4.2, Sec. 6). */
int kvo_decode_step(const kvo_model* m, const void* embed, const kvo_layer* layers,
                    const int32_t* tokens, const int32_t* positions, int32_t num_requests,
                    const int32_t* block_tables, int32_t max_blocks, kvo_arena* arena,
                    double* final_hidden);

/* Final RMSNorm (gain final_norm, rounded like every norm output) and LM head
 * lm_head [vocab, hidden]: logits_out[r][v] = fp32(sum_e W[v][e] a_r[e]), the
 * sum in fp64, for n rows of the final residual stream. */
int kvo_logits(const kvo_model* m, const void* final_norm, const void* lm_head,
               const double* hidden, int64_t n, float* logits_out);

/* Layer-0 rounded K and V rows (each num_kv_heads*head_dim elements of the
 * model dtype, written to k_out / v_out) for (token, position) pairs; layer 0
 * depends on nothing else, so sampled positions of a large batch can be
 * checked one by one. */
int kvo_layer0_kv(const kvo_model* m, const void* embed, const kvo_layer* layer0,
                  const int32_t* tokens, const int32_t* positions, int64_t n,
                  void* k_out, void* v_out);

/* Run layers [0, num_layers) of one request of n tokens without an arena
 * (scratch K/V), used to time the oracle on a bounded sample. */
int kvo_time_layers(const kvo_model* m, const void* embed, const kvo_layer* layers,
                    const int32_t* tokens, int32_t n, int32_t num_layers);

/* Rebuild from a retained prefix (partial recovery and shared-prefix reuse,
 * the two ways of not recomputing K/V the pool still holds): request r's
 * positions starts[r] .. lens[r]-1 are recomputed and written, while the K/V of
 * positions 0 .. starts[r]-1 are taken as already in the arena (its table
 * entries for them are read, their slots are not written).  tokens packs the
 * recomputed positions' tokens only: sum of (lens[r] - starts[r]).  Attention
 * of every recomputed position covers positions 0 .. p, reading the prefix
 * K/V from the arena.  With all starts 0 this is kvo_rebuild.  final_hidden
 * (optional) has one row per recomputed position.  Returns 0, or -1 on an
 * invalid argument (a start outside [0, len], a token or table entry out of
 * range). */
int kvo_rebuild_from(const kvo_model* m, const void* embed, const kvo_layer* layers,
                     const int32_t* tokens, const int32_t* lens, const int32_t* starts,
                     int32_t num_requests, const int32_t* block_tables, int32_t max_blocks,
                     kvo_arena* arena, double* final_hidden);

/* Commit digest of one block (flush-free recovery; the paper flushes the
 * whole pool because it cannot tell which KV contents survived intact, and
 * leaves fine-grained consistency tracking to future work: Sec. 4.2 flush
 * paragraph, Sec. 8 future work).  The digest covers slots 0 .. nslots-1 of
 * `block` in every layer and both planes.  Read those bytes as 32-bit
 * little-endian words u_0 .. u_{N-1} in the order (layer, K then V, slot, byte
 * within the slot row), N = num_layers * 2 * nslots * row_bytes / 4; then
 *     digest = sum over i of (u_i XOR (i * 0x9E3779B9 mod 2^32))^2  mod 2^64
 * (the square taken as a 64-bit product of two 32-bit values).  nslots = 0
 * gives 0.  Returns -1 in *ok on invalid arguments (row bytes not a multiple
 * of 4, block or nslots out of range), else 0. */
uint64_t kvo_block_digest(const kvo_model* m, const kvo_arena* a, int64_t block, int32_t nslots,
                          int* ok);

/* Verify the committed digests of a request set: request r occupies blocks
 * tables[r][0 .. ceil(lens[r]/B)-1]; block j of it covers min(B, lens[r]-j*B)
 * slots.  Entries are numbered request by request, block by block.  Writes
 * every entry's digest to digests (may be NULL) and, per request, the number
 * of leading blocks whose digest equals committed[entry] to intact.
 * Returns 0, or -1 on invalid arguments. */
int kvo_verify(const kvo_model* m, const kvo_arena* a, const int32_t* lens, int32_t R,
               const int32_t* tables, int32_t max_blocks, const uint64_t* committed,
               uint64_t* digests, int32_t* intact);

/* fp32 -> bf16 bits exactly as the oracle rounds (exported for its pins). */
uint16_t kvo_round_bf16(float x);

/* OpenMP threads the oracle runs with. */
int kvo_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
