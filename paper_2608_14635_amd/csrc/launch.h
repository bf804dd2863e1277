// Kernel launch interface between the host planner (abi.cpp) and the device
// code.  Plain structs of device pointers and sizes; no HIP types beyond
// hipStream_t.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvr {

enum Epi : int {
  EPI_QKV = 0,     // RoPE on q/k; Q -> workspace, K/V -> arena slots (+ V^T for attention)
  EPI_RESID = 1,   // X += acc (fp32 residual stream)
  EPI_SWIGLU = 2,  // Hf = silu(gate) * up
  EPI_STORE = 3,   // X = acc (fp32 output, e.g. transposed logits)
  EPI_PARTIAL = 4, // split-K pass: fp32 partial tile of one K range (see launch_gemm_bf16_splitk)
};

enum BMap : int {
  BMAP_PLAIN = 0,   // B rows n of one matrix
  BMAP_QKV = 1,     // rows [0,s0) of Wq, [s0,s1) of Wk, [s1,..) of Wv
  BMAP_GATEUP = 2,  // tile of BN rows = BN/2 rows of W_gate then the same BN/2 rows of W_up
};

struct EpiParams {
  // QKV
  void* q_out;            // [rows][nq*d]
  void* arena_k;          // this layer's K plane: [slots][nkv][d]
  void* arena_v;          // this layer's V plane
  void* vt;               // V^T (bf16 path, vt_offset layout) or null; row m at key krow(m)
  int64_t ldvt;
  void* kc;               // K copy [nkv][ldvt][d] (bf16 path) or null; row m at row krow(m)
  const int32_t* krow;    // per row: its key row in kc/vt (null = the row itself)
  const int64_t* slot;    // per wave-local row: arena slot index, -1 for padding rows
  const int32_t* pos;     // per wave-local token: position within its request
  const float2* rope;     // [max_pos][d/2] (cos, sin)
  int nq, nkv, d;
  // QKV variants: q/k/v biases (null = none) and per-head q/k RMSNorm gains
  const void* bq;
  const void* bk;
  const void* bv;
  const void* q_norm;     // null = no per-head norm
  const void* k_norm;
  float eps;
  // RESID
  float* x;               // [rows][ldx]
  int ldx;
  // SWIGLU
  void* hf;               // [rows][ldh]
  int ldh;
  int ffn;
};

struct GemmParams {
  const void* A;          // [M][K] activations, K contiguous
  int64_t lda;
  int M, K;
  const void* B0;         // weights [.][ldb] rows, K contiguous
  const void* B1;
  const void* B2;
  int64_t ldb;            // B row stride in elements (0 = K)
  int bmap;
  int s0, s1;             // BMAP_QKV split points (logical columns)
  int n_begin, n_end;     // logical column range of C computed by this launch
  EpiParams epi;
  // split-K (EPI_PARTIAL): K tiles [split*kt_per, ...) of each output tile go
  // to part + split*part_stride, row-major with part_ld columns
  int ksplit, kt_per;
  float* part;
  int64_t part_stride;
  int part_ld;
  int group_m;            // M tiles walked together by an XCD's workgroups (set by the launcher)
};

// Elementwise / small kernels
void launch_rope_table(float2* table, int max_pos, int d, double theta, hipStream_t s);
void launch_embed_norm(int dtype, const void* embed, const int32_t* tok, const void* gain,
                       float* x, void* a_out, int rows, int hidden, float eps, hipStream_t s);
void launch_rmsnorm(int dtype, const float* x, const void* gain, void* a_out, int rows,
                    int hidden, float eps, hipStream_t s);
int launch_probe(int* dev_flag, hipStream_t s);

// GEMMs with fused epilogues
void launch_gemm_bf16(int epi, const GemmParams& p, hipStream_t s);
void launch_gemm_f32(int epi, const GemmParams& p, hipStream_t s);
// Few-row products (the decode step): K split over enough workgroups to fill
// the chip, fp32 partials summed in split order by a second kernel that then
// applies the epilogue `epi`.  part holds part_cap floats.
void launch_gemm_bf16_splitk(int epi, const GemmParams& p, float* part, int64_t part_cap,
                             hipStream_t s);
int64_t gemm_bf16_splitk_part_elems(int M, int N, int K);
// Few-row product into the residual stream followed by the RMSNorm of the
// updated rows: X[m] += A[m] . B^T (split-K sums in split order, as
// launch_gemm_bf16_splitk with EPI_RESID), then a_out[m] = round(gain * X[m] /
// rms(X[m])) (bf16, row stride N).  Returns false, launching nothing, where
// the few-row kernel or the row width does not apply.
bool launch_gemm_bf16_splitk_resid_norm(const GemmParams& p, float* part, int64_t part_cap,
                                        const void* gain, void* a_out, float eps, hipStream_t s);
// Few-row product with K unsplit, fp32 C[M][N] = A . B^T written to out (row
// stride ldo), no epilogue; B rows follow p.bmap as for the other products.
// Returns false, launching nothing, unless M <= 64, K % 128 == 0 and N is a
// multiple of the 16-row blocks a wave owns (64 for M <= 16).
bool launch_gemm_bf16_rows(const GemmParams& p, float* out, int64_t ldo, hipStream_t s);

// Attention.  qblk: per q-block int4 {q_start, q_len, req_start, 0} in
// wave-local row indices, ordered longest-first.  Each request's rows start on
// a ROW_ALIGN boundary; the padding rows after it hold finite values.
// A q-block is (first query row, query count, key row of position 0 of its
// request, position of the first query): its queries attend key rows
// key_base .. key_base + position.  Query rows and key rows are separate
// index spaces (a rebuild from a retained prefix has key rows for the
// prefix but no query rows); they coincide when every request starts at 0.
struct AttnParams {
  const void* q;          // [rows][nq*d]
  const void* arena_k;    // this layer's K plane
  const void* arena_v;    // this layer's V plane (fp32 path)
  const void* vt;         // V^T (bf16 path, vt_offset layout)
  int64_t ldvt;
  const void* kc;         // K copy [nkv][ldvt][d] (bf16 path)
  const int64_t* kslot;   // per key row: arena slot (fp32 path reads the arena)
  const int4* qblk;
  int num_qblk;
  void* out;              // [rows][nq*d]
  int nq, nkv, d;
};
// bf16 attention workgroups are 8 waves: HW heads of one GQA group x QW blocks
// of 32 queries (HW = largest of 8/4/2/1 dividing the group size).
inline int attn_heads_per_wg(int group) {
  return group % 8 == 0 ? 8 : group % 4 == 0 ? 4 : group % 2 == 0 ? 2 : 1;
}
inline int attn_qblock(int dtype, int group) {
  return dtype == 1 ? 32 * (8 / attn_heads_per_wg(group)) : 128;
}
constexpr int ATTN_QBLOCK_MIN = 32;
constexpr int ROW_ALIGN = 64;  // each request's rows start on this boundary of the wave

// The V^T copy of the bf16 attention, per kv head: key tiles of VT_KEYS keys,
// each tile stored as [d][VT_KEYS] contiguously (16 KB at d = 128), so that a
// tile is one contiguous read and the QKV epilogue's writes of one tile stay
// in one DRAM region.  Offset (elements) of column col = kvh * d + e, key row
// `key`, for ldvt key rows per head (a multiple of VT_KEYS).
constexpr int VT_KEYS = 64;
__host__ __device__ __forceinline__ int64_t vt_offset(int col, int64_t key, int64_t ldvt, int d) {
  const int kvh = col / d, e = col % d;
  return (int64_t)kvh * d * ldvt + (key / VT_KEYS) * (int64_t)d * VT_KEYS + (int64_t)e * VT_KEYS +
         key % VT_KEYS;
}
void launch_attention_bf16(const AttnParams& p, hipStream_t s);
// Prefix keys of a rebuild from a retained prefix: segment (key row, count
// <= 64) copies the arena K/V of those key rows' slots into the K copy and
// V^T (bf16 path).
constexpr int GATHER_KEYS = 64;
void launch_prefix_gather(const int2* segs, int nseg, const int64_t* kslot, const void* plane_k,
                          const void* plane_v, void* kc, void* vt, int64_t ldvt, int nkv, int d,
                          hipStream_t s);
void launch_attention_f32(const AttnParams& p, int rows_total, hipStream_t s);

// Resumed decode (one token per request over the paged arena).
struct DecodeAttnParams {
  const void* q;          // [R][nq*d] rotated queries of the step
  const void* plane_k;    // this layer's K plane [slots][nkv][d]
  const void* plane_v;    // this layer's V plane
  const int32_t* tables;  // [R][max_blocks] block tables
  int max_blocks, block_size;
  const int32_t* ctx;     // [R] keys to attend (position + 1)
  int nq, nkv, d;
  int splits;             // key ranges per (request, kv head)
  float* part;            // [R][nq][splits][d + 2] partials (o, m, l)
  void* out;              // [R][nq*d] attention output
};
void launch_rope_rows(float2* table, const int32_t* positions, int rows, int d, double theta,
                      hipStream_t s);
int decode_attn_splits(int num_requests, int nkv, int64_t max_ctx);
void launch_decode_attention(int dtype, const DecodeAttnParams& p, int num_requests, hipStream_t s);
constexpr int ARGMAX_CHUNKS = 256;  // vocab chunks of the first argmax pass
void launch_argmax(const float* logits_t, int64_t ld, int vocab, int num_requests,
                   float2* partial, int32_t* next_tokens, float* logits_out, hipStream_t s);
// The same greedy choice over row-major logits [num_requests][ld].
void launch_argmax_rows(const float* logits, int64_t ld, int vocab, int num_requests,
                        float2* partial, int32_t* next_tokens, hipStream_t s);

// Block commit digests (flush-free recovery): one workgroup per entry reads
// the entry's covered slots in every plane and reduces the keyed sum of squares.
constexpr uint32_t DIGEST_KEY = 0x9E3779B9u;  // word-index multiplier of the key
struct DigestParams {
  const char* arena;        // arena base
  int64_t plane_bytes;      // bytes of one (layer, K|V) plane: num_blocks * block_size * row
  int64_t block_bytes;      // block_size * row
  int32_t row_bytes;        // one slot: nkv * d * element bytes (a multiple of 16)
  int32_t planes;           // 2 * num_layers
  const int2* entries;      // [n] (block id, covered slots)
  int64_t num_entries;
  const uint64_t* committed;  // [n] or null
  uint64_t* digests;        // [n] or null
  uint8_t* match;           // [n] digest == committed (written when committed is set)
};
void launch_block_digest(const DigestParams& p, hipStream_t s);
// intact[r] = index of request r's first entry (offsets[r] .. offsets[r+1]-1)
// whose match flag is 0, or its entry count when all match
void launch_leading_intact(const int32_t* offsets, int32_t num_requests, const uint8_t* match,
                           int32_t* intact, hipStream_t s);
// The entry list and request offsets of a verification built on the device
// from the raw lens [R] and block tables [R][max_blocks]: offsets[r] = sum of
// ceil(lens[q]/B) over q < r (offsets[R] = E); entry offsets[r] + j = (table
// entry j of request r, its covered slots min(B, lens[r] - j*B)).
void launch_verify_entries(const int32_t* lens, const int32_t* tables, int32_t num_requests,
                           int32_t max_blocks, int32_t block_size, int32_t* offsets, int2* entries,
                           hipStream_t s);

}  // namespace kvr
