// Block commit digests and the leading-intact count per request.
//
// A block's digest covers its first nslots slots in every (layer, K|V) plane:
// the covered bytes are read as little-endian 32-bit words u_i, numbered plane
// by plane, and digest = sum_i (u_i ^ (i * DIGEST_KEY mod 2^32))^2 mod 2^64.
// The sum is associative and commutative modulo 2^64, so the workgroup may
// reduce the terms in any order and still produce the exact value.
//
// The scan is HBM-bound: each covered byte is read once and costs a few
// integer operations (one 32x32->64 multiply-add per word).  One workgroup
// per entry streams its planes with 16-byte loads, eight in flight per lane.
#include <hip/hip_runtime.h>

#include "launch.h"

namespace kvr {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int DG_THREADS = 256;
constexpr int DG_UNROLL = 8;

__device__ __forceinline__ uint64_t sq_words(u32x4 v, uint32_t k) {
  const uint32_t x0 = v.x ^ k;
  const uint32_t x1 = v.y ^ (k + DIGEST_KEY);
  const uint32_t x2 = v.z ^ (k + 2u * DIGEST_KEY);
  const uint32_t x3 = v.w ^ (k + 3u * DIGEST_KEY);
  return (uint64_t)x0 * x0 + (uint64_t)x1 * x1 + (uint64_t)x2 * x2 + (uint64_t)x3 * x3;
}

__global__ __launch_bounds__(DG_THREADS) void block_digest_kernel(DigestParams p) {
  __shared__ uint64_t red[DG_THREADS];
  const int64_t e = blockIdx.x;
  const int2 ent = p.entries[e];
  const int64_t nbytes = (int64_t)ent.y * p.row_bytes;
  const int cpp = (int)(nbytes >> 4);            // 16-byte chunks per plane
  const uint32_t wpp = (uint32_t)(nbytes >> 2);  // words per plane (mod 2^32)
  const char* base = p.arena + (int64_t)ent.x * p.block_bytes;
  const int t = threadIdx.x;
  uint64_t acc = 0;
  for (int pl = 0; pl < p.planes; ++pl) {
    const u32x4* src = reinterpret_cast<const u32x4*>(base + (int64_t)pl * p.plane_bytes);
    const uint32_t ibase = (uint32_t)pl * wpp;
    int c0 = t;
    // full rounds: DG_UNROLL loads in flight per lane, no bounds checks
    for (; c0 + (DG_UNROLL - 1) * DG_THREADS < cpp; c0 += DG_THREADS * DG_UNROLL) {
      u32x4 v[DG_UNROLL];
#pragma unroll
      for (int u = 0; u < DG_UNROLL; ++u) v[u] = __builtin_nontemporal_load(src + c0 + u * DG_THREADS);
#pragma unroll
      for (int u = 0; u < DG_UNROLL; ++u)
        acc += sq_words(v[u], (ibase + 4u * (uint32_t)(c0 + u * DG_THREADS)) * DIGEST_KEY);
    }
    // ragged end of the plane
    for (; c0 < cpp; c0 += DG_THREADS)
      acc += sq_words(__builtin_nontemporal_load(src + c0), (ibase + 4u * (uint32_t)c0) * DIGEST_KEY);
  }
  red[t] = acc;
  __syncthreads();
#pragma unroll
  for (int w = DG_THREADS / 2; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  if (t == 0) {
    const uint64_t dg = red[0];
    if (p.digests) p.digests[e] = dg;
    if (p.committed) p.match[e] = dg == p.committed[e] ? 1 : 0;
  }
}

__global__ __launch_bounds__(DG_THREADS) void leading_intact_kernel(const int32_t* offsets,
                                                                    const uint8_t* match,
                                                                    int32_t* intact) {
  __shared__ int32_t red[DG_THREADS];
  const int r = blockIdx.x;
  const int32_t off = offsets[r], nb = offsets[r + 1] - off;
  const int t = threadIdx.x;
  int32_t first = nb;
  // the first mismatch among entries t, t+256, ...; the minimum over lanes is the first overall
  for (int32_t j = t; j < nb; j += DG_THREADS)
    if (!match[off + j]) {
      first = j;
      break;
    }
  red[t] = first;
  __syncthreads();
#pragma unroll
  for (int w = DG_THREADS / 2; w > 0; w >>= 1) {
    if (t < w) red[t] = min(red[t], red[t + w]);
    __syncthreads();
  }
  if (t == 0) intact[r] = red[0];
}

// Exclusive prefix sum of the per-request block counts in one workgroup, in
// chunks of DG_THREADS requests carried from one chunk to the next.
__global__ __launch_bounds__(DG_THREADS) void verify_offsets_kernel(const int32_t* lens, int32_t R,
                                                                    int32_t B, int32_t* offsets) {
  __shared__ int32_t sc[DG_THREADS];
  const int t = threadIdx.x;
  int32_t carry = 0;
  for (int32_t r0 = 0; r0 < R; r0 += DG_THREADS) {
    const int32_t r = r0 + t;
    const int32_t nb = r < R ? (lens[r] + B - 1) / B : 0;
    sc[t] = nb;
    __syncthreads();
    // Hillis-Steele inclusive scan
    for (int o = 1; o < DG_THREADS; o <<= 1) {
      const int32_t v = t >= o ? sc[t - o] : 0;
      __syncthreads();
      sc[t] += v;
      __syncthreads();
    }
    if (r < R) offsets[r] = carry + sc[t] - nb;
    carry += sc[DG_THREADS - 1];
    __syncthreads();
  }
  if (t == 0) offsets[R] = carry;
}

// One workgroup per request: its entries (block id, covered slots).
__global__ __launch_bounds__(DG_THREADS) void verify_entries_kernel(const int32_t* lens,
                                                                    const int32_t* tables,
                                                                    int32_t max_blocks, int32_t B,
                                                                    const int32_t* offsets,
                                                                    int2* entries) {
  const int32_t r = blockIdx.x;
  const int32_t off = offsets[r], nb = offsets[r + 1] - off, n = lens[r];
  const int32_t* tab = tables + (int64_t)r * max_blocks;
  for (int32_t j = threadIdx.x; j < nb; j += DG_THREADS)
    entries[off + j] = make_int2(tab[j], min(B, n - j * B));
}

}  // namespace

void launch_verify_entries(const int32_t* lens, const int32_t* tables, int32_t num_requests,
                           int32_t max_blocks, int32_t block_size, int32_t* offsets, int2* entries,
                           hipStream_t s) {
  if (num_requests <= 0) return;
  verify_offsets_kernel<<<dim3(1), dim3(DG_THREADS), 0, s>>>(lens, num_requests, block_size, offsets);
  verify_entries_kernel<<<dim3((unsigned)num_requests), dim3(DG_THREADS), 0, s>>>(
      lens, tables, max_blocks, block_size, offsets, entries);
}

void launch_block_digest(const DigestParams& p, hipStream_t s) {
  if (p.num_entries <= 0) return;
  block_digest_kernel<<<dim3((unsigned)p.num_entries), dim3(DG_THREADS), 0, s>>>(p);
}

void launch_leading_intact(const int32_t* offsets, int32_t num_requests, const uint8_t* match,
                           int32_t* intact, hipStream_t s) {
  if (num_requests <= 0) return;
  leading_intact_kernel<<<dim3((unsigned)num_requests), dim3(DG_THREADS), 0, s>>>(offsets, match,
                                                                                  intact);
}

}  // namespace kvr
