// Kernels of the resumed decode step (one new token per request over the
// rebuilt arena): the RoPE rows of the step's positions, paged split-K decode
// attention with its fixed-order combine, and the greedy argmax over the LM
// head's logits.
//
// Decode attention reads K and V straight from the paged arena: key j of
// request r lives at slot table[r][j/B]*B + j%B of the layer's K and V planes.
// A workgroup (4 waves) takes one (request, kv head, key range) and all g q
// heads of that kv head.  Per block of 64 keys it stages the K and V rows in
// LDS (coalesced 16-byte loads of whole rows), computes the g x 64 scores with
// one key per lane (row pitch padded by 16 bytes, so 16-lane LDS phases hit
// distinct banks; the next block is in flight in registers meanwhile, and
// the key range's block-table entries are staged in LDS once), runs the
// online softmax per head in the exp2 domain (one
// wave owns a head's running max and sum), and accumulates P.V with threads
// over (head, dim).  Each split writes (m, l, o[d]) partials; a second kernel
// merges the splits in index order, so results do not depend on timing.
// The step is HBM-bound on the context's K/V reads.  For bf16 models with
// head_dim 128 a second kernel does the same work with matrix-core scores
// and register-direct loads (decode_attn_mfma_kernel); the general one
// serves fp32 models and other head sizes.
#include <algorithm>

#include "common.h"
#include "launch.h"

namespace kvr {

namespace {

constexpr int DKB = 64;    // keys per staged block
constexpr int DNT = 256;   // 4 waves
constexpr int DMAXG = 16;  // q heads per kv head supported
constexpr int DMAXD = 128;
constexpr int TABN = 1024;  // block-table entries staged in LDS per workgroup
constexpr int DMAXS = 128;  // key ranges per (request, kv head) the combine supports

__global__ void rope_rows_kernel(float2* table, const int32_t* positions, int rows, int half,
                                 double theta, int d) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)rows * half) return;
  const int r = (int)(idx / half), i = (int)(idx % half);
  const double inv_freq = pow(theta, -(double)(2 * i) / (double)d);
  const double phi = (double)positions[r] * inv_freq;
  table[idx] = make_float2((float)cos(phi), (float)sin(phi));
}

__device__ __forceinline__ void load_vals8(const float* p, float* v) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void load_vals8(const bf16_t* p, float* v) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
  v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
  v[4] = __uint_as_float(u.z << 16); v[5] = __uint_as_float(u.z & 0xffff0000u);
  v[6] = __uint_as_float(u.w << 16); v[7] = __uint_as_float(u.w & 0xffff0000u);
}

template <typename T>
__global__ __launch_bounds__(DNT) void decode_attn_kernel(DecodeAttnParams p) {
  constexpr int PITCH = DMAXD * (int)sizeof(T) + 16;  // bytes per staged row
  __shared__ __attribute__((aligned(16))) char sk[DKB * PITCH];
  __shared__ __attribute__((aligned(16))) char sv[DKB * PITCH];
  __shared__ float sq[DMAXG * DMAXD];
  __shared__ float sp[DMAXG * DKB];
  __shared__ float s_m[DMAXG], s_l[DMAXG], s_alpha[DMAXG];
  __shared__ int s_tab[TABN];

  const int S = p.splits;
  int bid = blockIdx.x;
  const int split = bid % S;
  bid /= S;
  const int kvh = bid % p.nkv, r = bid / p.nkv;
  const int g = p.nq / p.nkv, d = p.d;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int ctx = p.ctx[r];
  const int chunk = ((ctx + S - 1) / S + DKB - 1) / DKB * DKB;
  const int k0 = split * chunk, k1 = min(ctx, k0 + chunk);
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)d);
  const int64_t row_elems = (int64_t)p.nkv * d;  // one token slot of a plane

  // queries of the g heads, fp32
  const T* qsrc = reinterpret_cast<const T*>(p.q) + (int64_t)r * p.nq * d + (int64_t)kvh * g * d;
  for (int i = tid; i < g * d; i += DNT) sq[i] = Elem<T>::load(qsrc, i);
  if (tid < g) {
    s_m[tid] = -INFINITY;
    s_l[tid] = 0.0f;
  }
  // P.V outputs of this thread: (head, dim) pairs o = tid + DNT * j
  constexpr int OMAX = DMAXG * DMAXD / DNT;
  float acc[OMAX];
#pragma unroll
  for (int j = 0; j < OMAX; ++j) acc[j] = 0.0f;
  const int* table = p.tables + (int64_t)r * p.max_blocks;
  const T* Kp = reinterpret_cast<const T*>(p.plane_k);
  const T* Vp = reinterpret_cast<const T*>(p.plane_v);
  const int units = d * (int)sizeof(T) / 16;  // 16-byte units per row
  __syncthreads();

  // block-table entries of the key range, staged once (entries past the
  // first TABN are read from the global table)
  const int B = p.block_size;
  const int b0 = k0 / B;
  if (k0 < k1)
    for (int i = tid; i <= (k1 - 1) / B - b0 && i < TABN; i += DNT) s_tab[i] = table[b0 + i];
  __syncthreads();

  // K/V of one 64-key block: DKB * units 16-byte pieces, PF per thread; the
  // next block is in flight in registers while this one is used from LDS
  // (a deeper register queue costs occupancy and was slower).
  constexpr int PF = DKB * (DMAXD * (int)sizeof(T) / 16) / DNT;
  uint4 ka[PF], va[PF];
  auto fetch = [&](uint4* kr, uint4* vr, int kb) {
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      const int i = tid + q * DNT;
      kr[q] = make_uint4(0, 0, 0, 0);
      vr[q] = make_uint4(0, 0, 0, 0);
      if (i < DKB * units) {
        const int key = i / units, u = i % units, j = kb + key;
        if (j < k1) {
          const int bi = j / B - b0;
          const int blk = bi < TABN ? s_tab[bi] : table[j / B];
          const int64_t off = ((int64_t)blk * B + j % B) * row_elems + (int64_t)kvh * d;
          kr[q] = reinterpret_cast<const uint4*>(Kp + off)[u];
          vr[q] = reinterpret_cast<const uint4*>(Vp + off)[u];
        }
      }
    }
  };
  auto park = [&](const uint4* kr, const uint4* vr) {
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      const int i = tid + q * DNT;
      if (i < DKB * units) {
        const int key = i / units, u = i % units;
        *reinterpret_cast<uint4*>(sk + key * PITCH + u * 16) = kr[q];
        *reinterpret_cast<uint4*>(sv + key * PITCH + u * 16) = vr[q];
      }
    }
  };
  // scores, online softmax and P.V of the block of keys kb.. parked in LDS
  auto attend = [&](int kb) {
    // ---- scores: one key per lane, heads h = wid, wid+4, ... ----
    const bool kvalid = kb + lane < k1;
    for (int h = wid; h < g; h += DNT / 64) {
      float s = 0.0f;
      const T* krow = reinterpret_cast<const T*>(sk + lane * PITCH);
      const float* qh = sq + h * d;
      for (int e = 0; e < d; e += 8) {
        float kv8[8];
        load_vals8(krow + e, kv8);
#pragma unroll
        for (int i = 0; i < 8; ++i) s = fmaf(qh[e + i], kv8[i], s);
      }
      s = kvalid ? s * scale_log2 : -INFINITY;
      float mx = s;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      const float m_old = s_m[h];
      const float m_new = fmaxf(m_old, mx);
      const float e = __builtin_amdgcn_exp2f(s - m_new);
      const float sum = wave_sum(e);
      sp[h * DKB + lane] = e;
      if (lane == 0) {
        const float alpha = __builtin_amdgcn_exp2f(m_old - m_new);
        s_alpha[h] = alpha;
        s_l[h] = s_l[h] * alpha + sum;
        s_m[h] = m_new;
      }
    }
    __syncthreads();
    // ---- O = O * alpha + P.V over the block's keys ----
#pragma unroll
    for (int j = 0; j < OMAX; ++j) {
      const int o = tid + DNT * j;
      if (o < g * d) {
        const int h = o / d, e = o % d;
        float a = acc[j] * s_alpha[h];
        const float* ph = sp + h * DKB;
        for (int key = 0; key < DKB; ++key)
          a = fmaf(ph[key], Elem<T>::load(reinterpret_cast<const T*>(sv + key * PITCH), e), a);
        acc[j] = a;
      }
    }
    __syncthreads();
  };
  if (k0 < k1) fetch(ka, va, k0);
  for (int kb = k0; kb < k1; kb += DKB) {
    park(ka, va);
    __syncthreads();
    if (kb + DKB < k1) fetch(ka, va, kb + DKB);
    attend(kb);
  }

  // ---- partials: [r][h][split][d + 2] = o[0..d), m, l ----
  const int stride = d + 2;
#pragma unroll
  for (int j = 0; j < OMAX; ++j) {
    const int o = tid + DNT * j;
    if (o < g * d) {
      const int h = o / d, e = o % d;
      const int hq = kvh * g + h;
      p.part[(((int64_t)r * p.nq + hq) * S + split) * stride + e] = acc[j];
    }
  }
  if (tid < g) {
    const int hq = kvh * g + tid;
    float* tail = p.part + (((int64_t)r * p.nq + hq) * S + split) * stride + d;
    tail[0] = s_m[tid];
    tail[1] = s_l[tid];
  }
}

// bf16, head_dim 128: one wave per (request, kv head, key range) over tiles
// of 16 keys (a tile never crosses an arena block when the block size is a
// multiple of 16).  Each lane loads 16-byte pieces of the keys' K and V rows
// straight into registers (a key's 256-byte head slice is four lanes' worth
// per instruction); the next tile's loads are issued before this tile's
// products (the copy into place at the end of the tile waits for them).
// Scores: S^T = K Q^T on v_mfma_f32_16x16x32_bf16 with the g q heads as the
// 16 columns (unused columns hold zero queries): lane (q, c) = (lane/16,
// lane%16) gets keys 4q..4q+3 of head c.  Online softmax per head in the exp2
// domain, rescaling only when a head's max rose by more than 2^DSLACK.  P.V in
// fp32 on the VALU: lane (q, c) owns dims 8c..8c+7 of keys 4q..4q+3 and
// reads every head's P of those keys from its wave's LDS area; the four lane
// groups' partial sums are added at the end.  Same (o, m, l) partials as the
// general kernel.
constexpr int DT = 16;           // keys per tile
constexpr float DSLACK = 8.0f;   // rescale slack, log2 units

template <int GM>
__global__ __launch_bounds__(256) void decode_attn_mfma_kernel(DecodeAttnParams p) {
  __shared__ __attribute__((aligned(16))) float s_p[4][GM * DT];
  __shared__ float s_a[4][16];
  const int S = p.splits, ngrp = (p.nkv + 3) / 4;
  int bid = blockIdx.x;
  const int split = bid % S;
  bid /= S;
  const int kgrp = bid % ngrp, r = bid / ngrp;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kvh = kgrp * 4 + wave;
  if (kvh >= p.nkv) return;  // whole waves
  const int g = p.nq / p.nkv;
  const int c = lane & 15, q = lane >> 4;
  const int ctx = p.ctx[r];
  const int chunk = ((ctx + S - 1) / S + DT - 1) / DT * DT;
  const int k0 = split * chunk, k1 = min(ctx, k0 + chunk);
  const float scale_log2 = 1.4426950408889634f / sqrtf(128.0f);
  const int64_t row_bytes = (int64_t)p.nkv * 128 * 2;
  const char* Kb = reinterpret_cast<const char*>(p.plane_k) + kvh * 256;
  const char* Vb = reinterpret_cast<const char*>(p.plane_v) + kvh * 256;
  const int* table = p.tables + (int64_t)r * p.max_blocks;
  const int B = p.block_size;

  // Q^T operand: head c (zero past g), dims 32t + 8q .. +7
  bf16x8 qf[4];
  {
    const bf16_t* qrow = reinterpret_cast<const bf16_t*>(p.q) +
                         ((int64_t)r * p.nq + kvh * g + min(c, g - 1)) * 128 + 8 * q;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      qf[t] = *reinterpret_cast<const bf16x8*>(qrow + 32 * t);
      if (c >= g) qf[t] = bf16x8{};
    }
  }
  float m_run = -INFINITY, l_run = 0.0f;
  float o[GM][8];
#pragma unroll
  for (int h = 0; h < GM; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.0f;
  float* sp = s_p[wave];

  auto load = [&](int kb, bf16x8* kr, bf16x8* vr) {
    const int64_t row0 = (int64_t)table[kb / B] * B + kb % B;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      kr[t] = *reinterpret_cast<const bf16x8*>(Kb + (row0 + c) * row_bytes + (32 * t + 8 * q) * 2);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vr[i] = *reinterpret_cast<const bf16x8*>(Vb + (row0 + 4 * q + i) * row_bytes + c * 16);
  };
  bf16x8 kf[4], vf[4];
  if (k0 < k1) load(k0, kf, vf);
  for (int kb = k0; kb < k1; kb += DT) {
    bf16x8 kn[4], vn[4];
    if (kb + DT < k1) load(kb + DT, kn, vn);
    f32x4 st = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int t = 0; t < 4; ++t) st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[t], qf[t], st, 0, 0, 0);
    // scores of keys 4q+j for head c; keys past the range are masked and
    // their V rows (which may hold any bits) zeroed
    float sc[4];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool ok = kb + 4 * q + j < k1;
      sc[j] = ok ? st[j] * scale_log2 : -INFINITY;
      if (!ok) vf[j] = bf16x8{};
      mx = fmaxf(mx, sc[j]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    if (__any(mx > m_run + DSLACK)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
      m_run = m_new;
      if (q == 0) s_a[wave][c] = alpha;
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        const float a = s_a[wave][h];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] *= a;
      }
    }
    float pr[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      pr[j] = __builtin_amdgcn_exp2f(sc[j] - m_run);
      l_run += pr[j];
    }
    if (c < GM) *reinterpret_cast<float4*>(sp + c * DT + 4 * q) = make_float4(pr[0], pr[1], pr[2], pr[3]);
    float4 ph[GM];
#pragma unroll
    for (int h = 0; h < GM; ++h) ph[h] = *reinterpret_cast<const float4*>(sp + h * DT + 4 * q);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v[8];
      const uint4 u = __builtin_bit_cast(uint4, vf[i]);
      v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
      v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
      v[4] = __uint_as_float(u.z << 16); v[5] = __uint_as_float(u.z & 0xffff0000u);
      v[6] = __uint_as_float(u.w << 16); v[7] = __uint_as_float(u.w & 0xffff0000u);
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        if (h < g) {
          const float w = i == 0 ? ph[h].x : i == 1 ? ph[h].y : i == 2 ? ph[h].z : ph[h].w;
#pragma unroll
          for (int e = 0; e < 8; ++e) o[h][e] = fmaf(w, v[e], o[h][e]);
        }
      }
    }
    if (kb + DT < k1) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        kf[t] = kn[t];
        vf[t] = vn[t];
      }
    }
  }
  // the four lane groups' sums; lanes of group 0 write head h's dims 8c..8c+7
  // and head c's (m, l)
  float l = l_run + __shfl_xor(l_run, 16, 64);
  l += __shfl_xor(l, 32, 64);
#pragma unroll
  for (int h = 0; h < GM; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      o[h][e] += __shfl_xor(o[h][e], 16, 64);
      o[h][e] += __shfl_xor(o[h][e], 32, 64);
    }
  if (q != 0) return;
  const int stride = 128 + 2;
#pragma unroll
  for (int h = 0; h < GM; ++h) {
    if (h < g) {
      float* dst = p.part + (((int64_t)r * p.nq + kvh * g + h) * S + split) * stride + 8 * c;
      *reinterpret_cast<float4*>(dst) = make_float4(o[h][0], o[h][1], o[h][2], o[h][3]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(o[h][4], o[h][5], o[h][6], o[h][7]);
    }
  }
  if (c < g) {
    float* tail = p.part + (((int64_t)r * p.nq + kvh * g + c) * S + split) * stride + 128;
    tail[0] = m_run;
    tail[1] = l;
  }
}

// Merge the splits of one (request, q head) in split order; round to T.
// The splits' weights exp2(m_s - M) are formed once (thread s) and shared
// through LDS; every output dim then sums its splits in index order.
template <typename T>
__global__ __launch_bounds__(DMAXD) void decode_combine_kernel(DecodeAttnParams p) {
  __shared__ float s_w[DMAXS], s_red[DMAXD];
  const int r = blockIdx.x / p.nq, h = blockIdx.x % p.nq;
  const int e = threadIdx.x, d = p.d, S = p.splits, stride = d + 2;
  const float* base = p.part + ((int64_t)r * p.nq + h) * S * stride;
  // M: maximum of the splits' m (order-free)
  float mloc = -INFINITY;
  for (int s = e; s < S; s += DMAXD) mloc = fmaxf(mloc, base[s * stride + d]);
  s_red[e] = mloc;
  __syncthreads();
  for (int w = DMAXD / 2; w > 0; w >>= 1) {
    if (e < w) s_red[e] = fmaxf(s_red[e], s_red[e + w]);
    __syncthreads();
  }
  const float M = s_red[0];
  for (int s = e; s < S; s += DMAXD) s_w[s] = __builtin_amdgcn_exp2f(base[s * stride + d] - M);
  __syncthreads();
  float L = 0.0f, o = 0.0f;
  int s = 0;
  for (; s + 4 <= S; s += 4) {
    float v[4], l[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      l[u] = base[(s + u) * stride + d + 1];
      v[u] = e < d ? base[(s + u) * stride + e] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      L = fmaf(l[u], s_w[s + u], L);
      o = fmaf(v[u], s_w[s + u], o);
    }
  }
  for (; s < S; ++s) {
    L = fmaf(base[s * stride + d + 1], s_w[s], L);
    if (e < d) o = fmaf(base[s * stride + e], s_w[s], o);
  }
  if (e < d) {
    T* out = reinterpret_cast<T*>(p.out) + (int64_t)r * p.nq * d + (int64_t)h * d;
    Elem<T>::store(out, e, o / L);
  }
}

// Greedy tokens from the transposed logits [vocab][ld], in two passes.
// (value, index) pairs merge by the larger value and, among equal values, the
// lower index, so the result is the lowest index among equal maxima whatever
// the merge order.
__device__ __forceinline__ void argmax_merge(float& best, int& bi, float b, int i) {
  if (i >= 0 && (bi < 0 || b > best || (b == best && i < bi))) {
    best = b;
    bi = i;
  }
}

// Pass 1: workgroup c scans a contiguous chunk of vocabulary rows.  With R <=
// 256 requests, the 256/R threads of request r (t % R == r) take rows t/R,
// t/R + 256/R, ... of the chunk, loading 8 rows before comparing (and, when
// asked, copying the logits out), then merge through LDS; larger batches
// keep one thread per request.  Pass 2 merges the chunks of each request.
__global__ __launch_bounds__(256) void argmax_partial_kernel(const float* logits_t, int64_t ld,
                                                             int vocab, int R, float2* partial,
                                                             float* logits_out) {
  __shared__ float s_best[256];
  __shared__ int s_idx[256];
  const int c = blockIdx.x;
  const int per = (vocab + ARGMAX_CHUNKS - 1) / ARGMAX_CHUNKS;
  const int v0 = c * per, v1 = min(vocab, v0 + per);
  if (R > 256) {
    for (int r = threadIdx.x; r < R; r += 256) {
      float best = -INFINITY;
      int bi = -1;
      for (int v = v0; v < v1; ++v) {
        const float z = logits_t[(int64_t)v * ld + r];
        if (logits_out) logits_out[(int64_t)r * vocab + v] = z;
        argmax_merge(best, bi, z, v);
      }
      partial[(int64_t)c * R + r] = make_float2(best, __int_as_float(bi));
    }
    return;
  }
  const int tpr = 256 / R, t = threadIdx.x, r = t % R, k = t / R;
  float best = -INFINITY;
  int bi = -1;
  if (k < tpr) {
    for (int vb = v0 + k; vb < v1; vb += 8 * tpr) {
      float z[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int v = vb + u * tpr;
        z[u] = v < v1 ? logits_t[(int64_t)v * ld + r] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int v = vb + u * tpr;
        if (v < v1) argmax_merge(best, bi, z[u], v);
      }
      if (logits_out) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int v = vb + u * tpr;
          if (v < v1) logits_out[(int64_t)r * vocab + v] = z[u];
        }
      }
    }
  }
  s_best[t] = best;
  s_idx[t] = bi;
  __syncthreads();
  if (t < R) {
    for (int j = 1; j < tpr; ++j) argmax_merge(best, bi, s_best[j * R + r], s_idx[j * R + r]);
    partial[(int64_t)c * R + r] = make_float2(best, __int_as_float(bi));
  }
}

// Pass 1 over row-major logits [R][ld]: workgroup c scans vocabulary chunk c
// of every request; wave w takes requests w, w+4, ..., its lanes consecutive
// entries (eight per lane in flight), and merges its lanes with shuffles.
__global__ __launch_bounds__(256) void argmax_rows_partial_kernel(const float* logits, int64_t ld,
                                                                  int vocab, int R, float2* partial) {
  const int c = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int per = (vocab + ARGMAX_CHUNKS - 1) / ARGMAX_CHUNKS;
  const int v0 = c * per, v1 = min(vocab, v0 + per);
  for (int r = w; r < R; r += 4) {
    const float* row = logits + (int64_t)r * ld;
    float best = -INFINITY;
    int bi = -1;
    for (int vb = v0 + lane; vb < v1; vb += 8 * 64) {
      float z[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) z[u] = vb + 64 * u < v1 ? row[vb + 64 * u] : 0.0f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (vb + 64 * u < v1) argmax_merge(best, bi, z[u], vb + 64 * u);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      argmax_merge(best, bi, ob, oi);
    }
    if (lane == 0) partial[(int64_t)c * R + r] = make_float2(best, __int_as_float(bi));
  }
}

// Pass 2: one wave per request; lane l merges chunks l, l+64, ..., then the
// wave merges its lanes.
__global__ __launch_bounds__(64) void argmax_final_kernel(const float2* partial, int R,
                                                          int32_t* next_tokens) {
  const int r = blockIdx.x, t = threadIdx.x;
  float best = -INFINITY;
  int bi = -1;
  for (int c = t; c < ARGMAX_CHUNKS; c += 64) {
    const float2 e = partial[(int64_t)c * R + r];
    argmax_merge(best, bi, e.x, __float_as_int(e.y));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    argmax_merge(best, bi, ob, oi);
  }
  if (t == 0) next_tokens[r] = bi < 0 ? 0 : bi;
}

}  // namespace

void launch_rope_rows(float2* table, const int32_t* positions, int rows, int d, double theta,
                      hipStream_t s) {
  const int half = d / 2;
  const int64_t n = (int64_t)rows * half;
  if (n <= 0) return;
  hipLaunchKernelGGL(rope_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, table,
                     positions, rows, half, theta, d);
}

int decode_attn_splits(int num_requests, int nkv, int64_t max_ctx) {
  // enough (request, kv head, key range) items to keep HBM busy (about 2048)
  // and ranges of at most about 2048 keys, so the longest request's waves
  // do not trail the rest (measured: 16 requests x 128K context and 64 x
  // 1.2M both run best at 16 ranges; shorter ranges spend their time on each
  // wave's fixed costs); at least 64 keys and at most 128 ranges per
  // (request, kv head).  Never more for more requests, so a workspace sized
  // for one request's split count fits any larger batch.
  const int64_t pairs = std::max<int64_t>(1, (int64_t)num_requests * nkv);
  const int64_t want = std::max<int64_t>((2048 + pairs - 1) / pairs, (max_ctx + 2047) / 2048);
  const int64_t cap = std::min<int64_t>(DMAXS, (max_ctx + 63) / 64);
  return (int)std::max<int64_t>(1, std::min(want, cap));
}

void launch_decode_attention(int dtype, const DecodeAttnParams& p, int num_requests,
                             hipStream_t s) {
  if (num_requests <= 0) return;
  const dim3 grid((unsigned)((int64_t)num_requests * p.nkv * p.splits));
  const dim3 cgrid((unsigned)((int64_t)num_requests * p.nq));
  const int g = p.nq / p.nkv;
  if (dtype == 1 && p.d == 128 && p.block_size % DT == 0 && g <= 16) {
    const dim3 mgrid((unsigned)((int64_t)num_requests * ((p.nkv + 3) / 4) * p.splits));
    if (g <= 4)
      hipLaunchKernelGGL(decode_attn_mfma_kernel<4>, mgrid, dim3(256), 0, s, p);
    else if (g <= 8)
      hipLaunchKernelGGL(decode_attn_mfma_kernel<8>, mgrid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL(decode_attn_mfma_kernel<16>, mgrid, dim3(256), 0, s, p);
    hipLaunchKernelGGL(decode_combine_kernel<bf16_t>, cgrid, dim3(DMAXD), 0, s, p);
  } else if (dtype == 1) {
    hipLaunchKernelGGL(decode_attn_kernel<bf16_t>, grid, dim3(DNT), 0, s, p);
    hipLaunchKernelGGL(decode_combine_kernel<bf16_t>, cgrid, dim3(DMAXD), 0, s, p);
  } else {
    hipLaunchKernelGGL(decode_attn_kernel<float>, grid, dim3(DNT), 0, s, p);
    hipLaunchKernelGGL(decode_combine_kernel<float>, cgrid, dim3(DMAXD), 0, s, p);
  }
}

void launch_argmax(const float* logits_t, int64_t ld, int vocab, int num_requests,
                   float2* partial, int32_t* next_tokens, float* logits_out, hipStream_t s) {
  if (num_requests <= 0) return;
  hipLaunchKernelGGL(argmax_partial_kernel, dim3(ARGMAX_CHUNKS), dim3(256), 0, s, logits_t, ld,
                     vocab, num_requests, partial, logits_out);
  hipLaunchKernelGGL(argmax_final_kernel, dim3(num_requests), dim3(64), 0, s, partial,
                     num_requests, next_tokens);
}

void launch_argmax_rows(const float* logits, int64_t ld, int vocab, int num_requests,
                        float2* partial, int32_t* next_tokens, hipStream_t s) {
  if (num_requests <= 0) return;
  hipLaunchKernelGGL(argmax_rows_partial_kernel, dim3(ARGMAX_CHUNKS), dim3(256), 0, s, logits, ld,
                     vocab, num_requests, partial);
  hipLaunchKernelGGL(argmax_final_kernel, dim3(num_requests), dim3(64), 0, s, partial,
                     num_requests, next_tokens);
}

}  // namespace kvr
