// Variable-length causal grouped-query attention of the rebuild.
//
// bf16 path (head_dim 128): one workgroup per (q-block of up to 128 queries of
// one request, q head); 4 wave64s each own 32 queries.  Key tiles of 64 keys
// are staged in LDS: K rows gathered from the arena slots through the slot
// table (the values the decode path would read), V from the V^T copy the QKV
// epilogue wrote.  Scores are computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16: a lane then owns one query column and 32 of the 64
// keys of the tile in registers, so the running max / sum of the online
// softmax are per-lane scalars completed by one cross-half exchange, and the
// probabilities P^T feed the P.V product (O^T = V^T P^T) directly from
// registers as the B operand, without a round trip through LDS.  exp2 with
// the scale folded in; P is rounded to bf16 for the MFMA; fp32 accumulation.
// q-blocks are scheduled longest-first; tiles entirely above a wave's
// diagonal are skipped.  Deterministic: fixed key order, no atomics.
//
// fp32 path: a plain online-softmax kernel (one wave per query, lanes across
// head dims) for fp32 models.
#include "common.h"
#include "launch.h"

namespace kvr {

namespace {

constexpr int QB = ATTN_QBLOCK;   // 128 queries per workgroup
constexpr int KB = 64;            // keys per tile
constexpr int D = 128;
constexpr int LDKS = D + 8;       // sK row, elements (272 B)
constexpr int LDVT = KB + 8;      // sVt row, elements (144 B)
constexpr int NT = 256;

__global__ __launch_bounds__(NT, 2) void attn_bf16_kernel(AttnParams p) {
  __shared__ __attribute__((aligned(16))) bf16_t sK[KB * LDKS];
  __shared__ __attribute__((aligned(16))) bf16_t sVt[D * LDVT];

  const int qb = blockIdx.x / p.nq, h = blockIdx.x % p.nq;
  const int kvh = h / (p.nq / p.nkv);
  const int4 blk = p.qblk[qb];
  const int q_start = blk.x, q_len = blk.y, req_start = blk.z;
  const int key_end = q_start + q_len;          // exclusive, wave-local token index
  const int nkeys = key_end - req_start;
  const int ntiles = (nkeys + KB - 1) / KB;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const bool wave_active = wid * 32 < q_len;
  const int qi = min(wid * 32 + col, q_len - 1);          // clamped query of this lane
  const int qpos = q_start + qi - req_start;              // its position in the request
  const int wave_last = min(wid * 32 + 31, q_len - 1);
  const int wave_max_pos = q_start + wave_last - req_start;

  const int ldq = p.nq * D;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(p.q);
  const bf16_t* Kp = reinterpret_cast<const bf16_t*>(p.arena_k);
  const bf16_t* Vt = reinterpret_cast<const bf16_t*>(p.vt);

  // Q^T fragments (B operand of S^T = K Q^T): lane holds 8 dims of its query per k-step
  bf16x8 qf[D / 16];
  {
    const bf16_t* qrow = Q + (int64_t)(q_start + qi) * ldq + h * D + half * 8;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16);
  }

  f32x16 acc_o[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc_o[t][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)D);

  // staging of the next tile: K 4 chunks, V^T 4 chunks of 16 B per thread
  uint4 rk[4], rv[4];
  auto fetch = [&](int kt) {
    const int kbase = req_start + kt * KB;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + NT * i;
      const int key = c >> 4, dch = c & 15;
      const int tok = kbase + key;
      if (tok < key_end) {
        const int64_t slot = p.slot[tok];
        rk[i] = *reinterpret_cast<const uint4*>(Kp + (slot * p.nkv + kvh) * D + dch * 8);
      } else {
        rk[i] = make_uint4(0, 0, 0, 0);
      }
      const int dd = c >> 3, kc = c & 7;
      const int t0 = kbase + kc * 8;
      const bf16_t* src = Vt + (int64_t)(kvh * D + dd) * p.ldvt + t0;
      if (t0 + 8 <= key_end) {
        rv[i] = *reinterpret_cast<const uint4*>(src);
      } else {
        uint16_t e[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) e[j] = (t0 + j < key_end) ? src[j] : (uint16_t)0;
        rv[i] = make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                           e[6] | (e[7] << 16));
      }
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + NT * i;
      *reinterpret_cast<uint4*>(sK + (c >> 4) * LDKS + (c & 15) * 8) = rk[i];
      *reinterpret_cast<uint4*>(sVt + (c >> 3) * LDVT + (c & 7) * 8) = rv[i];
    }
  };

  fetch(0);
  for (int kt = 0; kt < ntiles; ++kt) {
    __syncthreads();  // previous tile fully consumed
    stash();
    __syncthreads();
    if (kt + 1 < ntiles) fetch(kt + 1);

    if (wave_active && kt * KB <= wave_max_pos) {
      // ---- S^T for keys [0,32) and [32,64) of the tile ----
      f32x16 s[2];
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[k2][r] = 0.0f;
        const bf16_t* krow = sK + (k2 * 32 + col) * LDKS + half * 8;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(krow + ks * 16);
          s[k2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[k2], 0, 0, 0);
        }
      }
      // ---- mask, scale, online softmax (register r: key 8*(r/4) + 4*half + r%4) ----
      float mx = m_run;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kpos = kt * KB + k2 * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          const float v = kpos <= qpos ? s[k2][r] * scale_log2 : -INFINITY;
          s[k2][r] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float alpha = exp2f(m_run - mx);
      m_run = mx;
      float lsum = 0.0f;
      bf16x8 pf[4];
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = exp2f(s[k2][r] - mx);
          lsum += e;
          pf[k2 * 2 + (r >> 3)][r & 7] = (__bf16)e;
        }
      l_run = l_run * alpha + lsum;
#pragma unroll
      for (int t = 0; t < D / 32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc_o[t][r] *= alpha;
      // ---- O^T += V^T P^T; P^T slot j of chunk c is key 16c + 8*(j/4) + 4*half + j%4 ----
#pragma unroll
      for (int t = 0; t < D / 32; ++t) {
        const bf16_t* vrow = sVt + (t * 32 + col) * LDVT + 4 * half;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow + 16 * c);
          const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 16 * c + 8);
          const bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          acc_o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[c], acc_o[t], 0, 0, 0);
        }
      }
    }
  }

  if (!wave_active) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  const int q_local = wid * 32 + col;
  if (q_local >= q_len) return;
  bf16_t* orow = reinterpret_cast<bf16_t*>(p.out) + (int64_t)(q_start + q_local) * ldq + h * D;
  // O^T register r of d-tile t: dim 32t + 8*(r/4) + 4*half + r%4
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int dim = t * 32 + 8 * g + 4 * half;
      uint2 u;
      u.x = (uint32_t)f2bf(acc_o[t][4 * g + 0] * inv) | ((uint32_t)f2bf(acc_o[t][4 * g + 1] * inv) << 16);
      u.y = (uint32_t)f2bf(acc_o[t][4 * g + 2] * inv) | ((uint32_t)f2bf(acc_o[t][4 * g + 3] * inv) << 16);
      *reinterpret_cast<uint2*>(orow + dim) = u;
    }
}

// fp32: one wave per query of the q-block (strided over the 4 waves), lanes
// across head dims; plain online softmax over the visible keys.
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnParams p) {
  const int qb = blockIdx.x / p.nq, h = blockIdx.x % p.nq;
  const int kvh = h / (p.nq / p.nkv);
  const int4 blk = p.qblk[qb];
  const int q_start = blk.x, q_len = blk.y, req_start = blk.z;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int d = p.d;
  const float scale = 1.0f / sqrtf((float)d);
  const float* Q = reinterpret_cast<const float*>(p.q);
  const float* Kp = reinterpret_cast<const float*>(p.arena_k);
  const float* Vp = reinterpret_cast<const float*>(p.arena_v);
  const int ldq = p.nq * d;
  for (int qi = wid; qi < q_len; qi += 4) {
    const int tq = q_start + qi;
    float q[2], o[2] = {0.0f, 0.0f};
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int e = lane + 64 * t;
      q[t] = e < d ? Q[(int64_t)tq * ldq + h * d + e] : 0.0f;
    }
    float m = -INFINITY, l = 0.0f;
    for (int tk = req_start; tk <= tq; ++tk) {
      const int64_t row = (p.slot[tk] * p.nkv + kvh) * (int64_t)d;
      float part = 0.0f;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int e = lane + 64 * t;
        if (e < d) part += q[t] * Kp[row + e];
      }
      const float s = wave_sum(part) * scale;
      const float mn = fmaxf(m, s);
      const float a = __expf(m - mn), w = __expf(s - mn);
      l = l * a + w;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int e = lane + 64 * t;
        o[t] = o[t] * a + (e < d ? w * Vp[row + e] : 0.0f);
      }
      m = mn;
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int e = lane + 64 * t;
      if (e < d) reinterpret_cast<float*>(p.out)[(int64_t)tq * ldq + h * d + e] = o[t] / l;
    }
  }
}

}  // namespace

void launch_attention_bf16(const AttnParams& p, hipStream_t s) {
  if (p.num_qblk <= 0) return;
  hipLaunchKernelGGL(attn_bf16_kernel, dim3(p.num_qblk * p.nq), dim3(NT), 0, s, p);
}

void launch_attention_f32(const AttnParams& p, int, hipStream_t s) {
  if (p.num_qblk <= 0) return;
  hipLaunchKernelGGL(attn_f32_kernel, dim3(p.num_qblk * p.nq), dim3(256), 0, s, p);
}

}  // namespace kvr
