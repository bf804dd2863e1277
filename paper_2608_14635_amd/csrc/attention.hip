// Variable-length causal grouped-query attention of the rebuild.
//
// bf16 path (head_dim 128): a workgroup is 8 wave64s = HW q heads of one GQA
// group x QW blocks of 32 queries of one request (HW * QW = 8), so every K/V
// tile staged in LDS feeds 8 waves.  Key tiles of 64 keys stream into a
// 3-stage LDS ring with buffer_load_dwordx4 ... lds (two tiles in flight): K
// rows from a contiguous per-head copy of the stored K, V from the V^T copy
// (one contiguous 16 KB block per key tile), both written by the QKV epilogue
// with the values sent to the arena.  Scores are computed transposed,
// S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: a lane owns one query column
// and 32 of the tile's keys in registers, so the online softmax statistics are
// per-lane scalars completed by one exchange with the lane holding the
// column's other 32 keys (v_permlane32_swap), and P^T feeds O^T = V^T P^T
// straight from registers as the B operand.  K rows are placed in LDS with
// bits 2 and 3 of their index swapped, which makes the 8 keys of each P^T
// operand slot group contiguous in V^T, so every V^T operand is one 16-byte
// LDS read.  exp2 with the scale folded in; P rounded to bf16 for the MFMA,
// and the softmax denominator summed from the same rounded values (bf16 dot2
// with fp32 accumulation); fp32 accumulation; masking only on tiles that
// cross a wave's diagonal; the exponents are taken against an integer anchor
// (log2 units), raised and O rescaled by a power of two only when some lane's
// max rose by a factor above 2^8 since the last rescale.  q-blocks are
// scheduled longest-first.  Deterministic: fixed key order, no atomics.
//
// fp32 path: a plain online-softmax kernel (one wave per query, lanes across
// head dims) for fp32 models.
#include "common.h"
#include "launch.h"

namespace kvr {

namespace {

constexpr int D = 128;
constexpr int KB = 64;                       // keys per tile
constexpr int NW = 8, NT = 64 * NW;          // 8 waves per workgroup
constexpr int KTILE = KB * D * 2;            // 16 KB: 64 K rows of 256 B
constexpr int VTILE = D * KB * 2;            // 16 KB: 128 V^T rows of 128 B
constexpr int STAGE = KTILE + VTILE;
constexpr int NSTAGE = 3;
constexpr float RESCALE_SLACK = 8.0f;        // see the online softmax below
static_assert(KB == VT_KEYS, "a key tile is one tile of the V^T copy");
constexpr int READ_AHEAD = 4;                // LDS fragment reads in flight ahead of the MFMAs

typedef __attribute__((address_space(3))) void lds_void;

// LDS row r of a K tile holds key ksig(r): bits 2 and 3 swapped (an involution)
__device__ __forceinline__ int ksig(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }
// K row r: 16-byte unit u at slot u ^ (r & 15); V^T row d: unit u at slot u ^ vsw(d).
// Both make the MFMA operand reads (32 consecutive rows, one unit) conflict-free
// for 8- or 16-lane LDS read phases.
__device__ __forceinline__ int vsw(int d) { return (d & 7) ^ ((d >> 3) & 1); }

// v_permlane32_swap of a register with itself: one result holds the lower
// half's values in both halves, the other the upper half's, so a symmetric
// combination of the two is the lane's value combined with lane (lane ^ 32)'s
__device__ __forceinline__ float max_with_other_half(float x) {
  const unsigned u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_with_other_half(float x) {
  const unsigned u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

#define KVR_WAIT_VMCNT(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (((n) >> 4) << 14) | (0x7 << 4) | (0xF << 8))

constexpr int BUF_WORD3 = 0x00020000;  // gfx9 buffer descriptor: 32-bit data format

// Issue this wave's share (2 K blocks + 2 V^T blocks of 1 KB) of key tile
// starting at row kbase into ring stage `stage`.  Buffer loads with the LDS
// bit are counted by vmcnt only, so the fragment reads from LDS keep exact
// lgkm counts (global_load_lds would force lgkmcnt(0) before every MFMA).
// k_voff / v_voff: this lane's byte offsets within the head's K copy at key
// 0 / within a V^T key tile; the tile's offset is scalar.
__device__ __forceinline__ void issue_kv(char* smem, const bf16_t* Kc, const bf16_t* Vt,
                                         int head_bytes, int kbase, int stage, int wid,
                                         const int* k_voff, const int* v_voff) {
  char* st = smem + stage * STAGE;
  const auto rk = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(Kc), 0, head_bytes, BUF_WORD3);
  const auto rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(Vt), 0, head_bytes, BUF_WORD3);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int qk = wid + 8 * i;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(st + qk * 1024), 16, k_voff[i],
                                             kbase * D * 2, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(st + KTILE + qk * 1024), 16, v_voff[i],
                                             kbase * D * 2, 0, 0);  // key tile kbase / 64: 16 KB
  }
}

template <int HW>
__global__ __launch_bounds__(NT, 1) void attn_bf16_kernel(AttnParams p) {
  constexpr int QW = NW / HW;
  __shared__ __attribute__((aligned(1024))) char smem[NSTAGE * STAGE];

  const int g = p.nq / p.nkv, ngrp = g / HW;
  int bid = blockIdx.x;
  const int qb = bid / (p.nkv * ngrp);
  bid -= qb * p.nkv * ngrp;
  const int kvh = bid / ngrp, hgrp = bid % ngrp;
  const int4 blk = p.qblk[qb];
  const int q_start = blk.x, q_len = blk.y, key_base = blk.z, pos0 = blk.w;
  const int nkeys = pos0 + q_len;
  const int ntiles = (nkeys + KB - 1) / KB;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int qsub = wid / HW, h = kvh * g + hgrp * HW + wid % HW;
  const int half = lane >> 5, col = lane & 31;
  const bool wave_active = qsub * 32 < q_len;
  const int qi = min(qsub * 32 + col, q_len - 1);            // clamped query of this lane
  const int qpos = pos0 + qi;                                // its position in the request
  const int wave_first = pos0 + qsub * 32;
  const int wave_last = pos0 + min(qsub * 32 + 31, q_len - 1);

  const int ldq = p.nq * D;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(p.q);
  const bf16_t* Kc = reinterpret_cast<const bf16_t*>(p.kc) + (int64_t)kvh * p.ldvt * D;
  const bf16_t* Vt = reinterpret_cast<const bf16_t*>(p.vt) + (int64_t)kvh * D * p.ldvt;

  // Q^T fragments (B operand of S^T = K Q^T): lane holds 8 dims of its query per k-step
  bf16x8 qf[D / 16];
  {
    const bf16_t* qrow = Q + (int64_t)(q_start + qi) * ldq + h * D + half * 8;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qrow + ks * 16);
  }

  // direct-to-LDS loaders: wave w issues K instructions w, w+8 (4 rows each) and
  // V^T instructions w, w+8 (8 rows each)
  const int head_bytes = (int)(p.ldvt * D * 2);  // one head's K copy, and its V^T rows
  int k_voff[2], v_voff[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int qk = wid + 8 * i;
    const int lr = 4 * qk + (lane >> 4);                  // LDS row
    // key ksig(lr) lands there; unit (lane&15)^(lr&15) of it fills this lane's slot
    k_voff[i] = (ksig(lr) * D + ((lane & 15) ^ (lr & 15)) * 8) * 2;
    const int dv = 8 * qk + (lane >> 3);
    v_voff[i] = (dv * VT_KEYS + ((lane & 7) ^ vsw(dv)) * 8) * 2;  // within the key tile
  }

  f32x16 acc_o[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc_o[t][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)D);

  // fragment addressing
  const int kslot0 = (col & 15);   // LDS row 32*k2 + col has row&15 == col&15
  int vbase[D / 32], vsw_l[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t) {
    const int d = t * 32 + col;
    vbase[t] = KTILE + d * 128;
    vsw_l[t] = vsw(d);
  }
  // key offset (within a 32-key half) of accumulator register r: ksig(8*(r/4) + 4*half + r%4)

  issue_kv(smem, Kc, Vt, head_bytes, key_base, 0, wid, k_voff, v_voff);
  issue_kv(smem, Kc, Vt, head_bytes, key_base + min(1, ntiles - 1) * KB, 1, wid, k_voff, v_voff);
  for (int kt = 0; kt < ntiles; ++kt) {
    KVR_WAIT_VMCNT(4);                      // this wave's loads of tile kt have landed
    __builtin_amdgcn_s_barrier();           // ... and every other wave's; stage of kt-1 is free
    issue_kv(smem, Kc, Vt, head_bytes, key_base + min(kt + 2, ntiles - 1) * KB, (kt + 2) % NSTAGE,
             wid, k_voff, v_voff);
    const char* st = smem + (kt % NSTAGE) * STAGE;

    if (wave_active && kt * KB <= wave_last) {
      // ---- S^T for keys [0,32) and [32,64) of the tile (the two accumulation
      // chains alternate, so no MFMA waits on the one just issued) ----
      f32x16 s[2];
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[k2][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2) {
          const char* krow = st + (k2 * 32 + col) * 256;
          const bf16x8 kf =
              *reinterpret_cast<const bf16x8*>(krow + (((2 * ks + half) ^ kslot0) << 4));
          s[k2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[k2], 0, 0, 0);
        }
      // K fragment reads run READ_AHEAD ahead of the MFMAs that consume them
#pragma unroll
      for (int q = 0; q < READ_AHEAD; ++q) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
      for (int q = 0; q < 16 - READ_AHEAD; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, READ_AHEAD, 0);
      // ---- mask on diagonal tiles, online softmax ----
      // The running max m_run lives in the log2 domain (scores times
      // log2(e)/sqrt(d)); the scale is folded into the FMA that forms each
      // exponent, and exp2 is the bare v_exp_f32 (results below 2^-126 flush
      // to zero, far below bf16 resolution of P next to the row max's 1.0).
      // The softmax is VALU work that competes with the matrix core for issue,
      // so it is kept to one FMA, one exp, one add and half a convert per score.
      if (__builtin_expect(kt * KB + KB - 1 > wave_first, 0)) {
        // register r of half h holds tile key 32*k2 + ksig(8*(r/4) + 4h + r%4)
        // = 32*k2 + 8h + kc(r): compare kc(r) with the lane's limit
        const int lim = qpos - kt * KB - 8 * half;
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int kc = 32 * k2 + 16 * ((r >> 3) & 1) + 4 * ((r >> 2) & 1) + (r & 3);
            if (kc > lim) s[k2][r] = -INFINITY;
          }
      }
      // the lane's max as four independent chains (short dependency depth),
      // then the other half of its query column's keys via a lane swap
      // (IEEE maximum: v_maximum3_f32, with no quieting of the MFMA results)
      float mq[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        mq[j] = s[0][j];
#pragma unroll
        for (int i = 1; i < 8; ++i) mq[j] = __builtin_elementwise_maximum(mq[j], s[i >> 2][4 * (i & 3) + j]);
      }
      float mx = __builtin_elementwise_maximum(__builtin_elementwise_maximum(mq[0], mq[1]),
                                               __builtin_elementwise_maximum(mq[2], mq[3]));
      mx = max_with_other_half(mx) * scale_log2;
      // The reference max used for the exponents may lag the true running
      // max by up to RESCALE_SLACK (log2 units): P then reaches at most
      // 2^RESCALE_SLACK, which the fp32 sums and the final division by l
      // absorb exactly, while the 64-register rescale of O runs on few tiles.
      // The reference is an integer (the max rounded up), so every rescale
      // factor is an exact power of two and each key's rounded weight equals
      // bf16(2^(s - c)) for the row's final anchor c, whichever tile raised
      // it: rounding to bf16 commutes with scaling by a power of two.
      if (__any(mx > m_run + RESCALE_SLACK)) {
        const float m_new = ceilf(fmaxf(m_run, mx));
        const float alpha = m_run == -INFINITY ? 0.0f : ldexpf(1.0f, (int)(m_run - m_new));
        l_run *= alpha;
#pragma unroll
        for (int t = 0; t < D / 32; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc_o[t][r] *= alpha;
        m_run = m_new;
      }
      const float neg_m = -m_run;
      bf16x8 pf[4];
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          pf[k2 * 2 + (r >> 3)][r & 7] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[k2][r], scale_log2, neg_m));
      // row sums of the rounded P (exactly the weights the PV MFMA applies),
      // two values per instruction
      float lsum0 = 0.0f, lsum1 = 0.0f;
      const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        lsum0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf[c], pf[c], 0, 1), one2, lsum0, false);
        lsum1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf[c], pf[c], 2, 3), one2, lsum1, false);
        lsum0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf[c], pf[c], 4, 5), one2, lsum0, false);
        lsum1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf[c], pf[c], 6, 7), one2, lsum1, false);
      }
      l_run += lsum0 + lsum1;
      // ---- O^T += V^T P^T; P^T slot j of chunk c is key 16c + 8*half + j (the
      // four d-tiles' chains alternate) ----
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int t = 0; t < D / 32; ++t) {
          const bf16x8 vf = *reinterpret_cast<const bf16x8*>(st + vbase[t] +
                                                              (((2 * c + half) ^ vsw_l[t]) << 4));
          acc_o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[c], acc_o[t], 0, 0, 0);
        }
      // V^T fragment reads run READ_AHEAD ahead of their MFMAs
#pragma unroll
      for (int q = 0; q < READ_AHEAD; ++q) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
      for (int q = 0; q < 16 - READ_AHEAD; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, READ_AHEAD, 0);
    }
  }
  KVR_WAIT_VMCNT(0);  // trailing refetches complete before the workgroup retires

  if (!wave_active) return;
  const float l_tot = sum_with_other_half(l_run);
  const float inv = 1.0f / l_tot;
  const int q_local = qsub * 32 + col;
  if (q_local >= q_len) return;
  bf16_t* orow = reinterpret_cast<bf16_t*>(p.out) + (int64_t)(q_start + q_local) * ldq + h * D;
  // O^T register r of d-tile t: dim 32t + 8*(r/4) + 4*half + r%4
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int dim = t * 32 + 8 * gq + 4 * half;
      uint2 u;
      u.x = (uint32_t)f2bf(acc_o[t][4 * gq + 0] * inv) | ((uint32_t)f2bf(acc_o[t][4 * gq + 1] * inv) << 16);
      u.y = (uint32_t)f2bf(acc_o[t][4 * gq + 2] * inv) | ((uint32_t)f2bf(acc_o[t][4 * gq + 3] * inv) << 16);
      *reinterpret_cast<uint2*>(orow + dim) = u;
    }
}

// fp32: one wave per query of the q-block (strided over the 4 waves), lanes
// across head dims; plain online softmax over the visible keys.
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnParams p) {
  const int qb = blockIdx.x / p.nq, h = blockIdx.x % p.nq;
  const int kvh = h / (p.nq / p.nkv);
  const int4 blk = p.qblk[qb];
  const int q_start = blk.x, q_len = blk.y, key_base = blk.z, pos0 = blk.w;
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
    for (int j = 0; j <= pos0 + qi; ++j) {
      const int64_t row = (p.kslot[key_base + j] * p.nkv + kvh) * (int64_t)d;
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

// Prefix keys of a rebuild from a retained prefix, for the bf16 kernel above:
// workgroup (segment, kv head) copies up to 64 keys' K rows from the arena
// into the K copy and their V rows, through LDS, into V^T (8 consecutive
// keys of one dim per 16-byte store; segments start on a multiple of 8 key
// rows).  A segment with a negative count instead writes zeros to -count key
// rows (a multiple of 8): the rows between a request's last computed row and
// the end of its 64-aligned key region, which the last key tile reads and
// which must be finite since masked probabilities multiply them.
__global__ __launch_bounds__(256) void prefix_gather_kernel(const int2* segs, const int64_t* kslot,
                                                            const bf16_t* plane_k,
                                                            const bf16_t* plane_v, bf16_t* kc,
                                                            bf16_t* vt, int64_t ldvt, int nkv) {
  constexpr int GP = D + 8;  // LDS pitch, elements
  __shared__ __attribute__((aligned(16))) uint16_t sv[GATHER_KEYS * GP];
  const int seg = blockIdx.x / nkv, h = blockIdx.x % nkv;
  const int2 sg = segs[seg];
  const int kr0 = sg.x, cnt = sg.y;
  const int tid = threadIdx.x;
  if (cnt < 0) {  // uniform over the workgroup
    const int z = -cnt;
    const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
    for (int it = tid; it < z * (D / 8); it += 256)
      *reinterpret_cast<uint4*>(kc + ((int64_t)h * ldvt + kr0 + it / (D / 8)) * D + (it % (D / 8)) * 8) = zero;
    for (int it = tid; it < D * (z / 8); it += 256)
      *reinterpret_cast<uint4*>(vt + vt_offset(h * D + it % D, kr0 + (it / D) * 8, ldvt, D)) = zero;
    return;
  }
  const int64_t row_elems = (int64_t)nkv * D;
  for (int it = tid; it < cnt * (D / 8); it += 256) {
    const int k = it / (D / 8), u = it % (D / 8);
    const int64_t src = kslot[kr0 + k] * row_elems + (int64_t)h * D + u * 8;
    *reinterpret_cast<uint4*>(kc + ((int64_t)h * ldvt + kr0 + k) * D + u * 8) =
        *reinterpret_cast<const uint4*>(plane_k + src);
    *reinterpret_cast<uint4*>(sv + k * GP + u * 8) = *reinterpret_cast<const uint4*>(plane_v + src);
  }
  __syncthreads();
  for (int it = tid; it < D * (cnt / 8); it += 256) {
    const int e = it % D, k8 = (it / D) * 8;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)sv[(k8 + 2 * i) * GP + e] | ((uint32_t)sv[(k8 + 2 * i + 1) * GP + e] << 16);
    *reinterpret_cast<uint4*>(vt + vt_offset(h * D + e, kr0 + k8, ldvt, D)) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

}  // namespace

void launch_prefix_gather(const int2* segs, int nseg, const int64_t* kslot, const void* plane_k,
                          const void* plane_v, void* kc, void* vt, int64_t ldvt, int nkv, int d,
                          hipStream_t s) {
  if (nseg <= 0 || d != D) return;
  hipLaunchKernelGGL(prefix_gather_kernel, dim3((unsigned)(nseg * nkv)), dim3(256), 0, s, segs, kslot,
                     reinterpret_cast<const bf16_t*>(plane_k), reinterpret_cast<const bf16_t*>(plane_v),
                     reinterpret_cast<bf16_t*>(kc), reinterpret_cast<bf16_t*>(vt), ldvt, nkv);
}

void launch_attention_bf16(const AttnParams& p, hipStream_t s) {
  if (p.num_qblk <= 0) return;
  const int g = p.nq / p.nkv, hw = attn_heads_per_wg(g);
  const dim3 grid(p.num_qblk * p.nkv * (g / hw)), block(NT);
  switch (hw) {
    case 8: hipLaunchKernelGGL((attn_bf16_kernel<8>), grid, block, 0, s, p); break;
    case 4: hipLaunchKernelGGL((attn_bf16_kernel<4>), grid, block, 0, s, p); break;
    case 2: hipLaunchKernelGGL((attn_bf16_kernel<2>), grid, block, 0, s, p); break;
    default: hipLaunchKernelGGL((attn_bf16_kernel<1>), grid, block, 0, s, p); break;
  }
}

void launch_attention_f32(const AttnParams& p, int, hipStream_t s) {
  if (p.num_qblk <= 0) return;
  hipLaunchKernelGGL(attn_f32_kernel, dim3(p.num_qblk * p.nq), dim3(256), 0, s, p);
}

}  // namespace kvr
