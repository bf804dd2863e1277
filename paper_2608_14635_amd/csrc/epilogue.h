// Fused GEMM epilogues, shared by the bf16 MFMA GEMM and the fp32 GEMM.
//
// A tile's fp32 accumulators are first parked in LDS as sC[rows][ldc]; the
// routines below then read it in row-contiguous chunks so that every global
// store is a full 16-byte (bf16) or 32-byte (fp32) vector:
//   QKV    : NeoX RoPE on the q and k heads of the tile (pairs (i, i+d/2),
//            fp32 cos/sin from the per-position table), rounding to the model
//            dtype, Q rows to the workspace, K and V rows scattered to their
//            arena slots, and V^T columns for the attention kernel;
//   RESID  : X += acc on the fp32 residual stream;
//   STORE  : X = acc (the transposed logits of the decode step's LM head);
//   SWIGLU : h = silu(gate) * up from the two column halves of the tile (the
//            split-K path; the one-pass bf16 GEMM forms h from its accumulators).
#pragma once
#include "common.h"
#include "launch.h"

namespace kvr {

// Full-tile fast paths of the QKV epilogue for head dim 128 (every row of
// the tile below M).  Loads and stores share
// one wait counter on this GPU: once a store is pending, waiting for a load
// means waiting for everything, so each batch of rows loads all it needs
// (positions, slots, key rows, then the RoPE rows), forms every result and
// only then stores.  A thread keeps one (head, chunk of 8 rotary pairs).
template <typename T, int BN, int NT, int REGION>
__device__ __forceinline__ void epi_qkv_rot_full(const float* sC, int ldc, int rows, int m_base, int n0,
                                                 const EpiParams& e) {
  constexpr int D = 128, HALF = 64, CH = HALF / 8, PER_ROW = (BN / D) * CH, RSTEP = NT / PER_ROW, RB = 4;
  const int tid = threadIdx.x;
  const int hc = tid % PER_ROW, hh = hc / CH, c0 = (hc % CH) * 8;
  const int qcols = e.nq * D;
  const int kh = REGION == 1 ? (n0 - qcols) / D + hh : 0;
  // bias and per-head norm gain of this thread's columns (fixed per thread);
  // the norm's inverse RMS per (row, head) sits in column BN + hh
  const T* bias = reinterpret_cast<const T*>(REGION == 0 ? e.bq : e.bk);
  const T* gain = reinterpret_cast<const T*>(REGION == 0 ? e.q_norm : e.k_norm);
  const int hb = (REGION == 0 ? n0 : n0 - qcols) + hh * D;
  float ba[8], bb[8], ga[8], gb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) ba[i] = bb[i] = 0.0f, ga[i] = gb[i] = 1.0f;
  if (bias != nullptr) {
    ld8(bias + hb + c0, ba);
    ld8(bias + hb + c0 + HALF, bb);
  }
  if (gain != nullptr) {
    ld8(gain + c0, ga);
    ld8(gain + c0 + HALF, gb);
  }
  // a missing key-row map reads the positions instead (valid memory) and
  // the value is replaced by the row
  const bool has_krow = e.krow != nullptr;
  const int32_t* krow = has_krow ? e.krow : e.pos;
  for (int rb = tid / PER_ROW; rb < rows; rb += RSTEP * RB) {
    int pos[RB];
    int64_t sl[RB], kr[RB];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const int m = m_base + rb + b * RSTEP;
      pos[b] = e.pos[m];
      if (REGION == 1) {
        sl[b] = e.slot[m];
        const int k = krow[m];
        kr[b] = has_krow ? k : m;
      }
    }
    float2 cs[RB][8];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const float4* src = reinterpret_cast<const float4*>(e.rope + (int64_t)pos[b] * HALF + c0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 v = src[i];
        cs[b][2 * i] = make_float2(v.x, v.y);
        cs[b][2 * i + 1] = make_float2(v.z, v.w);
      }
    }
    float lo[RB][8], hi[RB][8];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const float* src = sC + (int64_t)(rb + b * RSTEP) * ldc + hh * D;
      const float inv = gain != nullptr ? sC[(int64_t)(rb + b * RSTEP) * ldc + BN + hh] : 1.0f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float a = src[c0 + i], bv = src[c0 + HALF + i];
        if (bias != nullptr) {
          a += ba[i];
          bv += bb[i];
        }
        if (gain != nullptr) {
          a = a * inv * ga[i];
          bv = bv * inv * gb[i];
        }
        const float2 t = cs[b][i];
        lo[b][i] = Elem<T>::round(a * t.x - bv * t.y);
        hi[b][i] = Elem<T>::round(bv * t.x + a * t.y);
        // padding rows: zeros in the K copy (keys past a request's end are
        // inert), nothing in the arena
        if (REGION == 1 && sl[b] < 0) lo[b][i] = hi[b][i] = 0.0f;
        asm volatile("" : "+v"(lo[b][i]), "+v"(hi[b][i]));
      }
    }
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const int64_t m = m_base + rb + b * RSTEP;
      if (REGION == 0) {
        T* dst = reinterpret_cast<T*>(e.q_out) + m * qcols + n0 + hh * D;
        store8(dst + c0, lo[b]);
        store8(dst + c0 + HALF, hi[b]);
      } else {
        if (e.kc != nullptr) {
          T* kd = reinterpret_cast<T*>(e.kc) + ((int64_t)kh * e.ldvt + kr[b]) * D;
          store8(kd + c0, lo[b]);
          store8(kd + c0 + HALF, hi[b]);
        }
        if (sl[b] >= 0) {
          T* dst = reinterpret_cast<T*>(e.arena_k) + (sl[b] * e.nkv + kh) * (int64_t)D;
          store8(dst + c0, lo[b]);
          store8(dst + c0 + HALF, hi[b]);
        }
      }
    }
  }
}

// V columns of a full tile without bias: arena rows (slots loaded a batch at
// a time before the stores), each row's padding flag and key row parked in
// the tile's spare columns BN, BN+1, then the V^T columns from LDS only.
template <typename T, int BN, int NT>
__device__ __forceinline__ void epi_qkv_v_full(float* sC, int ldc, int rows, int m_base, int n0,
                                               const EpiParams& e) {
  constexpr int PER_ROW = BN / 8, RSTEP = NT / PER_ROW, RB = 8;
  const int tid = threadIdx.x;
  const int c0 = (tid % PER_ROW) * 8;
  const int kcols = e.nkv * e.d, vbase = n0 - e.nq * e.d - kcols;
  const bool has_krow = e.krow != nullptr;
  const int32_t* krow = has_krow ? e.krow : e.pos;
  for (int rb = tid / PER_ROW; rb < rows; rb += RSTEP * RB) {
    int64_t sl[RB];
    int kr[RB];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const int m = m_base + rb + b * RSTEP;
      sl[b] = e.slot[m];
      const int k = krow[m];
      kr[b] = has_krow ? k : m;
      asm volatile("" : "+v"(sl[b]), "+v"(kr[b]));
    }
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const int r = rb + b * RSTEP;
      float* row = sC + (int64_t)r * ldc;
      if (c0 == 0) {
        row[BN] = sl[b] < 0 ? 1.0f : 0.0f;
        row[BN + 1] = __int_as_float(kr[b]);
      }
      if (sl[b] < 0) continue;  // padding row
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = row[c0 + i];
      store8(reinterpret_cast<T*>(e.arena_v) + sl[b] * (int64_t)kcols + vbase + c0, v);
    }
  }
  if (e.vt == nullptr) return;
  __syncthreads();
  // V^T (col, krow(m)): 8 consecutive rows of one column per item (their key
  // rows are consecutive and inside one key tile: a request's rows start on a
  // multiple of 8, and so do its suffix key rows); padding rows get zeros
  for (int it = tid; it < BN * (rows / 8); it += NT) {
    const int c = it % BN, rc = it / BN;
    const float* src = sC + (int64_t)(rc * 8) * ldc;
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = src[(int64_t)i * ldc + BN] != 0.0f ? 0.0f : src[(int64_t)i * ldc + c];
    const int64_t kr0 = __float_as_int(src[BN + 1]);
    store8(reinterpret_cast<T*>(e.vt) + vt_offset(vbase + c, kr0, e.ldvt, e.d), v);
  }
}

// QKV: the tile covers logical columns [n0, n0+BN) lying in one region
// (q: [0, nq*d), k: [nq*d, nq*d + nkv*d), v: after that) and BN % d == 0.
// Variants: biases are added to the accumulators first; with per-head q/k
// norms, a first pass writes each (row, head)'s inverse RMS into the spare
// columns BN.. of the parked tile (ldc >= BN + BN/d), then the rotary pass
// scales by it and by the gain.
template <typename T, int BN, int NT>
__device__ __forceinline__ void epi_qkv(float* sC, int ldc, int rows, int m_base, int M,
                                        int n0, const EpiParams& e) {
  const int tid = threadIdx.x;
  const int d = e.d, half = d >> 1;
  const int qcols = e.nq * d, kcols = e.nkv * d;
  const int region = n0 < qcols ? 0 : (n0 < qcols + kcols ? 1 : 2);
  const bool full = d == 128 && m_base + rows <= M && BN % 128 == 0 && NT % ((BN / 128) * 8) == 0 &&
                    rows % (NT / ((BN / 128) * 8) * 4) == 0 && ldc >= BN + 2;
  if (full && region == 2 && NT % (BN / 8) == 0 && rows % (NT / (BN / 8) * 8) == 0) {
    const T* bias = reinterpret_cast<const T*>(e.bv);
    if (bias != nullptr) {
      // fold the bias into the parked tile once; both stores read it
      for (int it = tid; it < rows * BN; it += NT) {
        const int r = it / BN, c = it % BN;
        sC[(int64_t)r * ldc + c] += Elem<T>::load(bias, (n0 - qcols - kcols) + c);
      }
      __syncthreads();
    }
    epi_qkv_v_full<T, BN, NT>(sC, ldc, rows, m_base, n0, e);
    return;
  }
  if (region < 2) {
    // column base of the tile within its region (q: head-major q columns,
    // k: head-major k columns), bias and norm gain of the region
    const int rbase = region == 0 ? n0 : n0 - qcols;
    const T* bias = reinterpret_cast<const T*>(region == 0 ? e.bq : e.bk);
    const T* gain = reinterpret_cast<const T*>(region == 0 ? e.q_norm : e.k_norm);
    const int heads = BN / d, chunks = half / 8;
    if (gain != nullptr) {
      // eight consecutive lanes per (row, head), each summing d/8 squares
      const int seg = d / 8;
      for (int it = tid; it < rows * heads * 8; it += NT) {
        const int pr = it >> 3, part = it & 7;
        const int r = pr / heads, hh = pr % heads;
        const float* src = sC + (int64_t)r * ldc + hh * d + part * seg;
        const int bb = rbase + hh * d + part * seg;
        float ss = 0.0f;
        for (int i = 0; i < seg; i += 4) {
          float b4[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
          if (bias) {
#pragma unroll
            for (int k = 0; k < 4; ++k) b4[k] = Elem<T>::load(bias, bb + i + k);
          }
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const float v = src[i + k] + b4[k];
            ss += v * v;
          }
        }
        ss += __shfl_xor(ss, 1, 64);
        ss += __shfl_xor(ss, 2, 64);
        ss += __shfl_xor(ss, 4, 64);
        if (part == 0) sC[(int64_t)r * ldc + BN + hh] = 1.0f / sqrtf(ss / (float)d + e.eps);
      }
      __syncthreads();
    }
    if (full) {
      if (region == 0)
        epi_qkv_rot_full<T, BN, NT, 0>(sC, ldc, rows, m_base, n0, e);
      else
        epi_qkv_rot_full<T, BN, NT, 1>(sC, ldc, rows, m_base, n0, e);
      return;
    }
    // items: (row, head in tile, chunk of 8 rotary pairs)
    const int per_row = heads * chunks;
    for (int it = tid; it < rows * per_row; it += NT) {
      const int r = it / per_row, hc = it % per_row;
      const int hh = hc / chunks, c0 = (hc % chunks) * 8;
      const int m = m_base + r;
      if (m >= M) continue;
      const float* src = sC + (int64_t)r * ldc + hh * d;
      const int p = e.pos[m];
      const float2* cs = e.rope + (int64_t)p * half + c0;
      const int hb = rbase + hh * d;
      const float inv = gain != nullptr ? sC[(int64_t)r * ldc + BN + hh] : 1.0f;
      float lo[8], hi[8], ba[8], bb[8], ga[8], gb[8];
      if (bias) {
        ld8(bias + hb + c0, ba);
        ld8(bias + hb + c0 + half, bb);
      }
      if (gain != nullptr) {
        ld8(gain + c0, ga);
        ld8(gain + c0 + half, gb);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float a = src[c0 + i], b = src[c0 + half + i];
        if (bias) {
          a += ba[i];
          b += bb[i];
        }
        if (gain != nullptr) {
          a = a * inv * ga[i];
          b = b * inv * gb[i];
        }
        const float2 t = cs[i];
        lo[i] = Elem<T>::round(a * t.x - b * t.y);
        hi[i] = Elem<T>::round(b * t.x + a * t.y);
      }
      T* dst;
      if (region == 0) {
        dst = reinterpret_cast<T*>(e.q_out) + (int64_t)m * qcols + n0 + hh * d;
      } else {
        const int kh = (n0 - qcols) / d + hh;
        const int64_t sl = e.slot[m];
        if (e.kc != nullptr) {
          // contiguous per-head copy for attention; padding rows hold zeros so
          // that keys past a request's end are inert whatever their residual holds
          const int64_t kr = e.krow != nullptr ? e.krow[m] : m;
          T* kd = reinterpret_cast<T*>(e.kc) + ((int64_t)kh * e.ldvt + kr) * d;
          if (sl < 0) {
#pragma unroll
            for (int i = 0; i < 8; ++i) lo[i] = hi[i] = 0.0f;
          }
          store8(kd + c0, lo);
          store8(kd + c0 + half, hi);
        }
        if (sl < 0) continue;  // padding row: nothing goes to the arena
        dst = reinterpret_cast<T*>(e.arena_k) + (sl * e.nkv + kh) * (int64_t)d;
      }
      store8(dst + c0, lo);
      store8(dst + c0 + half, hi);
    }
  } else {
    const int vbase = n0 - qcols - kcols;  // first V column (head-major) of the tile
    const T* bias = reinterpret_cast<const T*>(e.bv);
    if (bias != nullptr) {
      // fold the bias into the parked tile once; both stores below read it
      for (int it = tid; it < rows * BN; it += NT) {
        const int r = it / BN, c = it % BN;
        sC[(int64_t)r * ldc + c] += Elem<T>::load(bias, vbase + c);
      }
      __syncthreads();
    }
    const int per_row = BN / 8;
    for (int it = tid; it < rows * per_row; it += NT) {
      const int r = it / per_row, c0 = (it % per_row) * 8;
      const int m = m_base + r;
      if (m >= M) continue;
      const int64_t sl = e.slot[m];
      if (sl < 0) continue;  // padding row
      const float* src = sC + (int64_t)r * ldc + c0;
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = src[i];
      const int col = vbase + c0;  // = kh * d + e
      T* dst = reinterpret_cast<T*>(e.arena_v) + sl * (int64_t)kcols + col;
      store8(dst, v);
    }
    if (e.vt != nullptr) {
      // V^T (col, krow(m)): 8 consecutive rows of one column per item (their key
      // rows are consecutive and inside one key tile: a request's rows start
      // on a multiple of 8, and so do its suffix key rows); padding rows get
      // zeros, so attention reads inert values past a request's last key
      const int rchunks = rows / 8;
      for (int it = tid; it < BN * rchunks; it += NT) {
        const int c = it % BN, rc = it / BN;
        const int m0 = m_base + rc * 8;
        if (m0 >= M) continue;
        const float* src = sC + (int64_t)(rc * 8) * ldc + c;
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = e.slot[m0 + i] < 0 ? 0.0f : src[(int64_t)i * ldc];
        const int64_t kr0 = e.krow != nullptr ? e.krow[m0] : m0;
        store8(reinterpret_cast<T*>(e.vt) + vt_offset(vbase + c, kr0, e.ldvt, d), v);
      }
    }
  }
}

// RESID: X += acc on the fp32 residual stream, read and written nontemporally
// (once per product; it should not evict the operand panels other tiles are
// streaming through L2).  Loads and stores share one wait counter on this
// GPU, and once a store is pending every wait for a load becomes a wait for
// all: so a batch of rows is loaded, summed and only then stored, with no
// store between a load and its use.  A thread keeps one 4-column chunk; rows
// are NT/(BN/4) apart.  Tiles cut by M take the plain row-by-row loop.
template <int BN, int NT>
__device__ __forceinline__ void epi_resid(const float* sC, int ldc, int rows, int m_base, int M,
                                          int n0, const EpiParams& e) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  constexpr int PER_ROW = BN / 4, RSTEP = NT / PER_ROW, RB = 16;
  const int tid = threadIdx.x;
  const int c0 = (tid % PER_ROW) * 4, r0 = tid / PER_ROW;
  if (m_base + rows <= M && rows % (RSTEP * RB) == 0) {
    for (int rb = 0; rb < rows; rb += RSTEP * RB) {
      f32x4* xp = reinterpret_cast<f32x4*>(e.x + (int64_t)(m_base + rb + r0) * e.ldx + n0 + c0);
      const int64_t step = (int64_t)RSTEP * e.ldx / 4;  // f32x4 units between this thread's rows
      f32x4 xv[RB];
#pragma unroll
      for (int b = 0; b < RB; ++b) xv[b] = __builtin_nontemporal_load(xp + b * step);
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        const float* src = sC + (int64_t)(rb + r0 + b * RSTEP) * ldc + c0;
        xv[b].x += src[0];
        xv[b].y += src[1];
        xv[b].z += src[2];
        xv[b].w += src[3];
        asm volatile("" : "+v"(xv[b]));  // the sum is formed here, before any store
      }
#pragma unroll
      for (int b = 0; b < RB; ++b) __builtin_nontemporal_store(xv[b], xp + b * step);
    }
    return;
  }
  for (int it = tid; it < rows * PER_ROW; it += NT) {
    const int r = it / PER_ROW, c = (it % PER_ROW) * 4;
    const int m = m_base + r;
    if (m >= M) continue;
    f32x4* xp = reinterpret_cast<f32x4*>(e.x + (int64_t)m * e.ldx + n0 + c);
    const float* src = sC + (int64_t)r * ldc + c;
    f32x4 xv = __builtin_nontemporal_load(xp);
    xv.x += src[0];
    xv.y += src[1];
    xv.z += src[2];
    xv.w += src[3];
    __builtin_nontemporal_store(xv, xp);
  }
}

// STORE: X = acc (fp32), columns [n0, n0 + BN) of rows < M.
template <int BN, int NT>
__device__ __forceinline__ void epi_store(const float* sC, int ldc, int rows, int m_base, int M,
                                          int n0, const EpiParams& e) {
  const int tid = threadIdx.x;
  const int per_row = BN / 4;
  for (int it = tid; it < rows * per_row; it += NT) {
    const int r = it / per_row, c0 = (it % per_row) * 4;
    const int m = m_base + r;
    if (m >= M) continue;
    const float* src = sC + (int64_t)r * ldc + c0;
    *reinterpret_cast<float4*>(e.x + (int64_t)m * e.ldx + n0 + c0) =
        make_float4(src[0], src[1], src[2], src[3]);
  }
}

// SWIGLU: tile columns [0, BN/2) are gate rows j0.., [BN/2, BN) the same up rows.
template <typename T, int BN, int NT>
__device__ __forceinline__ void epi_swiglu(const float* sC, int ldc, int rows, int m_base, int M,
                                           int j0, const EpiParams& e) {
  const int tid = threadIdx.x;
  constexpr int HB = BN / 2;
  const int per_row = HB / 8;
#pragma unroll 4
  for (int it = tid; it < rows * per_row; it += NT) {
    const int r = it / per_row, c0 = (it % per_row) * 8;
    const int m = m_base + r;
    if (m >= M || j0 + c0 >= e.ffn) continue;
    const float* src = sC + (int64_t)r * ldc + c0;
    float h[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = Elem<T>::round(silu(src[i]) * src[HB + i]);
    T* dst = reinterpret_cast<T*>(e.hf) + (int64_t)m * e.ldh + j0 + c0;
    if (j0 + c0 + 8 <= e.ffn) {
      store8(dst, h);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (j0 + c0 + i < e.ffn) Elem<T>::store(dst, i, h[i]);
    }
  }
}

}  // namespace kvr
