// bf16 GEMM C[M, N] = A[M, K] . B[N, K]^T on gfx950 matrix cores, with the
// rebuild's epilogues fused (RoPE + K/V scatter, residual add, SwiGLU).
//
// Tile 256 x 256 x 64 per workgroup of WAVES wave64s (4: a 2 x 2 layout of
// 128 x 128 wave tiles; 8: a 2 x 4 layout of 128 x 64 wave tiles, two waves
// per SIMD), each wave tile made of 32 x 32 v_mfma_f32_32x32x16_bf16 tiles.
// Both operands are K-contiguous, so every MFMA operand is one 16-byte LDS
// read.  Operand tiles stream from global memory straight into a 5-slot LDS
// ring with buffer_load_dwordx4 ... lds (no register staging), three slots
// (96 KB) in flight per CU.  Workgroups are remapped so that each XCD
// (dispatch round-robins workgroups over the 8 XCDs) works on a contiguous
// range of tiles, walked in groups of a few M-tiles so that the 32 CUs of
// an XCD share A rows and B columns in their L2 (8 M-tiles x 4 N-tiles at a
// time; 4 x 8 when there are at most 16 N-tiles, which measured 3-4 % faster
// on the 4096-column products, whose long A panels then stay in the MALL).
// Every output element is produced by exactly one workgroup with a fixed K
// order: results are deterministic run to run.
#include <algorithm>

#include "common.h"
#include "epilogue.h"
#include "launch.h"

namespace kvr {

namespace {

#ifndef KVR_GEMM_WAVES
#define KVR_GEMM_WAVES 4
#endif

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int WAVES = KVR_GEMM_WAVES;
constexpr int NT = 64 * WAVES;
constexpr int WN = WAVES / 2;        // waves along N (2 along M)
constexpr int FI = 4;                // 32-row MFMA tiles per wave (128 rows)
constexpr int FJ = (BN / WN) / 32;   // 32-column MFMA tiles per wave
constexpr int LDC = BN + 4;          // epilogue fp32 tile row, elements
constexpr int EPI_BYTES = 128 * LDC * 4;
static_assert(WAVES == 4 || WAVES == 8, "2 x 2 or 2 x 4 wave layout");

// LDS layout of one 256-row x 64-k operand tile: 1 KB blocks of 8 rows of
// 128 bytes; in a block, row j holds its 16-byte k-units u at slot
// u ^ swz(j, block).  A direct-to-LDS load writes 64 lanes x 16 B
// contiguously, so one instruction fills one block with 8 lanes per row
// (each row's 128 bytes are one coalesced segment: one full L2 line per
// request, which moves twice the bytes per request of 64-byte rows).  The
// swizzle makes the MFMA operand reads (32 consecutive rows, one k-unit)
// conflict-free whether the LDS serves 8 or 16 lanes of a b128 read per pass.
//
// The ring holds NSLOT operand tiles.  Slot sequence number s carries the A
// tile (s even) or the B tile (s odd) of K tile s/2 and lives at ring position
// s % NSLOT.  While K tile kt is multiplied, its two slots are read and the
// loads of the next NSLOT-2 slots are in flight.
struct Ring {
  static constexpr int UPR = BK / 8;           // 16-byte units per row
  static constexpr int RPB = 1024 / (BK * 2);  // rows per 1 KB block
  static constexpr int BLOCKS = BM / RPB;      // blocks per operand tile
  static constexpr int HALF = BM * BK * 2;     // bytes per operand tile
  static constexpr int NSLOT = 5;              // 160 KB
  static constexpr int BYTES = NSLOT * HALF;
  static constexpr int LOADS = BLOCKS / WAVES; // per wave, per slot
  static __device__ __forceinline__ int swz(int j, int blk) { return (j ^ (blk & 1)) & 7; }
};

__device__ __forceinline__ const bf16_t* b_row_ptr(const GemmParams& p, int tile_n, int r) {
  const int64_t K = p.ldb ? p.ldb : p.K;
  if (p.bmap == BMAP_GATEUP) {
    const int j = tile_n * (BN / 2) + (r & (BN / 2 - 1));
    const bf16_t* base = reinterpret_cast<const bf16_t*>(r < BN / 2 ? p.B0 : p.B1);
    return base + (int64_t)j * K;
  }
  const int n = p.n_begin + tile_n * BN + r;
  if (p.bmap == BMAP_QKV) {
    if (n < p.s0) return reinterpret_cast<const bf16_t*>(p.B0) + (int64_t)n * K;
    if (n < p.s1) return reinterpret_cast<const bf16_t*>(p.B1) + (int64_t)(n - p.s0) * K;
    return reinterpret_cast<const bf16_t*>(p.B2) + (int64_t)(n - p.s1) * K;
  }
  return reinterpret_cast<const bf16_t*>(p.B0) + (int64_t)n * K;
}

typedef __attribute__((address_space(3))) void lds_void;

// Operand sources of one workgroup as buffer resources.  Buffer loads with
// the LDS bit (buffer_load_dwordx4 ... lds) are tracked by the vector-memory
// counter alone, so the LDS reads of the fragments keep exact lgkm counts;
// the global_load_lds form would also be counted as an LDS access and force a
// full lgkmcnt(0) drain before every k-step.
//   A: one resource at the tile's first row; each load q has its own lane
//      offset (rows past M are clamped to row M-1, their results dropped).
//   B: rows 0..127 and 128..255 of the tile each sit in one weight matrix
//      (the QKV split points are multiples of 256 and a gate/up tile is 128
//      gate rows then 128 up rows; the one-pass gate/up product takes them in
//      quarters instead, see issue_slot); the block's row offset is scalar.
struct Loader {
  const void* a;            // tile row 0 of A
  const void* b_lo;         // tile row 0 of B
  const void* b_hi;         // tile row 128 of B
  int a_bytes, b_bytes;     // extents of the three resources
  int a_voff[Ring::LOADS];
  int b_voff;
  int b_block_bytes;        // bytes between consecutive 8-row blocks of B
  int k_base_bytes;         // first K column of this launch's K range, bytes
};

constexpr int BUF_WORD3 = 0x00020000;  // gfx9 buffer descriptor: 32-bit data format

// Issue loads q in [Q0, Q1) of one ring slot holding operand B (IS_B) or A at
// K tile kt, into ring position slot % NSLOT (wave `wid` fills blocks wid,
// wid+WAVES, ...).  GU: the B tile of the fused gate/up product holds its
// 128 gate rows and 128 up rows in quarters of 64 (gate j0.., up j0..,
// gate j0+64.., up j0+64..), so that each wave column's accumulators hold
// the gate and the up values of the same 64 outputs.
template <bool IS_B, int Q0, int Q1, bool GU>
__device__ __forceinline__ void issue_slot(char* smem, const Loader& L, int kt, int slot, int wid) {
  static_assert(!GU || WAVES == 4, "the gate/up quarter layout assumes 8 B blocks per wave");
  const int kbytes = L.k_base_bytes + kt * BK * 2;
  char* st = smem + (slot % Ring::NSLOT) * Ring::HALF;
#pragma unroll
  for (int q = Q0; q < Q1; ++q) {
    lds_void* dst = (lds_void*)(st + (wid + WAVES * q) * 1024);
    if constexpr (IS_B) {
      constexpr int HB = Ring::BLOCKS / 2;  // blocks per 128-row half
      // tile block wid + 4q sits in quarter q/2; gate quarters are 0 and 2
      const bool hi = GU ? ((q >> 1) & 1) != 0 : q >= Ring::LOADS / 2;
      const int blk = GU ? (q >> 2) * 8 + wid + 4 * (q & 1) : wid + WAVES * q - (hi ? HB : 0);
      const int soff = kbytes + blk * L.b_block_bytes;
      const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(hi ? L.b_hi : L.b_lo), 0,
                                                          L.b_bytes, BUF_WORD3);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, dst, 16, L.b_voff, soff, 0, 0);
    } else {
      const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(L.a), 0, L.a_bytes,
                                                          BUF_WORD3);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, dst, 16, L.a_voff[q], kbytes, 0, 0);
    }
  }
}

template <bool IS_B, bool GU>
__device__ __forceinline__ void issue_whole(char* smem, const Loader& L, int kt, int slot, int wid) {
  issue_slot<IS_B, 0, Ring::LOADS, GU>(smem, L, kt, slot, wid);
}

// Share of k-step KS in the load issue of a K tile's two slots s0 and s0+1:
// the first half of the k-steps issues slot s0, the second half slot s0+1.
template <int KS, bool S0_IS_B, bool GU>
__device__ __forceinline__ void issue_step(char* smem, const Loader& L, int k_s0, int k_s1, int s0,
                                           int wid) {
  constexpr int SPS = (BK / 16) / 2;  // k-steps per slot
  constexpr int QS = Ring::LOADS / SPS;
  if constexpr (KS < SPS)
    issue_slot<S0_IS_B, (KS % SPS) * QS, (KS % SPS + 1) * QS, GU>(smem, L, k_s0, s0, wid);
  else
    issue_slot<!S0_IS_B, (KS % SPS) * QS, (KS % SPS + 1) * QS, GU>(smem, L, k_s1, s0 + 1, wid);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding)
#define KVR_WAIT_VMCNT(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (((n) >> 4) << 14) | (0x7 << 4) | (0xF << 8))

// sched_group_barrier masks
constexpr int SG_MFMA = 0x008, SG_VMEM = 0x010, SG_DS_READ = 0x100;

template <int EPI>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmParams p, int tiles_m, int tiles_n) {
  constexpr int SMEM = Ring::BYTES > EPI_BYTES ? Ring::BYTES : EPI_BYTES;
  constexpr bool GU = EPI == EPI_SWIGLU;  // gate/up B tile in quarters, SwiGLU in registers
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  // ---- split-K pass: consecutive workgroups share a tile, one K range each ----
  const int ksplit = EPI == EPI_PARTIAL ? p.ksplit : 1;
  const int split = EPI == EPI_PARTIAL ? (int)(blockIdx.x % ksplit) : 0;
  // ---- tile coordinates: XCD-contiguous ranges, grouped along M ----
  const int num_tiles = tiles_m * tiles_n;
  int t = EPI == EPI_PARTIAL ? (int)(blockIdx.x / ksplit) : (int)blockIdx.x;
  const int full = (num_tiles / 8) * 8;
  if (t < full) t = (t % 8) * (num_tiles / 8) + t / 8;
  const int gm = p.group_m;
  const int group = t / (gm * tiles_n);
  const int first_m = group * gm;
  const int gsz = min(tiles_m - first_m, gm);
  const int tile_m = first_m + (t % (gm * tiles_n)) % gsz;
  const int tile_n = (t % (gm * tiles_n)) / gsz;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = tile_m * BM;

  // ---- direct-to-LDS loaders: wave w fills blocks w, w+WAVES, ... of A and of B ----
  const int lrow = lane / Ring::UPR;  // row within the block
  // k-unit that lands in this lane's 16-byte slot (swz depends on the block
  // only through its parity, which is the wave's parity for every load)
  const int unit = (lane % Ring::UPR) ^ Ring::swz(lrow, wave);
  Loader L;
  {
    const int64_t ldb = p.ldb ? p.ldb : p.K;
    const int rows_a = min(BM, p.M - m0);
    L.a = reinterpret_cast<const bf16_t*>(p.A) + (int64_t)m0 * p.lda;
    L.a_bytes = (int)(rows_a * p.lda * 2);
#pragma unroll
    for (int q = 0; q < Ring::LOADS; ++q) {
      const int r = min((wave + WAVES * q) * Ring::RPB + lrow, rows_a - 1);
      L.a_voff[q] = (int)(r * p.lda * 2) + unit * 16;
    }
    L.b_bytes = (int)((BN / 2) * ldb * 2);
    L.b_lo = b_row_ptr(p, tile_n, 0);
    L.b_hi = b_row_ptr(p, tile_n, BN / 2);
    L.b_voff = (int)(lrow * ldb * 2) + unit * 16;
    L.b_block_bytes = (int)(Ring::RPB * ldb * 2);
    L.k_base_bytes = EPI == EPI_PARTIAL ? split * p.kt_per * BK * 2 : 0;
  }

  f32x16 acc[FI][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int KT = EPI == EPI_PARTIAL ? min(p.kt_per, p.K / BK - split * p.kt_per) : p.K / BK;
#pragma unroll
  for (int s = 0; s < Ring::NSLOT - 2; ++s) {
    if (s & 1)
      issue_whole<true, GU>(smem, L, min(s >> 1, KT - 1), s, wave);
    else
      issue_whole<false, GU>(smem, L, min(s >> 1, KT - 1), s, wave);
  }

  // fragment reads: lane%32 picks the row, lane/32 the 8-wide k half
  const int fr = lane & 31, fhalf = lane >> 5;
  const int fj = fr % Ring::RPB;
  int a_base[FI], b_base[FJ], a_sw[FI], b_sw[FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i) {
    const int ra = wm * 128 + i * 32 + fr;
    a_base[i] = (ra / Ring::RPB) * 1024 + fj * BK * 2;
    a_sw[i] = Ring::swz(fj, ra / Ring::RPB);
  }
#pragma unroll
  for (int j = 0; j < FJ; ++j) {
    const int rb = wn * (BN / WN) + j * 32 + fr;
    b_base[j] = (rb / Ring::RPB) * 1024 + fj * BK * 2;
    b_sw[j] = Ring::swz(fj, rb / Ring::RPB);
  }

  // Slots issued during K tile kt: s0 (the operand of parity NSLOT) and s1.
  // NSLOT-2 slots are always in flight (past the end, the last K tile is
  // fetched again into a position no later K tile reads), so both slots of a
  // K tile have landed once at most NSLOT-4 slots' loads are pending.
  constexpr bool S0_IS_B = (Ring::NSLOT & 1) != 0;
  constexpr int KS = BK / 16;                    // k-steps per K tile
  constexpr int MF = FI * FJ;                    // MFMAs per k-step
  constexpr int NRD = FI + FJ;                   // fragment reads per k-step
  constexpr int NLOAD = 2 * Ring::LOADS / KS;    // buffer loads per k-step
  constexpr int NRD2 = (NRD + 1) / 2;            // MFMAs carrying the next K tile's reads
  // MFMAs of the last k-step issued before its barrier
  constexpr int PBAR = MF - (NRD2 > MF / 4 ? NRD2 : MF / 4);
  static_assert(KS % 2 == 0 && NLOAD <= PBAR && NRD2 <= MF - PBAR && NRD + NLOAD <= MF,
                "k-step schedule");
  constexpr int LANDED = (Ring::NSLOT - 4) * Ring::LOADS;

  // K tile 0 lands; every wave sees every wave's loads after the barrier (a
  // bare s_barrier: __syncthreads() would also drain the loads in flight).
  KVR_WAIT_VMCNT(LANDED);
  __builtin_amdgcn_s_barrier();
  bf16x8 af[2][FI], bfr[2][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
    af[0][i] = *reinterpret_cast<const bf16x8*>(smem + a_base[i] + ((fhalf ^ a_sw[i]) << 4));
#pragma unroll
  for (int j = 0; j < FJ; ++j)
    bfr[0][j] = *reinterpret_cast<const bf16x8*>(smem + Ring::HALF + b_base[j] + ((fhalf ^ b_sw[j]) << 4));
  __builtin_amdgcn_sched_barrier(0);

  for (int kt = 0; kt < KT; ++kt) {
    const int s0 = 2 * kt + Ring::NSLOT - 2;
    const int k_s0 = min(s0 >> 1, KT - 1), k_s1 = min((s0 + 1) >> 1, KT - 1);
    const char* sta = smem + ((2 * kt) % Ring::NSLOT) * Ring::HALF;
    const char* stb = smem + ((2 * kt + 1) % Ring::NSLOT) * Ring::HALF;
    const char* sta_n = smem + ((2 * kt + 2) % Ring::NSLOT) * Ring::HALF;
    const char* stb_n = smem + ((2 * kt + 3) % Ring::NSLOT) * Ring::HALF;
    // The fragments of k-step ks+1 are read from LDS while the MFMAs of k-step
    // ks run, and the instruction stream interleaves them one by one with the
    // MFMAs (an MFMA keeps the pipe busy for 32 cycles while the next
    // instruction issues): (MFMA, LDS read) pairs, then (MFMA, buffer load)
    // pairs for the k-step's share of the next slots' loads.  The barrier that
    // hands K tile kt+1 over sits inside the last k-step of K tile kt, after
    // PBAR of its MFMAs: by then every fragment of K tile kt is in registers,
    // so the slots of K tile kt may be refilled, and the first fragments of
    // K tile kt+1 are read behind the remaining MFMAs instead of stalling the
    // start of the next K tile.
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < KS) {
        // in the order the next k-step's MFMAs consume them: A0, B0..B3, A1..
        const int cn = 2 * (ks + 1) + fhalf;
        af[cur ^ 1][0] = *reinterpret_cast<const bf16x8*>(sta + a_base[0] + ((cn ^ a_sw[0]) << 4));
#pragma unroll
        for (int j = 0; j < FJ; ++j)
          bfr[cur ^ 1][j] = *reinterpret_cast<const bf16x8*>(stb + b_base[j] + ((cn ^ b_sw[j]) << 4));
#pragma unroll
        for (int i = 1; i < FI; ++i)
          af[cur ^ 1][i] = *reinterpret_cast<const bf16x8*>(sta + a_base[i] + ((cn ^ a_sw[i]) << 4));
      }
      if (ks == 0) issue_step<0, S0_IS_B, GU>(smem, L, k_s0, k_s1, s0, wave);
      if (ks == 1) issue_step<1, S0_IS_B, GU>(smem, L, k_s0, k_s1, s0, wave);
      if (ks == 2) issue_step<2, S0_IS_B, GU>(smem, L, k_s0, k_s1, s0, wave);
      if (ks == 3) issue_step<3, S0_IS_B, GU>(smem, L, k_s0, k_s1, s0, wave);
      const int m_end = ks + 1 < KS ? MF : PBAR;
#pragma unroll
      for (int m = 0; m < m_end; ++m)
        acc[m / FJ][m % FJ] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            af[cur][m / FJ], bfr[cur][m % FJ], acc[m / FJ][m % FJ], 0, 0, 0);
      if (ks + 1 < KS) {
#pragma unroll
        for (int q = 0; q < NRD; ++q) {
          __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
          __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
        }
#pragma unroll
        for (int q = 0; q < NLOAD; ++q) {
          __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
          __builtin_amdgcn_sched_group_barrier(SG_VMEM, 1, 0);
        }
        if (MF - NRD - NLOAD > 0) __builtin_amdgcn_sched_group_barrier(SG_MFMA, MF - NRD - NLOAD, 0);
        __builtin_amdgcn_sched_barrier(0);
      } else {
        // (MFMA, buffer load) x NLOAD, MFMAs up to PBAR; barrier; the first
        // fragments of K tile kt+1 behind the remaining MFMAs, two per MFMA.
        // On the last K tile the wait, the barrier and the reads are harmless
        // leftovers.
#pragma unroll
        for (int q = 0; q < NLOAD; ++q) {
          __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
          __builtin_amdgcn_sched_group_barrier(SG_VMEM, 1, 0);
        }
        if (PBAR - NLOAD > 0) __builtin_amdgcn_sched_group_barrier(SG_MFMA, PBAR - NLOAD, 0);
        __builtin_amdgcn_sched_barrier(0);
        KVR_WAIT_VMCNT(LANDED);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        af[0][0] = *reinterpret_cast<const bf16x8*>(sta_n + a_base[0] + ((fhalf ^ a_sw[0]) << 4));
#pragma unroll
        for (int j = 0; j < FJ; ++j)
          bfr[0][j] = *reinterpret_cast<const bf16x8*>(stb_n + b_base[j] + ((fhalf ^ b_sw[j]) << 4));
#pragma unroll
        for (int i = 1; i < FI; ++i)
          af[0][i] = *reinterpret_cast<const bf16x8*>(sta_n + a_base[i] + ((fhalf ^ a_sw[i]) << 4));
#pragma unroll
        for (int m = PBAR; m < MF; ++m)
          acc[m / FJ][m % FJ] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              af[cur][m / FJ], bfr[cur][m % FJ], acc[m / FJ][m % FJ], 0, 0, 0);
#pragma unroll
        for (int q = 0; q < NRD2; ++q) {
          __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
          __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 2, 0);
        }
        if (MF - PBAR - NRD2 > 0) __builtin_amdgcn_sched_group_barrier(SG_MFMA, MF - PBAR - NRD2, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  KVR_WAIT_VMCNT(0);  // the trailing refetches land before the ring becomes the C tile

  if constexpr (GU) {
    // ---- SwiGLU from the accumulators: tile columns wn*128 + [0, 64) hold
    // the gate and wn*128 + [64, 128) the up values of outputs
    // j0 + wn*64 + [0, 64) (the quarter layout of the B tile); a lane has one
    // output column of each 32-column tile and 16 of its rows ----
    const int j0 = tile_n * (BN / 2);
    const int oc0 = j0 + wn * 64 + (lane & 31);
    const int row0 = m0 + wm * 128 + 4 * (lane >> 5);
    bf16_t* hf = reinterpret_cast<bf16_t*>(p.epi.hf) + (int64_t)row0 * p.epi.ldh + oc0;
    if (m0 + BM <= p.M && j0 + BN / 2 <= p.epi.ffn) {
      // (two-byte stores: each instruction writes 64-byte row segments, whose
      // other halves the same wave writes next; a transpose within quads of
      // lanes for 8-byte stores measured 1 % slower)
#pragma unroll
      for (int i = 0; i < FI; ++i)
#pragma unroll
        for (int j = 0; j < FJ / 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int dr = i * 32 + 8 * (r >> 2) + (r & 3);
            hf[(int64_t)dr * p.epi.ldh + j * 32] = f2bf(silu(acc[i][j][r]) * acc[i][j + 2][r]);
          }
    } else {
#pragma unroll
      for (int i = 0; i < FI; ++i)
#pragma unroll
        for (int j = 0; j < FJ / 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int dr = i * 32 + 8 * (r >> 2) + (r & 3);
            if (row0 + dr < p.M && oc0 + j * 32 < p.epi.ffn)
              hf[(int64_t)dr * p.epi.ldh + j * 32] = f2bf(silu(acc[i][j][r]) * acc[i][j + 2][r]);
          }
    }
    return;
  }

  // ---- epilogue: two passes of 128 rows through LDS ----
  __syncthreads();  // all waves are done with the ring before it becomes the C tile
  float* sC = reinterpret_cast<float*>(smem);
  for (int pass = 0; pass < 2; ++pass) {
    if (m0 + pass * 128 >= p.M) break;  // no valid rows left in this tile
    if (wm == pass) {
      // accumulator register r of tile (i, j): row 8*(r/4) + 4*(lane/32) + r%4, col lane%32
#pragma unroll
      for (int i = 0; i < FI; ++i)
#pragma unroll
        for (int j = 0; j < FJ; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            const int col = wn * (BN / WN) + j * 32 + (lane & 31);
            sC[row * LDC + col] = acc[i][j][r];
          }
    }
    __syncthreads();
    const int m_base = m0 + pass * 128;
    if (EPI == EPI_QKV) {
      epi_qkv<bf16_t, BN, NT>(sC, LDC, 128, m_base, p.M, p.n_begin + tile_n * BN, p.epi);
    } else if (EPI == EPI_RESID) {
      epi_resid<BN, NT>(sC, LDC, 128, m_base, p.M, p.n_begin + tile_n * BN, p.epi);
    } else if (EPI == EPI_STORE) {
      epi_store<BN, NT>(sC, LDC, 128, m_base, p.M, p.n_begin + tile_n * BN, p.epi);
    } else if (EPI == EPI_PARTIAL) {
      EpiParams e = p.epi;
      e.x = p.part + split * p.part_stride;
      e.ldx = p.part_ld;
      epi_store<BN, NT>(sC, LDC, 128, m_base, p.M, tile_n * BN, e);
    } else {
      epi_swiglu<bf16_t, BN, NT>(sC, LDC, 128, m_base, p.M, tile_n * (BN / 2), p.epi);
    }
    __syncthreads();
  }
}

// Split-K partials summed in split order (slice 0, then += slice 1, ...),
// then the fused epilogue, in 32-row x 256-column pieces, exactly as the
// one-pass GEMM would apply it.
constexpr int SK_ROWS = 32;

// Sums the ksplit partials of IPT float4 items (item i at src[i], splits
// stride apart) in split order, with SPB splits of every item loaded before
// any is added, so the loads of a thread overlap instead of waiting one by one.
template <int IPT, int SPB>
__device__ __forceinline__ void sum_splits(const float* const (&src)[IPT], const bool (&valid)[IPT],
                                           int ksplit, int64_t stride, float4 (&a)[IPT]) {
  for (int sp0 = 0; sp0 < ksplit; sp0 += SPB) {
    float4 v[IPT][SPB];
#pragma unroll
    for (int i = 0; i < IPT; ++i)
#pragma unroll
      for (int j = 0; j < SPB; ++j)
        if (valid[i] && sp0 + j < ksplit) v[i][j] = *reinterpret_cast<const float4*>(src[i] + (sp0 + j) * stride);
#pragma unroll
    for (int i = 0; i < IPT; ++i)
#pragma unroll
      for (int j = 0; j < SPB; ++j) {
        if (!valid[i] || sp0 + j >= ksplit) continue;
        if (sp0 + j == 0) {
          a[i] = v[i][j];
        } else {
          a[i].x += v[i][j].x;
          a[i].y += v[i][j].y;
          a[i].z += v[i][j].z;
          a[i].w += v[i][j].w;
        }
      }
  }
}

// TW: the epilogue's tile width, BN or (QKV, head dim dividing 128) 128 for
// twice the workgroups
template <int EPI, int TW>
__global__ __launch_bounds__(256) void splitk_epi_kernel(GemmParams p, int tiles_n) {
  __shared__ __attribute__((aligned(16))) float sC[SK_ROWS * LDC];
  const int tile_n = blockIdx.x % tiles_n, m0 = (blockIdx.x / tiles_n) * SK_ROWS;
  const int tid = threadIdx.x;
  constexpr int IPT = SK_ROWS * (TW / 4) / 256;
  const float* src[IPT];
  bool valid[IPT];
  float4 a[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int it = tid + i * 256, r = it / (TW / 4), c = (it % (TW / 4)) * 4;
    valid[i] = m0 + r < p.M;
    src[i] = p.part + (int64_t)min(m0 + r, p.M - 1) * p.part_ld + tile_n * TW + c;
    a[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
  sum_splits<IPT, 4>(src, valid, p.ksplit, p.part_stride, a);
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int it = tid + i * 256, r = it / (TW / 4), c = (it % (TW / 4)) * 4;
    *reinterpret_cast<float4*>(sC + r * LDC + c) = a[i];
  }
  __syncthreads();
  if (EPI == EPI_QKV) {
    epi_qkv<bf16_t, TW, 256>(sC, LDC, SK_ROWS, m0, p.M, p.n_begin + tile_n * TW, p.epi);
  } else if (EPI == EPI_RESID) {
    epi_resid<BN, 256>(sC, LDC, SK_ROWS, m0, p.M, p.n_begin + tile_n * BN, p.epi);
  } else if (EPI == EPI_STORE) {
    epi_store<BN, 256>(sC, LDC, SK_ROWS, m0, p.M, p.n_begin + tile_n * BN, p.epi);
  } else {
    epi_swiglu<bf16_t, BN, 256>(sC, LDC, SK_ROWS, m0, p.M, tile_n * (BN / 2), p.epi);
  }
}

// ---- products of few rows (resumed decode) ----
// C[M <= 64, N] = A . B^T, weight-stationary: a wave owns NBW blocks of 16
// output columns (16 weight rows each) and one K range.  It streams those rows
// once with 16-byte loads (per 128-k chunk a lane takes 64 contiguous bytes of
// its row) and multiplies them with every row of A on
// v_mfma_f32_16x16x32_bf16 (16-row tiles of A; rows past M are clamped and
// their results dropped).  The A fragments of a chunk are loaded once for all
// NBW blocks: with one block per wave, the A loads (from L2) equal the weight
// bytes and bound the kernel.  In a chunk of 128 k, MFMA t takes the k values
// 32t+8q..+7 from lane group q = lane/16 (the matrix core's own operand
// layout), so each load instruction reads 64 contiguous bytes of each of 16
// rows and the next one the rest of those lines; the loads are plain (cached),
// as nontemporal ones would fetch the lines again.  The waves of one K range
// are consecutive, so a workgroup's waves read the same A lines.  No LDS and
// no padding work: HBM-bound on the weights.  Output: the fp32 partial sums of
// the K range, in the split-K partial layout.
constexpr int SK_CHUNK = 128;   // k per chunk
constexpr int SK_UNROLL = 2;    // chunks in flight per wave
constexpr int SK_MAX_M = 64;
// K is split into ranges for about SK_WAVES waves, at most 16 where the
// epilogue is elementwise (it sums the splits of every output in parallel)
// and 8 where it works on whole tiles, whose few workgroups read every split
// (measured best on the 8B shapes with weights not in the last-level cache)
constexpr int SK_WAVES = 2048, SK_MAX_SPLIT_ELEM = 16, SK_MAX_SPLIT_TILE = 8;

template <int MT, int NBW>
__global__ __launch_bounds__(256) void gemm_bf16_skinny_kernel(GemmParams p, int ngroups, int kc_per) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= ngroups * p.ksplit) return;  // whole waves
  const int grp = item % ngroups, split = item / ngroups;
  const int r16 = lane & 15, q = lane >> 4;
  const bf16_t* brow[NBW];
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const int nb = grp * NBW + b;
    brow[b] = b_row_ptr(p, nb / (BN / 16), (nb % (BN / 16)) * 16 + r16) + 8 * q;
  }
  const bf16_t* arow[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    arow[mt] = reinterpret_cast<const bf16_t*>(p.A) + (int64_t)min(mt * 16 + r16, p.M - 1) * p.lda + 8 * q;
  const int KC = p.K / SK_CHUNK;
  const int kc0 = split * kc_per, kc1 = min(KC, kc0 + kc_per);
  f32x4 acc[NBW][MT];
#pragma unroll
  for (int b = 0; b < NBW; ++b)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[b][mt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  // SK_UNROLL chunks of loads in flight (weights first), then their MFMAs
  for (int kc = kc0; kc < kc1; kc += SK_UNROLL) {
    bf16x8 bv[SK_UNROLL][NBW][4], av[SK_UNROLL][MT][4];
#pragma unroll
    for (int u = 0; u < SK_UNROLL; ++u) {
      if (kc + u < kc1) {
        const int ko = (kc + u) * SK_CHUNK;
#pragma unroll
        for (int b = 0; b < NBW; ++b)
#pragma unroll
          for (int t = 0; t < 4; ++t) bv[u][b][t] = *reinterpret_cast<const bf16x8*>(brow[b] + ko + 32 * t);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int t = 0; t < 4; ++t) av[u][mt][t] = *reinterpret_cast<const bf16x8*>(arow[mt] + ko + 32 * t);
      }
    }
#pragma unroll
    for (int u = 0; u < SK_UNROLL; ++u) {
      if (kc + u < kc1) {
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int b = 0; b < NBW; ++b)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              acc[b][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[u][mt][t], bv[u][b][t], acc[b][mt], 0, 0, 0);
      }
    }
  }
  // a lane holds rows 4q .. 4q+3 of each 16-row tile, at column r16 of a block
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const int nb = grp * NBW + b;
    float* out = p.part + split * p.part_stride + nb * 16 + r16;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = mt * 16 + 4 * q + j;
        if (m < p.M) out[(int64_t)m * p.part_ld] = acc[b][mt][j];
      }
  }
}

// Elementwise epilogues (residual add, store) of a split-K product: one
// float4 of the output per thread, the splits summed in index order exactly
// as splitk_epi_kernel sums them, so every output is parallel work.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_elem_kernel(GemmParams p) {
  const int ld4 = p.part_ld / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)p.M * ld4) return;
  const int m = (int)(i / ld4), col = (int)(i % ld4) * 4;
  float4* xp = reinterpret_cast<float4*>(p.epi.x + (int64_t)m * p.epi.ldx + p.n_begin + col);
  float4 xv = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (EPI == EPI_RESID) xv = *xp;
  const float* src[1] = {p.part + (int64_t)m * p.part_ld + col};
  const bool valid[1] = {true};
  float4 acc[1];
  sum_splits<1, 8>(src, valid, p.ksplit, p.part_stride, acc);
  const float4 a = acc[0];
  if (EPI == EPI_RESID) {
    xv.x += a.x;
    xv.y += a.y;
    xv.z += a.z;
    xv.w += a.w;
    *xp = xv;
  } else {
    *xp = a;
  }
}

// Residual sum and RMSNorm after a few-row product: workgroup m sums row m's
// split-K partials in split order into the residual row X (the values
// splitk_elem_kernel writes), then writes round(g * x / rms(x)) as the next
// product's A row.  Every load (X, partials, gain) comes before any store.
constexpr int RN_THREADS = 1024, RN_MAXI = 2;  // rows up to RN_THREADS * 4 * RN_MAXI wide
__global__ __launch_bounds__(RN_THREADS) void splitk_resid_norm_kernel(GemmParams p, const bf16_t* gain,
                                                                       bf16_t* a_out, float eps) {
  __shared__ float red[RN_THREADS / 64];
  const int m = blockIdx.x, tid = threadIdx.x;
  const int N = p.n_end - p.n_begin;
  float* xrow = p.epi.x + (int64_t)m * p.epi.ldx + p.n_begin;
  const float* src[RN_MAXI];
  bool valid[RN_MAXI];
  float4 acc[RN_MAXI], xv[RN_MAXI];
  uint2 gv[RN_MAXI];
#pragma unroll
  for (int i = 0; i < RN_MAXI; ++i) {
    const int col = (tid + i * RN_THREADS) * 4;
    valid[i] = col < N;
    const int cc = valid[i] ? col : 0;
    src[i] = p.part + (int64_t)m * p.part_ld + cc;
    xv[i] = valid[i] ? *reinterpret_cast<const float4*>(xrow + cc) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    gv[i] = valid[i] ? *reinterpret_cast<const uint2*>(gain + cc) : make_uint2(0u, 0u);
    acc[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
  sum_splits<RN_MAXI, 8>(src, valid, p.ksplit, p.part_stride, acc);
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < RN_MAXI; ++i) {
    if (!valid[i]) continue;
    xv[i].x += acc[i].x;
    xv[i].y += acc[i].y;
    xv[i].z += acc[i].z;
    xv[i].w += acc[i].w;
    ss += xv[i].x * xv[i].x + xv[i].y * xv[i].y + xv[i].z * xv[i].z + xv[i].w * xv[i].w;
  }
#pragma unroll
  for (int i = 0; i < RN_MAXI; ++i)
    if (valid[i]) *reinterpret_cast<float4*>(xrow + (tid + i * RN_THREADS) * 4) = xv[i];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < RN_THREADS / 64; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)N + eps);
#pragma unroll
  for (int i = 0; i < RN_MAXI; ++i) {
    if (!valid[i]) continue;
    const float g0 = __uint_as_float(gv[i].x << 16), g1 = __uint_as_float(gv[i].x & 0xffff0000u);
    const float g2 = __uint_as_float(gv[i].y << 16), g3 = __uint_as_float(gv[i].y & 0xffff0000u);
    uint2 o;
    o.x = (uint32_t)f2bf(g0 * xv[i].x * inv) | ((uint32_t)f2bf(g1 * xv[i].y * inv) << 16);
    o.y = (uint32_t)f2bf(g2 * xv[i].z * inv) | ((uint32_t)f2bf(g3 * xv[i].w * inv) << 16);
    *reinterpret_cast<uint2*>(a_out + (int64_t)m * N + (tid + i * RN_THREADS) * 4) = o;
  }
}

struct SkinnyPlan {
  int nbw, ngroups, ksplit, kc_per;
};

bool skinny_ok(int M, int K) { return M > 0 && M <= SK_MAX_M && K % SK_CHUNK == 0; }

// 16-row blocks per wave: as many as keep the A tiles and the blocks' loads
// in registers (MT tiles of A cost as much as MT blocks)
int skinny_nbw(int M) {
  const int mt = (M + 15) / 16;
  return mt == 1 ? 4 : mt == 2 ? 2 : 1;
}

SkinnyPlan skinny_plan(int M, int tiles_n, int K, int max_split) {
  SkinnyPlan sp;
  sp.nbw = skinny_nbw(M);
  sp.ngroups = tiles_n * (BN / 16) / sp.nbw;
  const int KC = K / SK_CHUNK;
  const int want = std::max(1, std::min({KC, max_split, SK_WAVES / std::max(1, sp.ngroups)}));
  sp.kc_per = (KC + want - 1) / want;
  sp.ksplit = (KC + sp.kc_per - 1) / sp.kc_per;
  return sp;
}

// q.ksplit K ranges of kc_per chunks over ngroups groups of 16-row blocks
void launch_skinny(const GemmParams& q, int ngroups, int kc_per, hipStream_t s) {
  const dim3 grid((unsigned)((ngroups * q.ksplit + 3) / 4)), block(256);
  switch ((q.M + 15) / 16) {
    case 1: hipLaunchKernelGGL((gemm_bf16_skinny_kernel<1, 4>), grid, block, 0, s, q, ngroups, kc_per); break;
    case 2: hipLaunchKernelGGL((gemm_bf16_skinny_kernel<2, 2>), grid, block, 0, s, q, ngroups, kc_per); break;
    case 3: hipLaunchKernelGGL((gemm_bf16_skinny_kernel<3, 1>), grid, block, 0, s, q, ngroups, kc_per); break;
    default: hipLaunchKernelGGL((gemm_bf16_skinny_kernel<4, 1>), grid, block, 0, s, q, ngroups, kc_per); break;
  }
}

struct SplitPlan {
  int tiles_m, tiles_n, ksplit, kt_per;
};

SplitPlan split_plan(int M, int N_tiles, int K) {
  SplitPlan sp;
  sp.tiles_m = (M + BM - 1) / BM;
  sp.tiles_n = N_tiles;
  const int KT = K / BK;
  const int tiles = std::max(1, sp.tiles_m * sp.tiles_n);
  const int want = std::max(1, std::min(KT, (256 + tiles - 1) / tiles));
  sp.kt_per = (KT + want - 1) / want;
  sp.ksplit = (KT + sp.kt_per - 1) / sp.kt_per;
  return sp;
}

int n_tiles_of(const GemmParams& p) {
  return p.bmap == BMAP_GATEUP ? p.epi.ffn / (BN / 2) : (p.n_end - p.n_begin) / BN;
}

int group_m_for(int tiles_n) { return tiles_n <= 24 ? 4 : 8; }

}  // namespace

int64_t gemm_bf16_splitk_part_elems(int M, int N, int K) {
  if (skinny_ok(M, K))  // the larger of the two caps: enough for either epilogue
    return (int64_t)skinny_plan(M, N / BN, K, SK_MAX_SPLIT_ELEM).ksplit * M * (N / BN) * BN;
  const SplitPlan sp = split_plan(M, N / BN, K);
  return (int64_t)sp.ksplit * M * sp.tiles_n * BN;
}

void launch_gemm_bf16(int epi, const GemmParams& p, hipStream_t s);

void launch_gemm_bf16_splitk(int epi, const GemmParams& p, float* part, int64_t part_cap,
                             hipStream_t s) {
  if (p.M <= 0) return;
  const int tiles_n = n_tiles_of(p);
  const int64_t ld = (int64_t)tiles_n * BN;
  GemmParams q = p;
  q.part = part;
  q.part_ld = (int)ld;
  q.part_stride = (int64_t)p.M * ld;
  const int max_split = epi == EPI_RESID || epi == EPI_STORE ? SK_MAX_SPLIT_ELEM : SK_MAX_SPLIT_TILE;
  if (skinny_ok(p.M, p.K) && (int64_t)skinny_plan(p.M, tiles_n, p.K, max_split).ksplit * p.M * ld <= part_cap) {
    const SkinnyPlan kp = skinny_plan(p.M, tiles_n, p.K, max_split);
    q.ksplit = kp.ksplit;
    launch_skinny(q, kp.ngroups, kp.kc_per, s);
  } else {
    const SplitPlan sp = split_plan(p.M, tiles_n, p.K);
    if (sp.ksplit <= 1 || (int64_t)sp.ksplit * p.M * ld > part_cap) {
      launch_gemm_bf16(epi, p, s);
      return;
    }
    q.group_m = group_m_for(sp.tiles_n);
    q.ksplit = sp.ksplit;
    q.kt_per = sp.kt_per;
    const dim3 grid((unsigned)(sp.tiles_m * sp.tiles_n * sp.ksplit)), block(NT);
    hipLaunchKernelGGL(gemm_bf16_kernel<EPI_PARTIAL>, grid, block, 0, s, q, sp.tiles_m, sp.tiles_n);
  }
  const dim3 egrid((unsigned)(((p.M + SK_ROWS - 1) / SK_ROWS) * tiles_n));
  const dim3 lgrid((unsigned)(((int64_t)p.M * (ld / 4) + 255) / 256));
  if (epi == EPI_QKV && p.epi.d > 0 && 128 % p.epi.d == 0) {
    const int tiles_h = tiles_n * (BN / 128);
    const dim3 hgrid((unsigned)(((p.M + SK_ROWS - 1) / SK_ROWS) * tiles_h));
    hipLaunchKernelGGL((splitk_epi_kernel<EPI_QKV, 128>), hgrid, dim3(256), 0, s, q, tiles_h);
  } else if (epi == EPI_QKV)
    hipLaunchKernelGGL((splitk_epi_kernel<EPI_QKV, BN>), egrid, dim3(256), 0, s, q, tiles_n);
  else if (epi == EPI_RESID)
    hipLaunchKernelGGL(splitk_elem_kernel<EPI_RESID>, lgrid, dim3(256), 0, s, q);
  else if (epi == EPI_STORE)
    hipLaunchKernelGGL(splitk_elem_kernel<EPI_STORE>, lgrid, dim3(256), 0, s, q);
  else
    hipLaunchKernelGGL((splitk_epi_kernel<EPI_SWIGLU, BN>), egrid, dim3(256), 0, s, q, tiles_n);
}

bool launch_gemm_bf16_splitk_resid_norm(const GemmParams& p, float* part, int64_t part_cap,
                                        const void* gain, void* a_out, float eps, hipStream_t s) {
  const int N = p.n_end - p.n_begin;
  if (p.bmap != BMAP_PLAIN || !skinny_ok(p.M, p.K) || N <= 0 || N % BN != 0 ||
      N > RN_THREADS * 4 * RN_MAXI)
    return false;
  const int tiles_n = N / BN;
  const int64_t ld = (int64_t)tiles_n * BN;
  const SkinnyPlan kp = skinny_plan(p.M, tiles_n, p.K, SK_MAX_SPLIT_ELEM);
  if ((int64_t)kp.ksplit * p.M * ld > part_cap) return false;
  GemmParams q = p;
  q.part = part;
  q.part_ld = (int)ld;
  q.part_stride = (int64_t)p.M * ld;
  q.ksplit = kp.ksplit;
  launch_skinny(q, kp.ngroups, kp.kc_per, s);
  hipLaunchKernelGGL(splitk_resid_norm_kernel, dim3((unsigned)p.M), dim3(RN_THREADS), 0, s, q,
                     (const bf16_t*)gain, (bf16_t*)a_out, eps);
  return true;
}

bool launch_gemm_bf16_rows(const GemmParams& p, float* out, int64_t ldo, hipStream_t s) {
  const int N = p.n_end - p.n_begin;
  if (!skinny_ok(p.M, p.K) || N <= 0) return false;
  const int nbw = skinny_nbw(p.M);
  if (N % (16 * nbw) != 0 || ldo < N) return false;
  GemmParams q = p;
  q.part = out;
  q.part_ld = (int)ldo;
  q.part_stride = 0;
  q.ksplit = 1;
  const int ngroups = N / 16 / nbw, kc_per = p.K / SK_CHUNK;
  launch_skinny(q, ngroups, kc_per, s);
  return true;
}

void launch_gemm_bf16(int epi, const GemmParams& p_in, hipStream_t s) {
  const int tiles_m = (p_in.M + BM - 1) / BM;
  const int tiles_n = n_tiles_of(p_in);
  const dim3 grid(tiles_m * tiles_n), block(NT);
  if (p_in.M <= 0 || tiles_n <= 0) return;
  GemmParams p = p_in;
  p.group_m = group_m_for(tiles_n);
  if (epi == EPI_QKV)
    hipLaunchKernelGGL(gemm_bf16_kernel<EPI_QKV>, grid, block, 0, s, p, tiles_m, tiles_n);
  else if (epi == EPI_RESID)
    hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESID>, grid, block, 0, s, p, tiles_m, tiles_n);
  else if (epi == EPI_STORE)
    hipLaunchKernelGGL(gemm_bf16_kernel<EPI_STORE>, grid, block, 0, s, p, tiles_m, tiles_n);
  else
    hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SWIGLU>, grid, block, 0, s, p, tiles_m, tiles_n);
}

}  // namespace kvr
