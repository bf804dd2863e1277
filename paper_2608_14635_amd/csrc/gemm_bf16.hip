// bf16 GEMM C[M, N] = A[M, K] . B[N, K]^T on gfx950 matrix cores, with the
// rebuild's epilogues fused (RoPE + K/V scatter, residual add, SwiGLU).
//
// Tile 256 x 256 x 32, 256 threads = 4 wave64s in a 2 x 2 layout, each wave
// owning 128 x 128 outputs as 4 x 4 v_mfma_f32_32x32x16_bf16 tiles (256 fp32
// accumulators per lane).  Both operands are K-contiguous, so every MFMA
// operand is one 16-byte LDS read.  Operand tiles stream from global memory
// straight into a 4-stage LDS ring with global_load_lds_dwordx4 (no register
// staging), keeping three K tiles (96 KB) in flight per CU to cover memory
// latency; one barrier per K tile.  Workgroups are remapped
// so that each XCD (dispatch round-robins workgroups over the 8 XCDs) works
// on a contiguous range of tiles, walked in groups of 8 M-tiles so that the
// 32 CUs of an XCD share A rows and B columns in their L2.
// Every output element is produced by exactly one workgroup with a fixed K
// order: results are deterministic run to run.
#include "common.h"
#include "epilogue.h"
#include "launch.h"

namespace kvr {

namespace {

constexpr int BM = 256, BN = 256;
constexpr int NT = 256;
constexpr int LDC = BN + 4;  // epilogue fp32 tile row, elements
constexpr int EPI_BYTES = 128 * LDC * 4;
constexpr int GROUP_M = 8;

// LDS layout of one 256-row x BK operand tile: 1 KB blocks of RPB rows of
// BK*2 bytes; in a block, row j holds its 16-byte k-units u at slot
// u ^ swz(j, block).  A direct-to-LDS load writes 64 lanes x 16 B
// contiguously, so one instruction fills one block with UPR lanes per row
// (each row's bytes are one coalesced segment).  The swizzle makes the MFMA
// operand reads (32 consecutive rows, one k-unit) conflict-free whether the
// LDS serves 8 or 16 lanes of a b128 read per pass.
template <int BK> struct Ring {
  static constexpr int UPR = BK / 8;                       // 16-byte units per row
  static constexpr int RPB = 1024 / (BK * 2);              // rows per 1 KB block
  static constexpr int BLOCKS = BM / RPB;                  // blocks per operand tile
  static constexpr int HALF = BM * BK * 2;                 // bytes per operand tile
  static constexpr int STAGE = 2 * HALF;
  static constexpr int NSTAGE = BK == 32 ? 4 : 2;          // 128 KB ring either way
  static constexpr int BYTES = NSTAGE * STAGE;
  static constexpr int LOADS = BLOCKS / 4;                 // per wave, per operand, per stage
  static __device__ __forceinline__ int swz(int j, int blk) {
    return BK == 32 ? (((j >> 1) ^ (j >> 3)) & 3) : ((j ^ (blk & 1)) & 7);
  }
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

// Issue the direct-to-LDS loads of K tile kt (wave `wid` fills blocks wid, wid+4, ...)
// K tile `kt` goes to the ring stage of tile `slot_kt` (they differ only for the
// refetches past the last tile).
template <int BK, int Q0 = 0, int Q1 = Ring<BK>::LOADS>
__device__ __forceinline__ void issue_tile(char* smem, const bf16_t* const* a_src,
                                           const bf16_t* const* b_src, int kt, int slot_kt,
                                           int wid) {
  using R = Ring<BK>;
  const int k0 = kt * BK;
  char* st = smem + (slot_kt % R::NSTAGE) * R::STAGE;
#pragma unroll
  for (int q = Q0; q < Q1; ++q) {
    __builtin_amdgcn_global_load_lds(a_src[q] + k0, (lds_void*)(st + (wid + 4 * q) * 1024), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(b_src[q] + k0, (lds_void*)(st + R::HALF + (wid + 4 * q) * 1024),
                                     16, 0, 0);
  }
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding)
#define KVR_WAIT_VMCNT(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (((n) >> 4) << 14) | (0x7 << 4) | (0xF << 8))

template <int EPI, int BK>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmParams p, int tiles_m, int tiles_n) {
  using R = Ring<BK>;
  constexpr int SMEM = R::BYTES > EPI_BYTES ? R::BYTES : EPI_BYTES;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  // ---- tile coordinates: XCD-contiguous ranges, grouped along M ----
  const int num_tiles = tiles_m * tiles_n;
  int t = blockIdx.x;
  const int full = (num_tiles / 8) * 8;
  if (t < full) t = (t % 8) * (num_tiles / 8) + t / 8;
  const int group = t / (GROUP_M * tiles_n);
  const int first_m = group * GROUP_M;
  const int gsz = min(tiles_m - first_m, GROUP_M);
  const int tile_m = first_m + (t % (GROUP_M * tiles_n)) % gsz;
  const int tile_n = (t % (GROUP_M * tiles_n)) / gsz;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;
  const int m0 = tile_m * BM;

  // ---- direct-to-LDS loaders: wave w fills blocks w, w+4, ... of A and of B ----
  const int lrow = lane / R::UPR;  // row within the block
  const bf16_t* A = reinterpret_cast<const bf16_t*>(p.A);
  const bf16_t* a_src[R::LOADS];
  const bf16_t* b_src[R::LOADS];
#pragma unroll
  for (int q = 0; q < R::LOADS; ++q) {
    const int blk = wid + 4 * q;
    const int r = blk * R::RPB + lrow;
    const int unit = (lane % R::UPR) ^ R::swz(lrow, blk);  // k-unit landing in this lane's slot
    // rows past M read a valid row; their results are dropped by the epilogue
    a_src[q] = A + (int64_t)min(m0 + r, p.M - 1) * p.lda + unit * 8;
    b_src[q] = b_row_ptr(p, tile_n, r) + unit * 8;
  }

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int KT = p.K / BK;
#pragma unroll
  for (int s = 0; s < R::NSTAGE - 1; ++s)
    issue_tile<BK>(smem, a_src, b_src, min(s, KT - 1), s, wid);

  // fragment reads: lane%32 picks the row, lane/32 the 8-wide k half
  const int fr = lane & 31, fhalf = lane >> 5;
  const int fj = fr % R::RPB;
  int a_base[4], b_base[4], a_sw[4], b_sw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ra = wm * 128 + i * 32 + fr, rb = wn * 128 + i * 32 + fr;
    a_base[i] = (ra / R::RPB) * 1024 + fj * BK * 2;
    b_base[i] = R::HALF + (rb / R::RPB) * 1024 + fj * BK * 2;
    a_sw[i] = R::swz(fj, ra / R::RPB);
    b_sw[i] = R::swz(fj, rb / R::RPB);
  }

  constexpr int PER_TILE = 2 * R::LOADS;  // load instructions per wave per K tile
  for (int kt = 0; kt < KT; ++kt) {
    // NSTAGE-1 tiles are always in flight (past the end, the last tile is
    // fetched again into a stage no later iteration reads), so tile kt has
    // landed once at most NSTAGE-2 tiles' loads are pending.
    KVR_WAIT_VMCNT((R::NSTAGE - 2) * PER_TILE);
    // every wave's loads of tile kt are in LDS and every wave is done reading the
    // stage of tile kt-1.  A bare s_barrier: __syncthreads() would also drain
    // the loads still in flight for the next tiles.
    __builtin_amdgcn_s_barrier();
    const int kn = min(kt + R::NSTAGE - 1, KT - 1), sn = kt + R::NSTAGE - 1;
    const char* st = smem + (kt % R::NSTAGE) * R::STAGE;
    // Fragments of k-step ks+1 are read from LDS while the MFMAs of k-step ks
    // run: the A fragments before its first MFMA, the B fragments after its
    // eighth, so that at most 12 LDS reads are ever pending (the lgkm counter
    // tops out at 15).  sched_barrier fences keep the compiler from sinking
    // the reads back next to their uses.
    bf16x8 af[2][4], bfr[2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[0][i] = *reinterpret_cast<const bf16x8*>(st + a_base[i] + ((fhalf ^ a_sw[i]) << 4));
      bfr[0][i] = *reinterpret_cast<const bf16x8*>(st + b_base[i] + ((fhalf ^ b_sw[i]) << 4));
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int cur = ks & 1;
      const int cn = 2 * (ks + 1) + fhalf;
      if (ks + 1 < BK / 16) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          af[cur ^ 1][i] = *reinterpret_cast<const bf16x8*>(st + a_base[i] + ((cn ^ a_sw[i]) << 4));
      }
      // spread the next tile's load issue over this tile's k-steps
      constexpr int QS = R::LOADS / (BK / 16);
      if (ks == 0) issue_tile<BK, 0 * QS, 1 * QS>(smem, a_src, b_src, kn, sn, wid);
      if (ks == 1) issue_tile<BK, 1 * QS, 2 * QS>(smem, a_src, b_src, kn, sn, wid);
      if (ks == 2) issue_tile<BK, 2 * QS, 3 * QS>(smem, a_src, b_src, kn, sn, wid);
      if (ks == 3) issue_tile<BK, 3 * QS, 4 * QS>(smem, a_src, b_src, kn, sn, wid);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#ifndef KVR_PROBE_NO_MFMA
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
#endif
        }
      __builtin_amdgcn_sched_barrier(0);
      if (ks + 1 < BK / 16) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          bfr[cur ^ 1][i] = *reinterpret_cast<const bf16x8*>(st + b_base[i] + ((cn ^ b_sw[i]) << 4));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 2; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#ifndef KVR_PROBE_NO_MFMA
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
#endif
        }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  KVR_WAIT_VMCNT(0);  // the trailing refetches land before the ring becomes the C tile

  // ---- epilogue: two passes of 128 rows through LDS ----
  __syncthreads();  // all waves are done with the ring before it becomes the C tile
  float* sC = reinterpret_cast<float*>(smem);
  for (int pass = 0; pass < 2; ++pass) {
    if (wm == pass) {
      // accumulator register r of tile (i, j): row 8*(r/4) + 4*(lane/32) + r%4, col lane%32
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            const int col = wn * 128 + j * 32 + (lane & 31);
            sC[row * LDC + col] = acc[i][j][r];
          }
    }
    __syncthreads();
    const int m_base = m0 + pass * 128;
    if (EPI == EPI_QKV) {
      epi_qkv<bf16_t, BN, NT>(sC, LDC, 128, m_base, p.M, p.n_begin + tile_n * BN, p.epi);
    } else if (EPI == EPI_RESID) {
      epi_resid<BN, NT>(sC, LDC, 128, m_base, p.M, p.n_begin + tile_n * BN, p.epi);
    } else {
      epi_swiglu<bf16_t, BN, NT>(sC, LDC, 128, m_base, p.M, tile_n * (BN / 2), p.epi);
    }
    __syncthreads();
  }
}

}  // namespace

#ifndef KVR_GEMM_BK
#define KVR_GEMM_BK 32
#endif

void launch_gemm_bf16(int epi, const GemmParams& p, hipStream_t s) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = p.bmap == BMAP_GATEUP ? p.epi.ffn / (BN / 2) : (p.n_end - p.n_begin) / BN;
  const dim3 grid(tiles_m * tiles_n), block(NT);
  if (p.M <= 0 || tiles_n <= 0) return;
  if (epi == EPI_QKV)
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI_QKV, KVR_GEMM_BK>), grid, block, 0, s, p, tiles_m, tiles_n);
  else if (epi == EPI_RESID)
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI_RESID, KVR_GEMM_BK>), grid, block, 0, s, p, tiles_m, tiles_n);
  else
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI_SWIGLU, KVR_GEMM_BK>), grid, block, 0, s, p, tiles_m, tiles_n);
}

}  // namespace kvr
