// bf16 GEMM C[M, N] = A[M, K] . B[N, K]^T on gfx950 matrix cores, with the
// rebuild's epilogues fused (RoPE + K/V scatter, residual add, SwiGLU).
//
// Tile 256 x 256 x 64, 256 threads = 4 wave64s in a 2 x 2 layout, each wave
// owning 128 x 128 outputs as 4 x 4 v_mfma_f32_32x32x16_bf16 tiles (256 fp32
// accumulators per lane).  Both operands are K-contiguous, so every MFMA
// operand is one 16-byte LDS read.  A and B tiles are double-buffered in LDS
// (rows padded to 144 B so the 32 rows read by one MFMA operand fall in
// distinct banks); the next K tile is fetched into registers while the
// current one is multiplied, one barrier per K step.  Workgroups are remapped
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

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int LDK = BK + 8;     // padded LDS row, elements
constexpr int NT = 256;
constexpr int LDC = BN + 4;     // epilogue fp32 tile row, elements
constexpr int STAGE_ELEMS = (BM + BN) * LDK;
constexpr int SMEM_BYTES = 2 * STAGE_ELEMS * 2;  // two stages of bf16
static_assert(128 * LDC * 4 <= SMEM_BYTES, "epilogue tile must fit the main-loop LDS");
constexpr int GROUP_M = 8;

__device__ __forceinline__ const bf16_t* b_row_ptr(const GemmParams& p, int tile_n, int r) {
  const int64_t K = p.K;
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

template <int EPI>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmParams p, int tiles_m, int tiles_n) {
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * STAGE_ELEMS];

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

  // ---- per-thread global load addresses: 8 chunks of 16 B for A and for B ----
  // (named registers rather than arrays so that nothing lands in scratch)
  const int lrow = tid >> 3, lcol = (tid & 7) * 8;
  const bf16_t* A = reinterpret_cast<const bf16_t*>(p.A);
#define KVR_REP8(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7)
#define KVR_ADDR(j)                                                                        \
  const bf16_t* a_src##j =                                                                 \
      A + (int64_t)min(m0 + lrow + 32 * j, p.M - 1) * p.lda + lcol;                        \
  const bf16_t* b_src##j = b_row_ptr(p, tile_n, lrow + 32 * j) + lcol;                     \
  uint4 ra##j, rb##j;
  KVR_REP8(KVR_ADDR)
  // rows past M read a valid row; their results are dropped by the epilogue

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int KT = p.K / BK;
#define KVR_GLOAD1(j)                                          \
  ra##j = *reinterpret_cast<const uint4*>(a_src##j + k_next);  \
  rb##j = *reinterpret_cast<const uint4*>(b_src##j + k_next);
#define KVR_SSTORE1(j)                                                       \
  *reinterpret_cast<uint4*>(sA_ + (lrow + 32 * j) * LDK + lcol) = ra##j;     \
  *reinterpret_cast<uint4*>(sB_ + (lrow + 32 * j) * LDK + lcol) = rb##j;
  {
    const int k_next = 0;
    KVR_REP8(KVR_GLOAD1)
    bf16_t* sA_ = smem;
    bf16_t* sB_ = sA_ + BM * LDK;
    KVR_REP8(KVR_SSTORE1)
  }
  __syncthreads();

  // MFMA operand rows: lane%32 picks the row, lane/32 the 8-wide k half
  const int frow = lane & 31, fk = (lane >> 5) * 8;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    // the last iteration re-fetches its own tile (always in bounds) to keep the loop branch-free
    const int k_next = (kt + 1 < KT ? kt + 1 : kt) * BK;
    KVR_REP8(KVR_GLOAD1)
    const bf16_t* sA = smem + cur * STAGE_ELEMS + (wm * 128 + frow) * LDK + fk;
    const bf16_t* sB = smem + cur * STAGE_ELEMS + BM * LDK + (wn * 128 + frow) * LDK + fk;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8*>(sA + i * 32 * LDK + ks * 16);
#pragma unroll
      for (int j = 0; j < 4; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(sB + j * 32 * LDK + ks * 16);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    {
      bf16_t* sA_ = smem + (cur ^ 1) * STAGE_ELEMS;
      bf16_t* sB_ = sA_ + BM * LDK;
      KVR_REP8(KVR_SSTORE1)
    }
    __syncthreads();
  }

#undef KVR_REP8
#undef KVR_ADDR
#undef KVR_GLOAD1
#undef KVR_SSTORE1
  // ---- epilogue: two passes of 128 rows through LDS ----
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

void launch_gemm_bf16(int epi, const GemmParams& p, hipStream_t s) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = p.bmap == BMAP_GATEUP ? p.epi.ffn / (BN / 2) : (p.n_end - p.n_begin) / BN;
  const dim3 grid(tiles_m * tiles_n), block(NT);
  if (p.M <= 0 || tiles_n <= 0) return;
  if (epi == EPI_QKV)
    hipLaunchKernelGGL(gemm_bf16_kernel<EPI_QKV>, grid, block, 0, s, p, tiles_m, tiles_n);
  else if (epi == EPI_RESID)
    hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESID>, grid, block, 0, s, p, tiles_m, tiles_n);
  else
    hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SWIGLU>, grid, block, 0, s, p, tiles_m, tiles_n);
}

}  // namespace kvr
