// fp32 GEMM C[M, N] = A[M, K] . B[N, K]^T on the vector ALUs, for fp32
// models, with the same fused epilogues as the bf16 path.  Tile 64 x 128 x 16,
// 256 threads, 4 x 8 outputs per thread; every load is bounds-checked, so
// ragged M, N (FFN widths that are not tile multiples) and K are handled.
// Deterministic: one workgroup per output tile, fixed K order.
#include "common.h"
#include "epilogue.h"
#include "launch.h"

namespace kvr {

namespace {

constexpr int BM = 64, BN = 128, BK = 16, NT = 256;
constexpr int LDA = BM + 4, LDB = BN + 4, LDC = BN + 4;

__device__ __forceinline__ const float* b_row_ptr_f32(const GemmParams& p, int tile_n, int r) {
  const int64_t K = p.K;
  if (p.bmap == BMAP_GATEUP) {
    const int j = tile_n * (BN / 2) + (r & (BN / 2 - 1));
    if (j >= p.epi.ffn) return nullptr;
    return reinterpret_cast<const float*>(r < BN / 2 ? p.B0 : p.B1) + (int64_t)j * K;
  }
  const int n = p.n_begin + tile_n * BN + r;
  if (n >= p.n_end) return nullptr;
  if (p.bmap == BMAP_QKV) {
    if (n < p.s0) return reinterpret_cast<const float*>(p.B0) + (int64_t)n * K;
    if (n < p.s1) return reinterpret_cast<const float*>(p.B1) + (int64_t)(n - p.s0) * K;
    return reinterpret_cast<const float*>(p.B2) + (int64_t)(n - p.s1) * K;
  }
  return reinterpret_cast<const float*>(p.B0) + (int64_t)n * K;
}

template <int EPI>
__global__ __launch_bounds__(NT) void gemm_f32_kernel(GemmParams p, int tiles_n) {
  __shared__ float sA[BK * LDA];
  __shared__ float sB[BK * LDB];
  __shared__ __attribute__((aligned(16))) float sC[BM * LDC];
  const int tile_m = blockIdx.x / tiles_n, tile_n = blockIdx.x % tiles_n;
  const int tid = threadIdx.x;
  const int m0 = tile_m * BM;
  const float* A = reinterpret_cast<const float*>(p.A);

  // loaders: A 64 rows x 16 k (4 per thread), B 128 rows x 16 k (8 per thread)
  const int la_row = tid >> 2, la_k = (tid & 3) * 4;
  const int am = m0 + la_row;
  const float* a_row = am < p.M ? A + (int64_t)am * p.lda : nullptr;
  const float* b_row0 = b_row_ptr_f32(p, tile_n, la_row);
  const float* b_row1 = b_row_ptr_f32(p, tile_n, la_row + 64);

  const int ty = tid >> 4, tx = tid & 15;  // rows ty*4.., cols tx*8..
  float acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0f;

  for (int k0 = 0; k0 < p.K; k0 += BK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = k0 + la_k + i;
      sA[(la_k + i) * LDA + la_row] = (a_row && k < p.K) ? a_row[k] : 0.0f;
      sB[(la_k + i) * LDB + la_row] = (b_row0 && k < p.K) ? b_row0[k] : 0.0f;
      sB[(la_k + i) * LDB + la_row + 64] = (b_row1 && k < p.K) ? b_row1[k] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float av[4], bv[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = sA[kk * LDA + ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 8; ++j) bv[j] = sB[kk * LDB + tx * 8 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) sC[(ty * 4 + i) * LDC + tx * 8 + j] = acc[i][j];
  __syncthreads();
  if (EPI == EPI_QKV)
    epi_qkv<float, BN, NT>(sC, LDC, BM, m0, p.M, p.n_begin + tile_n * BN, p.epi);
  else if (EPI == EPI_RESID)
    epi_resid<BN, NT>(sC, LDC, BM, m0, p.M, p.n_begin + tile_n * BN, p.epi);
  else if (EPI == EPI_STORE)
    epi_store<BN, NT>(sC, LDC, BM, m0, p.M, p.n_begin + tile_n * BN, p.epi);
  else
    epi_swiglu<float, BN, NT>(sC, LDC, BM, m0, p.M, tile_n * (BN / 2), p.epi);
}

}  // namespace

void launch_gemm_f32(int epi, const GemmParams& p, hipStream_t s) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = p.bmap == BMAP_GATEUP ? (p.epi.ffn + BN / 2 - 1) / (BN / 2)
                                            : (p.n_end - p.n_begin + BN - 1) / BN;
  if (p.M <= 0 || tiles_n <= 0) return;
  const dim3 grid(tiles_m * tiles_n), block(NT);
  if (epi == EPI_QKV)
    hipLaunchKernelGGL(gemm_f32_kernel<EPI_QKV>, grid, block, 0, s, p, tiles_n);
  else if (epi == EPI_RESID)
    hipLaunchKernelGGL(gemm_f32_kernel<EPI_RESID>, grid, block, 0, s, p, tiles_n);
  else if (epi == EPI_STORE)
    hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE>, grid, block, 0, s, p, tiles_n);
  else
    hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, block, 0, s, p, tiles_n);
}

}  // namespace kvr
