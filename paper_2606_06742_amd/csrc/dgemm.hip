// Batched fp64 tile GEMM on CDNA4 matrix cores (v_mfma_f64_16x16x4_f64).
//
// One 256-thread workgroup (four 64-lane waves) computes a 64 x 64 tile of C.
// Wave w owns the 32 x 32 quadrant (rows 32*(w&1), cols 32*(w>>1)) as 2 x 2
// MFMA blocks of 16 x 16. The K loop stages 64 x 16 slices of A and 16 x 64
// slices of B through LDS, stored k-major so that the MFMA operand fetch of a
// wave (lane l reads row/col l%16 of k-row l/16) is a contiguous LDS read.
//
// MFMA f64 16x16x4 operand layout (per lane l of the wave):
//   A: element (i = l%16, k = l/16);  B: element (k = l/16, j = l%16);
//   D: 4 accumulators, register r holds (i = 4*r + l/16, j = l%16).
#include "kmp_common.h"
#include "kmp_kernels.h"

namespace kmp {

typedef double dbl4 __attribute__((ext_vector_type(4)));

constexpr int TM = 64, TN = 64, TK = 16, LPAD = 4;

template <bool AK, bool BK>
__device__ __forceinline__ void load_tiles(int M, int N, int K, int i0, int j0, int k0,
                                           const double* __restrict__ A, int64_t lda,
                                           const double* __restrict__ B, int64_t ldb,
                                           double (*As)[TM + LPAD], double (*Bs)[TN + LPAD]) {
  const int t = threadIdx.x;
  // A slice: 64 (i) x 16 (k)
  if (AK) {
    const int i = t >> 2, kb = (t & 3) * 4;
    const int gi = i0 + i;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int gk = k0 + kb + q;
      As[kb + q][i] = (gi < M && gk < K) ? A[(int64_t)gi * lda + gk] : 0.0;
    }
  } else {
    const int k = t >> 4, ib = (t & 15) * 4;
    const int gk = k0 + k;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int gi = i0 + ib + q;
      As[k][ib + q] = (gi < M && gk < K) ? A[(int64_t)gk * lda + gi] : 0.0;
    }
  }
  // B slice: 16 (k) x 64 (j)
  if (BK) {
    const int j = t >> 2, kb = (t & 3) * 4;
    const int gj = j0 + j;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int gk = k0 + kb + q;
      Bs[kb + q][j] = (gj < N && gk < K) ? B[(int64_t)gj * ldb + gk] : 0.0;
    }
  } else {
    const int k = t >> 4, jb = (t & 15) * 4;
    const int gk = k0 + k;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int gj = j0 + jb + q;
      Bs[k][jb + q] = (gj < N && gk < K) ? B[(int64_t)gk * ldb + gj] : 0.0;
    }
  }
}

// Main loop shared by all variants: accumulates the 2 x 2 blocks of the
// calling wave. acc[bi][bj] covers rows wi+16*bi.., cols wj+16*bj...
template <bool AK, bool BK>
__device__ __forceinline__ void tile_mainloop(int M, int N, int K, int i0, int j0,
                                              const double* __restrict__ A, int64_t lda,
                                              const double* __restrict__ B, int64_t ldb,
                                              dbl4 (&acc)[2][2]) {
  __shared__ double As[TK][TM + LPAD];
  __shared__ double Bs[TK][TN + LPAD];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wi = (w & 1) * 32, wj = (w >> 1) * 32;
  const int li = lane & 15, lk = lane >> 4;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = dbl4{0.0, 0.0, 0.0, 0.0};
  for (int k0 = 0; k0 < K; k0 += TK) {
    __syncthreads();
    load_tiles<AK, BK>(M, N, K, i0, j0, k0, A, lda, B, ldb, As, Bs);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; kk += 4) {
      const double a0 = As[kk + lk][wi + li];
      const double a1 = As[kk + lk][wi + 16 + li];
      const double b0 = Bs[kk + lk][wj + li];
      const double b1 = Bs[kk + lk][wj + 16 + li];
      acc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc[1][1], 0, 0, 0);
    }
  }
}

template <bool AK, bool BK, bool CR>
__global__ __launch_bounds__(256) void dgemm_kernel(int M, int N, int K,
                                                     const double* __restrict__ A, int64_t lda, int64_t sA,
                                                     const double* __restrict__ B, int64_t ldb, int64_t sB,
                                                     double* __restrict__ C, int64_t ldc, int64_t sC,
                                                     double alpha, double beta) {
  const int b = blockIdx.z;
  A += (int64_t)b * sA;
  B += (int64_t)b * sB;
  C += (int64_t)b * sC;
  const int i0 = blockIdx.x * TM, j0 = blockIdx.y * TN;
  dbl4 acc[2][2];
  tile_mainloop<AK, BK>(M, N, K, i0, j0, A, lda, B, ldb, acc);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wi = (w & 1) * 32, wj = (w >> 1) * 32;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = i0 + wi + bi * 16 + mfma_row(lane, r);
        const int gj = j0 + wj + bj * 16 + mfma_col(lane);
        if (gi < M && gj < N) {
          const int64_t off = CR ? (int64_t)gi * ldc + gj : (int64_t)gj * ldc + gi;
          const double v = alpha * acc[bi][bj][r];
          C[off] = (beta == 0.0) ? v : v + beta * C[off];
        }
      }
}

// First path GEMM with the loss-derivative epilogue (A = Q row-major,
// B = T abar column-major, C = Z column-major).
__global__ __launch_bounds__(256) void dgemm_loss_kernel(int M, int N, int K,
                                                          const double* __restrict__ A, int64_t lda, int64_t sA,
                                                          const double* __restrict__ B, int64_t ldb, int64_t sB,
                                                          double* __restrict__ C, int64_t ldc, int64_t sC,
                                                          LossEpi e) {
  __shared__ double red[4][32];
  const int b = blockIdx.z;
  A += (int64_t)b * sA;
  B += (int64_t)b * sB;
  C += (int64_t)b * sC;
  const int i0 = blockIdx.x * TM, j0 = blockIdx.y * TN;
  dbl4 acc[2][2];
  tile_mainloop<true, true>(M, N, K, i0, j0, A, lda, B, ldb, acc);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wi = (w & 1) * 32, wj = (w >> 1) * 32;
  const int nv = e.nv[b];
  const double inv_nv = 1.0 / (double)nv;
  const double* y = e.y + (int64_t)b * e.sy;
  const double* bbar = e.bbar + (int64_t)b * e.sbb;
  const double* tau = e.tau + (int64_t)b * e.stau;
  double colsum[2] = {0.0, 0.0};
#pragma unroll
  for (int bj = 0; bj < 2; ++bj) {
    const int gj = j0 + wj + bj * 16 + (lane & 15);
    const bool cj = gj < N;
    const double bb = cj ? bbar[gj] : 0.0;
    const double tj = cj ? tau[gj] : 0.0;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = i0 + wi + bi * 16 + mfma_row(lane, r);
        if (gi < M && cj) {
          double z = 0.0;
          if (gi < nv) z = loss_psi(e.loss, y[gi], acc[bi][bj][r] + bb, e.delta, tj) * inv_nv;
          C[(int64_t)gj * ldc + gi] = z;
          colsum[bj] += z;
        }
      }
  }
  // reduce over the four 16-lane row groups (same column), fixed order
#pragma unroll
  for (int bj = 0; bj < 2; ++bj) {
    double v = colsum[bj];
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 32, 64);
    colsum[bj] = v;
  }
  if (lane < 16) {
    red[w][lane] = colsum[0];
    red[w][16 + lane] = colsum[1];
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    const int j = threadIdx.x;            // tile column
    const int wq = (j >> 5) * 2;          // waves 0,1 own cols 0..31; 2,3 own 32..63
    const int jj = j & 31;
    const double s = red[wq][jj] + red[wq + 1][jj];
    const int gj = j0 + j;
    if (gj < N) e.partial[(int64_t)b * e.spart + (int64_t)blockIdx.x * N + gj] = s;
  }
}

int gemm(hipStream_t s, const GemmArgs& g, bool ak, bool bk, bool cr) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return 0;
  dim3 grid((unsigned)ceil_div(g.M, TM), (unsigned)ceil_div(g.N, TN), (unsigned)g.batch);
  dim3 block(256);
#define KMP_GEMM_CASE(a, b, c)                                                              \
  if (ak == a && bk == b && cr == c) {                                                      \
    hipLaunchKernelGGL((dgemm_kernel<a, b, c>), grid, block, 0, s, g.M, g.N, g.K, g.A, g.lda, \
                       g.sA, g.B, g.ldb, g.sB, g.C, g.ldc, g.sC, g.alpha, g.beta);          \
    KMP_LAUNCH_CHECK();                                                                     \
    return 0;                                                                               \
  }
  KMP_GEMM_CASE(true, true, true)
  KMP_GEMM_CASE(true, true, false)
  KMP_GEMM_CASE(true, false, true)
  KMP_GEMM_CASE(true, false, false)
  KMP_GEMM_CASE(false, true, true)
  KMP_GEMM_CASE(false, true, false)
  KMP_GEMM_CASE(false, false, true)
  KMP_GEMM_CASE(false, false, false)
#undef KMP_GEMM_CASE
  return KMP_EINVAL;
}

int gemm_loss(hipStream_t s, const GemmArgs& g, const LossEpi& e) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return 0;
  dim3 grid((unsigned)ceil_div(g.M, TM), (unsigned)ceil_div(g.N, TN), (unsigned)g.batch);
  hipLaunchKernelGGL(dgemm_loss_kernel, grid, dim3(256), 0, s, g.M, g.N, g.K, g.A, g.lda, g.sA,
                     g.B, g.ldb, g.sB, g.C, g.ldc, g.sC, e);
  KMP_LAUNCH_CHECK();
  return 0;
}

}  // namespace kmp
