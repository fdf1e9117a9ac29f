// Batched fp64 tile GEMM on CDNA4 matrix cores (v_mfma_f64_16x16x4_f64).
//
// One 256-thread workgroup (four 64-lane waves) computes a BM x 64 tile of C
// (BM = 64, or 32 when 64-row tiles would leave compute units idle). Wave w
// owns rows (BM/2)*(w&1) .. and cols 32*(w>>1) .. as (BM/32) x 2 MFMA blocks
// of 16 x 16. The K loop stages BM x 32 slices of A and 32 x 64 slices of B
// through LDS, stored k-major so that the MFMA operand fetch of a wave (lane
// l reads row/col l%16 of k-row l/16) is a contiguous LDS read.
//
// MFMA f64 16x16x4 operand layout (per lane l of the wave):
//   A: element (i = l%16, k = l/16);  B: element (k = l/16, j = l%16);
//   D: 4 accumulators, register r holds (i = 4*r + l/16, j = l%16).
#include "kmp_common.h"
#include "kmp_kernels.h"

#include <algorithm>
#include <cstdint>

namespace kmp {

typedef double dbl4 __attribute__((ext_vector_type(4)));
typedef double dbl2 __attribute__((ext_vector_type(2)));

constexpr int TN = 64, LPAD = 4;

// Tile geometry: BM x 64 outputs per 256-thread block, K slices of BK.
// Four waves in a 2 x 2 grid; each wave owns (BM/2) x 32 outputs, i.e.
// MB = BM/32 row blocks by 2 column blocks of 16 x 16.
template <int BM, int BK>
struct Tile {
  static constexpr int MB = BM / 32;
  static constexpr int APT = BM * BK / 256;   // A elements per thread per slice
  static constexpr int BPT = BK * TN / 256;   // B elements per thread per slice
};

// Global -> register fetch of one K slice, and register -> LDS store.
// Splitting the two lets the next slice be in flight while the matrix
// cores work on the current one.
// For k-contiguous B (BKC) each thread loads from one column, whose base
// pointer bcol the caller resolves once (null for a column past the end).
//
// VEC: every tile row and K slice lies inside the operands (M >= BM, the
// last row tile moved back to end at M by the caller; the K range a
// multiple of BK; M, leading dimensions and batch strides even and bases
// 16-byte aligned, which the host checks), so each thread's run of
// consecutive elements is read with unchecked 16-byte loads.
template <int BM, int BK, bool AK, bool BKC, bool VEC = false>
__device__ __forceinline__ void fetch_slice(int M, int N, int K, int i0, int j0, int k0,
                                            const double* __restrict__ A, int64_t lda,
                                            const double* __restrict__ B, int64_t ldb,
                                            const double* __restrict__ bcol,
                                            double (&ra)[Tile<BM, BK>::APT],
                                            double (&rb)[Tile<BM, BK>::BPT]) {
  constexpr int APT = Tile<BM, BK>::APT, BPT = Tile<BM, BK>::BPT;
  const int t = threadIdx.x;
  if constexpr (VEC) {
    static_assert(BKC && APT % 2 == 0 && BPT % 2 == 0, "vector fetch: k-contiguous B, pairs");
    const double* pa;
    if (AK) {
      constexpr int TPR = BK / APT;
      pa = A + (int64_t)(i0 + t / TPR) * lda + k0 + (t % TPR) * APT;
    } else {
      constexpr int TPR = BM / APT;
      pa = A + (int64_t)(k0 + t / TPR) * lda + i0 + (t % TPR) * APT;
    }
#pragma unroll
    for (int q = 0; q < APT / 2; ++q) {
      const dbl2 v = *reinterpret_cast<const dbl2*>(pa + 2 * q);
      ra[2 * q] = v.x;
      ra[2 * q + 1] = v.y;
    }
    constexpr int TPRB = BK / BPT;
    const double* pb = bcol ? bcol + k0 + (t % TPRB) * BPT : nullptr;
#pragma unroll
    for (int q = 0; q < BPT / 2; ++q) {
      const dbl2 v = pb ? *reinterpret_cast<const dbl2*>(pb + 2 * q) : dbl2{0.0, 0.0};
      rb[2 * q] = v.x;
      rb[2 * q + 1] = v.y;
    }
    return;
  }
  if (AK) {                       // A[i*lda + k]: threads walk k within a row
    constexpr int TPR = BK / APT;
    const int i = t / TPR, kb = (t % TPR) * APT;
    const int gi = i0 + i;
#pragma unroll
    for (int q = 0; q < APT; ++q) {
      const int gk = k0 + kb + q;
      ra[q] = (gi < M && gk < K) ? A[(int64_t)gi * lda + gk] : 0.0;
    }
  } else {                        // A[k*lda + i]: threads walk i within a k row
    constexpr int TPR = BM / APT;
    const int k = t / TPR, ib = (t % TPR) * APT;
    const int gk = k0 + k;
#pragma unroll
    for (int q = 0; q < APT; ++q) {
      const int gi = i0 + ib + q;
      ra[q] = (gi < M && gk < K) ? A[(int64_t)gk * lda + gi] : 0.0;
    }
  }
  if (BKC) {                      // B[j*ldb + k], column base bcol
    constexpr int TPR = BK / BPT;
    const int kb = (t % TPR) * BPT;
#pragma unroll
    for (int q = 0; q < BPT; ++q) {
      const int gk = k0 + kb + q;
      rb[q] = (bcol && gk < K) ? bcol[gk] : 0.0;
    }
  } else {                        // B[k*ldb + j]
    constexpr int TPR = TN / BPT;
    const int k = t / TPR, jb = (t % TPR) * BPT;
    const int gk = k0 + k;
#pragma unroll
    for (int q = 0; q < BPT; ++q) {
      const int gj = j0 + jb + q;
      rb[q] = (gj < N && gk < K) ? B[(int64_t)gk * ldb + gj] : 0.0;
    }
  }
}

// LDS column of element (k, c) of a staged slice. The columns are permuted
// within aligned groups so that the lanes of one store instruction land in
// distinct banks: a slice fetched along k (RS consecutive k per thread, KC)
// has rows RS apart in one instruction, so bits 2-3 of the column take
// those of k / RS; one fetched along the columns (consecutive columns per
// thread) has columns 4 or more apart, so bits 0-1 take bits 4-5. The
// matrix-core reads (16 consecutive columns of one row per lane group)
// stay conflict free under either permutation.
template <bool KC, int RS>
__device__ __forceinline__ int lds_col(int k, int c) {
  return KC ? c ^ (((k / RS) & 3) << 2) : c ^ ((c >> 4) & 3);
}

template <int BM, int BK, bool AK, bool BKC>
__device__ __forceinline__ void store_slice(const double (&ra)[Tile<BM, BK>::APT],
                                            const double (&rb)[Tile<BM, BK>::BPT],
                                            double (*As)[BM + LPAD], double (*Bs)[TN + LPAD]) {
  constexpr int APT = Tile<BM, BK>::APT, BPT = Tile<BM, BK>::BPT;
  const int t = threadIdx.x;
  if (AK) {
    constexpr int TPR = BK / APT;
    const int i = t / TPR, kb = (t % TPR) * APT;
#pragma unroll
    for (int q = 0; q < APT; ++q) As[kb + q][lds_col<true, APT>(kb + q, i)] = ra[q];
  } else {
    constexpr int TPR = BM / APT;
    const int k = t / TPR, ib = (t % TPR) * APT;
#pragma unroll
    for (int q = 0; q < APT; ++q) As[k][lds_col<false, APT>(k, ib + q)] = ra[q];
  }
  if (BKC) {
    constexpr int TPR = BK / BPT;
    const int j = t / TPR, kb = (t % TPR) * BPT;
#pragma unroll
    for (int q = 0; q < BPT; ++q) Bs[kb + q][lds_col<true, BPT>(kb + q, j)] = rb[q];
  } else {
    constexpr int TPR = TN / BPT;
    const int k = t / TPR, jb = (t % TPR) * BPT;
#pragma unroll
    for (int q = 0; q < BPT; ++q) Bs[k][lds_col<false, BPT>(k, jb + q)] = rb[q];
  }
}

// Matrix-core products of one LDS stage into acc (see tile_mainloop).
template <int BM, int BK, bool AK, bool BKC>
__device__ __forceinline__ void tile_stage_mfma(const double (*As)[BM + LPAD],
                                                const double (*Bs)[TN + LPAD], int wi, int wj,
                                                int li, int lk, bool use1,
                                                dbl4 (&acc)[Tile<BM, BK>::MB][2]) {
  constexpr int MB = Tile<BM, BK>::MB;
  constexpr int APT = Tile<BM, BK>::APT, BPT = Tile<BM, BK>::BPT;
#pragma unroll
  for (int kk = 0; kk < BK; kk += 4) {
    double av[MB];
#pragma unroll
    for (int a = 0; a < MB; ++a)
      av[a] = As[kk + lk][lds_col<AK, APT>(kk + lk, wi + 16 * a + li)];
    const double b0 = Bs[kk + lk][lds_col<BKC, BPT>(kk + lk, wj + li)];
    const double b1 = Bs[kk + lk][lds_col<BKC, BPT>(kk + lk, wj + 16 + li)];
#pragma unroll
    for (int a = 0; a < MB; ++a) {
      acc[a][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[a], b0, acc[a][0], 0, 0, 0);
      if (use1) acc[a][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[a], b1, acc[a][1], 0, 0, 0);
    }
  }
}

// Main loop shared by all variants. acc[bi][bj] covers rows
// wi + 16 bi .., cols wj + 16 bj ... Two LDS stages, one barrier per slice.
// PF = 1: slice k+1 is fetched into registers before the MFMAs on slice k
// and stored into the other stage afterwards. PF = 2: two register sets;
// at the start of step k slice k+1 (fetched two steps earlier) goes to the
// free stage and slice k+3 is fetched into its registers, so every load
// has two steps of matrix work to arrive.
//
// cmap (k-contiguous B only, may be null) maps tile column j0 + j to the
// column cmap[j0 + j] of B; N then counts the mapped columns. A wave skips
// the matrix products of a 16-column block that lies wholly past N (a
// wave-uniform test), so a tile with few columns costs little more than
// its loads.
template <int BM, int BK, bool AK, bool BKC, int PF = 1, bool VEC = false>
__device__ __forceinline__ void tile_mainloop(int M, int N, int kbeg, int K, int i0, int j0,
                                              const double* __restrict__ A, int64_t lda,
                                              const double* __restrict__ B, int64_t ldb,
                                              const int* __restrict__ cmap,
                                              dbl4 (&acc)[Tile<BM, BK>::MB][2]) {
  constexpr int MB = Tile<BM, BK>::MB;
  __shared__ double As[2][BK][BM + LPAD];
  __shared__ double Bs[2][BK][TN + LPAD];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wi = (w & 1) * (BM / 2), wj = (w >> 1) * 32;
  const int li = lane & 15, lk = lane >> 4;
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = dbl4{0.0, 0.0, 0.0, 0.0};
  const double* bcol = nullptr;
  if (BKC) {
    const int gj = j0 + (int)threadIdx.x / (BK / Tile<BM, BK>::BPT);
    if (gj < N) bcol = B + (int64_t)(cmap ? cmap[gj] : gj) * ldb;
  }
  const bool use0 = j0 + wj < N, use1 = j0 + wj + 16 < N;
  const int nk = (K - kbeg + BK - 1) / BK;
  if constexpr (PF == 1) {
    double ra[Tile<BM, BK>::APT], rb[Tile<BM, BK>::BPT];
    fetch_slice<BM, BK, AK, BKC, VEC>(M, N, K, i0, j0, kbeg, A, lda, B, ldb, bcol, ra, rb);
    store_slice<BM, BK, AK, BKC>(ra, rb, As[0], Bs[0]);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      const bool more = kt + 1 < nk;
      if (more)
        fetch_slice<BM, BK, AK, BKC, VEC>(M, N, K, i0, j0, kbeg + (kt + 1) * BK, A, lda, B, ldb, bcol,
                                     ra, rb);
      if (use0) tile_stage_mfma<BM, BK, AK, BKC>(As[cur], Bs[cur], wi, wj, li, lk, use1, acc);
      if (more) store_slice<BM, BK, AK, BKC>(ra, rb, As[cur ^ 1], Bs[cur ^ 1]);
      __syncthreads();
    }
  } else {
    double ra0[Tile<BM, BK>::APT], rb0[Tile<BM, BK>::BPT];
    double ra1[Tile<BM, BK>::APT], rb1[Tile<BM, BK>::BPT];
    fetch_slice<BM, BK, AK, BKC, VEC>(M, N, K, i0, j0, kbeg, A, lda, B, ldb, bcol, ra0, rb0);
    store_slice<BM, BK, AK, BKC>(ra0, rb0, As[0], Bs[0]);
    if (nk > 1) fetch_slice<BM, BK, AK, BKC, VEC>(M, N, K, i0, j0, kbeg + BK, A, lda, B, ldb, bcol, ra0, rb0);
    if (nk > 2)
      fetch_slice<BM, BK, AK, BKC, VEC>(M, N, K, i0, j0, kbeg + 2 * BK, A, lda, B, ldb, bcol, ra1, rb1);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      // even step: slice kt in stage 0, slice kt+1 in (ra0, rb0)
      if (kt + 1 < nk) store_slice<BM, BK, AK, BKC>(ra0, rb0, As[1], Bs[1]);
      if (kt + 3 < nk)
        fetch_slice<BM, BK, AK, BKC, VEC>(M, N, K, i0, j0, kbeg + (kt + 3) * BK, A, lda, B, ldb, bcol,
                                     ra0, rb0);
      if (use0) tile_stage_mfma<BM, BK, AK, BKC>(As[0], Bs[0], wi, wj, li, lk, use1, acc);
      __syncthreads();
      if (kt + 1 >= nk) break;
      // odd step: slice kt+1 in stage 1, slice kt+2 in (ra1, rb1)
      if (kt + 2 < nk) store_slice<BM, BK, AK, BKC>(ra1, rb1, As[0], Bs[0]);
      if (kt + 4 < nk)
        fetch_slice<BM, BK, AK, BKC, VEC>(M, N, K, i0, j0, kbeg + (kt + 4) * BK, A, lda, B, ldb, bcol,
                                     ra1, rb1);
      if (use0) tile_stage_mfma<BM, BK, AK, BKC>(As[1], Bs[1], wi, wj, li, lk, use1, acc);
      __syncthreads();
    }
  }
}

// Main loop of the whole-tile case (VEC above) without a branch around a
// memory access, so that the wait before each LDS store holds only for the
// slice it stores while the next slice's loads stay in flight: the slice
// index of every prefetch is clamped to the last slice (the surplus loads
// re-read it), both LDS stages are written unconditionally (the stage
// written is never the one being read), and a column past N reads column
// cmap[0] (or 0) and is zeroed when stored to LDS. Two register sets, each slice
// fetched two steps before it is stored, as tile_mainloop with PF = 2.
template <int BM, int BK, bool AK>
__device__ __forceinline__ void tile_mainloop_vec(int N, int kbeg, int K, int i0, int j0,
                                                  const double* __restrict__ A, int64_t lda,
                                                  const double* __restrict__ B, int64_t ldb,
                                                  const int* __restrict__ cmap,
                                                  dbl4 (&acc)[Tile<BM, BK>::MB][2]) {
  constexpr int MB = Tile<BM, BK>::MB;
  constexpr int APT = Tile<BM, BK>::APT, BPT = Tile<BM, BK>::BPT;
  __shared__ double As[2][BK][BM + LPAD];
  __shared__ double Bs[2][BK][TN + LPAD];
  const int t = threadIdx.x;
  const int lane = t & 63;
  // the wave index read as a scalar: the column-block tests below are then
  // scalar branches around the matrix products, not lane masks
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wi = (w & 1) * (BM / 2), wj = (w >> 1) * 32;
  const int li = lane & 15, lk = lane >> 4;
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = dbl4{0.0, 0.0, 0.0, 0.0};
  const double* pa;
  if (AK) {
    constexpr int TPR = BK / APT;
    pa = A + (int64_t)(i0 + t / TPR) * lda + kbeg + (t % TPR) * APT;
  } else {
    constexpr int TPR = BM / APT;
    pa = A + (int64_t)(kbeg + t / TPR) * lda + i0 + (t % TPR) * APT;
  }
  const int64_t astep = AK ? BK : (int64_t)BK * lda;    // one slice further along K
  constexpr int TPRB = BK / BPT;
  const int gj = j0 + t / TPRB;
  const bool bact = gj < N;
  const double* pb = B + (int64_t)(cmap ? cmap[bact ? gj : 0] : (bact ? gj : 0)) * ldb + kbeg +
                     (t % TPRB) * BPT;
  const bool use0 = j0 + wj < N, use1 = j0 + wj + 16 < N;
  const int nk = (K - kbeg) / BK;
  dbl2 ra0[APT / 2], rb0[BPT / 2], ra1[APT / 2], rb1[BPT / 2];
  auto fetch = [&](int kt, dbl2 (&ra)[APT / 2], dbl2 (&rb)[BPT / 2]) {
    const int k = min(kt, nk - 1);
    const double* qa = pa + k * astep;
    const double* qb = pb + (int64_t)k * BK;
#pragma unroll
    for (int q = 0; q < APT / 2; ++q) ra[q] = *reinterpret_cast<const dbl2*>(qa + 2 * q);
#pragma unroll
    for (int q = 0; q < BPT / 2; ++q) rb[q] = *reinterpret_cast<const dbl2*>(qb + 2 * q);
  };
  auto store = [&](const dbl2 (&ra)[APT / 2], const dbl2 (&rb)[BPT / 2], double (*Asl)[BM + LPAD],
                   double (*Bsl)[TN + LPAD]) {
    if (AK) {
      constexpr int TPR = BK / APT;
      const int i = t / TPR, kb = (t % TPR) * APT;
#pragma unroll
      for (int q = 0; q < APT; ++q) Asl[kb + q][lds_col<true, APT>(kb + q, i)] = ra[q / 2][q % 2];
    } else {
      constexpr int TPR = BM / APT;
      const int k = t / TPR, ib = (t % TPR) * APT;
#pragma unroll
      for (int q = 0; q < APT; ++q) Asl[k][lds_col<false, APT>(k, ib + q)] = ra[q / 2][q % 2];
    }
    const int j = t / TPRB, kb = (t % TPRB) * BPT;
#pragma unroll
    for (int q = 0; q < BPT; ++q)
      Bsl[kb + q][lds_col<true, BPT>(kb + q, j)] = bact ? rb[q / 2][q % 2] : 0.0;
  };
  if (nk <= 0) return;
  fetch(0, ra0, rb0);
  store(ra0, rb0, As[0], Bs[0]);
  fetch(1, ra0, rb0);
  // keep slice 1's loads older than slice 2's, as in the loop (the waits
  // are counted in issue order)
  __builtin_amdgcn_sched_barrier(0);
  fetch(2, ra1, rb1);
  __syncthreads();
  for (int kt = 0; kt < nk; kt += 2) {
    // even step: slice kt in stage 0, slice kt+1 in (ra0, rb0)
    store(ra0, rb0, As[1], Bs[1]);
    fetch(kt + 3, ra0, rb0);
    if (use0) tile_stage_mfma<BM, BK, AK, true>(As[0], Bs[0], wi, wj, li, lk, use1, acc);
    __syncthreads();
    if (kt + 1 >= nk) break;
    // odd step: slice kt+1 in stage 1, slice kt+2 in (ra1, rb1)
    store(ra1, rb1, As[0], Bs[0]);
    fetch(kt + 4, ra1, rb1);
    if (use0) tile_stage_mfma<BM, BK, AK, true>(As[1], Bs[1], wi, wj, li, lk, use1, acc);
    __syncthreads();
  }
}

template <int BM, int BK, bool AK, bool BKC, bool CR>
__global__ __launch_bounds__(256) void dgemm_kernel(int M, int N, int K,
                                                     const double* __restrict__ A, int64_t lda, int64_t sA,
                                                     const double* __restrict__ B, int64_t ldb, int64_t sB,
                                                     double* __restrict__ C, int64_t ldc, int64_t sC,
                                                     double alpha, double beta) {
  constexpr int MB = Tile<BM, BK>::MB;
  const int b = blockIdx.z;
  A += (int64_t)b * sA;
  B += (int64_t)b * sB;
  C += (int64_t)b * sC;
  const int i0 = blockIdx.x * BM, j0 = blockIdx.y * TN;
  dbl4 acc[MB][2];
  tile_mainloop<BM, BK, AK, BKC>(M, N, 0, K, i0, j0, A, lda, B, ldb, nullptr, acc);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wi = (w & 1) * (BM / 2), wj = (w >> 1) * 32;
#pragma unroll
  for (int bi = 0; bi < MB; ++bi)
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
// B = T abar column-major, C = Z column-major). The per-tile column sums
// of z are written to partial[b][tile][c] (BM rows per tile).
template <int BM, int BK>
__global__ __launch_bounds__(256) void dgemm_loss_kernel(int M, int N, int K,
                                                          const double* __restrict__ A, int64_t lda, int64_t sA,
                                                          const double* __restrict__ B, int64_t ldb, int64_t sB,
                                                          double* __restrict__ C, int64_t ldc, int64_t sC,
                                                          LossEpi e) {
  constexpr int MB = Tile<BM, BK>::MB;
  __shared__ double red[4][32];
  const int b = blockIdx.z;
  A += (int64_t)b * sA;
  B += (int64_t)b * sB;
  C += (int64_t)b * sC;
  const int i0 = blockIdx.x * BM, j0 = blockIdx.y * TN;
  dbl4 acc[MB][2];
  tile_mainloop<BM, BK, true, true>(M, N, 0, K, i0, j0, A, lda, B, ldb, nullptr, acc);
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wi = (w & 1) * (BM / 2), wj = (w >> 1) * 32;
  const int nv = e.nv[b];
  const double* y = e.y + (int64_t)b * e.sy;
  const double* bbar = e.bbar + (int64_t)b * e.sbb;
  const double* tau = e.tau + (int64_t)b * e.stau;
  const int* cnv = e.cnv + (int64_t)b * e.sbb;
  const int32_t* rfold = e.rfold ? e.rfold + (int64_t)b * e.sy : nullptr;
  const int32_t* cfold = e.cfold ? e.cfold + (int64_t)b * e.sbb : nullptr;
  double colsum[2] = {0.0, 0.0};
#pragma unroll
  for (int bj = 0; bj < 2; ++bj) {
    const int gj = j0 + wj + bj * 16 + mfma_col(lane);
    const bool cj = gj < N;
    const double bb = cj ? bbar[gj] : 0.0;
    const double tj = cj ? tau[gj] : 0.0;
    const double inv_nv = cj ? 1.0 / (double)cnv[gj] : 0.0;
    const int32_t hf = (cj && cfold) ? cfold[gj] : -1;
#pragma unroll
    for (int bi = 0; bi < MB; ++bi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = i0 + wi + bi * 16 + mfma_row(lane, r);
        if (gi < M && cj) {
          double z = 0.0;
          if (gi < nv && !(rfold && rfold[gi] == hf))
            z = loss_psi(e.loss, y[gi], acc[bi][bj][r] + bb, e.delta, tj) * inv_nv;
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

// Split-K partial products for the path GEMMs: block z = b * S + s computes
// the K range [s*Kc, min(K, (s+1)*Kc)) of batch b and stores its BM x 64
// tile of A B (column-major, ldc) into part + s*sP + b*sC. The S partials
// are added later in a fixed order, so results do not depend on timing.
// Only the active columns of a batch are computed: tile column k < nact[b]
// is column cmap[b*cstride + k] of B and of the partials (the other columns
// of the partials are left as they were); tiles past nact[b] exit at once.
// With IDENT (cmap and nact null), all cstride columns, in order.
template <int BM, int BK, bool AK, bool IDENT, int PF = 1, bool VEC = false>
__global__ __launch_bounds__(256) void dgemm_partial_kernel(int M, int K, int S, int Kc,
                                                             const double* __restrict__ A, int64_t lda, int64_t sA,
                                                             const double* __restrict__ B, int64_t ldb, int64_t sB,
                                                             double* __restrict__ part, int64_t ldc, int64_t sC,
                                                             int64_t sP, const int* __restrict__ cmap_all,
                                                             const int* __restrict__ nact, int cstride) {
  constexpr int MB = Tile<BM, BK>::MB;
  const int b = blockIdx.z / S, sk = blockIdx.z % S;
  const int N = IDENT ? cstride : nact[b];
  const int i0 = blockIdx.x * BM, j0 = blockIdx.y * TN;
  if (j0 >= N) return;
  const int* cmap = IDENT ? nullptr : cmap_all + (int64_t)b * cstride;
  A += (int64_t)b * sA;
  B += (int64_t)b * sB;
  double* C = part + (int64_t)sk * sP + (int64_t)b * sC;
  const int kbeg = sk * Kc;
  const int kend = min(K, kbeg + Kc);
  // whole-tile path: a last row tile that would reach past M is moved back
  // to end at M (M >= BM) and stores only its own rows
  const int il = VEC ? min(i0, M - BM) : i0;
  dbl4 acc[MB][2];
  if (kbeg < kend) {
    if constexpr (VEC)
      tile_mainloop_vec<BM, BK, AK>(N, kbeg, kend, il, j0, A, lda, B, ldb, cmap, acc);
    else
      tile_mainloop<BM, BK, AK, true, PF>(M, N, kbeg, kend, i0, j0, A, lda, B, ldb, cmap, acc);
  } else {
#pragma unroll
    for (int a = 0; a < MB; ++a) acc[a][0] = acc[a][1] = dbl4{0.0, 0.0, 0.0, 0.0};
  }
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wi = (w & 1) * (BM / 2), wj = (w >> 1) * 32;
#pragma unroll
  for (int bi = 0; bi < MB; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = il + wi + bi * 16 + mfma_row(lane, r);
        const int gj = j0 + wj + bj * 16 + mfma_col(lane);
        if (gi >= i0 && gi < M && gj < N) C[(int64_t)(IDENT ? gj : cmap[gj]) * ldc + gi] = acc[bi][bj][r];
      }
}

// The same split-K partial products with the four waves of a workgroup
// stacked by rows: wave w owns rows (BM/4) w .. of a BM x TW tile and all
// TW/16 of its column blocks, so that an A operand read from LDS serves
// TW/16 products (two in the 2 x 2 arrangement above) and, with 64 or fewer
// active columns, every wave has the same share of the products (in the
// 2 x 2 arrangement the waves of the second 32 columns idle while a batch
// has 32 or fewer, and do half the products at 33 to 48). Two shapes:
//  - 64 x 128 while most active columns are in batches with 65 to 128
//    of them (and none has more): such a batch's columns take one tile
//    instead of two, each A row tile being streamed once;
//  - 128 x 64 otherwise (M >= 128).
// Whole-tile path only (the conditions of VEC above); the main loop has no
// branch around a memory access, as in tile_mainloop_vec. Measured at 10
// groups of order 9024 (split-K 4, both operand orders): 100 active
// columns each, 64 x 128 3.2 ms against 3.5-3.8 ms for the 2 x 2 64 x 64
// tile in the same runs; 30 columns each, 128 x 64 1.6 ms against 1.8 ms;
// 12 each 1.2 against 1.26; 60 each equal. Each output element takes the
// same products in the same order as in dgemm_partial_kernel.
template <int BM, int TW, bool AK>
__global__ __launch_bounds__(256) void dgemm_partial_rows_kernel(int M, int K, int S, int Kc,
                                                                  const double* __restrict__ A, int64_t lda, int64_t sA,
                                                                  const double* __restrict__ B, int64_t ldb, int64_t sB,
                                                                  double* __restrict__ part, int64_t ldc, int64_t sC,
                                                                  int64_t sP, const int* __restrict__ cmap_all,
                                                                  const int* __restrict__ nact, int cstride) {
  constexpr int BK = 16, MB = BM / 64, NB = TW / 16;
  constexpr int APT = BM * BK / 256, BPT = BK * TW / 256;   // per thread and slice
  __shared__ double As[2][BK][BM + LPAD];
  __shared__ double Bs[2][BK][TW + LPAD];
  const int b = blockIdx.z / S, sk = blockIdx.z % S;
  const int N = nact[b];
  const int i0 = blockIdx.x * BM, j0 = blockIdx.y * TW;
  if (j0 >= N) return;
  const int* cmap = cmap_all + (int64_t)b * cstride;
  A += (int64_t)b * sA;
  B += (int64_t)b * sB;
  double* C = part + (int64_t)sk * sP + (int64_t)b * sC;
  const int kbeg = sk * Kc;
  const int kend = min(K, kbeg + Kc);
  // a last row tile that would reach past M is moved back to end at M
  const int il = min(i0, M - BM);
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wi = (BM / 4) * w;
  const int li = lane & 15, lk = lane >> 4;
  const int nblk = max(0, min(NB, (N - j0 + 15) / 16));   // blocks holding active columns
  dbl4 acc[MB][NB];
#pragma unroll
  for (int x = 0; x < MB; ++x)
#pragma unroll
    for (int y = 0; y < NB; ++y) acc[x][y] = dbl4{0.0, 0.0, 0.0, 0.0};
  const double* pa;
  if (AK) {
    constexpr int TPR = BK / APT;
    pa = A + (int64_t)(il + t / TPR) * lda + kbeg + (t % TPR) * APT;
  } else {
    constexpr int TPR = BM / APT;
    pa = A + (int64_t)(kbeg + t / TPR) * lda + il + (t % TPR) * APT;
  }
  const int64_t astep = AK ? BK : (int64_t)BK * lda;
  constexpr int TPRB = BK / BPT;
  const int gj = j0 + t / TPRB;
  const bool bact = gj < N;
  const double* pb = B + (int64_t)cmap[bact ? gj : 0] * ldb + kbeg + (t % TPRB) * BPT;
  const int nk = (kend - kbeg) / BK;
  dbl2 ra0[APT / 2], rb0[BPT / 2], ra1[APT / 2], rb1[BPT / 2];
  auto fetch = [&](int kt, dbl2 (&ra)[APT / 2], dbl2 (&rb)[BPT / 2]) {
    const int k = min(kt, nk - 1);
    const double* qa = pa + k * astep;
    const double* qb = pb + (int64_t)k * BK;
#pragma unroll
    for (int q = 0; q < APT / 2; ++q) ra[q] = *reinterpret_cast<const dbl2*>(qa + 2 * q);
#pragma unroll
    for (int q = 0; q < BPT / 2; ++q) rb[q] = *reinterpret_cast<const dbl2*>(qb + 2 * q);
  };
  auto store = [&](const dbl2 (&ra)[APT / 2], const dbl2 (&rb)[BPT / 2], double (*Asl)[BM + LPAD],
                   double (*Bsl)[TW + LPAD]) {
    if (AK) {
      constexpr int TPR = BK / APT;
      const int i = t / TPR, kb = (t % TPR) * APT;
#pragma unroll
      for (int q = 0; q < APT; ++q) Asl[kb + q][lds_col<true, APT>(kb + q, i)] = ra[q / 2][q % 2];
    } else {
      constexpr int TPR = BM / APT;
      const int k = t / TPR, ib = (t % TPR) * APT;
#pragma unroll
      for (int q = 0; q < APT; ++q) Asl[k][lds_col<false, APT>(k, ib + q)] = ra[q / 2][q % 2];
    }
    const int j = t / TPRB, kb = (t % TPRB) * BPT;
#pragma unroll
    for (int q = 0; q < BPT; ++q)
      Bsl[kb + q][lds_col<true, BPT>(kb + q, j)] = bact ? rb[q / 2][q % 2] : 0.0;
  };
  auto products = [&](const double (*Asl)[BM + LPAD], const double (*Bsl)[TW + LPAD]) {
#pragma unroll
    for (int kk = 0; kk < BK; kk += 4) {
      double av[MB], bv[NB];
#pragma unroll
      for (int x = 0; x < MB; ++x) av[x] = Asl[kk + lk][lds_col<AK, APT>(kk + lk, wi + 16 * x + li)];
#pragma unroll
      for (int y = 0; y < NB; ++y) bv[y] = Bsl[kk + lk][lds_col<true, BPT>(kk + lk, 16 * y + li)];
#pragma unroll
      for (int y = 0; y < NB; ++y)
        if (y < nblk)
#pragma unroll
          for (int x = 0; x < MB; ++x)
            acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[x], bv[y], acc[x][y], 0, 0, 0);
    }
  };
  if (nk > 0) {
    fetch(0, ra0, rb0);
    store(ra0, rb0, As[0], Bs[0]);
    fetch(1, ra0, rb0);
    // keep slice 1's loads older than slice 2's (the waits count in issue order)
    __builtin_amdgcn_sched_barrier(0);
    fetch(2, ra1, rb1);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      store(ra0, rb0, As[1], Bs[1]);
      fetch(kt + 3, ra0, rb0);
      products(As[0], Bs[0]);
      __syncthreads();
      if (kt + 1 >= nk) break;
      store(ra1, rb1, As[0], Bs[0]);
      fetch(kt + 4, ra1, rb1);
      products(As[1], Bs[1]);
      __syncthreads();
    }
  }
#pragma unroll
  for (int x = 0; x < MB; ++x)
#pragma unroll
    for (int y = 0; y < NB; ++y)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gi = il + wi + 16 * x + mfma_row(lane, r);
        const int gc = j0 + 16 * y + mfma_col(lane);
        if (gi >= i0 && gi < M && gc < N) C[(int64_t)cmap[gc] * ldc + gi] = acc[x][y][r];
      }
}

// Loss epilogue over split-K partials of f: for row i < M of batch b and
// active column c = cmap[b*N + k], k < nact[b], F = sum_s part_s[c][i] +
// bbar[c]; Z[c][i] = psi(y_i, F)/cnv[c] (0 at padding rows and at rows held
// out of column c); partial[b][tile][c]
// = sum of Z over the 64 rows of the tile (lanes = rows, so the column sums
// are wave reductions). Wave w of workgroup (tile, j, b) takes the active
// column k = 4 j + w.
__global__ __launch_bounds__(256) void loss_epilogue_kernel(int M, int N, int S,
                                                             const double* __restrict__ part,
                                                             int64_t ldc, int64_t sC, int64_t sP,
                                                             double* __restrict__ Z, LossEpi e,
                                                             const int* __restrict__ cmap_all,
                                                             const int* __restrict__ nact) {
  const int b = blockIdx.z;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int i = blockIdx.x * 64 + lane;
  const int nv = e.nv[b];
  const double yi = (i < nv) ? e.y[(int64_t)b * e.sy + i] : 0.0;
  const int32_t fi = (e.rfold && i < nv) ? e.rfold[(int64_t)b * e.sy + i] : -2;
  const double* bbar = e.bbar + (int64_t)b * e.sbb;
  const double* tau = e.tau + (int64_t)b * e.stau;
  const int* cmap = cmap_all + (int64_t)b * N;
  const int k = 4 * (int)blockIdx.y + w;
  if (k < nact[b]) {
    const int c = cmap[k];
    const double inv_nv = 1.0 / (double)e.cnv[(int64_t)b * e.sbb + c];
    const bool held = e.cfold && fi == e.cfold[(int64_t)b * e.sbb + c];
    double z = 0.0;
    if (i < M) {
      double f = 0.0;
      for (int sk = 0; sk < S; ++sk) f += part[(int64_t)sk * sP + (int64_t)b * sC + (int64_t)c * ldc + i];
      if (i < nv && !held) z = loss_psi(e.loss, yi, f + bbar[c], e.delta, tau[c]) * inv_nv;
      Z[(int64_t)b * sC + (int64_t)c * ldc + i] = z;
    }
    const double cs = wave_sum(z);
    if (lane == 0) e.partial[(int64_t)b * e.spart + (int64_t)blockIdx.x * N + c] = cs;
  }
}

// Output tiles of 64 rows unless that leaves the chip under-filled (fewer
// than two blocks per compute unit), then 32.
static int pick_bm(const GemmArgs& g) {
  const int64_t tiles64 = ceil_div(g.M, 64) * ceil_div(g.N, TN) * g.batch;
  return tiles64 < 512 ? 32 : 64;
}

int gemm(hipStream_t s, const GemmArgs& g, bool ak, bool bk, bool cr) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return 0;
  const int bm = pick_bm(g);
  dim3 grid((unsigned)ceil_div(g.M, bm), (unsigned)ceil_div(g.N, TN), (unsigned)g.batch);
  dim3 block(256);
#define KMP_GEMM_CASE(BMV, a, b, c)                                                          \
  if (bm == BMV && ak == a && bk == b && cr == c) {                                          \
    hipLaunchKernelGGL((dgemm_kernel<BMV, 32, a, b, c>), grid, block, 0, s, g.M, g.N, g.K, g.A, \
                       g.lda, g.sA, g.B, g.ldb, g.sB, g.C, g.ldc, g.sC, g.alpha, g.beta);     \
    KMP_LAUNCH_CHECK();                                                                      \
    return 0;                                                                                \
  }
#define KMP_GEMM_CASES(BMV)                \
  KMP_GEMM_CASE(BMV, true, true, true)     \
  KMP_GEMM_CASE(BMV, true, true, false)    \
  KMP_GEMM_CASE(BMV, true, false, true)    \
  KMP_GEMM_CASE(BMV, true, false, false)   \
  KMP_GEMM_CASE(BMV, false, true, true)    \
  KMP_GEMM_CASE(BMV, false, true, false)   \
  KMP_GEMM_CASE(BMV, false, false, true)   \
  KMP_GEMM_CASE(BMV, false, false, false)
  KMP_GEMM_CASES(32)
  KMP_GEMM_CASES(64)
#undef KMP_GEMM_CASES
#undef KMP_GEMM_CASE
  return KMP_EINVAL;
}

int gemm_loss_tile_rows(const GemmArgs& g) { return pick_bm(g); }

// Compute units of the current device (queried once per device).
static int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
      n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

// Split-K parts for dgemm_partial_kernel: the S that minimises the rounds
// of resident workgroups (per_cu per compute unit: four for the 64 x 64
// tile, bound by LDS; three for the 64 x 128 one) times the K
// range per part, over the tiles that do work (tiles <= 0: all of them);
// ties go to the larger S (the finer workgroups balance better: with 10
// groups of order 9024 and 100 columns each, the smallest S among ties ran
// 4 % slower). Each part keeps at least 2 slices
// of 16: at small orders the K loop is a short dependent chain, and at
// order 192 four parts instead of one took the iteration from 35.5 to
// 28.1 us.
int splitk_parts(const GemmArgs& g, int64_t tiles, int per_cu) {
  if (tiles <= 0) tiles = ceil_div(g.M, 64) * ceil_div(g.N, TN) * g.batch;
  const int64_t slots = (int64_t)per_cu * device_cus();
  int best = 1;
  int64_t best_cost = -1;
  for (int S = 1; S <= kMaxSplitK; ++S) {
    if (S > 1 && g.K / S < 2 * 16) break;
    const int64_t cost = ceil_div(tiles * S, slots) * ceil_div(g.K, S);
    if (best_cost < 0 || cost <= best_cost) { best = S; best_cost = cost; }
  }
  return best;
}

// The stacked-row tiles were measured at order 9024 only, so smaller
// orders keep the 2 x 2 tile.
PartTile pick_part_tile(int M, int G, int C, const int* na, int64_t* tiles, int* per_cu) {
  int64_t t64 = 0, tw = 0, tt = 0, cwide = 0, cnarrow = 0;
  bool wide = C > 64;
  for (int g = 0; g < G; ++g) {
    const int n = na ? na[g] : C;
    t64 += ceil_div(M, 64) * ceil_div(n, 64);
    tw += ceil_div(M, 64) * ceil_div(n, 128);
    tt += ceil_div(M, 128) * ceil_div(n, 64);
    if (n > 128) wide = false;
    (n > 64 ? cwide : cnarrow) += n;
  }
  // the 64 x 128 tile while most active columns are in groups of 65 to 128
  if (cwide <= cnarrow) wide = false;
  if (M < 4096 || t64 == 0) {
    *tiles = t64;
    *per_cu = 4;
    return PartTile::k64x64;
  }
  *per_cu = 3;
  *tiles = wide ? tw : tt;
  return wide ? PartTile::k64x128 : PartTile::k128x64;
}

int gemm_partial(hipStream_t s, const GemmArgs& g, bool a_kcontig, int S, double* part, int64_t sP,
                 const int* cmap, const int* nact, PartTile tile) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return 0;
  const int Kc = (int)round_up(ceil_div(g.K, S), 16);
  dim3 grid((unsigned)ceil_div(g.M, 64), (unsigned)ceil_div(g.N, TN), (unsigned)(g.batch * S));
  const bool ident = cmap == nullptr;
  if (ident != (nact == nullptr)) {
    set_error("gemm_partial: cmap and nact must both be given or both be null");
    return KMP_EINVAL;
  }
  // whole K slices, at least one row tile and 16-byte aligned operands:
  // unchecked vector loads (a ragged last row tile is moved back in the kernel)
  const bool vec = g.M >= 64 && g.M % 2 == 0 && g.K % 16 == 0 && g.lda % 2 == 0 && g.ldb % 2 == 0 &&
                   g.sA % 2 == 0 && g.sB % 2 == 0 && (reinterpret_cast<uintptr_t>(g.A) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(g.B) & 15) == 0;
  if (tile != PartTile::k64x64 && vec && !ident && g.M >= 128) {
    const bool w = tile == PartTile::k64x128;
    grid.x = (unsigned)ceil_div(g.M, w ? 64 : 128);
    grid.y = (unsigned)ceil_div(g.N, w ? 128 : 64);
#define KMP_ROWS_CASE(BMV, TWV, AKV)                                                              \
  hipLaunchKernelGGL((dgemm_partial_rows_kernel<BMV, TWV, AKV>), grid, dim3(256), 0, s, g.M, g.K, S, \
                     Kc, g.A, g.lda, g.sA, g.B, g.ldb, g.sB, part, g.ldc, g.sC, sP, cmap, nact, g.N)
    if (w && a_kcontig) KMP_ROWS_CASE(64, 128, true);
    else if (w) KMP_ROWS_CASE(64, 128, false);
    else if (a_kcontig) KMP_ROWS_CASE(128, 64, true);
    else KMP_ROWS_CASE(128, 64, false);
#undef KMP_ROWS_CASE
    KMP_LAUNCH_CHECK();
    return 0;
  }
#define KMP_PART_CASE(AKV, IDV, VV)                                                              \
  if (a_kcontig == AKV && ident == IDV && vec == VV)                                             \
    hipLaunchKernelGGL((dgemm_partial_kernel<64, 16, AKV, IDV, 2, VV>), grid, dim3(256), 0, s, g.M, \
                       g.K, S, Kc, g.A, g.lda, g.sA, g.B, g.ldb, g.sB, part, g.ldc, g.sC, sP, cmap, \
                       nact, g.N);
  KMP_PART_CASE(true, false, true)
  KMP_PART_CASE(false, false, true)
  KMP_PART_CASE(true, true, true)
  KMP_PART_CASE(false, true, true)
  KMP_PART_CASE(true, false, false)
  KMP_PART_CASE(false, false, false)
  KMP_PART_CASE(true, true, false)
  KMP_PART_CASE(false, true, false)
#undef KMP_PART_CASE
  KMP_LAUNCH_CHECK();
  return 0;
}

int loss_epilogue(hipStream_t s, int M, int N, int batch, int S, const double* part, int64_t ldc,
                  int64_t sC, int64_t sP, double* Z, const LossEpi& e, const int* cmap,
                  const int* nact) {
  if (M <= 0 || N <= 0 || batch <= 0) return 0;
  dim3 grid((unsigned)ceil_div(M, 64), (unsigned)ceil_div(N, 4), (unsigned)batch);
  hipLaunchKernelGGL(loss_epilogue_kernel, grid, dim3(256), 0, s, M, N, S, part, ldc, sC, sP, Z, e,
                     cmap, nact);
  KMP_LAUNCH_CHECK();
  return 0;
}

int gemm_loss(hipStream_t s, const GemmArgs& g, const LossEpi& e) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return 0;
  const int bm = pick_bm(g);
  dim3 grid((unsigned)ceil_div(g.M, bm), (unsigned)ceil_div(g.N, TN), (unsigned)g.batch);
  if (bm == 32)
    hipLaunchKernelGGL((dgemm_loss_kernel<32, 32>), grid, dim3(256), 0, s, g.M, g.N, g.K, g.A,
                       g.lda, g.sA, g.B, g.ldb, g.sB, g.C, g.ldc, g.sC, e);
  else
    hipLaunchKernelGGL((dgemm_loss_kernel<64, 32>), grid, dim3(256), 0, s, g.M, g.N, g.K, g.A,
                       g.lda, g.sA, g.B, g.ldb, g.sB, g.C, g.ldc, g.sC, e);
  KMP_LAUNCH_CHECK();
  return 0;
}

}  // namespace kmp
