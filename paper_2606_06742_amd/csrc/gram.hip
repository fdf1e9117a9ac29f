// Gram + fold gather: RBF kernel blocks written straight into per-fold
// matrices. The inner products x_r . x_c are an fp64 MFMA contraction over
// the feature dimension; the epilogue forms the squared distance by the norm
// expansion |x_r|^2 + |x_c|^2 - 2 x_r.x_c (clamped at 0) and applies
// exp(-dist^2 / (2 sigma^2)) for every requested bandwidth, so one distance
// tile feeds all bandwidths. Diagonal entries (same point) are exactly 1,
// padding entries (negative index) exactly 0.
#include "kmp_common.h"
#include "kmp_kernels.h"

namespace kmp {

typedef double dbl4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void row_norms_kernel(const double* __restrict__ X, int64_t n,
                                                         int64_t d, int64_t ldx, double* __restrict__ nrm) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const double* x = X + i * ldx;
  double s = 0.0;
  for (int64_t k = 0; k < d; ++k) s = fma(x[k], x[k], s);
  nrm[i] = s;
}

int row_norms(hipStream_t s, const double* X, int64_t n, int64_t d, int64_t ldx, double* nrm) {
  if (n <= 0) return 0;
  hipLaunchKernelGGL(row_norms_kernel, dim3((unsigned)ceil_div(n, 256)), dim3(256), 0, s, X, n, d,
                     ldx, nrm);
  KMP_LAUNCH_CHECK();
  return 0;
}

// out[0] = number of non-finite entries of X (n x d, ldx), out[1] = of y;
// one workgroup (16 wavefronts: rows over waves, columns over lanes), fixed
// order, no atomics.
__global__ __launch_bounds__(1024) void count_nonfinite_kernel(const double* __restrict__ X,
                                                                int64_t n, int64_t d, int64_t ldx,
                                                                const double* __restrict__ y,
                                                                int* __restrict__ out) {
  __shared__ double red[2][16];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double cx = 0.0, cy = 0.0;
  for (int64_t i = w; i < n; i += 16) {
    const double* xr = X + i * ldx;
    for (int64_t k = lane; k < d; k += 64) cx += isfinite(xr[k]) ? 0.0 : 1.0;
  }
  for (int64_t i = threadIdx.x; i < n; i += 1024) cy += isfinite(y[i]) ? 0.0 : 1.0;
  cx = wave_sum(cx);
  cy = wave_sum(cy);
  if (lane == 0) {
    red[0][w] = cx;
    red[1][w] = cy;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    double c = 0.0;
    for (int q = 0; q < 16; ++q) c += red[threadIdx.x][q];
    out[threadIdx.x] = (int)c;
  }
}

int count_nonfinite(hipStream_t s, const double* X, int64_t n, int64_t d, int64_t ldx,
                    const double* y, int* out) {
  hipLaunchKernelGGL(count_nonfinite_kernel, dim3(1), dim3(1024), 0, s, X, n, d, ldx, y, out);
  KMP_LAUNCH_CHECK();
  return 0;
}

constexpr int GT = 64, GK = 16, GPAD = 4, MAXS = 8;

__global__ __launch_bounds__(256) void rbf_blocks_kernel(
    const double* __restrict__ X, int64_t d, int64_t ldx, const double* __restrict__ nrm,
    const int32_t* __restrict__ idx_r, int64_t sr, int64_t m, const int32_t* __restrict__ idx_c,
    int64_t sc, int64_t p, const double* __restrict__ inv2s2, int S, double* __restrict__ out,
    int64_t sout_s, int64_t sout_q, int64_t ld) {
  __shared__ double As[GK][GT + GPAD];
  __shared__ double Bs[GK][GT + GPAD];
  __shared__ int32_t ri[GT], ci[GT];
  const int q = blockIdx.z;
  const int64_t i0 = (int64_t)blockIdx.x * GT, j0 = (int64_t)blockIdx.y * GT;
  const int t = threadIdx.x;
  if (t < GT) {
    const int64_t gi = i0 + t;
    ri[t] = gi < m ? idx_r[q * sr + gi] : -1;
  } else if (t < 2 * GT) {
    const int64_t gj = j0 + (t - GT);
    ci[t - GT] = gj < p ? idx_c[q * sc + gj] : -1;
  }
  const int lane = t & 63, w = t >> 6;
  const int wi = (w & 1) * 32, wj = (w >> 1) * 32;
  const int li = lane & 15, lk = lane >> 4;
  dbl4 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = dbl4{0.0, 0.0, 0.0, 0.0};
  for (int64_t k0 = 0; k0 < d; k0 += GK) {
    __syncthreads();
    {
      const int r = t >> 2, kb = (t & 3) * 4;
      const int32_t xr = ri[r], xc = ci[r];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t gk = k0 + kb + u;
        As[kb + u][r] = (xr >= 0 && gk < d) ? X[(int64_t)xr * ldx + gk] : 0.0;
        Bs[kb + u][r] = (xc >= 0 && gk < d) ? X[(int64_t)xc * ldx + gk] : 0.0;
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GK; kk += 4) {
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
  __syncthreads();
  double f2[MAXS];
  for (int s = 0; s < S; ++s) f2[s] = inv2s2[s];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int li2 = wi + bi * 16 + mfma_row(lane, r);
        const int lj2 = wj + bj * 16 + mfma_col(lane);
        const int64_t gi = i0 + li2, gj = j0 + lj2;
        if (gi >= m || gj >= p) continue;
        const int32_t xr = ri[li2], xc = ci[lj2];
        double dist2 = 0.0;
        if (xr >= 0 && xc >= 0) {
          dist2 = nrm[xr] + nrm[xc] - 2.0 * acc[bi][bj][r];
          dist2 = dist2 > 0.0 ? dist2 : 0.0;
        }
        double* o = out + (int64_t)q * sout_q + gi * ld + gj;
        for (int s = 0; s < S; ++s) {
          double v;
          if (xr < 0 || xc < 0) v = 0.0;
          else if (xr == xc) v = 1.0;
          else v = exp(-dist2 * f2[s]);
          o[(int64_t)s * sout_s] = v;
        }
      }
}

// out[i] = a.v[i] for i < count (small parameter arrays written without a
// host-to-device copy: the values travel as a kernel argument).
__global__ void store_small_kernel(Small8 a, int count, double* __restrict__ out) {
  const int i = threadIdx.x;
  if (i < count) out[i] = a.v[i];
}

int store_small(hipStream_t s, const double* vals, int count, double* out) {
  if (count < 0 || count > 8) {
    set_error("store_small: at most 8 values");
    return KMP_EINVAL;
  }
  Small8 a{};
  for (int i = 0; i < count; ++i) a.v[i] = vals[i];
  hipLaunchKernelGGL(store_small_kernel, dim3(1), dim3(64), 0, s, a, count, out);
  KMP_LAUNCH_CHECK();
  return 0;
}

int rbf_blocks(hipStream_t s, const double* X, int64_t d, int64_t ldx, const double* nrm,
               const int32_t* idx_r, int64_t sr, int64_t m, const int32_t* idx_c, int64_t sc,
               int64_t p, int nb, const double* inv2s2, int S, double* out, int64_t sout_s,
               int64_t sout_q, int64_t ld) {
  if (m <= 0 || p <= 0 || nb <= 0) return 0;
  if (S < 1 || S > MAXS) {
    set_error("rbf_blocks: at most 8 bandwidths per launch");
    return KMP_EINVAL;
  }
  dim3 grid((unsigned)ceil_div(m, GT), (unsigned)ceil_div(p, GT), (unsigned)nb);
  hipLaunchKernelGGL(rbf_blocks_kernel, grid, dim3(256), 0, s, X, d, ldx, nrm, idx_r, sr, m, idx_c,
                     sc, p, inv2s2, S, out, sout_s, sout_q, ld);
  KMP_LAUNCH_CHECK();
  return 0;
}

}  // namespace kmp
