// Per-fold factorisation K_v = Q T Q' (T symmetric tridiagonal, Q orthogonal).
//
// The paper factorises the kernel matrix once and reuses the factor for
// every lambda (Appendix A.3, one eigendecomposition). Here the one-time
// factorisation is the Householder reduction to tridiagonal form (Golub &
// Van Loan, Matrix Computations, Alg. 8.3.1), blocked as in LAPACK dsytrd /
// dlatrd: within a panel of nb columns only the current column is brought up
// to date; the symmetric rank-2nb update of the trailing matrix is deferred
// to one matrix-core GEMM per panel. The resolvent (2 lambda I + K/(n kappa))
// is then applied through T by a tridiagonal solve, which is exactly the
// spectral formula with the eigenvectors of T folded in.
//
// All G matrices of a batch advance together (blockIdx selects the matrix).
// Storage per matrix: A (N x N row-major, symmetric, full storage). After
// step j, row j of A holds the Householder vector v_j (v_j[i] = 0 for i <= j,
// v_j[j+1] = 1), which the compact-WY accumulation of Q reads back.
#include "kmp_common.h"
#include "kmp_kernels.h"

#include <algorithm>

namespace kmp {

constexpr int TB = 512;   // threads per block of the one-workgroup-per-matrix kernels
constexpr int TW = 8;     // waves per block

// One workgroup per matrix. Step j of the panel starting at p (jj = j - p):
//  1. (jj > 0) finish w_{jj-1} = w_raw - (tau/2)(w_raw' v) v   (dlatrd)
//  2. bring column j up to date with the panel's rank-2 updates
//  3. Householder vector of column j below the diagonal (dlarfg)
//  4. dot products W_k'v, V_k'v (k < jj) for the symv corrections; the
//     V_k'v are also the panel's Gram entries, kept for the WY factor
// Loops over k are unrolled with independent accumulators so that many
// loads are in flight (the panel rows live in L2).
__global__ __launch_bounds__(TB) void tri_col_kernel(double* __restrict__ A, double* __restrict__ P,
                                                     double* __restrict__ dots,
                                                     double* __restrict__ taus,
                                                     double* __restrict__ diag,
                                                     double* __restrict__ off,
                                                     double* __restrict__ pgram, int N, int nb, int j,
                                                     int jj) {
  __shared__ double red[TW];
  __shared__ double sh[2];
  __shared__ double coef[128];
  const int g = blockIdx.x;
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  double* Ag = A + (int64_t)g * N * N;
  double* Pg = P + (int64_t)g * 3 * nb * N;
  double* Vr = Pg;                    // rows 0..nb-1   : v_k
  double* Wr = Pg + (int64_t)nb * N;  // rows nb..2nb-1 : w_k
  double* V2 = Pg + (int64_t)2 * nb * N;
  double* dg = dots + (int64_t)g * 2 * nb;
  const double* tg = taus + (int64_t)g * N;
  const int p0 = j - jj;
  double* gr = pgram + (int64_t)g * N * nb + (int64_t)p0 * nb;   // this panel's nb x nb Gram

  // 1. finish the previous w (its v has support rows >= j)
  if (jj > 0) {
    const double* v = Vr + (int64_t)(jj - 1) * N;
    double* wr = Wr + (int64_t)(jj - 1) * N;
    double s = 0.0;
    for (int i = j + t; i < N; i += TB) s = fma(wr[i], v[i], s);
    s = block_sum<TW>(s, red);
    const double c = -0.5 * tg[j - 1] * s;
    for (int i = j + t; i < N; i += TB) wr[i] = fma(c, v[i], wr[i]);
    __syncthreads();
  }
  // coefficients W_k[j], V_k[j] of the pending rank-2 updates
  if (t < jj) coef[t] = Wr[(int64_t)t * N + j];
  else if (t >= 64 && t < 64 + jj) coef[t] = Vr[(int64_t)(t - 64) * N + j];
  __syncthreads();

  // 2. a = A[j:, j] - sum_k (V_k W_k[j] + W_k V_k[j]); A[j][i] by symmetry.
  // Each thread updates up to RPT of its rows at once, k unrolled by 8, so
  // that 2*8*RPT independent loads are in flight.
  constexpr int RPT = 4;
  double* rowj = Ag + (int64_t)j * N;
  double ss = 0.0;
  double aj = 0.0, a1 = 0.0;
  for (int base = j + t; base < N; base += TB * RPT) {
    double acc[RPT];
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      const int i = base + r * TB;
      acc[r] = i < N ? rowj[i] : 0.0;
    }
    for (int k0 = 0; k0 < jj; k0 += 8) {
#pragma unroll
      for (int kq = 0; kq < 8; ++kq) {
        const int k = k0 + kq;
        if (k < jj) {
          const double cw = coef[k], cv = coef[64 + k];
          const double* vk = Vr + (int64_t)k * N;
          const double* wk = Wr + (int64_t)k * N;
#pragma unroll
          for (int r = 0; r < RPT; ++r) {
            const int i = base + r * TB;
            if (i < N) acc[r] = fma(-vk[i], cw, fma(-wk[i], cv, acc[r]));
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      const int i = base + r * TB;
      if (i < N) {
        rowj[i] = acc[r];
        if (i == j) aj = acc[r];
        else if (i == j + 1) a1 = acc[r];
        else ss = fma(acc[r], acc[r], ss);
      }
    }
  }
  if (t == 0) sh[0] = aj;
  if (t == 1) sh[1] = a1;
  ss = block_sum<TW>(ss, red);   // its barriers publish sh[] and rowj[]
  const double dj = sh[0];
  const double alpha = (j + 1 < N) ? sh[1] : 0.0;
  double tau = 0.0, beta = alpha, scale = 0.0;
  if (j + 1 < N && ss > 0.0) {
    beta = -copysign(sqrt(alpha * alpha + ss), alpha);
    tau = (beta - alpha) / beta;
    scale = 1.0 / (alpha - beta);
  }
  if (t == 0) {
    diag[(int64_t)g * N + j] = dj;
    off[(int64_t)g * N + j] = (j + 1 < N) ? beta : 0.0;
    taus[(int64_t)g * N + j] = tau;
    gr[jj * nb + jj] = (j + 1 < N) ? 1.0 + ss * scale * scale : 0.0;   // v_j'v_j
  }
  // 3. v: zeros up to j, 1 at j+1, scaled a below. Stored in P (rows jj and
  // 2nb+jj) and in row j of A (for the accumulation of Q); W row jj is
  // cleared up to j so the symv only fills rows > j.
  double* vj = Vr + (int64_t)jj * N;
  double* vj2 = V2 + (int64_t)jj * N;
  double* wj = Wr + (int64_t)jj * N;
  for (int i = t; i < N; i += TB) {
    double v = 0.0;
    if (j + 1 < N) {
      if (i == j + 1) v = 1.0;
      else if (i > j + 1) v = (scale != 0.0) ? rowj[i] * scale : 0.0;
    }
    vj[i] = v;
    vj2[i] = v;
    rowj[i] = v;                      // row j of A now holds v_j (0 at and left of j)
    if (i <= j) wj[i] = 0.0;
  }
  __syncthreads();
  // 4. dot products, four k at a time per wave
  const int nk = 2 * jj;
  for (int k0 = 4 * w; k0 < nk; k0 += 4 * TW) {
    double s[4] = {0.0, 0.0, 0.0, 0.0};
    const double* src[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int k = k0 + q < nk ? k0 + q : k0;
      src[q] = (k < jj) ? (Wr + (int64_t)k * N) : (Vr + (int64_t)(k - jj) * N);
    }
#pragma unroll 4
    for (int i = j + 1 + lane; i < N; i += 64) {
      const double vi = vj[i];
#pragma unroll
      for (int q = 0; q < 4; ++q) s[q] = fma(src[q][i], vi, s[q]);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double r = wave_sum(s[q]);
      const int k = k0 + q;
      if (lane == 0 && k < nk) {
        dg[k] = r;                     // dg[k<jj] = W_k'v, dg[jj+k] = V_k'v
        if (k >= jj) gr[(k - jj) * nb + jj] = r;
      }
    }
  }
}

// w_raw = tau * (A[j+1:, j+1:] v - V (W'v) - W (V'v)) for rows > j. Four
// rows per wave: lanes stride the columns of the row-major trailing matrix
// (coalesced, two column blocks in flight), then the rank-2jj corrections
// are spread over the lanes.
constexpr int SR = 4;           // rows per wave
constexpr int SW = 4;           // waves per block
__global__ __launch_bounds__(SW * 64) void tri_symv_kernel(const double* __restrict__ A,
                                                           double* __restrict__ P,
                                                           const double* __restrict__ dots,
                                                           const double* __restrict__ taus, int N,
                                                           int nb, int j, int jj) {
  const int g = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const double* Ag = A + (int64_t)g * N * N;
  double* Pg = P + (int64_t)g * 3 * nb * N;
  const double* Vr = Pg;
  double* Wr = Pg + (int64_t)nb * N;
  const double* v = Vr + (int64_t)jj * N;
  const double* dg = dots + (int64_t)g * 2 * nb;
  const double tau = taus[(int64_t)g * N + j];
  const int r0 = j + 1 + (blockIdx.x * SW + w) * SR;
  if (r0 >= N) return;
  double acc[SR];
#pragma unroll
  for (int q = 0; q < SR; ++q) acc[q] = 0.0;
  const double* rowp[SR];
#pragma unroll
  for (int q = 0; q < SR; ++q) rowp[q] = Ag + (int64_t)(r0 + q < N ? r0 + q : r0) * N;
#pragma unroll 2
  for (int c = j + 1 + lane; c < N; c += 64) {
    const double vc = v[c];
#pragma unroll
    for (int q = 0; q < SR; ++q) acc[q] = fma(rowp[q][c], vc, acc[q]);
  }
#pragma unroll
  for (int q = 0; q < SR; ++q) acc[q] = wave_sum(acc[q]);
  // corrections: lane = 16*q + kl handles row q, terms k = kl, kl+16, ...
  const int q = lane >> 4, kl = lane & 15;
  const int r = r0 + q;
  double corr = 0.0;
  if (r < N)
    for (int k = kl; k < jj; k += 16)
      corr = fma(Vr[(int64_t)k * N + r], dg[k], fma(Wr[(int64_t)k * N + r], dg[jj + k], corr));
  corr += __shfl_xor(corr, 1, 64);
  corr += __shfl_xor(corr, 2, 64);
  corr += __shfl_xor(corr, 4, 64);
  corr += __shfl_xor(corr, 8, 64);
  double mine = acc[0];
#pragma unroll
  for (int qq = 1; qq < SR; ++qq)
    if (q == qq) mine = acc[qq];
  if (kl == 0 && r < N) Wr[(int64_t)jj * N + r] = tau * (mine - corr);
}

// Finish the last w of a panel (step 1 of tri_col_kernel alone).
__global__ __launch_bounds__(TB) void tri_finish_kernel(double* __restrict__ P,
                                                        const double* __restrict__ taus, int N,
                                                        int nb, int jlast, int jjlast) {
  __shared__ double red[TW];
  const int g = blockIdx.x, t = threadIdx.x;
  double* Pg = P + (int64_t)g * 3 * nb * N;
  const double* v = Pg + (int64_t)jjlast * N;
  double* wr = Pg + (int64_t)(nb + jjlast) * N;
  double s = 0.0;
  for (int i = jlast + 1 + t; i < N; i += TB) s = fma(wr[i], v[i], s);
  s = block_sum<TW>(s, red);
  const double c = -0.5 * taus[(int64_t)g * N + jlast] * s;
  for (int i = jlast + 1 + t; i < N; i += TB) wr[i] = fma(c, v[i], wr[i]);
}

__global__ void set_identity_kernel(double* __restrict__ Q, int N, int64_t total) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int64_t e = idx % ((int64_t)N * N);
  Q[idx] = (e / N == e % N) ? 1.0 : 0.0;
}

// Compact-WY factor of the panel's reflectors (LAPACK dlarft, forward,
// columnwise): H_p ... H_{p+nb-1} = I - V T V', T upper triangular,
// T[i][i] = tau_i, T[0:i, i] = -tau_i T[0:i, 0:i] (V[:, 0:i]' v_i). The
// Gram entries V' v_i were recorded by the reduction (pgram); column i of T
// is formed by nb threads in parallel, columns in sequence.
__global__ __launch_bounds__(64) void form_t_kernel(const double* __restrict__ pgram,
                                                    const double* __restrict__ taus,
                                                    double* __restrict__ tmat, int N, int nbs,
                                                    int nb, int p) {
  __shared__ double T[64][65];
  __shared__ double gcol[64];
  const int g = blockIdx.x, r = threadIdx.x;
  const double* gr = pgram + (int64_t)g * N * nbs + (int64_t)p * nbs;
  const double* tg = taus + (int64_t)g * N;
  if (r < nb)
    for (int c = 0; c < nb; ++c) T[r][c] = 0.0;
  __syncthreads();
  for (int i = 0; i < nb; ++i) {
    const double ti = (p + i < N) ? tg[p + i] : 0.0;
    if (r < i) gcol[r] = gr[r * nbs + i];
    __syncthreads();
    double s = 0.0;
    if (r < i)
      for (int c = r; c < i; ++c) s = fma(T[r][c], gcol[c], s);
    __syncthreads();
    if (r < i) T[r][i] = -ti * s;
    if (r == i) T[i][i] = ti;
    __syncthreads();
  }
  double* Tg = tmat + (int64_t)g * nbs * nbs;
  if (r < nb)
    for (int c = 0; c < nb; ++c) Tg[r * nb + c] = T[r][c];
}

size_t tridiag_panel_doubles(int G, int N, int nb) {
  return (size_t)G * (3 * (size_t)nb * N + 2 * nb + (size_t)nb * nb + 3 * (size_t)nb * N);
}

// Sum over matrices of f(valid order) for the work counters.
template <typename F>
static double over_groups(const TridiagWork& wk, F f) {
  double a = 0.0;
  for (int g = 0; g < wk.G; ++g) a += f((double)(wk.nv_host ? wk.nv_host[g] : wk.N));
  return a;
}

int tridiagonalize(hipStream_t s, const TridiagWork& wk) {
  const int G = wk.G, N = wk.N, nb = wk.nb;
  if (G <= 0 || N <= 0) return 0;
  if (nb > 64 || N % nb != 0) {
    set_error("tridiagonalize: panel width must divide N and be <= 64");
    return KMP_EINVAL;
  }
  int rc;
  KMP_HIP_TRY(hipMemsetAsync(wk.panel, 0, sizeof(double) * (size_t)G * 3 * nb * N, s));
  for (int p = 0; p < N; p += nb) {
    const int pe = (p + nb < N) ? p + nb : N;
    for (int j = p; j < pe; ++j) {
      const int jj = j - p;
      kc_begin(KMP_KC_TRI_COL, s);
      hipLaunchKernelGGL(tri_col_kernel, dim3(G), dim3(TB), 0, s, wk.A, wk.panel, wk.dots, wk.tau,
                         wk.diag, wk.off, wk.pgram, N, nb, j, jj);
      KMP_LAUNCH_CHECK();
      // panel rows (2jj) read twice, finish/update/store of ~6 vectors
      kc_end(KMP_KC_TRI_COL, s,
             over_groups(wk, [&](double n) { return 8.0 * std::max(0.0, n - j) * (4.0 * jj + 6.0); }),
             over_groups(wk, [&](double n) { return 2.0 * std::max(0.0, n - j) * (4.0 * jj + 4.0); }));
      const int rows = N - j - 1;
      if (rows > 0) {
        kc_begin(KMP_KC_TRI_SYMV, s);
        hipLaunchKernelGGL(tri_symv_kernel, dim3((unsigned)ceil_div(rows, SR * SW), G), dim3(SW * 64),
                           0, s, wk.A, wk.panel, wk.dots, wk.tau, N, nb, j, jj);
        KMP_LAUNCH_CHECK();
        // the trailing matrix is read once (m^2 doubles)
        kc_end(KMP_KC_TRI_SYMV, s, over_groups(wk, [&](double n) {
                 const double m = std::max(0.0, n - j - 1);
                 return 8.0 * (m * m + 2.0 * jj * m); }),
               over_groups(wk, [&](double n) {
                 const double m = std::max(0.0, n - j - 1);
                 return 2.0 * m * m + 4.0 * jj * m; }));
      }
    }
    if (pe < N) {
      hipLaunchKernelGGL(tri_finish_kernel, dim3(G), dim3(TB), 0, s, wk.panel, wk.tau, N, nb,
                         pe - 1, pe - 1 - p);
      KMP_LAUNCH_CHECK();
      // trailing update A[pe:, pe:] -= V W' + W V'  as one GEMM with K = 2nb
      GemmArgs ga;
      ga.M = N - pe; ga.N = N - pe; ga.K = 2 * nb; ga.batch = G;
      ga.A = wk.panel + pe; ga.lda = N; ga.sA = (int64_t)3 * nb * N;
      ga.B = wk.panel + (int64_t)nb * N + pe; ga.ldb = N; ga.sB = (int64_t)3 * nb * N;
      ga.C = wk.A + (int64_t)pe * N + pe; ga.ldc = N; ga.sC = (int64_t)N * N;
      ga.alpha = -1.0; ga.beta = 1.0;
      kc_begin(KMP_KC_TRI_SYR2K, s);
      if ((rc = gemm(s, ga, false, false, true)) != 0) return rc;
      kc_end(KMP_KC_TRI_SYR2K, s, over_groups(wk, [&](double n) {
               const double m = std::max(0.0, n - pe); return 16.0 * m * m; }),
             over_groups(wk, [&](double n) {
               const double m = std::max(0.0, n - pe); return 4.0 * nb * m * m; }));
    }
  }
  // Q = H_0 H_1 ... H_{N-2}, accumulated backwards panel by panel:
  // Q[p+1:, p+1:] -= V' (T (V Q[p+1:, p+1:]))
  const int64_t tot = (int64_t)G * N * N;
  hipLaunchKernelGGL(set_identity_kernel, dim3((unsigned)ceil_div(tot, 256)), dim3(256), 0, s,
                     wk.Q, N, tot);
  KMP_LAUNCH_CHECK();
  const int last = ((N - 2) / nb) * nb;
  for (int p = last; p >= 0; p -= nb) {
    const int m = N - p - 1;
    if (m <= 0) continue;
    const int kb = (p + nb <= N) ? nb : N - p;
    kc_begin(KMP_KC_QFORM, s);
    hipLaunchKernelGGL(form_t_kernel, dim3(G), dim3(64), 0, s, wk.pgram, wk.tau, wk.tmat, N, nb,
                       kb, p);
    KMP_LAUNCH_CHECK();
    GemmArgs g1;   // X = V[:, p+1:] Q[p+1:, p+1:]   (kb x m)
    g1.M = kb; g1.N = m; g1.K = m; g1.batch = G;
    g1.A = wk.A + (int64_t)p * N + p + 1; g1.lda = N; g1.sA = (int64_t)N * N;
    g1.B = wk.Q + (int64_t)(p + 1) * N + p + 1; g1.ldb = N; g1.sB = (int64_t)N * N;
    g1.C = wk.xbuf; g1.ldc = N; g1.sC = (int64_t)nb * N;
    if ((rc = gemm(s, g1, true, false, true)) != 0) return rc;
    GemmArgs g2;   // Y = T X
    g2.M = kb; g2.N = m; g2.K = kb; g2.batch = G;
    g2.A = wk.tmat; g2.lda = kb; g2.sA = (int64_t)nb * nb;
    g2.B = wk.xbuf; g2.ldb = N; g2.sB = (int64_t)nb * N;
    g2.C = wk.ybuf; g2.ldc = N; g2.sC = (int64_t)nb * N;
    if ((rc = gemm(s, g2, true, false, true)) != 0) return rc;
    GemmArgs g3;   // Q[p+1:, p+1:] -= V' Y
    g3.M = m; g3.N = m; g3.K = kb; g3.batch = G;
    g3.A = wk.A + (int64_t)p * N + p + 1; g3.lda = N; g3.sA = (int64_t)N * N;
    g3.B = wk.ybuf; g3.ldb = N; g3.sB = (int64_t)nb * N;
    g3.C = wk.Q + (int64_t)(p + 1) * N + p + 1; g3.ldc = N; g3.sC = (int64_t)N * N;
    g3.alpha = -1.0; g3.beta = 1.0;
    if ((rc = gemm(s, g3, false, false, true)) != 0) return rc;
    // Q block read by the first product, read and written by the update
    kc_end(KMP_KC_QFORM, s, over_groups(wk, [&](double n) {
             const double mm = std::max(0.0, n - p - 1); return 24.0 * mm * mm; }),
           over_groups(wk, [&](double n) {
             const double mm = std::max(0.0, n - p - 1); return 4.0 * kb * mm * mm + 2.0 * kb * kb * mm; }));
  }
  return 0;
}

}  // namespace kmp
