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
#include <vector>

namespace kmp {

constexpr int TB = 512;   // threads per block of the one-workgroup-per-matrix kernels
constexpr int TW = 8;     // waves per block
constexpr int SR = 2;     // symv: rows per wave
constexpr int SW = TW;    // symv: waves per block
constexpr int SRB = SR * SW;

// Sum of the symv blocks' partial dot products (fixed order, wave 0).
__device__ __forceinline__ double reduce_parts(const double* __restrict__ sp, int n, double* slot) {
  const int t = threadIdx.x;
  if (t < 64) {
    double s = 0.0;
    for (int q = t; q < n; q += 64) s += sp[q];
    s = wave_sum(s);
    if (t == 0) *slot = s;
  }
  __syncthreads();
  return *slot;
}

// One workgroup per matrix, step j of the panel starting at p (jj = j - p):
//  1. column j up to date: at a panel start it is row j of A (trailing
//     update done); otherwise the previous symv left
//     pnext = A[j][:] - sum_{k < jj-1} (V_k W_k[j] + W_k V_k[j]) and the
//     partial sums of w_raw'v, so the last rank-2 term is added with the
//     finished w_{jj-1} = w_raw - (tau/2)(w_raw'v) v   (dlatrd)
//  2. Householder vector of column j below the diagonal (dlarfg)
//  3. dot products W_k'v, V_k'v (k < jj) for the next symv's corrections
// Thread t owns rows j + t + TB*m (m < CR); the column stays in registers.
template <int CR>
__device__ __forceinline__ void col_role(int g, double* __restrict__ A, double* __restrict__ P,
                                         double* __restrict__ dots, double* __restrict__ taus,
                                         double* __restrict__ diag, double* __restrict__ off,
                                         const double* __restrict__ spart,
                                         const double* __restrict__ pnext, int N, int nb, int j,
                                         int jj, int nparts, double* red, double* sh) {
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  double* Ag = A + (int64_t)g * N * N;
  double* Pg = P + (int64_t)g * 3 * nb * N;
  double* Vr = Pg;                    // rows 0..nb-1   : v_k
  double* Wr = Pg + (int64_t)nb * N;  // rows nb..2nb-1 : w_k
  double* V2 = Pg + (int64_t)2 * nb * N;
  double* dg = dots + (int64_t)g * 2 * nb;
  double* rowj = Ag + (int64_t)j * N;

  // all loads of the column step are issued before the first barrier
  double a[CR];
  if (jj == 0) {
#pragma unroll
    for (int m = 0; m < CR; ++m) {
      const int r = j + t + TB * m;
      a[m] = r < N ? rowj[r] : 0.0;
    }
  } else {
    const double* vp = Vr + (int64_t)(jj - 1) * N;
    double* wp = Wr + (int64_t)(jj - 1) * N;
    const double* pn = pnext + (int64_t)g * N;
    double vr[CR], wr[CR], pr[CR];
#pragma unroll
    for (int m = 0; m < CR; ++m) {
      const int r = j + t + TB * m;
      const bool in = r < N;
      vr[m] = in ? vp[r] : 0.0;
      wr[m] = in ? wp[r] : 0.0;
      pr[m] = in ? pn[r] : 0.0;
    }
    const double tprev = taus[(int64_t)g * N + j - 1];
    const double wpj = wp[j];
    const double s = reduce_parts(spart + (int64_t)g * ((N + SRB - 1) / SRB), nparts, &sh[2]);
    const double c = 0.5 * tprev * s;
    const double wfj = wpj - c;               // finished w_{jj-1}[j]   (v_{jj-1}[j] = 1)
    // the finished w_{jj-1} replaces the raw one (own rows; every thread
    // has read wp[j] before the barrier inside reduce_parts)
#pragma unroll
    for (int m = 0; m < CR; ++m) {
      const int r = j + t + TB * m;
      const double wf = fma(-c, vr[m], wr[m]);
      if (r < N) wp[r] = wf;
      a[m] = pr[m] - fma(vr[m], wfj, wf);
    }
  }
  double ss = 0.0, aj = 0.0, a1 = 0.0;
#pragma unroll
  for (int m = 0; m < CR; ++m) {
    const int r = j + t + TB * m;
    if (r == j) aj = a[m];
    else if (r == j + 1) a1 = a[m];
    else if (r < N) ss = fma(a[m], a[m], ss);
  }
  if (t == 0) sh[0] = aj;
  if (t == 1) sh[1] = a1;
  ss = block_sum<TW>(ss, red);                  // its barriers publish sh[]
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
  }
  // v_j: zeros up to j, 1 at j+1, scaled a below; stored in P (rows jj and
  // 2nb+jj) and in row j of A (read back by the accumulation of Q). W row
  // jj is cleared up to j so the symv only fills rows > j.
  double* vj = Vr + (int64_t)jj * N;
  double* vj2 = V2 + (int64_t)jj * N;
  double* wj = Wr + (int64_t)jj * N;
#pragma unroll
  for (int m = 0; m < CR; ++m) {
    const int r = j + t + TB * m;
    double v = 0.0;
    if (r == j + 1) v = 1.0;
    else if (r > j + 1 && r < N) v = (scale != 0.0) ? a[m] * scale : 0.0;
    if (r < N) {
      vj[r] = v;
      vj2[r] = v;
      rowj[r] = v;
      if (r == j) wj[r] = 0.0;
    }
  }
  for (int i = t; i < j; i += TB) {
    vj[i] = 0.0;
    vj2[i] = 0.0;
    rowj[i] = 0.0;
    wj[i] = 0.0;
  }
  __syncthreads();                              // v_j stored before the products read it
  // dot products W_k'v, V_k'v (k < jj): wave w handles products 8w..8w+7
  // over all rows (lanes stride the rows, eight row blocks in flight), so
  // each reduction stays inside one wave. dg[k<jj] = W_k'v, dg[jj+k] = V_k'v.
  const int nk = 2 * jj;
  for (int k0 = 8 * w; k0 < nk; k0 += 8 * TW) {
    double acc[8];
    const double* src[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      acc[q] = 0.0;
      const int k = k0 + q < nk ? k0 + q : k0;
      src[q] = (k < jj) ? (Wr + (int64_t)k * N) : (Vr + (int64_t)(k - jj) * N);
    }
#pragma unroll 8
    for (int i = j + 1 + lane; i < N; i += 64) {
      const double vi = vj[i];
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] = fma(src[q][i], vi, acc[q]);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const double r = wave_sum(acc[q]);
      if (lane == 0 && k0 + q < nk) dg[k0 + q] = r;
    }
  }
}

// Step j's trailing product for rows r > j (four rows per wave, lanes
// striding the columns of the row-major matrix, two column blocks in
// flight):
//   w_raw[r] = tau (A[r, j+1:] v - sum_k (V_k[r] W_k'v + W_k[r] V_k'v)),
// the block's part of w_raw'v, and, when column j+1 is in the same panel,
//   pnext[r] = A[r][j+1] - sum_{k<jj} (V_k[r] W_k[j+1] + W_k[r] V_k[j+1]),
// which reuses the panel values loaded for the corrections.
__device__ __forceinline__ void symv_role(int g, int blk, const double* __restrict__ A,
                                          double* __restrict__ P, const double* __restrict__ dots,
                                          const double* __restrict__ taus, double* __restrict__ spart,
                                          double* __restrict__ pnext, int N, int nb, int j, int jj,
                                          int want_next, double* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const double* Ag = A + (int64_t)g * N * N;
  double* Pg = P + (int64_t)g * 3 * nb * N;
  const double* Vr = Pg;
  double* Wr = Pg + (int64_t)nb * N;
  const double* v = Vr + (int64_t)jj * N;
  const double* dg = dots + (int64_t)g * 2 * nb;
  const double tau = taus[(int64_t)g * N + j];
  const int r0 = j + 1 + (blk * SW + w) * SR;
  double acc[SR];
#pragma unroll
  for (int q = 0; q < SR; ++q) acc[q] = 0.0;
  const double* rowp[SR];
#pragma unroll
  for (int q = 0; q < SR; ++q) rowp[q] = Ag + (int64_t)(r0 + q < N ? r0 + q : N - 1) * N;
  if (r0 < N) {
#pragma unroll 2
    for (int c = j + 1 + lane; c < N; c += 64) {
      const double vc = v[c];
#pragma unroll
      for (int q = 0; q < SR; ++q) acc[q] = fma(rowp[q][c], vc, acc[q]);
    }
  }
#pragma unroll
  for (int q = 0; q < SR; ++q) acc[q] = wave_sum(acc[q]);
  // corrections: lane = (64/SR)*q + kl handles row q, terms k = kl, kl+64/SR, ...
  constexpr int LPR = 64 / SR;
  const int q = lane / LPR, kl = lane % LPR;
  const int r = r0 + q;
  double corr = 0.0, pn = 0.0;
  if (r < N) {
    for (int k = kl; k < jj; k += LPR) {
      const double vk = Vr[(int64_t)k * N + r], wk = Wr[(int64_t)k * N + r];
      corr = fma(vk, dg[k], fma(wk, dg[jj + k], corr));
      if (want_next) pn = fma(vk, Wr[(int64_t)k * N + j + 1], fma(wk, Vr[(int64_t)k * N + j + 1], pn));
    }
  }
#pragma unroll
  for (int o = 1; o < LPR; o <<= 1) {
    corr += __shfl_xor(corr, o, 64);
    pn += __shfl_xor(pn, o, 64);
  }
  double mine = acc[0];
#pragma unroll
  for (int qq = 1; qq < SR; ++qq)
    if (q == qq) mine = acc[qq];
  double contrib = 0.0;
  if (kl == 0 && r < N) {
    const double wr = tau * (mine - corr);
    Wr[(int64_t)jj * N + r] = wr;
    contrib = wr * v[r];
    if (want_next) pnext[(int64_t)g * N + r] = rowp[q][j + 1] - pn;
  }
  const double part = block_sum<SW>(contrib, red);
  if (threadIdx.x == 0) spart[(int64_t)g * ((N + SRB - 1) / SRB) + blk] = part;
}

// One launch = the column step of one set of matrices and the trailing
// product of another set: the first `ncol` blocks run col_role for groups
// cg0.., the rest symv_role for groups sg0.. (nparts blocks each). Running
// the latency-bound column step of one set beside the bandwidth-bound
// product of the other keeps the chip busy.
struct StepArgs {
  double* A; double* P; double* dots; double* taus; double* diag; double* off;
  double* spart; double* pnext;
  int N, nb;
  int ncol, cg0, cj, cjj, cparts;           // column role
  int nsym, sg0, sj, sjj, snext, sparts;    // product role (nsym groups)
};

template <int CR>
__global__ __launch_bounds__(TB) void tri_step_kernel(StepArgs a) {
  __shared__ double red[TW];
  __shared__ double sh[3];
  const int b = blockIdx.x;
  if (b < a.ncol) {
    col_role<CR>(a.cg0 + b, a.A, a.P, a.dots, a.taus, a.diag, a.off, a.spart, a.pnext, a.N, a.nb,
                 a.cj, a.cjj, a.cparts, red, sh);
  } else {
    const int q = b - a.ncol;
    symv_role(a.sg0 + q / a.sparts, q % a.sparts, a.A, a.P, a.dots, a.taus, a.spart, a.pnext, a.N,
              a.nb, a.sj, a.sjj, a.snext, red);
  }
}

// Finish the last w of a panel: w = w_raw - (tau/2)(w_raw'v) v.
__global__ __launch_bounds__(TB) void tri_finish_kernel(double* __restrict__ P,
                                                        const double* __restrict__ taus,
                                                        const double* __restrict__ spart, int N,
                                                        int nb, int jlast, int jjlast, int nparts,
                                                        int g0) {
  __shared__ double sh;
  const int g = g0 + blockIdx.x, t = threadIdx.x;
  double* Pg = P + (int64_t)g * 3 * nb * N;
  const double* v = Pg + (int64_t)jjlast * N;
  double* wr = Pg + (int64_t)(nb + jjlast) * N;
  const double s = reduce_parts(spart + (int64_t)g * ((N + SRB - 1) / SRB), nparts, &sh);
  const double c = -0.5 * taus[(int64_t)g * N + jlast] * s;
  for (int i = jlast + 1 + t; i < N; i += TB) wr[i] = fma(c, v[i], wr[i]);
}

// Q_g = I, one grid row per matrix (blockIdx.y) and a grid-stride loop, so
// that no launch dimension exceeds 2^32 work-items.
__global__ void set_identity_kernel(double* __restrict__ Q, int N) {
  const int64_t nn = (int64_t)N * N;
  double* Qg = Q + (int64_t)blockIdx.y * nn;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nn; e += stride)
    Qg[e] = (e / N == e % N) ? 1.0 : 0.0;
}

// Compact-WY factor of kb consecutive reflectors (LAPACK dlarft, forward):
// H_p ... H_{p+kb-1} = I - V T V' with T upper triangular. Built by
// recursive doubling from T[i][i] = tau_i: two adjacent blocks with factors
// T1, T2 combine into [[T1, -T1 (V1'V2) T2], [0, T2]], where V1'V2 is a block
// of the Gram matrix of the reflectors (gram, ld NBQ, valid for i, j < kb).
// Everything stays in LDS; six levels of small products for kb <= 64.
constexpr int NBQ = 64;
constexpr int FTT = 256;   // threads of form_t_kernel
// With nref > 0 the launch covers many blocks at once: grid row y is block
// y (reflectors p + NBQ y .., kb = min(NBQ, nref - p - NBQ y)), whose Gram
// and T sit at gram / tmat + y * bstride (+ g NBQ^2 within the block).
__global__ __launch_bounds__(FTT) void form_t_kernel(const double* __restrict__ gram,
                                                     const double* __restrict__ taus,
                                                     double* __restrict__ tmat, int N, int kb,
                                                     int p, int nref, int64_t bstride) {
  __shared__ double T[NBQ][NBQ + 1];
  __shared__ double Gs[NBQ][NBQ + 1];
  __shared__ double Ws[NBQ][NBQ + 1];
  const int g = blockIdx.x, t = threadIdx.x;
  if (nref > 0) {
    p += NBQ * blockIdx.y;
    kb = min(NBQ, nref - p);
    gram += (int64_t)blockIdx.y * bstride;
    tmat += (int64_t)blockIdx.y * bstride;
  }
  const double* gr = gram + (int64_t)g * NBQ * NBQ;
  for (int e = t; e < NBQ * NBQ; e += FTT) {
    const int a = e / NBQ, b = e % NBQ;
    Gs[a][b] = (a < kb && b < kb) ? gr[e] : 0.0;
    T[a][b] = (a == b && a < kb && p + a < N) ? taus[(int64_t)g * N + p + a] : 0.0;
  }
  __syncthreads();
  for (int sz = 1; sz < NBQ; sz *= 2) {
    // pairs of blocks [2qs, 2qs+s) and [2qs+s, 2qs+2s): 32*sz outputs
    const int outs = (NBQ / 2) * sz;
    for (int e = t; e < outs; e += FTT) {       // W = G12 T2
      const int q = e / (sz * sz), rem = e % (sz * sz);
      const int a = 2 * q * sz + rem / sz, b = 2 * q * sz + sz + rem % sz;
      double acc = 0.0;
      for (int c = 2 * q * sz + sz; c <= b; ++c) acc = fma(Gs[a][c], T[c][b], acc);
      Ws[a][b] = acc;
    }
    __syncthreads();
    for (int e = t; e < outs; e += FTT) {       // T12 = -T1 W
      const int q = e / (sz * sz), rem = e % (sz * sz);
      const int a = 2 * q * sz + rem / sz, b = 2 * q * sz + sz + rem % sz;
      double acc = 0.0;
      for (int c = a; c < 2 * q * sz + sz; ++c) acc = fma(T[a][c], Ws[c][b], acc);
      T[a][b] = -acc;
    }
    __syncthreads();
  }
  double* Tg = tmat + (int64_t)g * NBQ * NBQ;
  for (int e = t; e < NBQ * NBQ; e += FTT) Tg[e] = T[e / NBQ][e % NBQ];
}

int wy_form_t(hipStream_t s, const double* gram, const double* taus, double* tmat, int G, int N,
              int kb, int p) {
  hipLaunchKernelGGL(form_t_kernel, dim3(G), dim3(FTT), 0, s, gram, taus, tmat, N, kb, p, 0,
                     (int64_t)0);
  KMP_LAUNCH_CHECK();
  return 0;
}

int wy_form_t_blocks(hipStream_t s, const double* gram, const double* taus, double* tmat, int G,
                     int N, int nref, int nblk) {
  if (nblk <= 0) return 0;
  hipLaunchKernelGGL(form_t_kernel, dim3(G, nblk), dim3(FTT), 0, s, gram, taus, tmat, N, 0, 0,
                     nref, (int64_t)G * NBQ * NBQ);
  KMP_LAUNCH_CHECK();
  return 0;
}

int tridiag_parts(int N) { return (N + SRB - 1) / SRB; }

size_t tridiag_panel_doubles(int G, int N, int nb) {
  const size_t parts = (size_t)((N + SRB - 1) / SRB);
  return (size_t)G * (3 * (size_t)nb * N + 2 * nb + 2 * (size_t)NBQ * NBQ + 2 * (size_t)NBQ * N +
                      parts + (size_t)N);
}

// Sum over matrices of f(valid order) for the work counters.
template <typename F>
static double over_groups(const TridiagWork& wk, F f) {
  double a = 0.0;
  for (int g = 0; g < wk.G; ++g) a += f((double)(wk.nv_host ? wk.nv_host[g] : wk.N));
  return a;
}

// Column steps, panel updates and the accumulation of Q for nch independent
// sets of matrices, each on its own stream; launches are interleaved step
// by step so that every stream always has work queued.
int tridiagonalize_multi(const hipStream_t* ss, const TridiagWork* ws, int nch) {
  if (nch <= 0) return 0;
  const int N = ws[0].N, nb = ws[0].nb;
  for (int k = 0; k < nch; ++k)
    if (ws[k].N != N || ws[k].nb != nb) {
      set_error("tridiagonalize: all parts must share N and the panel width");
      return KMP_EINVAL;
    }
  if (nb > 64 || N % nb != 0 || N > TB * 16) {
    set_error("tridiagonalize: panel width must divide N, and N <= 8192 per matrix");
    return KMP_EINVAL;
  }
  int rc;
  for (int k = 0; k < nch; ++k)
    if (ws[k].G > 0)
      KMP_HIP_TRY(hipMemsetAsync(ws[k].panel, 0, sizeof(double) * (size_t)ws[k].G * 3 * nb * N, ss[k]));
  for (int k = 0; k < nch; ++k) {
    const TridiagWork& wk = ws[k];
    const hipStream_t s = ss[k];
    const int G = wk.G;
    if (G <= 0) continue;
    // two sets of matrices, the second half a step behind the first
    const int GA = (G + 1) / 2, GB = G - GA;
    int partsA = 0, partsB = 0;
    auto launch = [&](int ncol, int cg0, int cj, int nsym, int sg0, int sj) -> int {
      StepArgs a;
      a.A = wk.A; a.P = wk.panel; a.dots = wk.dots; a.taus = wk.tau; a.diag = wk.diag;
      a.off = wk.off; a.spart = wk.spart; a.pnext = wk.pnext; a.N = N; a.nb = nb;
      a.ncol = ncol; a.cg0 = cg0; a.cj = cj; a.cjj = cj - (cj / nb) * nb;
      a.cparts = (cg0 < GA) ? partsA : partsB;
      a.nsym = nsym; a.sg0 = sg0; a.sj = sj; a.sjj = sj - (sj / nb) * nb;
      a.snext = (nsym > 0 && a.sjj + 1 < nb && sj + 1 < N) ? 1 : 0;
      a.sparts = nsym > 0 ? (int)ceil_div(N - sj - 1, SRB) : 1;
      const unsigned blocks = (unsigned)(ncol + nsym * a.sparts);
      if (blocks == 0) return 0;
      const int rows_col = ncol > 0 ? N - cj : 0;
      if (ncol > 0) kc_begin(KMP_KC_PANEL, s);
      else kc_begin(KMP_KC_PANEL_WY, s);
      if (rows_col <= TB * 4) hipLaunchKernelGGL(tri_step_kernel<4>, dim3(blocks), dim3(TB), 0, s, a);
      else if (rows_col <= TB * 8) hipLaunchKernelGGL(tri_step_kernel<8>, dim3(blocks), dim3(TB), 0, s, a);
      else hipLaunchKernelGGL(tri_step_kernel<16>, dim3(blocks), dim3(TB), 0, s, a);
      KMP_LAUNCH_CHECK();
      // column steps: column (~4 vectors) and panel rows once; products:
      // the trailing matrix once (m^2 doubles) plus the panel rows
      double bytes = 0.0, flops = 0.0;
      for (int g = 0; g < ncol; ++g) {
        const double n = wk.nv_host ? wk.nv_host[cg0 + g] : N;
        bytes += 8.0 * std::max(0.0, n - cj) * (2.0 * a.cjj + 8.0);
        flops += 2.0 * std::max(0.0, n - cj) * (2.0 * a.cjj + 4.0);
      }
      for (int g = 0; g < nsym; ++g) {
        const double n = wk.nv_host ? wk.nv_host[sg0 + g] : N;
        const double m = std::max(0.0, n - sj - 1);
        bytes += 8.0 * (m * m + 2.0 * a.sjj * m);
        flops += 2.0 * m * m + 8.0 * a.sjj * m;
      }
      if (ncol > 0) kc_end(KMP_KC_PANEL, s, bytes, flops);
      else kc_end(KMP_KC_PANEL_WY, s, bytes, flops);
      if (nsym > 0) {
        if (sg0 < GA) partsA = a.sparts;
        else partsB = a.sparts;
      }
      return 0;
    };
    for (int p = 0; p < N; p += nb) {
      const int pe = (p + nb < N) ? p + nb : N;
      for (int j = p; j < pe; ++j) {
        const bool rows = (N - j - 1) > 0;
        // A: column j     B: product j-1 (same panel)
        if ((rc = launch(GA, 0, j, (j > p && GB > 0) ? GB : 0, GA, j - 1)) != 0) return rc;
        if (j == p) partsB = 0;
        // A: product j    B: column j
        if ((rc = launch(GB, GA, j, rows ? GA : 0, 0, j)) != 0) return rc;
        if (!rows) partsA = 0;
      }
      if (GB > 0 && N - pe > 0) {
        // B: product of the panel's last column
        if ((rc = launch(0, 0, 0, GB, GA, pe - 1)) != 0) return rc;
      }
      if (pe < N) {
        hipLaunchKernelGGL(tri_finish_kernel, dim3(GA), dim3(TB), 0, s, wk.panel, wk.tau, wk.spart,
                           N, nb, pe - 1, pe - 1 - p, partsA, 0);
        KMP_LAUNCH_CHECK();
        if (GB > 0) {
          hipLaunchKernelGGL(tri_finish_kernel, dim3(GB), dim3(TB), 0, s, wk.panel, wk.tau, wk.spart,
                             N, nb, pe - 1, pe - 1 - p, partsB, GA);
          KMP_LAUNCH_CHECK();
        }
        // trailing update A[pe:, pe:] -= V W' + W V'  as one GEMM with K = 2nb
        GemmArgs ga;
        ga.M = N - pe; ga.N = N - pe; ga.K = 2 * nb; ga.batch = G;
        ga.A = wk.panel + pe; ga.lda = N; ga.sA = (int64_t)3 * nb * N;
        ga.B = wk.panel + (int64_t)nb * N + pe; ga.ldb = N; ga.sB = (int64_t)3 * nb * N;
        ga.C = wk.A + (int64_t)pe * N + pe; ga.ldc = N; ga.sC = (int64_t)N * N;
        ga.alpha = -1.0; ga.beta = 1.0;
        kc_begin(KMP_KC_TRAIL, s);
        if ((rc = gemm(s, ga, false, false, true)) != 0) return rc;
        kc_end(KMP_KC_TRAIL, s, over_groups(wk, [&](double n) {
                 const double m = std::max(0.0, n - pe); return 16.0 * m * m; }),
               over_groups(wk, [&](double n) {
                 const double m = std::max(0.0, n - pe); return 4.0 * nb * m * m; }));
        partsA = partsB = 0;
      }
    }
  }
  // Q = H_0 H_1 ... H_{N-2}, accumulated backwards in blocks of NBQ
  // reflectors: Q[p+1:, p+1:] -= V' (T (V Q[p+1:, p+1:])).
  for (int k = 0; k < nch; ++k) {
    if (ws[k].G <= 0) continue;
    const int64_t bx = std::min<int64_t>(ceil_div((int64_t)N * N, 256), 1 << 20);
    hipLaunchKernelGGL(set_identity_kernel, dim3((unsigned)bx, (unsigned)ws[k].G), dim3(256), 0,
                       ss[k], ws[k].Q, N);
    KMP_LAUNCH_CHECK();
  }
  const int last = ((N - 2) / NBQ) * NBQ;
  for (int p = last; p >= 0; p -= NBQ) {
    const int m = N - p - 1;
    if (m <= 0) continue;
    const int kb = std::min(NBQ, N - 1 - p);
    for (int k = 0; k < nch; ++k) {
      const TridiagWork& wk = ws[k];
      const hipStream_t s = ss[k];
      const int G = wk.G;
      if (G <= 0) continue;
      kc_begin(KMP_KC_QFORM, s);
      GemmArgs g0;   // Gram of the block's reflectors (rows p..p+kb-1 of A)
      g0.M = kb; g0.N = kb; g0.K = m; g0.batch = G;
      g0.A = wk.A + (int64_t)p * N + p + 1; g0.lda = N; g0.sA = (int64_t)N * N;
      g0.B = wk.A + (int64_t)p * N + p + 1; g0.ldb = N; g0.sB = (int64_t)N * N;
      g0.C = wk.gram; g0.ldc = NBQ; g0.sC = (int64_t)NBQ * NBQ;
      if ((rc = gemm(s, g0, true, true, true)) != 0) return rc;
      hipLaunchKernelGGL(form_t_kernel, dim3(G), dim3(FTT), 0, s, wk.gram, wk.tau, wk.tmat, N, kb, p,
                         0, (int64_t)0);
      KMP_LAUNCH_CHECK();
      GemmArgs g1;   // X = V[:, p+1:] Q[p+1:, p+1:]   (kb x m)
      g1.M = kb; g1.N = m; g1.K = m; g1.batch = G;
      g1.A = wk.A + (int64_t)p * N + p + 1; g1.lda = N; g1.sA = (int64_t)N * N;
      g1.B = wk.Q + (int64_t)(p + 1) * N + p + 1; g1.ldb = N; g1.sB = (int64_t)N * N;
      g1.C = wk.xbuf; g1.ldc = N; g1.sC = (int64_t)NBQ * N;
      if ((rc = gemm(s, g1, true, false, true)) != 0) return rc;
      GemmArgs g2;   // Y = T X
      g2.M = kb; g2.N = m; g2.K = kb; g2.batch = G;
      g2.A = wk.tmat; g2.lda = NBQ; g2.sA = (int64_t)NBQ * NBQ;
      g2.B = wk.xbuf; g2.ldb = N; g2.sB = (int64_t)NBQ * N;
      g2.C = wk.ybuf; g2.ldc = N; g2.sC = (int64_t)NBQ * N;
      if ((rc = gemm(s, g2, true, false, true)) != 0) return rc;
      GemmArgs g3;   // Q[p+1:, p+1:] -= V' Y
      g3.M = m; g3.N = m; g3.K = kb; g3.batch = G;
      g3.A = wk.A + (int64_t)p * N + p + 1; g3.lda = N; g3.sA = (int64_t)N * N;
      g3.B = wk.ybuf; g3.ldb = N; g3.sB = (int64_t)NBQ * N;
      g3.C = wk.Q + (int64_t)(p + 1) * N + p + 1; g3.ldc = N; g3.sC = (int64_t)N * N;
      g3.alpha = -1.0; g3.beta = 1.0;
      if ((rc = gemm(s, g3, false, false, true)) != 0) return rc;
      // Q block read by the first product, read and written by the update
      kc_end(KMP_KC_QFORM, s, over_groups(wk, [&](double n) {
               const double mm = std::max(0.0, n - p - 1); return 24.0 * mm * mm; }),
             over_groups(wk, [&](double n) {
               const double mm = std::max(0.0, n - p - 1);
               return 4.0 * kb * mm * mm + 2.0 * kb * kb * mm; }));
    }
  }
  return 0;
}

int tridiagonalize(hipStream_t s, const TridiagWork& w) { return tridiagonalize_multi(&s, &w, 1); }

}  // namespace kmp
