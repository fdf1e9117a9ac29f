// Batched regularisation-path solver in the tridiagonal basis K_v = Q T Q'.
//
// Every column is one (tau, lambda) problem of one group (bandwidth, fold).
// With hats denoting Q' coordinates (a = Q'alpha), one iteration of the
// accelerated majorise-minimise method (Appendix A.1 update; Algorithm 1
// inner loop; Appendix A.3 block inverse of H) is
//
//   f      = Q (T abar) + bbar                      (first path GEMM)
//   z      = psi(y, f) / n_v,  d0 = 1'z             (its epilogue)
//   zhat   = Q' z                                   (second path GEMM)
//   w      = zhat + 2 lambda abar                   (= Q'(z + 2 lambda alpha))
//   t      = vhat' T w                              (= v' K (z + 2 lambda alpha))
//   x      = (2 lambda I + T/(n_v kappa))^{-1} w    (tridiagonal solve)
//   Da     = g (t - d0) vhat + x,   Db = g (d0 - t)
//   a_new  = abar - Da,             b_new = bbar - Db
//
// with vhat = (2 lambda I + T/(n_v kappa))^{-1} Q'1 / (n_v kappa) and
// g = 1/(2 lambda (Q'1)' vhat) precomputed once per smoothing stage. These
// are the paper's v and g taken as the exact Schur complement of the
// (n+1)-square majoriser H = [[1/kappa, 1'K/(n kappa)], [K1/(n kappa),
// 2 lambda K + K K/(n kappa)]], written in the basis Q instead of the
// eigenvectors. The column stops when n_v max(||w||_2, |d0|) <= tol at the
// extrapolated point, which it then keeps.
#include "kmp_common.h"
#include "kmp_kernels.h"

namespace kmp {

constexpr int PB = 256;   // threads per column workgroup
constexpr int PW = 4;

// ------------------------------------------------------------- small setup
__global__ void gather_labels_kernel(const double* __restrict__ y, const int32_t* __restrict__ tidx,
                                     int V, int S_b, int N, double* __restrict__ ylab) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t tot = (int64_t)S_b * V * N;
  if (idx >= tot) return;
  const int64_t i = idx % N;
  const int64_t g = idx / N;
  const int v = (int)(g % V);
  const int32_t src = tidx[(int64_t)v * N + i];
  ylab[idx] = src >= 0 ? y[src] : 0.0;
}

int gather_labels(hipStream_t s, const double* y, const int32_t* tidx, int V, int S_b, int N,
                  double* ylab) {
  const int64_t tot = (int64_t)S_b * V * N;
  hipLaunchKernelGGL(gather_labels_kernel, dim3((unsigned)ceil_div(tot, 256)), dim3(256), 0, s, y,
                     tidx, V, S_b, N, ylab);
  KMP_LAUNCH_CHECK();
  return 0;
}

// c = Q'1 over the valid rows of each group. Block (64 columns x 16 row
// groups): lanes read consecutive columns of a row (coalesced), the 16 row
// groups are added in a fixed order.
constexpr int OPC = 64, OPR = 16;
__global__ __launch_bounds__(OPC * OPR) void ones_projection_kernel(const double* __restrict__ Q,
                                                                    const int* __restrict__ nv,
                                                                    int N, double* __restrict__ cvec) {
  __shared__ double part[OPR][OPC];
  const int g = blockIdx.y;
  const int j = blockIdx.x * OPC + threadIdx.x, ry = threadIdx.y;
  const double* Qg = Q + (int64_t)g * N * N;
  const int m = nv[g];
  double s = 0.0;
  if (j < N)
    for (int i = ry; i < m; i += OPR) s += Qg[(int64_t)i * N + j];
  part[ry][threadIdx.x] = s;
  __syncthreads();
  if (ry == 0 && j < N) {
    double t = 0.0;
    for (int r = 0; r < OPR; ++r) t += part[r][threadIdx.x];
    cvec[(int64_t)g * N + j] = t;
  }
}

int group_ones_projection(hipStream_t s, const double* Q, const int* nv, int G, int N, double* cvec) {
  hipLaunchKernelGGL(ones_projection_kernel, dim3((unsigned)ceil_div(N, OPC), (unsigned)G),
                     dim3(OPC, OPR), 0, s, Q, nv, N, cvec);
  KMP_LAUNCH_CHECK();
  return 0;
}

int path_init_columns(hipStream_t s, const PathArrays& p) {
  const size_t cols = (size_t)p.G * p.C;
  const size_t vec = cols * p.N * sizeof(double);
  KMP_HIP_TRY(hipMemsetAsync(p.ahat, 0, vec, s));
  KMP_HIP_TRY(hipMemsetAsync(p.abar, 0, vec, s));
  KMP_HIP_TRY(hipMemsetAsync(p.bmat, 0, vec, s));
  KMP_HIP_TRY(hipMemsetAsync(p.beta, 0, cols * sizeof(double), s));
  KMP_HIP_TRY(hipMemsetAsync(p.bbar, 0, cols * sizeof(double), s));
  KMP_HIP_TRY(hipMemsetAsync(p.flag, 0, cols * sizeof(int), s));
  KMP_HIP_TRY(hipMemsetAsync(p.iters, 0, cols * sizeof(int), s));
  KMP_HIP_TRY(hipMemsetAsync(p.iters_total, 0, cols * sizeof(int), s));
  return 0;
}

// Sum over groups of f(valid rows) for the work counters.
template <typename F>
static double over_groups(const PathArrays& p, F f) {
  double a = 0.0;
  for (int g = 0; g < p.G; ++g) a += f((double)(p.nv_host ? p.nv_host[g] : p.N));
  return a;
}

// ---------------------------------------------------------- scan helpers
// Affine map x -> a x + b; compose(second, first) = second o first.
struct Aff {
  double a, b;
};
__device__ __forceinline__ Aff compose(Aff second, Aff first) {
  return Aff{second.a * first.a, fma(second.a, first.b, second.b)};
}

// Exclusive prefix composition across the block in thread order (thread t
// receives map_{t-1} o ... o map_0, identity for t = 0). `sh` holds PW Affs.
__device__ __forceinline__ Aff block_exclusive_scan(Aff m, Aff* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  Aff inc = m;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double pa = __shfl_up(inc.a, off, 64);
    const double pb = __shfl_up(inc.b, off, 64);
    if (lane >= off) inc = compose(inc, Aff{pa, pb});
  }
  // exclusive within the wave
  double ea = __shfl_up(inc.a, 1, 64), eb = __shfl_up(inc.b, 1, 64);
  Aff ex = lane == 0 ? Aff{1.0, 0.0} : Aff{ea, eb};
  __syncthreads();
  if (lane == 63) sh[w] = inc;
  __syncthreads();
  Aff pre{1.0, 0.0};
  for (int k = 0; k < w; ++k) pre = compose(sh[k], pre);
  return compose(ex, pre);
}

// Same in reverse thread order (thread t receives map_{t+1} o ... o map_last).
__device__ __forceinline__ Aff block_exclusive_scan_rev(Aff m, Aff* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  Aff inc = m;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double pa = __shfl_down(inc.a, off, 64);
    const double pb = __shfl_down(inc.b, off, 64);
    if (lane + off < 64) inc = compose(inc, Aff{pa, pb});
  }
  double ea = __shfl_down(inc.a, 1, 64), eb = __shfl_down(inc.b, 1, 64);
  Aff ex = lane == 63 ? Aff{1.0, 0.0} : Aff{ea, eb};
  __syncthreads();
  if (lane == 0) sh[w] = inc;
  __syncthreads();
  Aff pre{1.0, 0.0};
  for (int k = PW - 1; k > w; --k) pre = compose(sh[k], pre);
  return compose(ex, pre);
}

// Solve (L D L') x = w on the rows [i0, i0 + E) owned by this thread, L unit
// lower bidiagonal (l[i] = L[i+1][i]), dv = 1/D. lv holds l on the own rows,
// lprev = l[i0 - 1] (0 for the first thread). wv holds w on entry and x on
// exit. Both triangular solves are first-order affine recurrences, done as
// block-wide scans of affine maps.
template <int E>
__device__ __forceinline__ void ldl_solve(double (&wv)[E], const double (&lv)[E], double lprev,
                                          const double (&dv)[E], Aff* sh) {
  // forward: y_i = w_i - l_{i-1} y_{i-1}
  Aff m{1.0, 0.0};
  {
    double ca = 1.0, cb = 0.0, lp = lprev;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      ca = -lp * ca;
      cb = fma(-lp, cb, wv[e]);
      lp = lv[e];
    }
    m = Aff{ca, cb};
  }
  Aff pre = block_exclusive_scan(m, sh);
  {
    double yin = pre.b;                       // y_{i0-1} (maps applied to 0)
    double lp = lprev;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const double yi = fma(-lp, yin, wv[e]);
      wv[e] = yi;
      yin = yi;
      lp = lv[e];
    }
  }
  // diagonal
#pragma unroll
  for (int e = 0; e < E; ++e) wv[e] *= dv[e];
  // backward: x_i = z_i - l_i x_{i+1}
  {
    double ca = 1.0, cb = 0.0;
#pragma unroll
    for (int e = E - 1; e >= 0; --e) {
      ca = -lv[e] * ca;
      cb = fma(-lv[e], cb, wv[e]);
    }
    m = Aff{ca, cb};
  }
  pre = block_exclusive_scan_rev(m, sh);
  {
    double xin = pre.b;                       // x_{i0+E}
#pragma unroll
    for (int e = E - 1; e >= 0; --e) {
      const double xi = fma(-lv[e], xin, wv[e]);
      wv[e] = xi;
      xin = xi;
    }
  }
}

// y = T x for the own rows of a thread (T tridiagonal, diagonal Td, off-
// diagonal To[i] = T[i+1][i]); neighbours across threads through LDS.
template <int E>
__device__ __forceinline__ void tri_apply(const double (&x)[E], double (&y)[E], int i0, int N,
                                          const double* __restrict__ Tdg,
                                          const double* __restrict__ Tog, double* edge_lo,
                                          double* edge_hi) {
  const int t = threadIdx.x;
  __syncthreads();
  edge_lo[t] = x[0];
  edge_hi[t] = x[E - 1];
  __syncthreads();
  const double left = t > 0 ? edge_hi[t - 1] : 0.0;
  const double right = t + 1 < (int)blockDim.x ? edge_lo[t + 1] : 0.0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = i0 + e;
    double bv = 0.0;
    if (i < N) {
      const double xl = e > 0 ? x[e - 1] : left;
      const double xr = e + 1 < E ? x[e + 1] : right;
      bv = Tdg[i] * x[e];
      if (i > 0) bv = fma(Tog[i - 1], xl, bv);
      if (i + 1 < N) bv = fma(Tog[i], xr, bv);
    }
    y[e] = bv;
  }
}

// ------------------------------------------------------ per-stage factors
// One workgroup per column: LDL' of M = 2 lambda I + T/(n_v kappa) (the
// pivot recurrence is sequential, run by one thread over LDS-staged chunks
// of T), then vhat = M^{-1} c/(n_v kappa), u = T vhat, g = 1/(2 lambda
// c'vhat); restart the momentum (r = 1, abar = ahat, B = T ahat) and
// reactivate the columns that stopped in the previous stage.
template <int E>
__global__ __launch_bounds__(PB) void precompute_kernel(
    int N, int C, const int* __restrict__ nv, const double* __restrict__ Td,
    const double* __restrict__ To, const double* __restrict__ cvec, const double* __restrict__ lamv,
    double kappa, double* __restrict__ ldl_l, double* __restrict__ ldl_d, double* __restrict__ vhat,
    double* __restrict__ uvec, double* __restrict__ gcoef, const double* __restrict__ ahat,
    double* __restrict__ abar, double* __restrict__ bmat, const double* __restrict__ beta,
    double* __restrict__ bbar, double* __restrict__ rmom, int* __restrict__ flag,
    int* __restrict__ iters) {
  __shared__ double red[PW];
  __shared__ Aff sh[PW];
  __shared__ double sd[PB], so[PB], sl[PB], sdi[PB];
  __shared__ double edge_lo[PB], edge_hi[PB];
  const int64_t gc = blockIdx.x;
  const int g = (int)(gc / C);
  const int t = threadIdx.x;
  const int i0 = t * E;
  const int64_t base = gc * N;
  const double lam = lamv[gc];
  const double sc = 1.0 / ((double)nv[g] * kappa);
  const double* d = Td + (int64_t)g * N;
  const double* o = To + (int64_t)g * N;
  const double* c = cvec + (int64_t)g * N;
  // pivots: D_i = 2 lambda + T_ii sc - l_{i-1} T_{i,i-1} sc, l_i = T_{i+1,i} sc / D_i
  double lrun = 0.0, orun = 0.0;
  for (int c0 = 0; c0 < N; c0 += PB) {
    const int i = c0 + t;
    sd[t] = i < N ? d[i] : 0.0;
    so[t] = i < N ? o[i] : 0.0;
    __syncthreads();
    if (t == 0) {
      const int cnt = (N - c0 < PB) ? N - c0 : PB;
      for (int k = 0; k < cnt; ++k) {
        const double piv = fma(-lrun, orun, fma(sd[k], sc, 2.0 * lam));
        const double dinv = 1.0 / piv;
        orun = so[k] * sc;
        lrun = (c0 + k + 1 < N) ? orun * dinv : 0.0;
        sl[k] = lrun;
        sdi[k] = dinv;
      }
    }
    __syncthreads();
    if (i < N) {
      ldl_l[base + i] = sl[t];
      ldl_d[base + i] = sdi[t];
    }
    __syncthreads();
  }
  double lv[E], dv[E], wv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = i0 + e;
    lv[e] = i < N ? ldl_l[base + i] : 0.0;
    dv[e] = i < N ? ldl_d[base + i] : 0.0;
    wv[e] = i < N ? c[i] * sc : 0.0;
  }
  const double lprev = (i0 > 0 && i0 - 1 < N) ? ldl_l[base + i0 - 1] : 0.0;
  ldl_solve<E>(wv, lv, lprev, dv, sh);
  double u[E];
  tri_apply<E>(wv, u, i0, N, d, o, edge_lo, edge_hi);
  double cv = 0.0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = i0 + e;
    if (i < N) {
      vhat[base + i] = wv[e];
      uvec[base + i] = u[e];
      cv = fma(c[i], wv[e], cv);
    }
  }
  cv = block_sum<PW>(cv, red);
  // stage restart of the accelerated iteration
  double ah[E], bm[E];
#pragma unroll
  for (int e = 0; e < E; ++e) ah[e] = (i0 + e < N) ? ahat[base + i0 + e] : 0.0;
  tri_apply<E>(ah, bm, i0, N, d, o, edge_lo, edge_hi);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = i0 + e;
    if (i < N) {
      abar[base + i] = ah[e];
      bmat[base + i] = bm[e];
    }
  }
  if (t == 0) {
    gcoef[gc] = 1.0 / (2.0 * lam * cv);
    bbar[gc] = beta[gc];
    rmom[gc] = 1.0;
    if (flag[gc] == 1 || flag[gc] == 2) flag[gc] = 0;
    iters[gc] = 0;
  }
}

int path_stage_precompute(hipStream_t s, const PathArrays& p, double kappa) {
  const unsigned cols = (unsigned)(p.G * p.C);
  kc_begin(KMP_KC_PRECOMPUTE, s);
#define KMP_PRE(EE)                                                                              \
  hipLaunchKernelGGL(precompute_kernel<EE>, dim3(cols), dim3(PB), 0, s, p.N, p.C, p.nv, p.Tdiag, \
                     p.Toff, p.cvec, p.lam, kappa, p.ldl_l, p.ldl_d, p.vhat, p.uvec, p.gcoef,    \
                     p.ahat, p.abar, p.bmat, p.beta, p.bbar, p.rmom, p.flag, p.iters)
  if (p.N <= PB * 1) KMP_PRE(1);
  else if (p.N <= PB * 2) KMP_PRE(2);
  else if (p.N <= PB * 4) KMP_PRE(4);
  else if (p.N <= PB * 8) KMP_PRE(8);
  else if (p.N <= PB * 16) KMP_PRE(16);
  else if (p.N <= PB * 32) KMP_PRE(32);
  else {
    set_error("path: more than 8192 training points per fold is not supported yet");
    return KMP_EINVAL;
  }
#undef KMP_PRE
  KMP_LAUNCH_CHECK();
  // reads T, c, ahat; writes l, 1/d, vhat, u, abar, T ahat
  kc_end(KMP_KC_PRECOMPUTE, s, over_groups(p, [&](double n) { return 8.0 * n * p.C * 8.0; }),
         over_groups(p, [&](double n) { return 20.0 * n * p.C; }));
  return 0;
}

// ------------------------------------------------------- the update (K2)
// One workgroup per column; thread t owns rows [t*E, t*E + E).
template <int E>
__global__ __launch_bounds__(PB) void update_kernel(
    int N, int C, int RT, const int* __restrict__ nvv, const double* __restrict__ Td,
    const double* __restrict__ To, const double* __restrict__ lamv,
    const double* __restrict__ zpart, int S2, int64_t sP, double* __restrict__ ahat,
    double* __restrict__ abar,
    double* __restrict__ bmat, const double* __restrict__ ldl_l, const double* __restrict__ ldl_d,
    const double* __restrict__ vhat, const double* __restrict__ uvec,
    const double* __restrict__ gcoef, const double* __restrict__ partial,
    double* __restrict__ beta, double* __restrict__ bbar, double* __restrict__ rmom,
    double* __restrict__ kktv, int* __restrict__ flag, int* __restrict__ iters,
    int* __restrict__ iters_total, double tol, int max_iter, int restart) {
  __shared__ double red[PW];
  __shared__ Aff sh[PW];
  __shared__ double edge_lo[PB], edge_hi[PB];
  const int64_t gc = blockIdx.x;
  if (flag[gc] != 0) return;
  const int g = (int)(gc / C), c = (int)(gc % C);
  const int t = threadIdx.x;
  const int i0 = t * E;
  const int64_t base = gc * N;
  const double lam = lamv[gc];
  const double nvd = (double)nvv[g];
  const double* Tdg = Td + (int64_t)g * N;
  const double* Tog = To + (int64_t)g * N;

  double d0 = 0.0;
  {
    const double* pg = partial + (int64_t)g * RT * C + c;
    for (int r = 0; r < RT; ++r) d0 += pg[(int64_t)r * C];
  }
  double wv[E], ab[E], ah[E];
  double tl = 0.0, n2 = 0.0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = i0 + e;
    if (i < N) {
      ab[e] = abar[base + i];
      ah[e] = ahat[base + i];
      double zh = 0.0;
      for (int sk = 0; sk < S2; ++sk) zh += zpart[(int64_t)sk * sP + base + i];
      wv[e] = fma(2.0 * lam, ab[e], zh);
      tl = fma(uvec[base + i], wv[e], tl);
      n2 = fma(wv[e], wv[e], n2);
    } else {
      ab[e] = ah[e] = wv[e] = 0.0;
    }
  }
  const double tsum = block_sum<PW>(tl, red);
  const double n2sum = block_sum<PW>(n2, red);
  const double kkt = nvd * fmax(sqrt(n2sum), fabs(d0));
  const double bb = bbar[gc];
  if (!(kkt == kkt) || kkt > 1e300) {          // non-finite
    if (t == 0) { flag[gc] = 3; kktv[gc] = kkt; }
    return;
  }
  if (kkt <= tol) {                            // certified at the extrapolated point
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (i0 + e < N) ahat[base + i0 + e] = ab[e];
    if (t == 0) { beta[gc] = bb; flag[gc] = 1; kktv[gc] = kkt; }
    return;
  }
  double lv[E], dv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    lv[e] = (i0 + e < N) ? ldl_l[base + i0 + e] : 0.0;
    dv[e] = (i0 + e < N) ? ldl_d[base + i0 + e] : 0.0;
  }
  const double lprev = (i0 > 0 && i0 - 1 < N) ? ldl_l[base + i0 - 1] : 0.0;
  ldl_solve<E>(wv, lv, lprev, dv, sh);
  // step, new iterate and the restart test
  const double gco = gcoef[gc];
  const double sa = gco * (tsum - d0);
  const double db = gco * (d0 - tsum);
  const double bn = bb - db;
  const double bold = beta[gc];
  double rd = 0.0;
  double an[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = i0 + e;
    double da = 0.0;
    if (i < N) da = fma(sa, vhat[base + i], wv[e]);
    an[e] = ab[e] - da;
    rd = fma(da, an[e] - ah[e], rd);
  }
  rd = block_sum<PW>(rd, red) + db * (bn - bold);
  const double r = rmom[gc];
  const double rn = (restart && rd > 0.0) ? 1.0 : 0.5 * (1.0 + sqrt(1.0 + 4.0 * r * r));
  const double coef = (rn - 1.0) / (0.5 * (1.0 + sqrt(1.0 + 4.0 * rn * rn)));
  double nb_[E];
#pragma unroll
  for (int e = 0; e < E; ++e) nb_[e] = fma(coef, an[e] - ah[e], an[e]);
  edge_lo[t] = nb_[0];
  edge_hi[t] = nb_[E - 1];
  __syncthreads();
  const double left = t > 0 ? edge_hi[t - 1] : 0.0;
  const double right = t + 1 < PB ? edge_lo[t + 1] : 0.0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = i0 + e;
    if (i < N) {
      const double xl = e > 0 ? nb_[e - 1] : left;
      const double xr = e + 1 < E ? nb_[e + 1] : right;
      double bv = Tdg[i] * nb_[e];
      if (i > 0) bv = fma(Tog[i - 1], xl, bv);
      if (i + 1 < N) bv = fma(Tog[i], xr, bv);
      ahat[base + i] = an[e];
      abar[base + i] = nb_[e];
      bmat[base + i] = bv;
    }
  }
  if (t == 0) {
    beta[gc] = bn;
    bbar[gc] = fma(coef, bn - bold, bn);
    rmom[gc] = rn;
    kktv[gc] = kkt;
    const int it = iters[gc] + 1;
    iters[gc] = it;
    iters_total[gc] += 1;
    if (it >= max_iter) flag[gc] = 2;
  }
}

int path_iteration(hipStream_t s, const PathArrays& p, double delta, double kappa, double tol,
                   int max_iter, int restart) {
  (void)kappa;
  int rc;
  const int RT = (int)ceil_div(p.N, 64);
  const int64_t sC = (int64_t)p.N * p.C;
  const int64_t sP = (int64_t)p.G * sC;
  // f = Q (T abar) as split-K partials, then z = psi(y, f + bbar)/n_v with
  // 64-row column sums
  GemmArgs g1;
  g1.M = p.N; g1.N = p.C; g1.K = p.N; g1.batch = p.G;
  g1.A = p.Q; g1.lda = p.N; g1.sA = (int64_t)p.N * p.N;
  g1.B = p.bmat; g1.ldb = p.N; g1.sB = sC;
  g1.ldc = p.N; g1.sC = sC;
  const int S1 = splitk_parts(g1);
  LossEpi e;
  e.loss = p.loss; e.delta = delta;
  e.y = p.ylab; e.sy = p.N; e.nv = p.nv;
  e.bbar = p.bbar; e.sbb = p.C; e.tau = p.tau; e.stau = p.C;
  e.partial = p.partial; e.spart = (int64_t)RT * p.C;
  const double gflops = over_groups(p, [&](double n) { return 2.0 * n * n * p.C; });
  const double gbytes = over_groups(p, [&](double n) { return 8.0 * (n * n + 2.0 * n * p.C); });
  kc_begin(KMP_KC_GEMM_F, s);
  if ((rc = gemm_partial(s, g1, true, S1, p.fpart, sP)) != 0) return rc;
  if ((rc = loss_epilogue(s, p.N, p.C, p.G, S1, p.fpart, p.N, sC, sP, p.zmat, e)) != 0) return rc;
  kc_end(KMP_KC_GEMM_F, s, gbytes, gflops);
  // zhat = Q' z as split-K partials (added by the update kernel)
  GemmArgs g2;
  g2.M = p.N; g2.N = p.C; g2.K = p.N; g2.batch = p.G;
  g2.A = p.Q; g2.lda = p.N; g2.sA = (int64_t)p.N * p.N;
  g2.B = p.zmat; g2.ldb = p.N; g2.sB = sC;
  g2.ldc = p.N; g2.sC = sC;
  const int S2 = splitk_parts(g2);
  kc_begin(KMP_KC_GEMM_ZHAT, s);
  if ((rc = gemm_partial(s, g2, false, S2, p.zpart, sP)) != 0) return rc;
  kc_end(KMP_KC_GEMM_ZHAT, s, gbytes, gflops);
  const unsigned cols = (unsigned)(p.G * p.C);
  kc_begin(KMP_KC_UPDATE, s);
#define KMP_UPD(EE)                                                                              \
  hipLaunchKernelGGL(update_kernel<EE>, dim3(cols), dim3(PB), 0, s, p.N, p.C, RT, p.nv, p.Tdiag, \
                     p.Toff, p.lam, p.zpart, S2, sP, p.ahat, p.abar, p.bmat, p.ldl_l, p.ldl_d,   \
                     p.vhat,                                                                     \
                     p.uvec, p.gcoef, p.partial, p.beta, p.bbar, p.rmom, p.kkt, p.flag, p.iters, \
                     p.iters_total, tol, max_iter, restart)
  if (p.N <= PB * 1) KMP_UPD(1);
  else if (p.N <= PB * 2) KMP_UPD(2);
  else if (p.N <= PB * 4) KMP_UPD(4);
  else if (p.N <= PB * 8) KMP_UPD(8);
  else if (p.N <= PB * 16) KMP_UPD(16);
  else if (p.N <= PB * 32) KMP_UPD(32);
  else {
    set_error("path: more than 8192 training points per fold is not supported yet");
    return KMP_EINVAL;
  }
#undef KMP_UPD
  KMP_LAUNCH_CHECK();
  // per column element: read zhat, abar, ahat, l, 1/d, vhat, u; write ahat,
  // abar, T abar (80 bytes), counted for every column of the launch
  kc_end(KMP_KC_UPDATE, s, over_groups(p, [&](double n) { return 80.0 * n * p.C; }),
         over_groups(p, [&](double n) { return 30.0 * n * p.C; }));
  return 0;
}

__global__ void count_active_kernel(const int* __restrict__ flag, int64_t cols, int* __restrict__ out) {
  __shared__ double red[PW];
  double c = 0.0;
  for (int64_t i = threadIdx.x; i < cols; i += blockDim.x) c += (flag[i] == 0) ? 1.0 : 0.0;
  c = block_sum<PW>(c, red);
  if (threadIdx.x == 0) *out = (int)c;
}

int path_count_active(hipStream_t s, const PathArrays& p) {
  hipLaunchKernelGGL(count_active_kernel, dim3(1), dim3(PB), 0, s, p.flag, (int64_t)p.G * p.C,
                     p.active_count);
  KMP_LAUNCH_CHECK();
  return 0;
}

// --------------------------------------------------------------- finalize
// B = T ahat for every column (T tridiagonal per group).
__global__ void tri_mult_kernel(int N, int C, int64_t total, const double* __restrict__ Td,
                                const double* __restrict__ To, const double* __restrict__ x,
                                double* __restrict__ y) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int64_t col = idx / N;
  const int i = (int)(idx % N);
  const int g = (int)(col / C);
  const double* d = Td + (int64_t)g * N;
  const double* o = To + (int64_t)g * N;
  const double* xc = x + col * N;
  double v = d[i] * xc[i];
  if (i > 0) v = fma(o[i - 1], xc[i - 1], v);
  if (i + 1 < N) v = fma(o[i], xc[i + 1], v);
  y[idx] = v;
}

// One workgroup per column: objective on the training points, CV sums on the
// held-out points, scatter of alpha into the output layout.
__global__ __launch_bounds__(256) void cv_reduce_kernel(
    int n, int N, int Mh, int C, int V, int Qt, int L, int s0, int loss, double delta,
    const double* __restrict__ y, const int32_t* __restrict__ tidx,
    const int32_t* __restrict__ hidx, const int* __restrict__ nvv, const double* __restrict__ lamv,
    const double* __restrict__ tauv, const double* __restrict__ alpha_loc,
    const double* __restrict__ ftrain, const double* __restrict__ fheld,
    const double* __restrict__ betav, const int* __restrict__ flag,
    const int* __restrict__ iters_total, double* __restrict__ alpha_out,
    double* __restrict__ beta_out, double* __restrict__ obj_out, double* __restrict__ cv_out,
    int32_t* __restrict__ err_out, int32_t* __restrict__ it_out, int32_t* __restrict__ st_out) {
  __shared__ double red[PW];
  const int64_t gc = blockIdx.x;
  const int g = (int)(gc / C), c = (int)(gc % C);
  const int v = g % V, sl = g / V;
  const int q = c / L, l = c % L;
  const int64_t cell = (((int64_t)(s0 + sl) * Qt + q) * V + v) * L + l;
  const int nv = nvv[g];
  const double lam = lamv[gc], tau = tauv[gc], b = betav[gc];
  const double* A = alpha_loc + gc * N;
  const double* ft = ftrain + gc * N;
  const double* fh = fheld + gc * Mh;
  const int32_t* T = tidx + (int64_t)v * N;
  const int32_t* H = hidx + (int64_t)v * Mh;
  double* aout = alpha_out + cell * n;
  double ls = 0.0, pen = 0.0;
  for (int j = threadIdx.x; j < nv; j += blockDim.x) {
    const int32_t i = T[j];
    const double kf = ft[j];                 // (K_v alpha)_j
    ls += loss_value(loss, y[i], kf + b, delta, tau);
    pen = fma(A[j], kf, pen);
    aout[i] = A[j];
  }
  double cs = 0.0, ce = 0.0;
  for (int k = threadIdx.x; k < Mh; k += blockDim.x) {
    const int32_t i = H[k];
    if (i < 0) continue;
    const double fi = fh[k] + b;
    cs += loss_eval(loss, y[i], fi, tau);
    if (loss != 2 && y[i] * fi <= 0.0) ce += 1.0;
  }
  ls = block_sum<PW>(ls, red);
  pen = block_sum<PW>(pen, red);
  cs = block_sum<PW>(cs, red);
  ce = block_sum<PW>(ce, red);
  if (threadIdx.x == 0) {
    beta_out[cell] = b;
    obj_out[cell] = ls / (double)nv + lam * pen;
    cv_out[cell] = cs;
    if (err_out) err_out[cell] = (int32_t)ce;
    if (it_out) it_out[cell] = iters_total[gc];
    if (st_out) {
      const int fl = flag[gc];
      st_out[cell] = fl == 1 ? 0 : (fl == 3 ? 2 : 1);
    }
  }
}

int path_finalize(hipStream_t s, const PathArrays& p, const FinalArgs& fa) {
  int rc;
  kc_begin(KMP_KC_FINALIZE, s);
  const int64_t sNC = (int64_t)p.N * p.C;
  // alpha_loc = Q ahat (into zmat)
  GemmArgs g;
  g.M = p.N; g.N = p.C; g.K = p.N; g.batch = p.G;
  g.A = p.Q; g.lda = p.N; g.sA = (int64_t)p.N * p.N;
  g.B = p.ahat; g.ldb = p.N; g.sB = sNC;
  g.C = p.zmat; g.ldc = p.N; g.sC = sNC;
  if ((rc = gemm(s, g, true, true, false)) != 0) return rc;
  // training predictions K_v alpha = Q (T ahat)
  const int64_t tot = (int64_t)p.G * sNC;
  hipLaunchKernelGGL(tri_mult_kernel, dim3((unsigned)ceil_div(tot, 256)), dim3(256), 0, s, p.N, p.C,
                     tot, p.Tdiag, p.Toff, p.ahat, p.bmat);
  KMP_LAUNCH_CHECK();
  GemmArgs gt = g;
  gt.B = p.bmat;
  gt.C = fa.ftrain;
  if ((rc = gemm(s, gt, true, true, false)) != 0) return rc;
  // held-out kernel blocks K[H_v, T_v] (into the factor buffer, no longer
  // needed), then held-out predictions K[H_v, T_v] alpha
  if ((rc = rbf_blocks(s, fa.X, fa.d, fa.ldx, fa.nrm, fa.hidx, fa.Mh, fa.Mh, fa.tidx, p.N, p.N,
                       fa.V, fa.inv2s2, fa.S_b, fa.kh, (int64_t)fa.V * p.N * p.N,
                       (int64_t)p.N * p.N, p.N)) != 0)
    return rc;
  GemmArgs gh;
  gh.M = fa.Mh; gh.N = p.C; gh.K = p.N; gh.batch = p.G;
  gh.A = fa.kh; gh.lda = p.N; gh.sA = (int64_t)p.N * p.N;
  gh.B = p.zmat; gh.ldb = p.N; gh.sB = sNC;
  gh.C = fa.fbuf; gh.ldc = fa.Mh; gh.sC = (int64_t)fa.Mh * p.C;
  if ((rc = gemm(s, gh, true, true, false)) != 0) return rc;
  hipLaunchKernelGGL(cv_reduce_kernel, dim3((unsigned)(p.G * p.C)), dim3(256), 0, s, fa.n, p.N,
                     fa.Mh, p.C, fa.V, fa.Qt, fa.L, fa.s0, p.loss, fa.delta, fa.y, fa.tidx, fa.hidx,
                     p.nv, p.lam, p.tau, p.zmat, fa.ftrain, fa.fbuf, p.beta, p.flag, p.iters_total,
                     fa.alpha, fa.beta_out, fa.objective, fa.cv_sum, fa.cv_err, fa.iters, fa.status);
  KMP_LAUNCH_CHECK();
  // three N x C x N products (alpha, training f, held-out f on Mh rows), the
  // held-out kernel block (2d flops per entry) and the column reads/writes
  kc_end(KMP_KC_FINALIZE, s,
         over_groups(p, [&](double n) {
           return 8.0 * (2.0 * n * n + 5.0 * n * p.C + 2.0 * fa.Mh * n + fa.Mh * p.C); }),
         over_groups(p, [&](double n) {
           return 4.0 * n * n * p.C + 2.0 * fa.Mh * n * (p.C + fa.d); }));
  return 0;
}

}  // namespace kmp
