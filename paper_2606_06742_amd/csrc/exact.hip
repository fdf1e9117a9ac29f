// Finite smoothing to the exact hinge SVM (Appendix A.1; Algorithm 1's outer
// loop ends when the SVM's KKT conditions hold).
//
// From the delta-smoothed solution of each column, the exact minimiser of
//   P(alpha, beta) = (1/n) sum_i (1 - y_i f_i)_+ + lambda alpha' K alpha
// is recovered on the point sets it induces. With a_i = 2 n lambda y_i alpha_i
// the SVM's KKT conditions are a_i in [0, 1], sum_i y_i a_i = 0 and, per point,
// u_i = y_i f_i < 1 with a_i = 1 (set L), u_i > 1 with a_i = 0 (set R), or
// u_i = 1 (set E). Given the sets, u_i = 1 on E and the balance sum y a = 0
// are a linear system in (a_E, beta):
//   c y_i sum_{j in E} y_j K_ij a_j + y_i beta = 1 - c y_i sum_{j in L} y_j K_ij,
//   sum_{j in E} y_j a_j = - sum_{j in L} y_j,            c = 1/(2 n lambda),
// solved per column by LU with partial pivoting in one workgroup. The
// solution is the SVM's minimiser when every condition holds; otherwise the
// violators change sets (a_E below 0 to R, above 1 to L, points of L or R
// whose margin crosses 1 to E) and the system is solved again. The first
// sets are the smoothed solution's: L below the quadratic zone, E inside,
// R above. With no point in E the sets fix a, the balance must hold by
// itself and beta may take any value that keeps every point on its side.
//
// Kernel matrices come from the observation-space Gram the finalize builds
// (row-major, order N per group); the products K w run as GEMMs between the
// kernels here.
#include "kmp_common.h"
#include "kmp_kernels.h"

namespace kmp {

constexpr int XB = 256;   // threads per column workgroup
constexpr int XW = XB / 64;

// state[i] of every row of every column from u = y (f + beta) at the final
// delta: 0 below the zone (L), 1 inside (E), 2 above (R), 3 padding. The
// working intercept starts at the smoothed one.
__global__ __launch_bounds__(XB) void exact_init_kernel(int N, int C, const int* __restrict__ nv,
                                                        double delta, const double* __restrict__ ylab,
                                                        const double* __restrict__ f,
                                                        const double* __restrict__ beta,
                                                        int32_t* __restrict__ state,
                                                        double* __restrict__ beta_x,
                                                        int* __restrict__ xflag) {
  const int64_t gc = blockIdx.y;
  const int g = (int)(gc / C);
  const int i = blockIdx.x * XB + threadIdx.x;
  if (i == 0) {
    xflag[gc] = 0;
    beta_x[gc] = beta[gc];
  }
  if (i >= N) return;
  int st = 3;
  if (i < nv[g]) {
    const double u = ylab[(int64_t)g * N + i] * (f[gc * N + i] + beta[gc]);
    st = u <= 1.0 - delta ? 0 : (u >= 1.0 + delta ? 2 : 1);
  }
  state[gc * N + i] = st;
}

// Block-wide exclusive prefix of a per-thread count (fixed order), and total.
__device__ __forceinline__ int block_scan(int v, int* sh, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  __syncthreads();
  if (lane == 63) sh[w] = incl;
  __syncthreads();
  int base = 0, tot = 0;
  for (int k = 0; k < XW; ++k) {
    if (k < w) base += sh[k];
    tot += sh[k];
  }
  *total = tot;
  return base + incl - v;
}

// Per column (skipping the settled ones): the list of E rows in index order,
// |E|, the L weights w_j = y_j [j in L] for the product K w, and sum_L y_j.
// More E rows than emax: the column is marked as beyond the solver (-1).
__global__ __launch_bounds__(XB) void exact_sets_kernel(int N, int C, int emax,
                                                        const double* __restrict__ ylab,
                                                        const int32_t* __restrict__ state,
                                                        int32_t* __restrict__ elist,
                                                        int* __restrict__ ne_out,
                                                        double* __restrict__ wl,
                                                        double* __restrict__ sumyl,
                                                        int* __restrict__ xflag) {
  __shared__ int sh[XW];
  __shared__ double red[XW];
  const int64_t gc = blockIdx.x;
  if (xflag[gc] != 0) return;
  const int g = (int)(gc / C);
  const double* y = ylab + (int64_t)g * N;
  const int32_t* st = state + gc * N;
  int32_t* el = elist + gc * N;
  double* w = wl + gc * N;
  int base = 0;
  double sl = 0.0;
  for (int i0 = 0; i0 < N; i0 += XB) {
    const int i = i0 + threadIdx.x;
    const int s = i < N ? st[i] : 3;
    if (i < N) {
      const double wv = s == 0 ? y[i] : 0.0;
      w[i] = wv;
      sl += wv;
    }
    int tot = 0;
    const int pos = block_scan(s == 1 ? 1 : 0, sh, &tot);
    if (s == 1) el[base + pos] = i;
    base += tot;
  }
  sl = block_sum<XW>(sl, red);
  if (threadIdx.x == 0) {
    ne_out[gc] = base;
    sumyl[gc] = sl;
    if (base > emax) xflag[gc] = -1;
  }
}

// Per column: assemble the (|E| + 1)-square system in sys (row-major, ld m),
// solve it by LU with partial pivoting, and write the candidate alpha
// (c y_j a_j: a = 1 on L, a_E from the solve, 0 on R and padding) and beta.
// A pivot below 1e-300 marks the column as failed (-2). With E empty only
// alpha is written: the intercept keeps the last solve's value (the
// smoothed one before any), so the point that next joins E is chosen
// against the current iterate; a fixed intercept there lets a point enter
// E, leave it for R and enter again without end.
__global__ __launch_bounds__(XB) void exact_solve_kernel(
    int N, int C, int64_t sys_stride, const int* __restrict__ nv, const double* __restrict__ lamv,
    const int* __restrict__ cnv, const double* __restrict__ ylab, const double* __restrict__ K,
    const int32_t* __restrict__ state, const int32_t* __restrict__ elist,
    const int* __restrict__ ne_in, const double* __restrict__ fl,
    const double* __restrict__ sumyl, double* __restrict__ sys, double* __restrict__ alpha,
    double* __restrict__ beta_x, int* __restrict__ xflag) {
  __shared__ double rv[XB];
  __shared__ int ri[XB];
  __shared__ double piv_sh;
  __shared__ int pr_sh;
  const int64_t gc = blockIdx.x;
  if (xflag[gc] != 0) return;
  const int g = (int)(gc / C);
  const int t = threadIdx.x;
  const int ne = ne_in[gc], m = ne + 1;
  const double c = 1.0 / (2.0 * (double)cnv[gc] * lamv[gc]);
  const double* y = ylab + (int64_t)g * N;
  const double* Kg = K + (int64_t)g * N * N;
  const int32_t* el = elist + gc * N;
  const int32_t* st = state + gc * N;
  double* M = sys + gc * sys_stride;         // m x m, then the right-hand side (m)
  double* rhs = M + (int64_t)m * m;
  double* ax = alpha + gc * N;
  const int n = nv[g];
  if (ne > 0) {
    for (int64_t e = t; e < (int64_t)m * m; e += XB) {
      const int r = (int)(e / m), s = (int)(e % m);
      double v;
      if (r < ne && s < ne) {
        const int i = el[r], j = el[s];
        v = c * y[i] * y[j] * Kg[(int64_t)i * N + j];
      } else if (r < ne) {
        v = y[el[r]];
      } else if (s < ne) {
        v = y[el[s]];
      } else {
        v = 0.0;
      }
      M[e] = v;
    }
    for (int r = t; r < m; r += XB)
      rhs[r] = r < ne ? 1.0 - c * y[el[r]] * fl[gc * N + el[r]] : -sumyl[gc];
    __syncthreads();
    // LU with partial pivoting, right-looking; the row exchanges are applied
    // to the right-hand side as they happen
    for (int k = 0; k < m; ++k) {
      double best = -1.0;
      int bi = k;
      for (int r = k + t; r < m; r += XB) {
        const double a = fabs(M[(int64_t)r * m + k]);
        if (a > best) { best = a; bi = r; }
      }
      rv[t] = best;
      ri[t] = bi;
      __syncthreads();
      for (int off = XB / 2; off > 0; off >>= 1) {
        if (t < off) {
          const double a = rv[t + off];
          const int b = ri[t + off];
          if (a > rv[t] || (a == rv[t] && b < ri[t])) { rv[t] = a; ri[t] = b; }
        }
        __syncthreads();
      }
      if (t == 0) {
        pr_sh = ri[0];
        piv_sh = rv[0];
      }
      __syncthreads();
      const int p = pr_sh;
      if (!(piv_sh > 1e-300)) {
        if (t == 0) xflag[gc] = -2;
        return;
      }
      if (p != k) {
        for (int s = t; s < m; s += XB) {
          const double a = M[(int64_t)k * m + s];
          M[(int64_t)k * m + s] = M[(int64_t)p * m + s];
          M[(int64_t)p * m + s] = a;
        }
        if (t == 0) {
          const double a = rhs[k];
          rhs[k] = rhs[p];
          rhs[p] = a;
        }
      }
      __syncthreads();
      const double d = M[(int64_t)k * m + k];
      const int rest = m - k - 1;
      // multipliers in column k, then the trailing update (row r, column s)
      for (int r = k + 1 + t; r < m; r += XB) M[(int64_t)r * m + k] /= d;
      __syncthreads();
      for (int64_t e = t; e < (int64_t)rest * (rest + 1); e += XB) {
        const int r = k + 1 + (int)(e / (rest + 1));
        const int s = k + 1 + (int)(e % (rest + 1));
        const double l = M[(int64_t)r * m + k];
        if (s < m) M[(int64_t)r * m + s] = fma(-l, M[(int64_t)k * m + s], M[(int64_t)r * m + s]);
        else rhs[r] = fma(-l, rhs[k], rhs[r]);
      }
      __syncthreads();
    }
    // back substitution, one row at a time with a block reduction
    for (int k = m - 1; k >= 0; --k) {
      double s = 0.0;
      for (int j = k + 1 + t; j < m; j += XB) s = fma(M[(int64_t)k * m + j], rhs[j], s);
      rv[t] = s;
      __syncthreads();
      for (int off = XB / 2; off > 0; off >>= 1) {
        if (t < off) rv[t] += rv[t + off];
        __syncthreads();
      }
      if (t == 0) rhs[k] = (rhs[k] - rv[0]) / M[(int64_t)k * m + k];
      __syncthreads();
    }
  }
  // candidate alpha: a = 1 on L, a_E from the solve, 0 elsewhere
  for (int i = t; i < N; i += XB) {
    const int s = st[i];
    ax[i] = (i < n && s == 0) ? c * y[i] : 0.0;
  }
  __syncthreads();
  for (int r = t; r < ne; r += XB) {
    const int i = el[r];
    ax[i] = c * y[i] * rhs[r];
  }
  if (t == 0 && ne > 0) beta_x[gc] = rhs[ne];
}

// Per column: the KKT check of the candidate, with f = K alpha (fx) and
// u = y (f + beta). All conditions within tol: settled (1). Otherwise the
// violators change sets for the next round. With E empty: the balance must
// hold and beta is clamped into the interval that keeps every point on its
// side; if the balance fails or the interval is empty, the point nearest
// the margin joins E. Unsettled columns are counted in *pending.
__global__ __launch_bounds__(XB) void exact_check_kernel(
    int N, int C, double tol, const int* __restrict__ nv, const double* __restrict__ lamv,
    const int* __restrict__ cnv, const double* __restrict__ ylab, const double* __restrict__ fx,
    const double* __restrict__ alpha, double* __restrict__ beta_x, const int* __restrict__ ne_in,
    const double* __restrict__ sumyl, int32_t* __restrict__ state, int* __restrict__ xflag,
    int* __restrict__ pending) {
  __shared__ double red[XW];
  __shared__ double rv[XB];
  __shared__ int ri[XB];
  const int64_t gc = blockIdx.x;
  if (xflag[gc] != 0) return;
  const int g = (int)(gc / C);
  const int t = threadIdx.x;
  const int n = nv[g];
  const double c = 1.0 / (2.0 * (double)cnv[gc] * lamv[gc]);
  const double* y = ylab + (int64_t)g * N;
  const double* f = fx + gc * N;
  const double* ax = alpha + gc * N;
  int32_t* st = state + gc * N;
  const int ne = ne_in[gc];
  double b = beta_x[gc];
  if (ne == 0) {
    // bounds on beta: y_i beta <= 1 - y_i g_i on L, >= on R
    double lo = -1e300, hi = 1e300;
    for (int i = t; i < n; i += XB) {
      const int s = st[i];
      const double tt = 1.0 - y[i] * f[i];
      if (s == 0) { if (y[i] > 0) hi = fmin(hi, tt); else lo = fmax(lo, -tt); }
      else if (s == 2) { if (y[i] > 0) lo = fmax(lo, tt); else hi = fmin(hi, -tt); }
    }
    rv[t] = hi;
    __syncthreads();
    for (int off = XB / 2; off > 0; off >>= 1) {
      if (t < off) rv[t] = fmin(rv[t], rv[t + off]);
      __syncthreads();
    }
    hi = rv[0];
    __syncthreads();
    rv[t] = lo;
    __syncthreads();
    for (int off = XB / 2; off > 0; off >>= 1) {
      if (t < off) rv[t] = fmax(rv[t], rv[t + off]);
      __syncthreads();
    }
    lo = rv[0];
    __syncthreads();
    const bool balanced = fabs(sumyl[gc]) <= tol * n;
    if (balanced && lo <= hi + tol) {
      if (t == 0) {
        beta_x[gc] = fmin(fmax(b, lo), hi);
        xflag[gc] = 1;
      }
      return;
    }
    // the point nearest the margin joins E (smallest index on ties)
    double best = 1e300;
    int bi = N;
    for (int i = t; i < n; i += XB) {
      const double d = fabs(y[i] * (f[i] + b) - 1.0);
      if (d < best) { best = d; bi = i; }
    }
    rv[t] = best;
    ri[t] = bi;
    __syncthreads();
    for (int off = XB / 2; off > 0; off >>= 1) {
      if (t < off && (rv[t + off] < rv[t] || (rv[t + off] == rv[t] && ri[t + off] < ri[t]))) {
        rv[t] = rv[t + off];
        ri[t] = ri[t + off];
      }
      __syncthreads();
    }
    if (t == 0) {
      if (ri[0] < n) st[ri[0]] = 1;
      atomicAdd(pending, 1);
    }
    return;
  }
  double bad = 0.0;
  for (int i = t; i < n; i += XB) {
    const int s = st[i];
    const double u = y[i] * (f[i] + b);
    int ns = s;
    if (s == 1) {
      const double a = ax[i] / (c * y[i]);
      if (a < -tol) ns = 2;
      else if (a > 1.0 + tol) ns = 0;
    } else if (s == 0) {
      if (u > 1.0 + tol) ns = 1;
    } else if (s == 2) {
      if (u < 1.0 - tol) ns = 1;
    }
    if (ns != s) {
      st[i] = ns;
      bad += 1.0;
    }
  }
  bad = block_sum<XW>(bad, red);
  if (t == 0) {
    if (bad == 0.0) xflag[gc] = 1;
    else atomicAdd(pending, 1);
  }
}

// The settled columns take the exact solution: alpha_loc, f (without beta)
// and beta.
__global__ __launch_bounds__(XB) void exact_commit_kernel(int N, const int* __restrict__ xflag,
                                                          const double* __restrict__ alpha,
                                                          const double* __restrict__ fx,
                                                          const double* __restrict__ beta_x,
                                                          double* __restrict__ alpha_loc,
                                                          double* __restrict__ ftrain,
                                                          double* __restrict__ beta) {
  const int64_t gc = blockIdx.y;
  if (xflag[gc] != 1) return;
  const int i = blockIdx.x * XB + threadIdx.x;
  if (i < N) {
    alpha_loc[gc * N + i] = alpha[gc * N + i];
    ftrain[gc * N + i] = fx[gc * N + i];
  }
  if (i == 0) beta[gc] = beta_x[gc];
}

int exact_init(hipStream_t s, const ExactArgs& x) {
  hipLaunchKernelGGL(exact_init_kernel, dim3((unsigned)ceil_div(x.N, XB), (unsigned)x.cols), dim3(XB),
                     0, s, x.N, x.C, x.nv, x.delta, x.ylab, x.ftrain, x.beta, x.state, x.beta_x, x.xflag);
  KMP_LAUNCH_CHECK();
  return 0;
}

int exact_sets(hipStream_t s, const ExactArgs& x) {
  hipLaunchKernelGGL(exact_sets_kernel, dim3((unsigned)x.cols), dim3(XB), 0, s, x.N, x.C, x.emax,
                     x.ylab, x.state, x.elist, x.ne, x.wl, x.sumyl, x.xflag);
  KMP_LAUNCH_CHECK();
  return 0;
}

int exact_solve(hipStream_t s, const ExactArgs& x) {
  hipLaunchKernelGGL(exact_solve_kernel, dim3((unsigned)x.cols), dim3(XB), 0, s, x.N, x.C,
                     x.sys_stride, x.nv, x.lam, x.cnv, x.ylab, x.K, x.state, x.elist, x.ne, x.fl,
                     x.sumyl, x.sys, x.alpha, x.beta_x, x.xflag);
  KMP_LAUNCH_CHECK();
  return 0;
}

int exact_check(hipStream_t s, const ExactArgs& x) {
  hipLaunchKernelGGL(exact_check_kernel, dim3((unsigned)x.cols), dim3(XB), 0, s, x.N, x.C, x.tol,
                     x.nv, x.lam, x.cnv, x.ylab, x.fx, x.alpha, x.beta_x, x.ne, x.sumyl, x.state,
                     x.xflag, x.pending);
  KMP_LAUNCH_CHECK();
  return 0;
}

int exact_commit(hipStream_t s, const ExactArgs& x, double* alpha_loc, double* ftrain,
                 double* beta) {
  hipLaunchKernelGGL(exact_commit_kernel, dim3((unsigned)ceil_div(x.N, XB), (unsigned)x.cols),
                     dim3(XB), 0, s, x.N, x.xflag, x.alpha, x.fx, x.beta_x, alpha_loc, ftrain, beta);
  KMP_LAUNCH_CHECK();
  return 0;
}

}  // namespace kmp
