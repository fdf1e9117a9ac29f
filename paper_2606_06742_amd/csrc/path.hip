// Batched regularisation-path solver in the band basis K_v = Q B Q'.
//
// Every column is one (tau, lambda) problem of one group (bandwidth, fold).
// With hats denoting Q' coordinates (a = Q'alpha), one iteration of the
// accelerated majorise-minimise method (Appendix A.1 update; Algorithm 1
// inner loop; Appendix A.3 block inverse of H) is
//
//   f      = (Q B) abar + bbar                      (first path GEMM; Q B
//                                                     formed once per factor)
//   z      = psi(y, f) / n_v,  d0 = 1'z             (its epilogue)
//   zhat   = Q' z                                   (second path GEMM)
//   w      = zhat + 2 lambda abar                   (= Q'(z + 2 lambda alpha))
//   t      = vhat' B w                              (= v' K (z + 2 lambda alpha))
//   x      = (2 lambda I + B/(n_v kappa))^{-1} w    (banded solve)
//   Da     = g (t - d0) vhat + x,   Db = g (d0 - t)
//   a_new  = abar - Da,             b_new = bbar - Db
//
// with vhat = (2 lambda I + B/(n_v kappa))^{-1} Q'1 / (n_v kappa) and
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
// Sum over groups of f(valid rows, columns in the group's active list) for
// the work counters of the iteration kernels (groups with none are skipped).
template <typename F>
static double over_active(const PathArrays& p, F f) {
  double a = 0.0;
  for (int g = 0; g < p.G; ++g) {
    const double c = p.nact_host ? (double)p.nact_host[g] : (double)p.C;
    if (c > 0.0) a += f((double)(p.nv_host ? p.nv_host[g] : p.N), c);
  }
  return a;
}

// ------------------------------------------------------------ band solver
// One wavefront per column. The column's working vector lives in LDS (xs,
// N doubles); elementwise work spreads rows over the lanes as i = lane + 64 k.
//
// Per column and smoothing stage, M = 2 lambda I + B/(n_v kappa) (B banded,
// lower bandwidth BND) is factored blockwise in BND x BND blocks,
//   M = L D L',  L unit lower block-bidiagonal with diagonal blocks L_I and
//   subdiagonal blocks C_I = L_{I,I-1} (upper triangular: the band),
//   S_I = M_II - C_I D_{I-1} C_I',  S_I = L_I D_I L_I',
//   C_{I+1} = M_{I+1,I} L_I^{-T} D_I^{-1},
// and stored per block as one BND x BND tile V_I with V_I[a][j] =
// (L_I^{-1})[a][j] for j < a and C_I[a][j] for j >= a (the two triangles
// are complementary), element (a, j) of block I at V[j*N + BND*I + a]. With
// it both triangular solves are two small products per block:
//   forward   r = w_I - C_I y_{I-1},   y_I = L_I^{-1} r
//   backward  s = z_I - C_{I+1}' x_{I+1},   x_I = L_I^{-T} s.
constexpr int BND = kBand;

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Sum over the four 16-lane rows of the wavefront: lane (a, g) (a = lane
// mod 16, g = lane / 16) receives sum_g' v(a, g'), added as (row 0 + row 1)
// + (row 2 + row 3) in every lane. gfx950's permlane16 swap exchanges the
// odd rows of its first operand with the even rows of its second, permlane32
// the upper half of the first with the lower half of the second.
__device__ __forceinline__ double swap_sum16(double v) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const auto lo = __builtin_amdgcn_permlane16_swap((unsigned)b, (unsigned)b, false, false);
  const auto hi = __builtin_amdgcn_permlane16_swap((unsigned)(b >> 32), (unsigned)(b >> 32), false, false);
  return __longlong_as_double((long long)(((unsigned long long)hi[0] << 32) | lo[0])) +
         __longlong_as_double((long long)(((unsigned long long)hi[1] << 32) | lo[1]));
}
__device__ __forceinline__ double swap_sum32(double v) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const auto lo = __builtin_amdgcn_permlane32_swap((unsigned)b, (unsigned)b, false, false);
  const auto hi = __builtin_amdgcn_permlane32_swap((unsigned)(b >> 32), (unsigned)(b >> 32), false, false);
  return __longlong_as_double((long long)(((unsigned long long)hi[0] << 32) | lo[0])) +
         __longlong_as_double((long long)(((unsigned long long)hi[1] << 32) | lo[1]));
}
__device__ __forceinline__ double row4_sum(double v) { return swap_sum32(swap_sum16(v)); }

// xs <- M^{-1} xs (xs: N doubles of LDS) from the stored factor (Vc: the
// BND x N tiles, Dc: 1/D). Each block product of 16 terms per row is split
// over the wavefront: lane (a, g) takes row a and terms j = 4g .. 4g+3, and
// row4_sum adds the four parts, so a block step is four FMAs, two swaps and
// one LDS exchange per triangular factor. The lane's four tile entries of
// the next SPF blocks are loaded ahead into registers, so the recurrence
// does not wait on device memory: a block step takes far less than a load's
// latency under load, so the loads of several steps must be in flight (the
// vector-memory counter allows 63 per wave: 4 loads per forward step and 5
// per backward step here). The depth also sets the registers of the
// per-column update kernel: at 10 it stays within 256, so two of its
// workgroups share a compute unit (at 12 it took 272 and one workgroup per
// compute unit, which doubled the update time above 256 active columns). Forward tiles are read by rows
// (V[j*N + 16 I + a], j = 4g+t), backward tiles by columns
// (V[a*N + 16 I + j]) as the transposed factors need.
constexpr int SPF = 10;

// Element i of the solve's vector: xs[i], or xs[N - 1 - i] for the sweeps
// of the twisted solve that run from the last row (REV).
template <bool REV>
__device__ __forceinline__ double& xel(double* xs, int N, int i) {
  return REV ? xs[N - 1 - i] : xs[i];
}

// One forward block step of the LDS solve: rg holds the lane's four entries
// of tile I and receives those of tile min(I + SPF, NB - 1). Branch free, so
// that the loads of the following steps stay in flight across it. With
// LAST only r = w_I - C_I y_{I-1} is formed, into slot (lead lanes).
template <bool REV = false, bool LAST = false>
__device__ __forceinline__ void band_fwd_step(const double* __restrict__ Vc, double* xs, int N,
                                              int NB, int I, int a, int g, bool lead,
                                              double (&rg)[4], double* slot = nullptr) {
  double cn[4], lm[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const double v = rg[t];
    cn[t] = (4 * g + t >= a && I > 0) ? -v : 0.0;   // C_I (upper triangle, diagonal included)
    lm[t] = (4 * g + t < a) ? v : 0.0;              // strict lower part of L_I^{-1}
  }
  const int In = min(I + SPF, NB - 1);
#pragma unroll
  for (int t = 0; t < 4; ++t) rg[t] = Vc[(int64_t)(4 * g + t) * N + BND * In + a];
  double p0 = lead ? xel<REV>(xs, N, BND * I + a) : 0.0, p1 = 0.0;
  const int yb = BND * max(I - 1, 0) + 4 * g;
  p0 = fma(cn[0], xel<REV>(xs, N, yb), p0);
  p1 = fma(cn[1], xel<REV>(xs, N, yb + 1), p1);
  p0 = fma(cn[2], xel<REV>(xs, N, yb + 2), p0);
  p1 = fma(cn[3], xel<REV>(xs, N, yb + 3), p1);
  const double r = row4_sum(p0 + p1);
  if constexpr (LAST) {
    if (lead) slot[a] = r;
    return;
  }
  xel<REV>(xs, N, BND * I + a) = r;    // the four lanes of row a store the same value
  wave_sync();
  const int rb = BND * I + 4 * g;
  double q0 = lead ? r : 0.0, q1 = 0.0;
  q0 = fma(lm[0], xel<REV>(xs, N, rb), q0);
  q1 = fma(lm[1], xel<REV>(xs, N, rb + 1), q1);
  q0 = fma(lm[2], xel<REV>(xs, N, rb + 2), q0);
  q1 = fma(lm[3], xel<REV>(xs, N, rb + 3), q1);
  const double yv = row4_sum(q0 + q1);
  xel<REV>(xs, N, BND * I + a) = yv;
  wave_sync();
}

// One backward block step (block I = NB - 1 - tt); vprev holds the lane's
// entries (4g+t, a) of tile I + 1.
template <bool REV = false>
__device__ __forceinline__ void band_bwd_step(const double* __restrict__ Vc,
                                              const double* __restrict__ Dc, double* xs, int N,
                                              int NB, int tt, int a, int g, bool lead,
                                              double (&rg)[4], double& dr, double (&vprev)[4]) {
  const int I = NB - 1 - tt;
  double cn[4], lm[4], vv[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    vv[t] = rg[t];
    cn[t] = (a >= 4 * g + t && tt > 0) ? -vprev[t] : 0.0;   // C_{I+1}' row a
    lm[t] = (4 * g + t > a) ? vv[t] : 0.0;                  // strict upper part of L_I^{-T}
  }
  const double dv = dr;
  const int In = max(I - SPF, 0);
#pragma unroll
  for (int t = 0; t < 4; ++t) rg[t] = Vc[(int64_t)a * N + BND * In + 4 * g + t];
  dr = Dc[BND * In + a];
  double p0 = lead ? dv * xel<REV>(xs, N, BND * I + a) : 0.0, p1 = 0.0;
  const int xb = BND * min(I + 1, NB - 1) + 4 * g;
  p0 = fma(cn[0], xel<REV>(xs, N, xb), p0);
  p1 = fma(cn[1], xel<REV>(xs, N, xb + 1), p1);
  p0 = fma(cn[2], xel<REV>(xs, N, xb + 2), p0);
  p1 = fma(cn[3], xel<REV>(xs, N, xb + 3), p1);
  const double sv = row4_sum(p0 + p1);
  xel<REV>(xs, N, BND * I + a) = sv;
  wave_sync();
  const int sb = BND * I + 4 * g;
  double q0 = lead ? sv : 0.0, q1 = 0.0;
  q0 = fma(lm[0], xel<REV>(xs, N, sb), q0);
  q1 = fma(lm[1], xel<REV>(xs, N, sb + 1), q1);
  q0 = fma(lm[2], xel<REV>(xs, N, sb + 2), q0);
  q1 = fma(lm[3], xel<REV>(xs, N, sb + 3), q1);
  const double xv = row4_sum(q0 + q1);
  xel<REV>(xs, N, BND * I + a) = xv;
  wave_sync();
#pragma unroll
  for (int t = 0; t < 4; ++t) vprev[t] = vv[t];
}

// The sweeps run whole groups of SPF blocks without a branch (block
// p of a group in ring slot p), then the remaining NB mod SPF blocks.
__device__ __forceinline__ void band_solve(const double* __restrict__ Vc,
                                           const double* __restrict__ Dc, double* xs, int N,
                                           int lane) {
  const int NB = N / BND;
  const int NBm = NB - NB % SPF;
  const int a = lane & 15, g = lane >> 4;
  const bool lead = g == 0;
  double ring[SPF][4];
  // forward: y_I = L_I^{-1} (w_I - C_I y_{I-1}), y overwrites w in xs
#pragma unroll
  for (int p = 0; p < SPF; ++p) {
    const int Ib = min(p, NB - 1);
#pragma unroll
    for (int t = 0; t < 4; ++t) ring[p][t] = Vc[(int64_t)(4 * g + t) * N + BND * Ib + a];
  }
  for (int I0 = 0; I0 < NBm; I0 += SPF) {
#pragma unroll
    for (int p = 0; p < SPF; ++p) band_fwd_step(Vc, xs, N, NB, I0 + p, a, g, lead, ring[p]);
  }
#pragma unroll
  for (int p = 0; p < SPF; ++p)
    if (NBm + p < NB) band_fwd_step(Vc, xs, N, NB, NBm + p, a, g, lead, ring[p]);
  wave_sync();
  // backward: x_I = L_I^{-T} (D_I^{-1} y_I - C_{I+1}' x_{I+1}), x overwrites y
  double dring[SPF];
#pragma unroll
  for (int p = 0; p < SPF; ++p) {
    const int Ib = max(NB - 1 - p, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) ring[p][t] = Vc[(int64_t)a * N + BND * Ib + 4 * g + t];
    dring[p] = Dc[BND * Ib + a];
  }
  double vprev[4] = {0.0, 0.0, 0.0, 0.0};     // entries (4g+t, a) of the tile of block I+1
  for (int T0 = 0; T0 < NBm; T0 += SPF) {
#pragma unroll
    for (int p = 0; p < SPF; ++p)
      band_bwd_step(Vc, Dc, xs, N, NB, T0 + p, a, g, lead, ring[p], dring[p], vprev);
  }
#pragma unroll
  for (int p = 0; p < SPF; ++p)
    if (NBm + p < NB) band_bwd_step(Vc, Dc, xs, N, NB, NBm + p, a, g, lead, ring[p], dring[p], vprev);
  wave_sync();
}

// Twisted form of the same solve, for a workgroup of two or more
// wavefronts: the top-down factors of blocks 0 .. k (k = NB/2) and those of
// the reversed matrix (rows and columns in reverse order: the bottom-up
// factors of blocks NB-1 .. k) meet at block k, where
//   Z = M_kk - C_k D_{k-1} C_k' - (the same term from below)
// (the two Schur complements of block k, less M_kk once). With
// r = w_k - C_k y_{k-1} from the top sweep and r~ from the bottom one,
// x_k = Z^{-1} (r + r~ - w_k); from x_k the backward sweeps run outwards.
// Wavefront 0 takes the top half, wavefront 1 the bottom half, so the
// dependent chain is about half as long as in band_solve, for the same
// tiles read. Vr, Dr: the reversed matrix's factors (block J of it at
// 16 J, in its own row order); tw: L_Z^{-1} (16 x 16, row-major, strict
// lower part) and 1/D_Z; tslot: 48 doubles of LDS. Every wavefront of the
// workgroup calls it (it holds two barriers); the caller synchronises
// after it before reading xs.

// forward sweep over blocks 0 .. n-1, then r of block n into slot
template <bool REV>
__device__ __forceinline__ void band_sweep_fwd(const double* __restrict__ Vc, double* xs, int N,
                                               int n, int a, int g, bool lead, double* slot) {
  const int NBe = n + 1;
  const int nm = n - n % SPF;
  double ring[SPF][4];
#pragma unroll
  for (int p = 0; p < SPF; ++p) {
    const int Ib = min(p, n);
#pragma unroll
    for (int t = 0; t < 4; ++t) ring[p][t] = Vc[(int64_t)(4 * g + t) * N + BND * Ib + a];
  }
  for (int I0 = 0; I0 < nm; I0 += SPF) {
#pragma unroll
    for (int p = 0; p < SPF; ++p) band_fwd_step<REV>(Vc, xs, N, NBe, I0 + p, a, g, lead, ring[p]);
  }
#pragma unroll
  for (int p = 0; p < SPF; ++p) {
    if (nm + p < n) band_fwd_step<REV>(Vc, xs, N, NBe, nm + p, a, g, lead, ring[p]);
    else if (nm + p == n) band_fwd_step<REV, true>(Vc, xs, N, NBe, n, a, g, lead, ring[p], slot);
  }
}

// backward sweep over blocks n-1 .. 0, block n's solution already in xs
template <bool REV>
__device__ __forceinline__ void band_sweep_bwd(const double* __restrict__ Vc,
                                               const double* __restrict__ Dc, double* xs, int N,
                                               int n, int a, int g, bool lead) {
  const int NBe = n + 1;
  // slot p serves the steps tt = p (mod SPF), tt = 1 .. n (block n - tt)
  double ring[SPF][4], dring[SPF];
#pragma unroll
  for (int p = 0; p < SPF; ++p) {
    const int Ib = max(n - (p > 0 ? p : SPF), 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) ring[p][t] = Vc[(int64_t)a * N + BND * Ib + 4 * g + t];
    dring[p] = Dc[BND * Ib + a];
  }
  double vprev[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) vprev[t] = Vc[(int64_t)a * N + BND * n + 4 * g + t];
#pragma unroll
  for (int p = 1; p < SPF; ++p)
    if (p <= n) band_bwd_step<REV>(Vc, Dc, xs, N, NBe, p, a, g, lead, ring[p], dring[p], vprev);
  int T0 = SPF;
  for (; T0 + SPF - 1 <= n; T0 += SPF) {
#pragma unroll
    for (int p = 0; p < SPF; ++p)
      band_bwd_step<REV>(Vc, Dc, xs, N, NBe, T0 + p, a, g, lead, ring[p], dring[p], vprev);
  }
#pragma unroll
  for (int p = 0; p < SPF; ++p)
    if (T0 + p <= n) band_bwd_step<REV>(Vc, Dc, xs, N, NBe, T0 + p, a, g, lead, ring[p], dring[p], vprev);
}

// x_k = Z^{-1} (r + r~ - w_k) = L_Z^{-T} D_Z^{-1} L_Z^{-1} (.), one wavefront
__device__ __forceinline__ void band_twist_block(const double* __restrict__ tw, double* xs,
                                                 double* tslot, int k, int a, int g, bool lead) {
  double* rhs = tslot + 2 * BND;
  // r~ is in the bottom sweep's row order
  if (lead) rhs[a] = tslot[a] + tslot[BND + (BND - 1 - a)] - xs[BND * k + a];
  wave_sync();
  double q0 = lead ? rhs[a] : 0.0, q1 = 0.0;
#pragma unroll
  for (int t = 0; t < 4; t += 2) {
    const int j0 = 4 * g + t, j1 = j0 + 1;
    q0 = fma((j0 < a) ? tw[a * BND + j0] : 0.0, rhs[j0], q0);
    q1 = fma((j1 < a) ? tw[a * BND + j1] : 0.0, rhs[j1], q1);
  }
  const double u = row4_sum(q0 + q1) * tw[BND * BND + a];     // D_Z^{-1} L_Z^{-1} rhs
  wave_sync();
  if (lead) rhs[a] = u;
  wave_sync();
  double s0 = lead ? u : 0.0, s1 = 0.0;
#pragma unroll
  for (int t = 0; t < 4; t += 2) {
    const int j0 = 4 * g + t, j1 = j0 + 1;
    s0 = fma((j0 > a) ? tw[j0 * BND + a] : 0.0, rhs[j0], s0);
    s1 = fma((j1 > a) ? tw[j1 * BND + a] : 0.0, rhs[j1], s1);
  }
  const double x = row4_sum(s0 + s1);
  if (lead) xs[BND * k + a] = x;
}

__device__ __forceinline__ void band_solve_twist(const double* __restrict__ Vt,
                                                 const double* __restrict__ Dt,
                                                 const double* __restrict__ Vr,
                                                 const double* __restrict__ Dr,
                                                 const double* __restrict__ tw, double* xs,
                                                 double* tslot, int N, int wv, int lane) {
  const int NB = N / BND, k = NB / 2, J = NB - 1 - k;
  const int a = lane & 15, g = lane >> 4;
  const bool lead = g == 0;
  if (wv == 0) band_sweep_fwd<false>(Vt, xs, N, k, a, g, lead, tslot);
  else if (wv == 1) band_sweep_fwd<true>(Vr, xs, N, J, a, g, lead, tslot + BND);
  __syncthreads();
  if (wv == 0) band_twist_block(tw, xs, tslot, k, a, g, lead);
  __syncthreads();
  if (wv == 0) band_sweep_bwd<false>(Vt, Dt, xs, N, k, a, g, lead);
  else if (wv == 1) band_sweep_bwd<true>(Vr, Dr, xs, N, J, a, g, lead);
}

// Fences that order device-memory stores of some lanes of a wavefront
// before loads of the same addresses by other lanes of it.
__device__ __forceinline__ void grid_vec_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// The same solve for orders whose vector does not fit in LDS. Row r =
// BND I + a belongs to lane row a of the wavefront: its input is wsc * win[r]
// (device memory written before the solve; the four lanes of the row load
// the same address and the lead lane (a, 0) keeps the value), the forward result
// y_r is kept in device memory (ysc[r], stored by the four lanes of the row
// with the same value and read back by them in the backward sweep), and the
// solution goes to wout(r, x_r, lead), called by every lane, the lead lane
// flagged. The blocks that the other lanes need are staged in an LDS ring of
// two BND-double slots (block I in slot I & 1). Within the solve a lane
// reads back from device memory only what it wrote itself (the input is
// written before the solve, with a fence when by the same launch). As in
// band_solve, the sweeps
// run whole groups of SPFG blocks through branch-free steps (prefetch index
// clamped, the first block as a select, stores unconditional) and the
// remaining blocks after them, and every prefetched value is a plain load
// that is first used SPFG steps later: the loads complete in issue order,
// so a branch around them, or arithmetic on a value just loaded, makes the
// step wait for every load in flight, and each step then took as long as a
// device-memory load.
// Prefetch depth of the device-memory solve (5 loads per forward step, 6
// per backward step).
constexpr int SPFG = 10;

template <bool REV = false, bool LAST = false>
__device__ __forceinline__ void bandg_fwd_step(const double* __restrict__ Vc,
                                               const double* __restrict__ win, double wsc,
                                               double* ysc, double* ring, int N, int NB, int I,
                                               int a, int g, bool lead, double (&rg)[4],
                                               double& wr, double* slot = nullptr) {
  double cn[4], lm[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const double v = rg[t];
    cn[t] = (4 * g + t >= a && I > 0) ? -v : 0.0;
    lm[t] = (4 * g + t < a) ? v : 0.0;
  }
  double p0 = lead ? wsc * wr : 0.0, p1 = 0.0;
  const int In = min(I + SPFG, NB - 1);
#pragma unroll
  for (int t = 0; t < 4; ++t) rg[t] = Vc[(int64_t)(4 * g + t) * N + BND * In + a];
  wr = xel<REV>(const_cast<double*>(win), N, BND * In + a);
  double* cur = ring + BND * (I & 1);
  const double* yp = ring + BND * ((I + 1) & 1) + 4 * g;   // block I - 1 (zeros before block 0)
  p0 = fma(cn[0], yp[0], p0);
  p1 = fma(cn[1], yp[1], p1);
  p0 = fma(cn[2], yp[2], p0);
  p1 = fma(cn[3], yp[3], p1);
  const double r = row4_sum(p0 + p1);
  if constexpr (LAST) {
    if (lead) slot[a] = r;
    return;
  }
  cur[a] = r;
  wave_sync();
  const double* rp = cur + 4 * g;
  double q0 = lead ? r : 0.0, q1 = 0.0;
  q0 = fma(lm[0], rp[0], q0);
  q1 = fma(lm[1], rp[1], q1);
  q0 = fma(lm[2], rp[2], q0);
  q1 = fma(lm[3], rp[3], q1);
  const double yv = row4_sum(q0 + q1);
  cur[a] = yv;
  xel<REV>(ysc, N, BND * I + a) = yv;
  wave_sync();
}

template <typename WOut, bool REV = false>
__device__ __forceinline__ void bandg_bwd_step(const double* __restrict__ Vc,
                                               const double* __restrict__ Dc, const double* ysc,
                                               double* ring, int N, int NB, int tt, int a, int g,
                                               bool lead, double (&rg)[4], double& dr, double& wr,
                                               double (&vprev)[4], WOut wout) {
  const int I = NB - 1 - tt;
  double cn[4], lm[4], vv[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    vv[t] = rg[t];
    cn[t] = (a >= 4 * g + t && tt > 0) ? -vprev[t] : 0.0;
    lm[t] = (4 * g + t > a) ? vv[t] : 0.0;
  }
  double p0 = lead ? dr * wr : 0.0, p1 = 0.0;
  const int In = max(I - SPFG, 0);
#pragma unroll
  for (int t = 0; t < 4; ++t) rg[t] = Vc[(int64_t)a * N + BND * In + 4 * g + t];
  dr = Dc[BND * In + a];
  wr = xel<REV>(const_cast<double*>(ysc), N, BND * In + a);
  double* cur = ring + BND * (I & 1);
  const double* xp = ring + BND * ((I + 1) & 1) + 4 * g;   // block I + 1
  p0 = fma(cn[0], xp[0], p0);
  p1 = fma(cn[1], xp[1], p1);
  p0 = fma(cn[2], xp[2], p0);
  p1 = fma(cn[3], xp[3], p1);
  const double sv = row4_sum(p0 + p1);
  cur[a] = sv;
  wave_sync();
  const double* sp = cur + 4 * g;
  double q0 = lead ? sv : 0.0, q1 = 0.0;
  q0 = fma(lm[0], sp[0], q0);
  q1 = fma(lm[1], sp[1], q1);
  q0 = fma(lm[2], sp[2], q0);
  q1 = fma(lm[3], sp[3], q1);
  const double xv = row4_sum(q0 + q1);
  cur[a] = xv;
  wout(REV ? N - 1 - (BND * I + a) : BND * I + a, xv, lead);
  wave_sync();
#pragma unroll
  for (int t = 0; t < 4; ++t) vprev[t] = vv[t];
}

template <typename WOut>
__device__ __forceinline__ void band_solve_g(const double* __restrict__ Vc,
                                             const double* __restrict__ Dc,
                                             const double* __restrict__ win, double wsc,
                                             double* ysc, double* ring, int N, int lane,
                                             WOut wout) {
  const int NB = N / BND;
  const int NBm = NB - NB % SPFG;
  const int a = lane & 15, g = lane >> 4;
  const bool lead = g == 0;
  // the slot read as block -1 holds zeros (its products are zero multiples)
  ring[BND + a] = 0.0;
  wave_sync();
  double rt[SPFG][4], wr[SPFG];
#pragma unroll
  for (int p = 0; p < SPFG; ++p) {
    const int Ib = min(p, NB - 1);
#pragma unroll
    for (int t = 0; t < 4; ++t) rt[p][t] = Vc[(int64_t)(4 * g + t) * N + BND * Ib + a];
    wr[p] = win[BND * Ib + a];
  }
  for (int I0 = 0; I0 < NBm; I0 += SPFG) {
#pragma unroll
    for (int p = 0; p < SPFG; ++p)
      bandg_fwd_step(Vc, win, wsc, ysc, ring, N, NB, I0 + p, a, g, lead, rt[p], wr[p]);
  }
#pragma unroll
  for (int p = 0; p < SPFG; ++p)
    if (NBm + p < NB)
      bandg_fwd_step(Vc, win, wsc, ysc, ring, N, NB, NBm + p, a, g, lead, rt[p], wr[p]);
  wave_sync();
  double dring[SPFG];
#pragma unroll
  for (int p = 0; p < SPFG; ++p) {
    const int Ib = max(NB - 1 - p, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) rt[p][t] = Vc[(int64_t)a * N + BND * Ib + 4 * g + t];
    dring[p] = Dc[BND * Ib + a];
    wr[p] = ysc[BND * Ib + a];
  }
  double vprev[4] = {0.0, 0.0, 0.0, 0.0};
  for (int T0 = 0; T0 < NBm; T0 += SPFG) {
#pragma unroll
    for (int p = 0; p < SPFG; ++p)
      bandg_bwd_step(Vc, Dc, ysc, ring, N, NB, T0 + p, a, g, lead, rt[p], dring[p], wr[p], vprev,
                     wout);
  }
#pragma unroll
  for (int p = 0; p < SPFG; ++p)
    if (NBm + p < NB)
      bandg_bwd_step(Vc, Dc, ysc, ring, N, NB, NBm + p, a, g, lead, rt[p], dring[p], wr[p], vprev,
                     wout);
  wave_sync();
}

// Twisted form of the device-memory solve (see band_solve_twist): the two
// wavefronts of a column run the sweeps over blocks 0 .. k (role 0) and,
// on the reversed factors and with reversed indices, NB-1 .. k (role 1),
// each with its own ring; role 0 solves the twist block, writes x_k to
// device memory and into both rings, and the backward sweeps run outwards.
// Every wavefront of the workgroup calls it (two barriers); live is false
// for a column that skips the solve (its wavefronts only take the
// barriers). tslot: 48 doubles of LDS per column.
template <bool REV>
__device__ __forceinline__ void bandg_sweep_fwd(const double* __restrict__ Vc,
                                                const double* __restrict__ win, double* ysc,
                                                double* ring, int N, int n, int a, int g,
                                                bool lead, double* slot) {
  const int NBe = n + 1;
  const int nm = n - n % SPFG;
  ring[BND + a] = 0.0;                            // the slot read as block -1
  wave_sync();
  double rt[SPFG][4], wr[SPFG];
#pragma unroll
  for (int p = 0; p < SPFG; ++p) {
    const int Ib = min(p, n);
#pragma unroll
    for (int t = 0; t < 4; ++t) rt[p][t] = Vc[(int64_t)(4 * g + t) * N + BND * Ib + a];
    wr[p] = xel<REV>(const_cast<double*>(win), N, BND * Ib + a);
  }
  for (int I0 = 0; I0 < nm; I0 += SPFG) {
#pragma unroll
    for (int p = 0; p < SPFG; ++p)
      bandg_fwd_step<REV>(Vc, win, 1.0, ysc, ring, N, NBe, I0 + p, a, g, lead, rt[p], wr[p]);
  }
#pragma unroll
  for (int p = 0; p < SPFG; ++p) {
    if (nm + p < n)
      bandg_fwd_step<REV>(Vc, win, 1.0, ysc, ring, N, NBe, nm + p, a, g, lead, rt[p], wr[p]);
    else if (nm + p == n)
      bandg_fwd_step<REV, true>(Vc, win, 1.0, ysc, ring, N, NBe, n, a, g, lead, rt[p], wr[p], slot);
  }
}

template <bool REV, typename WOut>
__device__ __forceinline__ void bandg_sweep_bwd(const double* __restrict__ Vc,
                                                const double* __restrict__ Dc, const double* ysc,
                                                double* ring, int N, int n, int a, int g,
                                                bool lead, WOut wout) {
  const int NBe = n + 1;
  double rt[SPFG][4], dring[SPFG], wr[SPFG];
#pragma unroll
  for (int p = 0; p < SPFG; ++p) {
    const int Ib = max(n - (p > 0 ? p : SPFG), 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) rt[p][t] = Vc[(int64_t)a * N + BND * Ib + 4 * g + t];
    dring[p] = Dc[BND * Ib + a];
    wr[p] = xel<REV>(const_cast<double*>(ysc), N, BND * Ib + a);
  }
  double vprev[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) vprev[t] = Vc[(int64_t)a * N + BND * n + 4 * g + t];
#pragma unroll
  for (int p = 1; p < SPFG; ++p)
    if (p <= n)
      bandg_bwd_step<WOut, REV>(Vc, Dc, ysc, ring, N, NBe, p, a, g, lead, rt[p], dring[p], wr[p],
                                vprev, wout);
  int T0 = SPFG;
  for (; T0 + SPFG - 1 <= n; T0 += SPFG) {
#pragma unroll
    for (int p = 0; p < SPFG; ++p)
      bandg_bwd_step<WOut, REV>(Vc, Dc, ysc, ring, N, NBe, T0 + p, a, g, lead, rt[p], dring[p],
                                wr[p], vprev, wout);
  }
#pragma unroll
  for (int p = 0; p < SPFG; ++p)
    if (T0 + p <= n)
      bandg_bwd_step<WOut, REV>(Vc, Dc, ysc, ring, N, NBe, T0 + p, a, g, lead, rt[p], dring[p],
                                wr[p], vprev, wout);
}

template <typename WOut>
__device__ __forceinline__ void band_solve_g_twist(
    const double* __restrict__ Vt, const double* __restrict__ Dt, const double* __restrict__ Vr,
    const double* __restrict__ Dr, const double* __restrict__ tw, const double* __restrict__ win,
    double* ysc, double* ring0, double* ring1, double* tslot, int N, int role, bool live,
    int lane, WOut wout) {
  const int NB = N / BND, k = NB / 2, J = NB - 1 - k;
  const int a = lane & 15, g = lane >> 4;
  const bool lead = g == 0;
  if (live) {
    if (role == 0) bandg_sweep_fwd<false>(Vt, win, ysc, ring0, N, k, a, g, lead, tslot);
    else bandg_sweep_fwd<true>(Vr, win, ysc, ring1, N, J, a, g, lead, tslot + BND);
  }
  __syncthreads();
  if (live && role == 0) {
    double* rhs = tslot + 2 * BND;
    if (lead) rhs[a] = tslot[a] + tslot[BND + (BND - 1 - a)] - win[BND * k + a];
    wave_sync();
    double q0 = lead ? rhs[a] : 0.0, q1 = 0.0;
#pragma unroll
    for (int t = 0; t < 4; t += 2) {
      const int j0 = 4 * g + t, j1 = j0 + 1;
      q0 = fma((j0 < a) ? tw[a * BND + j0] : 0.0, rhs[j0], q0);
      q1 = fma((j1 < a) ? tw[a * BND + j1] : 0.0, rhs[j1], q1);
    }
    const double u = row4_sum(q0 + q1) * tw[BND * BND + a];
    wave_sync();
    if (lead) rhs[a] = u;
    wave_sync();
    double s0 = lead ? u : 0.0, s1 = 0.0;
#pragma unroll
    for (int t = 0; t < 4; t += 2) {
      const int j0 = 4 * g + t, j1 = j0 + 1;
      s0 = fma((j0 > a) ? tw[j0 * BND + a] : 0.0, rhs[j0], s0);
      s1 = fma((j1 > a) ? tw[j1 * BND + a] : 0.0, rhs[j1], s1);
    }
    const double x = row4_sum(s0 + s1);
    if (lead) {
      ring0[BND * (k & 1) + a] = x;
      ring1[BND * (J & 1) + (BND - 1 - a)] = x;
    }
    wout(BND * k + a, x, lead);
  }
  __syncthreads();
  if (live) {
    if (role == 0) bandg_sweep_bwd<false>(Vt, Dt, ysc, ring0, N, k, a, g, lead, wout);
    else bandg_sweep_bwd<true>(Vr, Dr, ysc, ring1, N, J, a, g, lead, wout);
  }
}

// Columns (wavefronts) per workgroup and where the solve keeps its vector.
// With the vector in LDS a workgroup holds one N-vector per column plus
// `extra` doubles of per-column tiles, and four columns share a workgroup
// when they fit in 64 KiB, else each has its own. Orders above what one
// workgroup's LDS holds (lds_vec_max: the device's LDS per workgroup, 160 KiB
// on gfx950, less a margin for the kernels' static arrays; never below 8192
// rows), or every order with KMP_FLAG_GLOBAL_SOLVE, keep the vector in device
// memory and only a two-block ring in LDS.
constexpr int PTILE = 2 * BND * (BND + 1) + 5 * BND + (BND + 1) * BND;   // LDS of one column's LDL' sweep
constexpr int RING = 2 * BND;                          // LDS ring of the device-memory solve
constexpr int kLdsVecFloor = 8192;
static int lds_vec_max() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return kLdsVecFloor;
  if (cached[dev] == 0) {
    int bytes = 0;
    if (hipDeviceGetAttribute(&bytes, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
      bytes = 0;
    const int rows = (bytes - 2048) / (int)sizeof(double) / 64 * 64;
    cached[dev] = rows > kLdsVecFloor ? rows : kLdsVecFloor;
  }
  return cached[dev];
}
static bool path_global_vec(const PathArrays& p) { return p.global_solve || p.N > lds_vec_max(); }
static int path_lds_doubles(const PathArrays& p, int extra, bool gv) {
  return gv ? extra + RING : p.N + extra;
}
static int path_lds_doubles(const PathArrays& p, int extra) {
  return path_lds_doubles(p, extra, path_global_vec(p));
}
static int path_waves(const PathArrays& p, int extra, bool gv) {
  const size_t per = sizeof(double) * (size_t)path_lds_doubles(p, extra, gv);
  return 4 * per <= 64 * 1024 ? 4 : 1;
}
static int path_waves(const PathArrays& p, int extra) { return path_waves(p, extra, path_global_vec(p)); }

// Compute units and LDS bytes per compute unit of the current device
// (queried once per device; zero when the query fails).
struct CuShape {
  int cus = 0, lds = 0;
};
static CuShape cu_shape() {
  static CuShape cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return CuShape{};
  if (cached[dev].cus == 0) {
    int cus = 0, lds = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
            hipSuccess)
      return CuShape{};
    cached[dev].cus = cus;
    cached[dev].lds = lds;
  }
  return cached[dev];
}

// Where this iteration's update keeps the solve's vector. The LDS form
// (update_column_kernel: one column per workgroup, its N doubles in LDS,
// at most 256 registers per lane) keeps two columns per compute unit at
// most, fewer when LDS allows fewer; the device-memory form
// (solve_step_twist_kernel: two columns per workgroup, two workgroups per
// compute unit by its registers) keeps four. When more columns are active than
// the LDS form holds at once, the device-memory form needs fewer rounds and
// is taken (10 groups of order 9024: above 512 active columns 623 against
// 717 us per iteration; below, the LDS form's shorter steps win: 280
// against 380 us).
// The counts are the host's copy of the last poll, which only overestimates
// the active columns.
static bool iteration_global_vec(const PathArrays& p) {
  if (path_global_vec(p)) return true;
  if (!p.nact_host) return false;
  const CuShape d = cu_shape();
  if (d.cus <= 0 || d.lds <= 0) return false;
  int64_t act = 0;
  for (int g = 0; g < p.G; ++g) act += p.nact_host[g];
  const int64_t per_wg = (int64_t)sizeof(double) * p.N + 2048;
  const int64_t res_lds = std::max<int64_t>(1, std::min<int64_t>(2, d.lds / per_wg));
  return ceil_div(act, 4 * (int64_t)d.cus) < ceil_div(act, res_lds * d.cus);
}

// ---------------------------------------------------- band products B x
// One workgroup per (row tile of BT rows, column): the tile of x with a halo
// of BND rows each side is staged in LDS (zero outside 0 .. N-1), and
// thread i adds the 2 BND + 1 band terms of row i,
//   (B x)[i] = B[i][i] x[i] + sum_r B[i][i-r] x[i-r] + B[i+r][i] x[i+r],
// with band loads coalesced across the tile (bg[r*N + j] = B[j+r][j], zero
// for j + r >= N, so the upper terms past the end vanish by themselves).
constexpr int BT = 256;

__device__ __forceinline__ double band_tile_row(const double* __restrict__ bg, const double* xt,
                                                int N, int i, int li) {
  double y0 = bg[i] * xt[li + BND], y1 = 0.0;
#pragma unroll
  for (int r = 1; r <= BND; ++r) {
    const int il = (i - r >= 0) ? i - r : 0;        // xt is zero above row 0
    y0 = fma(bg[(int64_t)r * N + il], xt[li + BND - r], y0);
    y1 = fma(bg[(int64_t)r * N + i], xt[li + BND + r], y1);
  }
  return y0 + y1;
}

__global__ __launch_bounds__(BT) void band_apply_kernel(int N, int C,
                                                        const double* __restrict__ band,
                                                        const double* __restrict__ x,
                                                        double* __restrict__ y) {
  __shared__ double xt[BT + 2 * BND];
  const int64_t col = blockIdx.y;
  const double* bg = band + (int64_t)(col / C) * (BND + 1) * N;
  const double* xc = x + col * N;
  const int t0 = blockIdx.x * BT;
  for (int j = threadIdx.x; j < BT + 2 * BND; j += BT) {
    const int r = t0 - BND + j;
    xt[j] = (r >= 0 && r < N) ? xc[r] : 0.0;
  }
  __syncthreads();
  const int i = t0 + threadIdx.x;
  if (i < N) y[col * N + i] = band_tile_row(bg, xt, N, i, threadIdx.x);
}

// y = B x for every column of the path arrays (x, y: column-major N-vectors).
static int band_apply(hipStream_t s, const PathArrays& p, const double* x, double* y) {
  const int64_t cols = (int64_t)p.G * p.C;
  hipLaunchKernelGGL(band_apply_kernel, dim3((unsigned)ceil_div(p.N, BT), (unsigned)cols), dim3(BT),
                     0, s, p.N, p.C, p.band, x, y);
  KMP_LAUNCH_CHECK();
  return 0;
}

// Q B, the A operand of the first path GEMM (f = (Q B) abar then needs no
// band product per iteration): row i of Q B is B applied to row i of Q (B
// symmetric, band[r][j] = B[j+r][j]). One workgroup per BT columns and QBR
// rows of a group; each thread keeps the 2 BND + 1 band entries of its
// column in registers and each row's piece of Q, with BND columns on either
// side, passes through LDS.
constexpr int QBR = 32;
__global__ __launch_bounds__(BT) void form_qb_kernel(int N, const double* __restrict__ Q,
                                                     const double* __restrict__ band,
                                                     double* __restrict__ QB) {
  __shared__ double qt[BT + 2 * BND];
  const int g = blockIdx.z;
  const int j0 = blockIdx.x * BT, j = j0 + threadIdx.x;
  const int i0 = blockIdx.y * QBR, i1 = min(i0 + QBR, N);
  const double* bg = band + (int64_t)g * (BND + 1) * N;
  const double* Qg = Q + (int64_t)g * N * N;
  double* Og = QB + (int64_t)g * N * N;
  const bool cj = j < N;
  // column j of B: B[j][j], B[j+r][j] = band[r][j], B[j-r][j] = band[r][j-r]
  const double b0 = cj ? bg[j] : 0.0;
  double bu[BND], bl[BND];
#pragma unroll
  for (int r = 1; r <= BND; ++r) {
    bu[r - 1] = (cj && j + r < N) ? bg[(int64_t)r * N + j] : 0.0;
    bl[r - 1] = (cj && j - r >= 0) ? bg[(int64_t)r * N + j - r] : 0.0;
  }
  for (int i = i0; i < i1; ++i) {
    const double* qr = Qg + (int64_t)i * N;
    for (int t = threadIdx.x; t < BT + 2 * BND; t += BT) {
      const int c = j0 - BND + t;
      qt[t] = (c >= 0 && c < N) ? qr[c] : 0.0;
    }
    __syncthreads();
    if (cj) {
      const int l = threadIdx.x + BND;
      double y0 = b0 * qt[l], y1 = 0.0;
#pragma unroll
      for (int r = 1; r <= BND; ++r) {
        y0 = fma(bu[r - 1], qt[l + r], y0);
        y1 = fma(bl[r - 1], qt[l - r], y1);
      }
      Og[(int64_t)i * N + j] = y0 + y1;
    }
    __syncthreads();
  }
}

int form_qb(hipStream_t s, const double* Q, const double* band, int N, int G, double* QB) {
  if (N <= 0 || G <= 0) return 0;
  hipLaunchKernelGGL(form_qb_kernel, dim3((unsigned)ceil_div(N, BT), (unsigned)ceil_div(N, QBR),
                                          (unsigned)G),
                     dim3(BT), 0, s, N, Q, band, QB);
  KMP_LAUNCH_CHECK();
  return 0;
}

// ------------------------------------------------------ per-stage factors
// ldl_factor_kernel, one wavefront per column: the blockwise LDL' of
// M = 2 lambda I + B/(n_v kappa) (stored as above). It reads the band,
// lambda and n_v only, so a stage's factors can be formed as soon as the
// band is known, before c = Q'1 is. Per 16-row block I:
//   S = M_II - C_I D_{I-1} C_I';
//   S = L D L' by a right-looking sweep whose row operations also turn an
//   identity into L^{-1} (the product of the elimination steps);
//   C_{I+1} = M_{I+1,I} L^{-T} D^{-1}.
// The band tile of block I+1 (rows 0 .. 16 of its 16 columns) is loaded
// while block I is worked on and passes through LDS.
constexpr int FW = 4;                  // wavefronts (columns) per workgroup
__global__ __launch_bounds__(64 * FW) void ldl_factor_kernel(
    int N, int C, int64_t cols, const int* __restrict__ nv, const double* __restrict__ band,
    const double* __restrict__ lamv, double kappa, double* __restrict__ Vfac,
    double* __restrict__ Dfac) {
  __shared__ double tiles[FW * PTILE];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t gc = (int64_t)blockIdx.x * FW + wv;
  if (gc >= cols) return;
  constexpr int TL = BND + 1;            // LDS row of a 16 x 16 tile
  double* Cs = tiles + wv * PTILE;       // C_I (upper triangular)
  double* Xs = Cs + BND * TL;            // L_I^{-1} (unit lower triangular)
  double* colb = Xs + BND * TL;          // column k of the sweep
  double* wrow = colb + BND;             // row k of the inverse being formed
  double* rdv = wrow + BND;              // 1 / D_I
  double* dbuf = rdv + BND;              // D_I and D_{I-1}, by the parity of I
  double* Bt = dbuf + 2 * BND;           // band tile of block I: Bt[r * BND + j] = B[i0+j+r][i0+j]
  const int g = (int)(gc / C);
  const double lam = lamv[gc];
  const double sc = 1.0 / ((double)nv[gc] * kappa);   // the column's loss normaliser
  const double* bg = band + (int64_t)g * (BND + 1) * N;
  double* Vc = Vfac + gc * (int64_t)BND * N;
  double* Dc = Dfac + gc * (int64_t)N;
  // lane (a, qg): row a of each 16 x 16 tile, columns 4 qg .. 4 qg + 3
  const int a = lane & (BND - 1), qg = lane >> 4;
  const int NB = N / BND;
  // the (BND + 1) x BND band tile of block I, element e = lane + 64 q
  constexpr int BTQ = ((BND + 1) * BND + 63) / 64;
  const auto load_tile = [&](int I, double* bt) {
    const int i0 = BND * I;
#pragma unroll
    for (int q = 0; q < BTQ; ++q) {
      const int e = lane + 64 * q;
      bt[q] = (e < (BND + 1) * BND) ? bg[(int64_t)(e / BND) * N + i0 + e % BND] : 0.0;
    }
  };
  for (int e = lane; e < BND * TL; e += 64) Cs[e] = 0.0;
  if (lane < 2 * BND) dbuf[lane] = 0.0;
  double bt[BTQ];
  load_tile(0, bt);
  for (int I = 0; I < NB; ++I) {
    const int i0 = BND * I;
    const double* dp = dbuf + ((I + 1) & 1) * BND;   // D_{I-1}
    double* dc = dbuf + (I & 1) * BND;               // D_I
    wave_sync();
#pragma unroll
    for (int q = 0; q < BTQ; ++q)
      if (lane + 64 * q < (BND + 1) * BND) Bt[lane + 64 * q] = bt[q];
    load_tile(I + 1 < NB ? I + 1 : I, bt);
    wave_sync();
    double s4[4], w4[4];
    {
      double cr[BND];
#pragma unroll
      for (int j = 0; j < BND; ++j) cr[j] = Cs[a * TL + j] * dp[j];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int c = 4 * qg + t;
        const double bv = (c <= a) ? Bt[(a - c) * BND + c] : Bt[(c - a) * BND + a];
        const double m = fma(sc, bv, (c == a) ? 2.0 * lam : 0.0);
        double acc0 = 0.0, acc1 = 0.0;
#pragma unroll
        for (int j = 0; j < BND; j += 2) {
          acc0 = fma(cr[j], Cs[c * TL + j], acc0);
          acc1 = fma(cr[j + 1], Cs[c * TL + j + 1], acc1);
        }
        s4[t] = m - (acc0 + acc1);
        w4[t] = (c == a) ? 1.0 : 0.0;
      }
    }
    // the sweep: column k of S and row k of the inverse through LDS; rows
    // below k take off l_ak times row k (S: trailing entries, W: all)
#pragma unroll 1
    for (int kq = 0; kq < BND / 4; ++kq) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const int k = 4 * kq + kt;
        wave_sync();
        if (qg == kq) colb[a] = s4[kt];
        if (a == k) {
#pragma unroll
          for (int t = 0; t < 4; ++t) wrow[4 * qg + t] = w4[t];
        }
        wave_sync();
        const double rk = rcp_newton(colb[k]);
        const double ca = colb[a];
        double cj[4], wk[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          cj[t] = colb[4 * qg + t];
          wk[t] = wrow[4 * qg + t];
        }
        // entries outside the trailing block (a <= k or j <= k), and the
        // inverse rows a <= k, take off a zero multiple: every lane runs
        // the same straight-line code
        const double cam = (a > k) ? ca : 0.0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const double cjm = (4 * qg + t > k) ? cj[t] : 0.0;
          s4[t] = fma(-(cam * cjm), rk, s4[t]);
        }
        const double la = ca * rk;                    // L[a][k] for a > k
        const double lw = cam * rk;
#pragma unroll
        for (int t = 0; t < 4; ++t) w4[t] = fma(-lw, wk[t], w4[t]);
        s4[kt] = ((qg == kq) & (a > k)) ? la : s4[kt];
      }
    }
    // D_I, 1/D_I and L_I^{-1} to LDS
    if (qg == (a >> 2)) {
      const double da = s4[a & 3];
      dc[a] = da;
      rdv[a] = rcp_newton(da);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) Xs[a * TL + 4 * qg + t] = w4[t];
    wave_sync();
    // the tile (L^{-1} below the diagonal, C_I on and above) and 1/D
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int j = 4 * qg + t;
      Vc[(int64_t)j * N + i0 + a] = (j < a) ? w4[t] : Cs[a * TL + j];
    }
    if (qg == 0) Dc[i0 + a] = rdv[a];
    // C_{I+1}[a][c] = sum_{j=a..c} M_{I+1,I}[a][j] X[c][j] / D[c], with
    // B[i0+16+a][i0+j] = Bt[(16+a-j) BND + j] for j >= a
    double cn[4] = {0.0, 0.0, 0.0, 0.0};
    if (I + 1 < NB) {
      double mn[BND];
#pragma unroll
      for (int j = 0; j < BND; ++j) mn[j] = (j >= a) ? Bt[(BND + a - j) * BND + j] : 0.0;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int c = 4 * qg + t;
        double acc0 = 0.0, acc1 = 0.0;
#pragma unroll
        for (int j = 0; j < BND; j += 2) {
          acc0 = fma(mn[j], Xs[c * TL + j], acc0);
          acc1 = fma(mn[j + 1], Xs[c * TL + j + 1], acc1);
        }
        cn[t] = (c >= a) ? sc * (acc0 + acc1) * rdv[c] : 0.0;
      }
    }
    wave_sync();
#pragma unroll
    for (int t = 0; t < 4; ++t) Cs[a * TL + 4 * qg + t] = cn[t];
  }
}

// stage_vectors_kernel, one wavefront per column, after the factors:
// vhat = M^{-1} c/(n_v kappa), g = 1/(2 lambda c'vhat); restart the momentum
// (r = 1, abar = ahat) and reactivate the columns that stopped in the
// previous stage (u = B vhat follows in band_apply_kernel).
template <bool GV>
__global__ __launch_bounds__(256) void stage_vectors_kernel(
    int N, int C, int64_t cols, const int* __restrict__ nv, const double* __restrict__ cvec,
    const double* __restrict__ lamv, double kappa, const double* __restrict__ Vfac,
    const double* __restrict__ Dfac, double* __restrict__ vhat, double* __restrict__ gcoef,
    const double* __restrict__ ahat, double* __restrict__ abar, const double* __restrict__ beta,
    double* __restrict__ bbar, double* __restrict__ rmom, int* __restrict__ flag,
    int* __restrict__ iters) {
  extern __shared__ double lds_dyn[];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t gc = (int64_t)blockIdx.x * (blockDim.x >> 6) + wv;
  if (gc >= cols) return;
  double* xs = lds_dyn + (int64_t)wv * (GV ? RING : N);   // vector or ring
  const int g = (int)(gc / C);
  const double lam = lamv[gc];
  const double sc = 1.0 / ((double)nv[gc] * kappa);   // the column's loss normaliser
  const double* cg = cvec + (int64_t)g * N;
  const double* Vc = Vfac + gc * (int64_t)BND * N;
  const double* Dc = Dfac + gc * (int64_t)N;
  const int64_t base = gc * (int64_t)N;
  double cv = 0.0;
  if constexpr (GV) {
    // input c sc, forward results kept in vhat, then vhat = x
    double* vg = vhat + base;
    band_solve_g(Vc, Dc, cg, sc, vg, xs, N, lane, [&](int r, double x, bool) { vg[r] = x; });
    // x was written by the lanes of its rows and is read by every lane
    grid_vec_sync();
#pragma unroll 8
    for (int i = lane; i < N; i += 64) cv = fma(cg[i], vg[i], cv);
  } else {
#pragma unroll 8
    for (int i = lane; i < N; i += 64) xs[i] = cg[i] * sc;
    wave_sync();
    band_solve(Vc, Dc, xs, N, lane);
#pragma unroll 8
    for (int i = lane; i < N; i += 64) {
      const double v = xs[i];
      vhat[base + i] = v;
      cv = fma(cg[i], v, cv);
    }
  }
  cv = wave_sum(cv);
#pragma unroll 8
  for (int i = lane; i < N; i += 64) abar[base + i] = ahat[base + i];
  if (lane == 0) {
    gcoef[gc] = 1.0 / (2.0 * lam * cv);
    bbar[gc] = beta[gc];
    rmom[gc] = 1.0;
    if (flag[gc] == 1 || flag[gc] == 2) flag[gc] = 0;
    iters[gc] = 0;
  }
}

// The band of the matrix with rows and columns in reverse order:
// Brev[c+d][c] = B[N-1-c-d][N-1-c] = band[d][N-1-c-d] (symmetric B), zero
// past the last row.
__global__ void reverse_band_kernel(const double* __restrict__ band, int N, int64_t total,
                                    double* __restrict__ brev) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = e / N;                 // g * (BND + 1) + d
    const int c = (int)(e % N), d = (int)(row % (BND + 1));
    const int src = N - 1 - c - d;
    brev[e] = (src >= 0) ? band[row * N + src] : 0.0;
  }
}

// The twist block of band_solve_twist for every column: k = NB/2,
// J = NB-1-k,
//   Z = M_kk - C_k D_{k-1} C_k' - P (C~_J D~_{J-1} C~_J') P
// (C, D: the top-down factors; C~, D~: those of the reversed matrix, whose
// block J is block k with its rows in reverse order, P that reversal;
// both factor arrays hold 1/D), then Z = L D L' by unpivoted row
// elimination (Z is symmetric positive definite), the same operations
// turning an identity into L^{-1}. Stored at tw + gc * (BND*BND + BND):
// L^{-1} row-major, then 1/D. One wavefront per column; lane a < 16 holds
// row a.
constexpr int TWS = BND * BND + BND;
__global__ __launch_bounds__(64 * FW) void twist_factor_kernel(
    int N, int C, int64_t cols, const int* __restrict__ nv, const double* __restrict__ band,
    const double* __restrict__ lamv, double kappa, const double* __restrict__ Vt,
    const double* __restrict__ Dt, const double* __restrict__ Vr, const double* __restrict__ Dr,
    double* __restrict__ tw) {
  __shared__ double zr[FW][BND][BND + 1];
  __shared__ double wr[FW][BND][BND + 1];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t gc = (int64_t)blockIdx.x * FW + wv;
  if (gc >= cols) return;                       // per wavefront: no barrier below
  const int g = (int)(gc / C);
  const double lam = lamv[gc];
  const double sc = 1.0 / ((double)nv[gc] * kappa);
  const double* bg = band + (int64_t)g * (BND + 1) * N;
  const int NB = N / BND, k = NB / 2, J = NB - 1 - k;
  const double* Vc = Vt + gc * (int64_t)BND * N;
  const double* Dc = Dt + gc * (int64_t)N;
  const double* Vq = Vr + gc * (int64_t)BND * N;
  const double* Dq = Dr + gc * (int64_t)N;
  const int a = lane;
  double z[BND], w[BND];
  if (a < BND) {
    const int ar = BND - 1 - a;                 // row a of block k in the reversed order
#pragma unroll
    for (int c = 0; c < BND; ++c) {
      const double bv = (c <= a) ? bg[(int64_t)(a - c) * N + BND * k + c]
                                 : bg[(int64_t)(c - a) * N + BND * k + a];
      double v = fma(sc, bv, (c == a) ? 2.0 * lam : 0.0);
      const int cr = BND - 1 - c;
      double st = 0.0, sb = 0.0;
      if (k > 0)
        for (int j = max(a, c); j < BND; ++j)   // C_k upper triangular
          st = fma(Vc[(int64_t)j * N + BND * k + a] * Vc[(int64_t)j * N + BND * k + c],
                   1.0 / Dc[BND * (k - 1) + j], st);
      if (J > 0)
        for (int j = max(ar, cr); j < BND; ++j)
          sb = fma(Vq[(int64_t)j * N + BND * J + ar] * Vq[(int64_t)j * N + BND * J + cr],
                   1.0 / Dq[BND * (J - 1) + j], sb);
      z[c] = v - st - sb;
      w[c] = (c == a) ? 1.0 : 0.0;
    }
  }
  for (int p = 0; p < BND; ++p) {
    wave_sync();
    if (a == p) {
#pragma unroll
      for (int c = 0; c < BND; ++c) {
        zr[wv][p][c] = z[c];
        wr[wv][p][c] = w[c];
      }
    }
    wave_sync();
    if (a < BND && a > p) {
      const double l = z[p] / zr[wv][p][p];
#pragma unroll
      for (int c = 0; c < BND; ++c) {
        z[c] = fma(-l, zr[wv][p][c], z[c]);
        w[c] = fma(-l, wr[wv][p][c], w[c]);
      }
    }
  }
  if (a < BND) {
    double* out = tw + gc * (int64_t)TWS;
#pragma unroll
    for (int c = 0; c < BND; ++c) out[a * BND + c] = w[c];
    out[BND * BND + a] = 1.0 / z[a];
  }
}

int path_stage_factor(hipStream_t s, const PathArrays& p, double kappa) {
  const int64_t cols = (int64_t)p.G * p.C;
  kc_begin(KMP_KC_PRECOMPUTE, s);
  hipLaunchKernelGGL(ldl_factor_kernel, dim3((unsigned)ceil_div(cols, FW)), dim3(64 * FW), 0, s, p.N,
                     p.C, cols, p.cnv, p.band, p.lam, kappa, p.ldl_l, p.ldl_d);
  KMP_LAUNCH_CHECK();
  // the twisted solves' data: the factors of the reversed matrix and the
  // twist block
  {
    const int64_t tb = (int64_t)p.G * (BND + 1) * p.N;
    hipLaunchKernelGGL(reverse_band_kernel, dim3((unsigned)std::min<int64_t>(ceil_div(tb, 256), 4096)),
                       dim3(256), 0, s, p.band, p.N, tb, p.band_rev);
    KMP_LAUNCH_CHECK();
    hipLaunchKernelGGL(ldl_factor_kernel, dim3((unsigned)ceil_div(cols, FW)), dim3(64 * FW), 0, s,
                       p.N, p.C, cols, p.cnv, p.band_rev, p.lam, kappa, p.ldl_lr, p.ldl_dr);
    KMP_LAUNCH_CHECK();
    hipLaunchKernelGGL(twist_factor_kernel, dim3((unsigned)ceil_div(cols, FW)), dim3(64 * FW), 0, s,
                       p.N, p.C, cols, p.cnv, p.band, p.lam, kappa, p.ldl_l, p.ldl_d, p.ldl_lr,
                       p.ldl_dr, p.twist);
    KMP_LAUNCH_CHECK();
  }
  // reads the band, writes the factor tiles and 1/d (BND + 1 per element),
  // in both directions
  kc_end(KMP_KC_PRECOMPUTE, s,
         2.0 * over_groups(p, [&](double n) { return 8.0 * n * p.C * (BND + 1.0); }),
         2.0 * over_groups(p, [&](double n) { return 4.0 * BND * BND * n * p.C; }));
  return 0;
}

int path_stage_vectors(hipStream_t s, const PathArrays& p, double kappa) {
  const int64_t cols = (int64_t)p.G * p.C;
  const int cw = path_waves(p, 0);
  const size_t lds = sizeof(double) * (size_t)cw * path_lds_doubles(p, 0);
  const void* kfn = path_global_vec(p) ? (const void*)stage_vectors_kernel<true>
                                       : (const void*)stage_vectors_kernel<false>;
  KMP_HIP_TRY(hipFuncSetAttribute(kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
  kc_begin(KMP_KC_PRECOMPUTE, s);
  if (path_global_vec(p))
    hipLaunchKernelGGL(stage_vectors_kernel<true>, dim3((unsigned)ceil_div(cols, cw)), dim3(64 * cw),
                       lds, s, p.N, p.C, cols, p.cnv, p.cvec, p.lam, kappa, p.ldl_l, p.ldl_d, p.vhat,
                       p.gcoef, p.ahat, p.abar, p.beta, p.bbar, p.rmom, p.flag, p.iters);
  else
    hipLaunchKernelGGL(stage_vectors_kernel<false>, dim3((unsigned)ceil_div(cols, cw)), dim3(64 * cw),
                       lds, s, p.N, p.C, cols, p.cnv, p.cvec, p.lam, kappa, p.ldl_l, p.ldl_d, p.vhat,
                       p.gcoef, p.ahat, p.abar, p.beta, p.bbar, p.rmom, p.flag, p.iters);
  KMP_LAUNCH_CHECK();
  int rc;
  if ((rc = band_apply(s, p, p.vhat, p.uvec)) != 0) return rc;
  // the solve reads the factor (BND + 1 per element) and c, writes vhat;
  // ahat to abar; then u = B vhat (read one vector, write one)
  kc_end(KMP_KC_PRECOMPUTE, s, over_groups(p, [&](double n) { return 8.0 * n * p.C * (BND + 7.0); }),
         over_groups(p, [&](double n) { return (4.0 * BND + 2.0 * (2 * BND + 1)) * n * p.C; }));
  return 0;
}

// ------------------------------------------------------- the update (K2)
// Element loops load UL rows per lane before using them, so a lane keeps UL
// loads of each stream in flight.
constexpr int UL = 8;

// The update with the solve's vector in device memory (orders above the
// LDS capacity, or when it keeps more columns resident): two columns per
// 256-thread workgroup, wavefronts 2c and 2c+1 for column c. Wavefront 2c:
//   d0 = 1'z (from the loss epilogue's tile sums), w = zhat + 2 lambda abar
//   (split-K parts of zhat added in order) into the column's e vector,
//   t = u'w, ||w||; the KKT test at the extrapolated point;
// both: x = M^{-1} w by the twisted device-memory solve (x over w in e);
// wavefront 2c: the step Da = g (t - d0) vhat + x, a+ = abar - Da,
//   e = a+ - ahat, the restart test sum Da'e + Db (b+ - beta) > 0, the
//   momentum r and its coefficient; then ahat = a+ and abar = a+ +
//   coef (a+ - ahat) (the first path GEMM multiplies Q B by abar, so no
//   band product follows), and the column's scalars.
// A column that stops before the solve (inactive, converged at the
// extrapolated point, non-finite) still takes the workgroup's barriers, so
// nothing returns early.
__global__ __launch_bounds__(256) void solve_step_twist_kernel(
    int N, int C, int64_t cols, int RT, const int* __restrict__ nvv,
    const double* __restrict__ lamv, const double* __restrict__ zpart, int S2, int64_t sP,
    double* __restrict__ ahat, double* __restrict__ abar, const double* __restrict__ Vfac,
    const double* __restrict__ Dfac, const double* __restrict__ Vrev,
    const double* __restrict__ Drev, const double* __restrict__ twist,
    const double* __restrict__ vhat, const double* __restrict__ uvec,
    const double* __restrict__ gcoef, const double* __restrict__ partial,
    double* __restrict__ beta, double* __restrict__ bbar, double* __restrict__ rmom,
    double* __restrict__ kktv, int* __restrict__ flag, int* __restrict__ iters,
    int* __restrict__ iters_total, double* __restrict__ anew, double* __restrict__ estep,
    double tol, int max_iter, int restart) {
  __shared__ double rings[4][RING];
  __shared__ double tslot[2][3 * BND];
  __shared__ int go[2];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int pr = wv >> 1, role = wv & 1;
  const int64_t gc = (int64_t)blockIdx.x * 2 + pr;
  const bool exists = gc < cols;
  bool live = exists && flag[gc] == 0;
  const int64_t gcs = exists ? gc : 0;                 // a valid column for the pointers
  const int g = (int)(gcs / C), c = (int)(gcs % C);
  const int64_t base = gcs * (int64_t)N;
  double d0 = 0.0, tsum = 0.0, kkt = 0.0;
  if (role == 0 && live) {
    const double lam = lamv[gc];
    const double nvd = (double)nvv[gc];
    {
      const double* pg = partial + (int64_t)g * RT * C + c;
      for (int r = lane; r < RT; r += 64) d0 += pg[(int64_t)r * C];
      d0 = wave_sum(d0);
    }
    double tl = 0.0, n2 = 0.0;
    for (int i0 = 0; i0 < N; i0 += 64 * UL) {
      double zs[UL], ab[UL], uv[UL];
#pragma unroll
      for (int q = 0; q < UL; ++q) {
        const int i = i0 + lane + 64 * q;
        const int64_t ic = base + ((i < N) ? i : N - 1);
        double z = zpart[ic];
#pragma unroll
        for (int sk = 1; sk < kMaxSplitK; ++sk) {
          const double zz = zpart[(sk < S2 ? sk : 0) * sP + ic];
          z += (sk < S2) ? zz : 0.0;
        }
        zs[q] = z;
        ab[q] = abar[ic];
        uv[q] = uvec[ic];
      }
#pragma unroll
      for (int q = 0; q < UL; ++q) {
        const int i = i0 + lane + 64 * q;
        if (i < N) {
          const double w = fma(2.0 * lam, ab[q], zs[q]);
          estep[base + i] = w;
          tl = fma(uv[q], w, tl);
          n2 = fma(w, w, n2);
        }
      }
    }
    tsum = wave_sum(tl);
    const double n2sum = wave_sum(n2);
    kkt = nvd * fmax(sqrt(n2sum), fabs(d0));
    if (!(n2sum == n2sum) || !(d0 == d0) || !(kkt <= 1e300)) {
      if (lane == 0) { flag[gc] = 3; kktv[gc] = kkt; }
      live = false;
    } else if (kkt <= tol) {                            // certified at the extrapolated point
#pragma unroll 8
      for (int i = lane; i < N; i += 64) ahat[base + i] = abar[base + i];
      if (lane == 0) { beta[gc] = bbar[gc]; flag[gc] = 1; kktv[gc] = kkt; }
      live = false;
    }
  }
  if (role == 0 && lane == 0) go[pr] = live ? 1 : 0;
  __syncthreads();                                      // w in e and the decision
  live = go[pr] != 0;
  double* xg = estep + base;
  band_solve_g_twist(Vfac + gcs * (int64_t)BND * N, Dfac + base, Vrev + gcs * (int64_t)BND * N,
                     Drev + base, twist + gcs * (int64_t)TWS, xg, anew + base, rings[2 * pr],
                     rings[2 * pr + 1], tslot[pr], N, role, live, lane,
                     [&](int r, double x, bool) { xg[r] = x; });
  __syncthreads();                                      // x in e
  if (role != 0 || !live) return;
  const double gco = gcoef[gc];
  const double sa = gco * (tsum - d0);
  const double db = gco * (d0 - tsum);
  const double bb = bbar[gc];
  const double bn = bb - db;
  const double bold = beta[gc];
  double rd = 0.0;
  for (int i0 = 0; i0 < N; i0 += 64 * UL) {
    double vh[UL], ab[UL], ah[UL], xv[UL];
#pragma unroll
    for (int q = 0; q < UL; ++q) {
      const int i = i0 + lane + 64 * q;
      const int ii = (i < N) ? i : N - 1;
      const int64_t ic = base + ii;
      vh[q] = vhat[ic];
      ab[q] = abar[ic];
      ah[q] = ahat[ic];
      xv[q] = xg[ii];
    }
#pragma unroll
    for (int q = 0; q < UL; ++q) {
      const int i = i0 + lane + 64 * q;
      if (i < N) {
        const double da = fma(sa, vh[q], xv[q]);
        const double an = ab[q] - da;
        rd = fma(da, an - ah[q], rd);
        xg[i] = an;
      }
    }
  }
  rd = wave_sum(rd) + db * (bn - bold);
  const double r = rmom[gc];
  const double rn = (restart && rd > 0.0) ? 1.0 : 0.5 * (1.0 + sqrt(1.0 + 4.0 * r * r));
  const double coef = (rn - 1.0) / (0.5 * (1.0 + sqrt(1.0 + 4.0 * rn * rn)));
  for (int i0 = 0; i0 < N; i0 += 64 * UL) {
    double ah[UL], an[UL];
#pragma unroll
    for (int q = 0; q < UL; ++q) {
      const int i = i0 + lane + 64 * q;
      const int ii = (i < N) ? i : N - 1;
      ah[q] = ahat[base + ii];
      an[q] = xg[ii];
    }
#pragma unroll
    for (int q = 0; q < UL; ++q) {
      const int i = i0 + lane + 64 * q;
      if (i < N) {
        ahat[base + i] = an[q];
        abar[base + i] = fma(coef, an[q] - ah[q], an[q]);
      }
    }
  }
  if (lane == 0) {
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

// The update of one column per 256-thread workgroup, for orders whose
// vector fits in LDS (N <= lds_vec_max()): the element passes are spread over
// the four wavefronts (four times the loads in flight of one wavefront) and
// wavefront 0 alone runs the banded solve on the LDS vector:
//   w = zhat + 2 lambda abar (LDS), t = u'w, ||w||, d0; KKT decision;
//   x = M^{-1} w (wavefront 0); a+ = abar - g (t - d0) vhat - x,
//   e = a+ - ahat, restart test, momentum coefficient; a+ is kept in LDS
//   over x, then ahat = a+ and abar = a+ + coef e (no band product: the
//   first path GEMM multiplies Q B by abar).
// Reductions are block sums in a fixed order. LDS: N doubles.
__global__ __launch_bounds__(256) void update_column_kernel(
    int N, int C, int RT, const int* __restrict__ nvv, const double* __restrict__ lamv,
    const double* __restrict__ zpart, int S2, int64_t sP, double* __restrict__ ahat,
    double* __restrict__ abar, const double* __restrict__ Vfac, const double* __restrict__ Dfac,
    const double* __restrict__ Vrev, const double* __restrict__ Drev,
    const double* __restrict__ twist, const double* __restrict__ vhat,
    const double* __restrict__ uvec,
    const double* __restrict__ gcoef, const double* __restrict__ partial,
    double* __restrict__ beta, double* __restrict__ bbar, double* __restrict__ rmom,
    double* __restrict__ kktv, int* __restrict__ flag, int* __restrict__ iters,
    int* __restrict__ iters_total, double tol, int max_iter, int restart) {
  extern __shared__ double lds_dyn[];
  __shared__ double red[PW];
  __shared__ double tslot[3 * BND];
  const int t = threadIdx.x, wv = t >> 6, lane = t & 63;
  const int64_t gc = blockIdx.x;
  if (flag[gc] != 0) return;                            // uniform over the block
  double* xs = lds_dyn;                                 // w, then x
  const int g = (int)(gc / C), c = (int)(gc % C);
  const int64_t base = gc * (int64_t)N;
  const double lam = lamv[gc];
  const double nvd = (double)nvv[gc];                  // the column's loss normaliser
  double d0 = 0.0;
  {
    const double* pg = partial + (int64_t)g * RT * C + c;
    for (int r = t; r < RT; r += PB) d0 += pg[(int64_t)r * C];
  }
  double tl = 0.0, n2 = 0.0;
  for (int i0 = 0; i0 < N; i0 += PB * 4) {
    double zs[4], ab[4], uv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + t + PB * q;
      const int64_t ic = base + ((i < N) ? i : N - 1);
      double z = zpart[ic];
#pragma unroll
      for (int sk = 1; sk < kMaxSplitK; ++sk) {
        const double zz = zpart[(sk < S2 ? sk : 0) * sP + ic];
        z += (sk < S2) ? zz : 0.0;
      }
      zs[q] = z;
      ab[q] = abar[ic];
      uv[q] = uvec[ic];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + t + PB * q;
      if (i < N) {
        const double w = fma(2.0 * lam, ab[q], zs[q]);
        xs[i] = w;
        tl = fma(uv[q], w, tl);
        n2 = fma(w, w, n2);
      }
    }
  }
  d0 = block_sum<PW>(d0, red);
  const double tsum = block_sum<PW>(tl, red);
  const double n2sum = block_sum<PW>(n2, red);
  const double kkt = nvd * fmax(sqrt(n2sum), fabs(d0));
  const double bb = bbar[gc];
  // non-finite (uniform): tested on both terms, since fmax drops a NaN
  if (!(n2sum == n2sum) || !(d0 == d0) || !(kkt <= 1e300)) {
    if (t == 0) { flag[gc] = 3; kktv[gc] = kkt; }
    return;
  }
  if (kkt <= tol) {                                     // certified at the extrapolated point
    for (int i = t; i < N; i += PB) ahat[base + i] = abar[base + i];
    if (t == 0) { beta[gc] = bb; flag[gc] = 1; kktv[gc] = kkt; }
    return;
  }
  __syncthreads();                                      // w complete in LDS
  band_solve_twist(Vfac + gc * (int64_t)BND * N, Dfac + base, Vrev + gc * (int64_t)BND * N,
                   Drev + base, twist + gc * (int64_t)TWS, xs, tslot, N, wv, lane);
  __syncthreads();                                      // x complete in LDS
  const double gco = gcoef[gc];
  const double sa = gco * (tsum - d0);
  const double db = gco * (d0 - tsum);
  const double bn = bb - db;
  const double bold = beta[gc];
  double rd = 0.0;
  for (int i0 = 0; i0 < N; i0 += PB * 4) {
    double vh[4], ab[4], ah[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + t + PB * q;
      const int64_t ic = base + ((i < N) ? i : N - 1);
      vh[q] = vhat[ic];
      ab[q] = abar[ic];
      ah[q] = ahat[ic];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + t + PB * q;
      if (i < N) {
        const double da = fma(sa, vh[q], xs[i]);
        const double an = ab[q] - da;
        rd = fma(da, an - ah[q], rd);
        xs[i] = an;                                     // a+ over x, row by row
      }
    }
  }
  rd = block_sum<PW>(rd, red) + db * (bn - bold);
  const double r = rmom[gc];
  const double rn = (restart && rd > 0.0) ? 1.0 : 0.5 * (1.0 + sqrt(1.0 + 4.0 * r * r));
  const double coef = (rn - 1.0) / (0.5 * (1.0 + sqrt(1.0 + 4.0 * rn * rn)));
  // momentum: ahat = a+, abar = a+ + coef (a+ - ahat), each thread on the
  // rows whose a+ it kept
  for (int i0 = 0; i0 < N; i0 += PB * 4) {
    double ah[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + t + PB * q;
      ah[q] = ahat[base + ((i < N) ? i : N - 1)];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + t + PB * q;
      if (i < N) {
        const double an = xs[i];
        ahat[base + i] = an;
        abar[base + i] = fma(coef, an - ah[q], an);
      }
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
  // f = (Q B) abar as split-K partials, then z = psi(y, f + bbar)/n_v with
  // 64-row column sums
  GemmArgs g1;
  g1.M = p.N; g1.N = p.C; g1.K = p.N; g1.batch = p.G;
  g1.A = p.QB; g1.lda = p.N; g1.sA = (int64_t)p.N * p.N;
  g1.B = p.abar; g1.ldb = p.N; g1.sB = sC;
  g1.ldc = p.N; g1.sC = sC;
  // the tile shape and its work tiles (the counts are one poll behind:
  // any choice is exact)
  int64_t work_tiles = 0;
  int per_cu = 4;
  const PartTile tile = pick_part_tile(p.N, p.G, p.C, p.nact_host, &work_tiles, &per_cu);
  const int S1 = splitk_parts(g1, work_tiles, per_cu);
  LossEpi e;
  e.loss = p.loss; e.delta = delta;
  e.y = p.ylab; e.sy = p.N; e.nv = p.nv; e.cnv = p.cnv;
  e.bbar = p.bbar; e.sbb = p.C; e.tau = p.tau; e.stau = p.C;
  e.rfold = p.rfold; e.cfold = p.cfold;
  e.partial = p.partial; e.spart = (int64_t)RT * p.C;
  const double gflops = over_active(p, [&](double n, double c) { return 2.0 * n * n * c; });
  const double gbytes = over_active(p, [&](double n, double c) { return 8.0 * (n * n + 2.0 * n * c); });
  kc_begin(KMP_KC_GEMM_F, s);
  if ((rc = gemm_partial(s, g1, true, S1, p.fpart, sP, p.cmap, p.nact, tile)) != 0) return rc;
  if ((rc = loss_epilogue(s, p.N, p.C, p.G, S1, p.fpart, p.N, sC, sP, p.zmat, e, p.cmap,
                          p.nact)) != 0)
    return rc;
  kc_end(KMP_KC_GEMM_F, s, gbytes, gflops);
  // zhat = Q' z as split-K partials (added by the update kernel)
  GemmArgs g2;
  g2.M = p.N; g2.N = p.C; g2.K = p.N; g2.batch = p.G;
  g2.A = p.Q; g2.lda = p.N; g2.sA = (int64_t)p.N * p.N;
  g2.B = p.zmat; g2.ldb = p.N; g2.sB = sC;
  g2.ldc = p.N; g2.sC = sC;
  const int S2 = splitk_parts(g2, work_tiles, per_cu);
  kc_begin(KMP_KC_GEMM_ZHAT, s);
  if ((rc = gemm_partial(s, g2, false, S2, p.zpart, sP, p.cmap, p.nact, tile)) != 0) return rc;
  kc_end(KMP_KC_GEMM_ZHAT, s, gbytes, gflops);
  const int64_t cols = (int64_t)p.G * p.C;
  const bool gv = iteration_global_vec(p);
  // per column element: S2 zhat parts, abar (twice), u, the factor tiles
  // (BND each, forward and backward), 1/d, vhat and ahat (twice) read, ahat
  // and abar written. Flops: BND multiply-adds per row in each triangular
  // sweep, 16 elementwise.
  const auto upd_bytes = over_active(p, [&](double n, double c) { return 8.0 * (S2 + 2.0 * BND + 9.0) * n * c; });
  const auto upd_flops = over_active(p, [&](double n, double c) { return (4.0 * BND + 16.0) * n * c; });
  if (!gv) {
    // one workgroup per column, the momentum step included
    const size_t lds_u = sizeof(double) * (size_t)p.N;
    KMP_HIP_TRY(hipFuncSetAttribute((const void*)update_column_kernel,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_u));
    kc_begin(KMP_KC_UPDATE, s);
    hipLaunchKernelGGL(update_column_kernel, dim3((unsigned)cols), dim3(PB), lds_u, s, p.N, p.C, RT,
                       p.cnv, p.lam, p.zpart, S2, sP, p.ahat, p.abar, p.ldl_l, p.ldl_d, p.ldl_lr,
                       p.ldl_dr, p.twist, p.vhat,
                       p.uvec, p.gcoef, p.partial, p.beta, p.bbar, p.rmom, p.kkt, p.flag, p.iters,
                       p.iters_total, tol, max_iter, restart);
    KMP_LAUNCH_CHECK();
    kc_end(KMP_KC_UPDATE, s, upd_bytes, upd_flops);
    return 0;
  }
  // the vector in device memory: the twisted solve, two columns per
  // workgroup
  kc_begin(KMP_KC_UPDATE, s);
  hipLaunchKernelGGL(solve_step_twist_kernel, dim3((unsigned)ceil_div(cols, 2)), dim3(256), 0, s,
                     p.N, p.C, cols, RT, p.cnv, p.lam, p.zpart, S2, sP, p.ahat, p.abar, p.ldl_l,
                     p.ldl_d, p.ldl_lr, p.ldl_dr, p.twist, p.vhat, p.uvec, p.gcoef, p.partial,
                     p.beta, p.bbar, p.rmom, p.kkt, p.flag, p.iters, p.iters_total, p.anew,
                     p.estep, tol, max_iter, restart);
  KMP_LAUNCH_CHECK();
  kc_end(KMP_KC_UPDATE, s, upd_bytes, upd_flops);
  return 0;
}

// One workgroup: wave w lists the active columns of groups w, w + 4, ...
// in increasing order (a ballot per 64 columns, the lane's rank among the
// active lanes below it giving its slot), then the group counts are added
// in a fixed order for the total.
__global__ __launch_bounds__(PB) void compact_columns_kernel(int G, int C,
                                                             const int* __restrict__ flag,
                                                             int* __restrict__ cmap,
                                                             int* __restrict__ nact,
                                                             int* __restrict__ total) {
  __shared__ int cnt[PW];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int mine = 0;
  for (int g = wv; g < G; g += PW) {
    int base = 0;
    for (int c0 = 0; c0 < C; c0 += 64) {
      const int c = c0 + lane;
      const bool act = c < C && flag[(int64_t)g * C + c] == 0;
      const unsigned long long m = __ballot(act);
      const int rank = __popcll(m & ((1ull << lane) - 1ull));
      if (act) cmap[(int64_t)g * C + base + rank] = c;
      base += __popcll(m);
    }
    if (lane == 0) nact[g] = base;
    mine += base;
  }
  if (lane == 0) cnt[wv] = mine;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int w = 0; w < PW; ++w) t += cnt[w];
    *total = t;
  }
}

int path_compact(hipStream_t s, const PathArrays& p) {
  hipLaunchKernelGGL(compact_columns_kernel, dim3(1), dim3(PB), 0, s, p.G, p.C, p.flag, p.cmap,
                     p.nact, p.active_count);
  KMP_LAUNCH_CHECK();
  return 0;
}

// --------------------------------------------------------------- finalize
// One workgroup per column: objective on the training points (from
// ftrain = K_v alpha in observation space), CV sums on the held-out points,
// scatter of alpha into the output layout, status counts.
__global__ __launch_bounds__(256) void cv_reduce_kernel(
    int n, int N, int Mh, int C, int V, int Qt, int L, int s0, int loss, double delta,
    const double* __restrict__ y, const int32_t* __restrict__ tidx,
    const int32_t* __restrict__ hidx, const int* __restrict__ nvv, const double* __restrict__ lamv,
    const double* __restrict__ tauv, const double* __restrict__ alpha_loc,
    const double* __restrict__ ftrain, const double* __restrict__ fheld,
    const double* __restrict__ betav, const int* __restrict__ flag,
    const int* __restrict__ iters_total, double* __restrict__ alpha_out,
    double* __restrict__ beta_out, double* __restrict__ obj_out, double* __restrict__ cv_out,
    int32_t* __restrict__ err_out, int32_t* __restrict__ it_out, int32_t* __restrict__ st_out,
    int* __restrict__ stat_count, const int* __restrict__ xflag) {
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
    const int fl = flag[gc];
    int st = fl == 1 ? 0 : (fl == 3 ? 2 : 1);
    if (st == 0 && xflag && xflag[gc] != 1) st = 3;    // exact hinge solution not reached
    if (st_out) st_out[cell] = st;
    // cells that stopped at max_iter / went non-finite / kept the smoothed
    // solution, counted whether or not the caller asked for the status
    if (st != 0) atomicAdd(stat_count + (st - 1), 1);
  }
}

// Shared-factor finalize, one workgroup per column (group g = bandwidth,
// column c = (tau, fold, lambda)): the rows of the column's fold give the CV
// sums, the others the objective F = (1/n_v) sum loss + lambda alpha' K alpha
// (f = K alpha in observation space, alpha zero on the held-out rows); alpha
// is scattered with zeros at the held-out rows; status counts.
__global__ __launch_bounds__(256) void cv_reduce_shared_kernel(
    int n, int N, int C, int s0, int loss, double delta, const double* __restrict__ y,
    const int32_t* __restrict__ fold, const int* __restrict__ cnv,
    const int32_t* __restrict__ cfold, const double* __restrict__ lamv,
    const double* __restrict__ tauv, const double* __restrict__ alpha_loc,
    const double* __restrict__ fall, const double* __restrict__ betav,
    const int* __restrict__ flag, const int* __restrict__ iters_total,
    double* __restrict__ alpha_out, double* __restrict__ beta_out, double* __restrict__ obj_out,
    double* __restrict__ cv_out, int32_t* __restrict__ err_out, int32_t* __restrict__ it_out,
    int32_t* __restrict__ st_out, int* __restrict__ stat_count) {
  __shared__ double red[PW];
  const int64_t gc = blockIdx.x;
  const int g = (int)(gc / C), c = (int)(gc % C);
  const int64_t cell = (int64_t)(s0 + g) * C + c;
  const int32_t v = cfold[gc];
  const double lam = lamv[gc], tau = tauv[gc], b = betav[gc];
  const double* A = alpha_loc + gc * N;
  const double* f = fall + gc * N;
  double* aout = alpha_out + cell * n;
  double ls = 0.0, pen = 0.0, cs = 0.0, ce = 0.0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const double fi = f[i] + b;
    if (fold[i] == v) {
      cs += loss_eval(loss, y[i], fi, tau);
      if (loss != 2 && y[i] * fi <= 0.0) ce += 1.0;
      aout[i] = 0.0;
    } else {
      ls += loss_value(loss, y[i], fi, delta, tau);
      pen = fma(A[i], f[i], pen);
      aout[i] = A[i];
    }
  }
  ls = block_sum<PW>(ls, red);
  pen = block_sum<PW>(pen, red);
  cs = block_sum<PW>(cs, red);
  ce = block_sum<PW>(ce, red);
  if (threadIdx.x == 0) {
    beta_out[cell] = b;
    obj_out[cell] = ls / (double)cnv[gc] + lam * pen;
    cv_out[cell] = cs;
    if (err_out) err_out[cell] = (int32_t)ce;
    if (it_out) it_out[cell] = iters_total[gc];
    const int fl = flag[gc];
    const int st = fl == 1 ? 0 : (fl == 3 ? 2 : 1);
    if (st_out) st_out[cell] = st;
    if (st != 0) atomicAdd(stat_count + (st - 1), 1);
  }
}

// x[gc][i] = 0 on the rows held out of column gc (rfold[g][i] == cfold[gc])
// and on padding rows (rfold = -1).
__global__ __launch_bounds__(256) void mask_heldout_kernel(int N, int C,
                                                           const int32_t* __restrict__ rfold,
                                                           const int32_t* __restrict__ cfold,
                                                           double* __restrict__ x) {
  const int64_t gc = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= N) return;
  const int32_t rf = rfold[(gc / C) * N + i];
  if (rf < 0 || rf == cfold[gc]) x[gc * N + i] = 0.0;
}

// C = sum over S split-K parts (part s at part + s sP; column-major, ld
// ldc, matrix b at + b sC), added in part order.
__global__ __launch_bounds__(256) void sum_parts_kernel(int M, int Nc, int S,
                                                        const double* __restrict__ part, int64_t sP,
                                                        int64_t ldc, int64_t sC,
                                                        double* __restrict__ C) {
  const int b = blockIdx.z, j = blockIdx.y;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= M || j >= Nc) return;
  const int64_t o = (int64_t)b * sC + (int64_t)j * ldc + i;
  double v = part[o];
  for (int q = 1; q < S; ++q) v += part[(int64_t)q * sP + o];
  C[o] = v;
}

// C = A B (A k-contiguous, B k-contiguous columns, C column-major with the
// parts' layout) by split-K parts in scratch, then their ordered sum.
static int gemm_split(hipStream_t s, const GemmArgs& g, double* scratch, int64_t sP) {
  int rc;
  const int S = splitk_parts(g);
  if ((rc = gemm_partial(s, g, true, S, scratch, sP, nullptr, nullptr)) != 0) return rc;
  hipLaunchKernelGGL(sum_parts_kernel, dim3((unsigned)ceil_div(g.M, 256), (unsigned)g.N,
                                            (unsigned)g.batch),
                     dim3(256), 0, s, g.M, g.N, S, (const double*)scratch, sP, g.ldc, g.sC, g.C);
  KMP_LAUNCH_CHECK();
  return 0;
}

// Finite smoothing to the exact hinge SVM (exact.hip), between the training
// predictions and the held-out block of the finalize: the Gram K_v is in the
// factor buffer, alpha_loc in zmat, K alpha in ftrain. Each round: the point
// sets, the products K w_L, the per-column solves, the products K alpha and
// the KKT check; the host reads the count of open columns after each round.
// Settled columns then take the exact solution.
static int exact_recover(hipStream_t s, const PathArrays& p, const FinalArgs& fa,
                         const GemmArgs& gk, int64_t sP) {
  int rc;
  ExactArgs x = fa.ex;
  x.ftrain = fa.ftrain;
  x.beta = p.beta;
  if ((rc = exact_init(s, x)) != 0) return rc;
  GemmArgs gl = gk;            // K_v times a column block
  for (int round = 0; round < fa.exact_rounds; ++round) {
    if ((rc = exact_sets(s, x)) != 0) return rc;
    gl.B = x.wl;
    gl.C = x.fl;
    if ((rc = gemm_split(s, gl, p.zpart, sP)) != 0) return rc;
    if ((rc = exact_solve(s, x)) != 0) return rc;
    gl.B = x.alpha;
    gl.C = x.fx;
    if ((rc = gemm_split(s, gl, p.zpart, sP)) != 0) return rc;
    KMP_HIP_TRY(hipMemsetAsync(x.pending, 0, sizeof(int), s));
    if ((rc = exact_check(s, x)) != 0) return rc;
    KMP_HIP_TRY(hipMemcpyAsync(fa.pending_host, x.pending, sizeof(int), hipMemcpyDeviceToHost, s));
    KMP_HIP_TRY(hipStreamSynchronize(s));
    if (*fa.pending_host == 0) break;
  }
  return exact_commit(s, x, p.zmat, fa.ftrain, p.beta);
}

// Shared-factor finalize: alpha = Q ahat with the held-out rows of each
// column set to zero, f = K alpha with K built again from X over all points
// (training and held-out predictions from one product), then the reductions.
static int path_finalize_shared(hipStream_t s, const PathArrays& p, const FinalArgs& fa) {
  int rc;
  kc_begin(KMP_KC_FINALIZE, s);
  const int64_t sNC = (int64_t)p.N * p.C;
  const int64_t sP = (int64_t)p.G * sNC;
  const int64_t cols = (int64_t)p.G * p.C;
  GemmArgs g;
  g.M = p.N; g.N = p.C; g.K = p.N; g.batch = p.G;
  g.A = p.Q; g.lda = p.N; g.sA = (int64_t)p.N * p.N;
  g.B = p.ahat; g.ldb = p.N; g.sB = sNC;
  g.C = p.zmat; g.ldc = p.N; g.sC = sNC;
  if ((rc = gemm_split(s, g, p.fpart, sP)) != 0) return rc;
  hipLaunchKernelGGL(mask_heldout_kernel, dim3((unsigned)ceil_div(p.N, 256), (unsigned)cols),
                     dim3(256), 0, s, p.N, p.C, p.rfold, p.cfold, p.zmat);
  KMP_LAUNCH_CHECK();
  if ((rc = rbf_blocks(s, fa.X, fa.d, fa.ldx, fa.nrm, fa.tidx, p.N, p.N, fa.tidx, p.N, p.N, 1,
                       fa.inv2s2, fa.S_b, fa.kh, (int64_t)p.N * p.N, (int64_t)p.N * p.N, p.N)) != 0)
    return rc;
  GemmArgs gt = g;
  gt.A = fa.kh;
  gt.B = p.zmat;
  gt.C = fa.ftrain;
  if ((rc = gemm_split(s, gt, p.zpart, sP)) != 0) return rc;
  hipLaunchKernelGGL(cv_reduce_shared_kernel, dim3((unsigned)cols), dim3(256), 0, s, fa.n, p.N,
                     p.C, fa.s0, p.loss, fa.delta, fa.y, fa.fold, p.cnv, p.cfold, p.lam, p.tau,
                     p.zmat, fa.ftrain, p.beta, p.flag, p.iters_total, fa.alpha, fa.beta_out,
                     fa.objective, fa.cv_sum, fa.cv_err, fa.iters, fa.status, fa.stat_count);
  KMP_LAUNCH_CHECK();
  // alpha = Q ahat and f = K alpha; K written and read back (2d flops per
  // entry); the column reads and writes
  kc_end(KMP_KC_FINALIZE, s,
         over_groups(p, [&](double n) { return 8.0 * (3.0 * n * n + 5.0 * n * p.C); }),
         over_groups(p, [&](double n) { return 4.0 * n * n * p.C + 2.0 * n * n * fa.d; }));
  return 0;
}

int path_finalize(hipStream_t s, const PathArrays& p, const FinalArgs& fa) {
  if (fa.shared) return path_finalize_shared(s, p, fa);
  int rc;
  kc_begin(KMP_KC_FINALIZE, s);
  const int64_t sNC = (int64_t)p.N * p.C;
  const int64_t sP = (int64_t)p.G * sNC;    // between split-K parts in fpart / zpart
  // alpha_loc = Q ahat (into zmat)
  GemmArgs g;
  g.M = p.N; g.N = p.C; g.K = p.N; g.batch = p.G;
  g.A = p.Q; g.lda = p.N; g.sA = (int64_t)p.N * p.N;
  g.B = p.ahat; g.ldb = p.N; g.sB = sNC;
  g.C = p.zmat; g.ldc = p.N; g.sC = sNC;
  // (the parts of this product go to fpart, those of the next to zpart:
  // the training predictions are stored in fpart)
  if ((rc = gemm_split(s, g, p.fpart, sP)) != 0) return rc;
  // training predictions K_v alpha in observation space: K_v is built again
  // from X into the factor buffer (no longer needed) and multiplied by
  // alpha, so the objective does not carry the factorisation's rounding
  if ((rc = rbf_blocks(s, fa.X, fa.d, fa.ldx, fa.nrm, fa.tidx, p.N, p.N, fa.tidx, p.N, p.N,
                       fa.V, fa.inv2s2, fa.S_b, fa.kh, (int64_t)fa.V * p.N * p.N,
                       (int64_t)p.N * p.N, p.N)) != 0)
    return rc;
  GemmArgs gt = g;
  gt.A = fa.kh;
  gt.B = p.zmat;
  gt.C = fa.ftrain;
  if ((rc = gemm_split(s, gt, p.zpart, sP)) != 0) return rc;
  if (fa.exact && (rc = exact_recover(s, p, fa, gt, sP)) != 0) return rc;
  // held-out kernel blocks K[H_v, T_v] (into the same buffer), then held-out
  // predictions K[H_v, T_v] alpha (none in a refit)
  if (fa.Mh > 0 &&
      (rc = rbf_blocks(s, fa.X, fa.d, fa.ldx, fa.nrm, fa.hidx, fa.Mh, fa.Mh, fa.tidx, p.N, p.N,
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
                     fa.alpha, fa.beta_out, fa.objective, fa.cv_sum, fa.cv_err, fa.iters, fa.status,
                     fa.stat_count, fa.exact ? fa.ex.xflag : nullptr);
  KMP_LAUNCH_CHECK();
  // products alpha = Q ahat, f = K_v alpha and the held-out f (Mh rows); the
  // training and held-out kernel blocks written and read back (2d flops per
  // entry); the column reads and writes
  kc_end(KMP_KC_FINALIZE, s,
         over_groups(p, [&](double n) {
           return 8.0 * (3.0 * n * n + 4.0 * n * p.C + 2.0 * fa.Mh * n + fa.Mh * p.C); }),
         over_groups(p, [&](double n) {
           return 4.0 * n * n * p.C + 2.0 * n * n * fa.d + 2.0 * fa.Mh * n * (p.C + fa.d); }));
  return 0;
}

}  // namespace kmp
