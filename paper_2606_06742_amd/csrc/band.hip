// Per-fold factorisation K_v = Q B Q' with B symmetric banded (lower
// bandwidth kBand) and Q orthogonal.
//
// The paper factorises the kernel matrix once and reuses the factor for
// every lambda (Appendix A.3). Here the one-time factorisation stops at a
// band matrix: the resolvent (2 lambda I + K/(n kappa))^{-1} equals
// Q (2 lambda I + B/(n kappa))^{-1} Q' exactly, and the banded system is
// solved per column by a banded LDL' factorisation. Unlike the reduction to
// tridiagonal form, whose trailing matrix-vector product per column bounds it
// by memory latency and bandwidth, the reduction to band form is blocked:
// each panel of kBand columns is factored by a Householder QR (Golub & Van
// Loan Alg. 5.2.1; compact WY form, Schreiber & Van Loan 1989) and the
// trailing matrix receives one two-sided update built from matrix-core GEMMs
// (the first stage of the successive band reduction of Bischof, Lang & Sun,
// 2000, as in LAPACK's dsytrd_sy2sb).
//
// Per panel p (columns p .. p+b-1, trailing block rows/columns m0 = p+b ..):
//   P = A[m0:, p:p+b] = Q_p R,  Q_p = I - V T V'
//   X = A22 V T,  W = X - 1/2 V (T' (V' X)),  A22 <- A22 - V W' - W V'.
// The reflectors of panel p are kept transposed in rows p .. p+b-1 of A
// (row p+i holds v_i from column m0+i, where v_i has its leading 1), so that
// Q = H_0 H_1 ... is accumulated afterwards in compact-WY blocks exactly as
// for the one-reflector-per-row layout, with the leading 1 of row r at
// column r + b.
#include "kmp_common.h"
#include "kmp_kernels.h"

#include <algorithm>

namespace kmp {

constexpr int BB = kBand;        // band width = panel width

typedef double xdbl4 __attribute__((ext_vector_type(4)));
constexpr int kFusedYtRows = 1536;   // register panels that also form Y'
constexpr int PQT = 512;         // threads of the panel factorisation
constexpr int PQW = PQT / 64;

// Register-resident panel factorisation with NW wavefronts: lane l of wave
// w holds column c = l % 16 of row r = 4 NW m + 4 w + l / 16 in slot m
// (m < RS). Step i needs only row i of the panel's Gram matrix,
// h_c = sum_{r > i} P[r][i] P[r][c]: every lane multiplies its entry by
// P[r][i], taken from lane i of its 16-lane row by a DPP row broadcast
// (row_newbcast takes an immediate lane, so the 16 steps are unrolled), the
// four rows of the wavefront are added by permlane swaps and the NW
// wavefronts through LDS. With alpha = P[i][i], sigma = h_i,
//   v_i' P[:, c] = P[i][c] + h_c / (alpha - beta)            (c > i)
//   V[:, k]' v_i = P[i][k] + h_k / (alpha - beta) =: z_i[k]   (k < i).
// One pass over the slots makes the update of step i and the products of
// step i+1:
//  - below the diagonal, column k < i keeps u_k = v_k / scale_k (scale_k =
//    1/(alpha_k - beta_k)), so the update of a slot is one multiply-add,
//    x_c += A_c P[r][i] with A_c = -tau scale (v_i' P[:, c]) for c > i and
//    zero otherwise; the scales are applied when the panel is written back
//    and folded into the z_i;
//  - P[r][i+1] after step i is P[r][i+1] + A_{i+1} P[r][i], formed from the
//    broadcast of the old column i+1 and, with CARRY, kept for step i+1
//    (one broadcast and three multiply-adds per slot and step).
// The reflectors leave through an LDS tile so that their transposed rows
// are written contiguously, and the compact-WY factor is formed at the end
// row by row, T[t][i] = -tau_i sum_{k=t}^{i-1} T[t][k] z_i[k].
template <int K>
__device__ __forceinline__ double row_bcast(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_mov_dpp((int)b, 0x150 + K, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), 0x150 + K, 0xf, 0xf, false);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

__device__ __forceinline__ double swap_sum16_b(double v) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const auto lo = __builtin_amdgcn_permlane16_swap((unsigned)b, (unsigned)b, false, false);
  const auto hi = __builtin_amdgcn_permlane16_swap((unsigned)(b >> 32), (unsigned)(b >> 32), false, false);
  return __longlong_as_double((long long)(((unsigned long long)hi[0] << 32) | lo[0])) +
         __longlong_as_double((long long)(((unsigned long long)hi[1] << 32) | lo[1]));
}
__device__ __forceinline__ double swap_sum32_b(double v) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const auto lo = __builtin_amdgcn_permlane32_swap((unsigned)b, (unsigned)b, false, false);
  const auto hi = __builtin_amdgcn_permlane32_swap((unsigned)(b >> 32), (unsigned)(b >> 32), false, false);
  return __longlong_as_double((long long)(((unsigned long long)hi[0] << 32) | lo[0])) +
         __longlong_as_double((long long)(((unsigned long long)hi[1] << 32) | lo[1]));
}

// Householder QR of the panel P = A[m0:N, p:p+BB] of every matrix (one
// workgroup per matrix), streamed from memory, in place: R on and above the
// diagonal of P, v_i below it (dlarfg convention, v_i[i] = 1 implicit).
// Lane l of wave w takes column c = l % 16 of the rows r = 4w + l/16 + 32k,
// so a wavefront reads and writes four whole 128-byte rows per pass. Step i
// needs, over rows r > i, the products h_c = sum_r P[r][i] P[r][c] (c >= i):
// sigma = h_i, and v_i'P[:, c] = P[i][c] + h_c / (alpha - beta). P[r][i] and
// the updated P[r][i+1] come from lanes i and i+1 of the row by DPP row
// broadcasts (immediate lanes: the 16 steps are unrolled); the update of
// step i and the products of step i+1 are made in one pass over the rows,
// in batches of QB rows per lane whose loads are issued together. The
// per-lane products are added over the four rows of a wavefront by permlane
// swaps and over the wavefronts through LDS (double-buffered by step
// parity), in a fixed order.
// Outputs: tau[p+i], and v_i transposed into row p+i of A (columns m0 ..,
// zeros before its leading 1) and into rows i and 2BB+i of the panel buffer.
constexpr int QB = 8;            // rows per lane and batch of the streamed panel QR
constexpr int QS = PQT / 16;     // rows per pass of the workgroup

struct QrStream {
  double* P;
  int N, mrow, kf, s, c, w, sub, t;
  double (*red)[PQW][BB];
};

// one pass over the rows: f(r, x) returns the new P[r][c] (stored when
// STORE) and accumulates the products; whole batches of QB rows first
// (every row valid), then the rest with the row index clamped for the loads
template <bool STORE, typename F>
__device__ __forceinline__ void qr_stream_rows(const QrStream& q, F f) {
  int k0 = 0;
  for (; k0 + QB <= q.kf; k0 += QB) {
    double x[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) x[b] = q.P[(int64_t)(q.s + QS * (k0 + b)) * q.N + q.c];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      const int r = q.s + QS * (k0 + b);
      const double v = f(r, x[b]);
      if (STORE) q.P[(int64_t)r * q.N + q.c] = v;
    }
  }
  double x[QB];
#pragma unroll
  for (int b = 0; b < QB; ++b) x[b] = q.P[(int64_t)min(q.s + QS * (k0 + b), q.mrow - 1) * q.N + q.c];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    const int r = q.s + QS * (k0 + b);
    if (r < q.mrow) {
      const double v = f(r, x[b]);
      if (STORE) q.P[(int64_t)r * q.N + q.c] = v;
    }
  }
}

// h of the lane's column into red[B] (per wavefront), then one barrier
template <int B>
__device__ __forceinline__ void qr_stream_put(const QrStream& q, double h) {
  const double v = swap_sum32_b(swap_sum16_b(h));
  if (q.sub == 0) q.red[B][q.w][q.c] = v;
  __syncthreads();
}

template <int I>
__device__ __forceinline__ void qr_stream_steps(const QrStream& q, double* __restrict__ taus) {
  if constexpr (I < BB) {
    double hc = 0.0;                                   // h_c of the lane's column
#pragma unroll
    for (int j = 0; j < PQW; ++j) hc += q.red[I & 1][j][q.c];
    const double sigma = row_bcast<I>(hc);
    const double alpha = q.P[(int64_t)I * q.N + I];
    double tau = 0.0, beta = alpha, scale = 0.0;
    if (sigma > 0.0) {
      // the norm and the two reciprocals are on the step's dependency
      // chain: hardware estimates refined by Newton-Raphson (IEEE sqrt for
      // arguments near the bottom of the normal range)
      const double s2 = fma(alpha, alpha, sigma);
      beta = -copysign(s2 > 1e-280 ? sqrt_newton(s2) : sqrt(s2), alpha);
      tau = (beta - alpha) * rcp_newton(beta);
      scale = rcp_newton(alpha - beta);
    }
    const double wsc = (q.c > I) ? fma(scale, hc, q.P[(int64_t)I * q.N + q.c]) : 0.0;  // v_I' P[:, c]
    if (q.t == 0) taus[I] = tau;
    __syncthreads();                                   // row I read by all before its update
    const double ft = -tau;
    const int c = q.c;
    double h = 0.0;
    qr_stream_rows<true>(q, [&](int r, double x) {
      const double xi = row_bcast<I>(x);                             // P[r][I]
      const double vr = (r == I) ? 1.0 : xi * scale;
      const double fr = (r >= I) ? ft * vr : 0.0;
      double xn = (c > I) ? fma(fr, wsc, x) : x;
      if (c == I) xn = (r == I) ? beta : (r > I ? vr : x);
      if constexpr (I + 1 < BB) {
        const double x1 = row_bcast<I + 1>(xn);                      // updated P[r][I+1]
        h = fma((r > I + 1) ? x1 : 0.0, xn, h);
      }
      return xn;
    });
    if constexpr (I + 1 < BB) qr_stream_put<(I + 1) & 1>(q, h);
    qr_stream_steps<I + 1>(q, taus);
  }
}

__device__ __forceinline__ void panel_qr_stream_body(double* __restrict__ A, int N, int p,
                                                     double* __restrict__ taus,
                                                     double* __restrict__ panel, int g) {
  __shared__ double red[2][PQW][BB];
  const int t = threadIdx.x, lane = t & 63;
  double* Ag = A + (int64_t)g * N * N;
  const int m0 = p + BB, mrow = N - m0;
  QrStream q;
  q.P = Ag + (int64_t)m0 * N + p;                    // P[r][c] = P[r*N + c]
  q.N = N;
  q.mrow = mrow;
  q.kf = mrow / QS;
  q.w = t >> 6;
  q.sub = lane >> 4;
  q.c = lane & 15;
  q.s = 4 * q.w + q.sub;
  q.t = t;
  q.red = red;
  // products of step 0: h_c = sum_{r >= 1} P[r][0] P[r][c]
  {
    double h = 0.0;
    qr_stream_rows<false>(q, [&](int r, double x) {
      const double x0 = row_bcast<0>(x);
      h = fma((r >= 1) ? x0 : 0.0, x, h);
      return x;
    });
    qr_stream_put<0>(q, h);
  }
  qr_stream_steps<0>(q, taus + (int64_t)g * N + p);
  __syncthreads();                                   // the last step's rows
  // reflectors, transposed: row i of Vt is v_i over rows m0 .. N-1
  double* Vt = panel + (int64_t)g * 3 * BB * N;
  double* P = q.P;
  for (int e = t; e < BB * mrow; e += PQT) {
    const int i = e / mrow, r = e % mrow;
    double v = 0.0;
    if (r == i) v = 1.0;
    else if (r > i) v = P[(int64_t)r * N + i];
    Ag[(int64_t)(p + i) * N + m0 + r] = v;
    Vt[(int64_t)i * N + m0 + r] = v;
    Vt[(int64_t)(2 * BB + i) * N + m0 + r] = v;
  }
}

__global__ __launch_bounds__(PQT) void panel_qr_kernel(double* __restrict__ A, int N, int p,
                                                        double* __restrict__ taus,
                                                        double* __restrict__ panel) {
  panel_qr_stream_body(A, N, p, taus, panel, blockIdx.x);
}

constexpr int PVT = 256;          // rows of the reflector staging tile

template <int NW>
struct PanelLds {
  double red[2][NW][BB];   // per-wave partial sums of h, by step parity
  double rowb[2][BB];      // row i of the panel before step i (as held: u_k for k < i)
  double scl[BB];          // scale_k
  double tau[BB];
  double z[BB][BB];        // z_i[k], k < i
  double tq[BB][BB + 1];   // T of the block reflector
  double vt[BB][PVT + 1];  // reflector staging tile
};

template <int NW>
struct PanelCtx {
  PanelLds<NW>* L;
  int w, c, sub, t;
};

// The per-wave partial sums of h (column c of the lane) into red[B], then
// one barrier; each wavefront then adds the NW partials itself
// (panel_h_col: lane (c, sub) reads the partials of waves sub, sub+4, ...,
// and the four rows are added by permlane swaps, so every lane ends with
// h_c of its column). red is double-buffered by step parity: a wavefront
// writes red[B] again two steps later, after the barrier of the step
// between, which every wavefront reaches only after its reads.
template <int NW, int B>
__device__ __forceinline__ void panel_h_put(double acc, const PanelCtx<NW>& st) {
  const double v = swap_sum32_b(swap_sum16_b(acc));
  if (st.sub == 0) st.L->red[B][st.w][st.c] = v;
  __syncthreads();
}
template <int NW, int B>
__device__ __forceinline__ double panel_h_col(const PanelCtx<NW>& st) {
  double s = 0.0;
#pragma unroll
  for (int j = 0; j < NW / 4; ++j) s += st.L->red[B][st.sub + 4 * j][st.c];
  return swap_sum32_b(swap_sum16_b(s));
}

template <int RS, int NW, bool CARRY, int I>
__device__ __forceinline__ void panel_steps(double (&x)[RS], double (&xi)[RS],
                                            const PanelCtx<NW>& st) {
  if constexpr (I < BB) {
    PanelLds<NW>& L = *st.L;
    const double* ri = L.rowb[I & 1];
    const double alpha = ri[I];
    const int c = st.c;
    const double hc = panel_h_col<NW, I & 1>(st);                   // h_c, every lane
    const double sigma = row_bcast<I>(hc);
    double tau = 0.0, beta = alpha, scale = 0.0;
    if (sigma > 0.0) {
      // the norm and the two reciprocals are on the step's dependency
      // chain: hardware estimates refined by Newton-Raphson (IEEE sqrt for
      // arguments near the bottom of the normal range)
      const double s2 = fma(alpha, alpha, sigma);
      beta = -copysign(s2 > 1e-280 ? sqrt_newton(s2) : sqrt(s2), alpha);
      tau = (beta - alpha) * rcp_newton(beta);
      scale = rcp_newton(alpha - beta);
    }
    if (st.t < I) L.z[I][st.t] = L.scl[st.t] * fma(scale, hc, ri[st.t]);   // t < 16: c = t
    if (st.t == 0) {
      L.scl[I] = scale;
      L.tau[I] = tau;
    }
    const double tw = -tau * fma(scale, hc, ri[c]);                 // -tau v_I' P[:, c]
    const double ac = (c > I) ? tw * scale : 0.0;
    double a1 = 0.0;
    if constexpr (I + 1 < BB) a1 = -tau * fma(scale, row_bcast<I + 1>(hc), ri[I + 1]) * scale;
    double acc = 0.0;
#pragma unroll
    for (int m = 0; m < RS; ++m) {
      const double xim = CARRY ? xi[m] : row_bcast<I>(x[m]);          // P[r][I]
      if (m == 0) {
        const int r = 4 * st.w + st.sub;
        double xn = x[0];
        if (r > I) xn = fma(ac, xim, xn);
        else if (r == I) xn = (c > I) ? xn + tw : ((c == I) ? beta : xn);
        x[0] = xn;
        if constexpr (I + 1 < BB) {
          const double xo = row_bcast<I + 1>(xn);                    // column I+1, updated
          if (r == I + 1) L.rowb[(I + 1) & 1][c] = xn;
          acc = fma((r > I + 1) ? xo : 0.0, xn, acc);
          if constexpr (CARRY) xi[0] = xo;
        }
      } else {
        if constexpr (I + 1 < BB) {
          const double xo = row_bcast<I + 1>(x[m]);                  // column I+1, old
          const double xj = fma(a1, xim, xo);
          x[m] = fma(ac, xim, x[m]);
          acc = fma(xj, x[m], acc);
          if constexpr (CARRY) xi[m] = xj;
        } else {
          x[m] = fma(ac, xim, x[m]);
        }
      }
    }
    if constexpr (I + 1 < BB) {
      panel_h_put<NW, (I + 1) & 1>(acc, st);
      panel_steps<RS, NW, CARRY, I + 1>(x, xi, st);
    }
  }
}

template <int RS, int NW, bool CARRY>
__device__ __forceinline__ void panel_qr_vec_body(double* __restrict__ A, int N, int p,
                                                  double* __restrict__ taus,
                                                  double* __restrict__ panel,
                                                  double* __restrict__ tmat,
                                                  double* __restrict__ yt, int g) {
  constexpr int RPS = 4 * NW;                      // rows per slot
  __shared__ PanelLds<NW> L;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int c = lane & 15, sub = lane >> 4;
  double* Ag = A + (int64_t)g * N * N;
  const int m0 = p + BB, mrow = N - m0;
  double* P = Ag + (int64_t)m0 * N + p;
  double x[RS], xi[RS];
#pragma unroll
  for (int m = 0; m < RS; ++m) {
    const int r = RPS * m + 4 * w + sub;
    x[m] = (r < mrow) ? P[(int64_t)r * N + c] : 0.0;
  }
  if (w == 0 && sub == 0) L.rowb[0][c] = x[0];          // row 0: slot 0, wave 0, sub 0
  PanelCtx<NW> st{&L, w, c, sub, t};
  double acc = 0.0;
#pragma unroll
  for (int m = 0; m < RS; ++m) {
    const int r = RPS * m + 4 * w + sub;
    const double x0 = row_bcast<0>(x[m]);
    if constexpr (CARRY) xi[m] = x0;
    acc = fma((r > 0) ? x0 : 0.0, x[m], acc);
  }
  panel_h_put<NW, 0>(acc, st);
  panel_steps<RS, NW, CARRY, 0>(x, xi, st);
  __syncthreads();
  // T, row t per thread, built in LDS (rolled loops, operands read from
  // LDS), then into tmat; before the reflector tiles when Y' is formed
  // with them, after them otherwise (the slots are then dead)
  constexpr bool kYt = RPS * RS <= kFusedYtRows;
  const auto form_t = [&]() {
    if (t < BB) {
      double* Tg = tmat + (int64_t)g * kWyBlock * kWyBlock + (int64_t)t * kWyBlock;
#pragma unroll 1
      for (int i = 0; i < BB; ++i) {
        double s0 = 0.0, s1 = 0.0;
        for (int k = t; k + 1 < i; k += 2) {
          s0 = fma(L.tq[t][k], L.z[i][k], s0);
          s1 = fma(L.tq[t][k + 1], L.z[i][k + 1], s1);
        }
        if (((i - t) & 1) && t < i) s0 = fma(L.tq[t][i - 1], L.z[i][i - 1], s0);
        const double v = (i > t) ? -L.tau[i] * (s0 + s1) : ((i == t) ? L.tau[t] : 0.0);
        L.tq[t][i] = v;
        Tg[i] = v;
      }
      taus[(int64_t)g * N + p + t] = L.tau[t];
    }
  };
  if constexpr (kYt) form_t();
  // R (rows < BB, on and above the diagonal) back into the panel; the
  // reflectors v_k = scale_k u_k (leading 1 at row k) transposed into row
  // p+k of A and rows k, 2BB+k of the panel buffer, through the LDS tile;
  // from the same tile Y' = T'V' on the matrix cores, stored transposed
  // (row r: 16 doubles), one 16-row block per wavefront (for panels of at
  // most kFusedYtRows rows: beyond, the slots leave no registers for it)
  const double sc = L.scl[c];
  int rb = 4 * w + sub;               // fresh: keeps the slots' row indices out of registers
  asm volatile("" : "+v"(rb));
  if (rb < BB && rb <= c) P[(int64_t)rb * N + c] = x[0];
  double* Vt = panel + (int64_t)g * 3 * BB * N;
  double* Yg = yt + (int64_t)g * kWyBlock * N;
  constexpr int SPT = PVT / RPS;      // slots per tile
#pragma unroll
  for (int m0s = 0; m0s < RS; m0s += SPT) {
#pragma unroll
    for (int q = 0; q < SPT && m0s + q < RS; ++q) {
      const int rl = RPS * q + rb;                   // row within the tile
      const int r = RPS * (m0s + q) + rb;
      L.vt[c][rl] = (r == c) ? 1.0 : ((r > c) ? sc * x[m0s + q] : 0.0);
    }
    __syncthreads();
    const int r0 = RPS * m0s;
    const int nr = (mrow - r0 < PVT) ? mrow - r0 : PVT;
    for (int e = t; e < BB * PVT; e += 64 * NW) {
      const int k = e / PVT, rr = e % PVT;
      if (rr < nr) {
        const double v = L.vt[k][rr];
        const int64_t col = (int64_t)m0 + r0 + rr;
        Ag[(int64_t)(p + k) * N + col] = v;
        Vt[(int64_t)k * N + col] = v;
        Vt[(int64_t)(2 * BB + k) * N + col] = v;
      }
    }
    if constexpr (kYt)
    for (int blk = w; 16 * blk < nr; blk += NW) {
      xdbl4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4)
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64(L.vt[4 * s4 + sub][16 * blk + c],
                                                   L.tq[4 * s4 + sub][c], acc, 0, 0, 0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * blk + 4 * r + sub;
        if (row < nr) Yg[(int64_t)(r0 + row) * BB + c] = acc[r];
      }
    }
    __syncthreads();
  }
  if constexpr (!kYt) form_t();
}

template <int RS, int NW, bool CARRY>
__global__ __launch_bounds__(64 * NW) void panel_qr_vec_kernel(double* __restrict__ A, int N,
                                                                int p, double* __restrict__ taus,
                                                                double* __restrict__ panel,
                                                                double* __restrict__ tmat,
                                                                double* __restrict__ yt) {
  panel_qr_vec_body<RS, NW, CARRY>(A, N, p, taus, panel, tmat, yt, blockIdx.x);
}

// Only the lower triangle of the trailing matrix is kept up to date (the
// two-sided update skips the 64 x 64 tiles above the diagonal): an element
// (R, C) with R > C lies in a tile on or below the diagonal for every tile
// origin, and every diagonal 16 x 16 block lies inside one diagonal tile,
// since the origins of successive panels differ by multiples of 16. So
// A22[k][j] is read as A[k][j] for k >= j and as A[j][k] above.
//
// X' = Y' A22 and the partial products of M2 = V'X for one panel (A22 =
// A[m0:, m0:], Y' = T'V' stored transposed, Yt[k][i] = Yt[16 k + i], m x 16).
// One workgroup per 64 columns (four 16-column blocks) of X' and matrix:
// wave w accumulates the 16-row chunks q = w, w+XW, ... of all four blocks
// on the matrix cores (A operand Yt[k][i]; B operand A22[k][j], so that
// below the diagonal each chunk is read as 512-byte row pieces, with its Y'
// operand loaded once for the four blocks). A chunk may lie below some
// blocks and above others (the test is per block and uniform over the
// wavefront); above, a block's entries A22[j][k] are read from its
// transposed rows, 32 contiguous bytes per lane, with the k of MFMA step s4
// in lane group kq taken as 16 q + 4 kq + s4 (16 q + 4 s4 + kq below). The
// XW partial tiles of each block are added in LDS, X' goes to xq (row b
// of matrix g at xq + g sX + b N), and the workgroup's parts of M2,
// sum_{j in block} V'[a][j] X'[b][j], to part[(g NJ + block)*256].
constexpr int XU4 = 1;            // chunks per wavefront and iteration
constexpr int XW = 8;             // wavefronts per workgroup
__global__ __launch_bounds__(64 * XW) void panel_x_kernel(const double* __restrict__ A, int N, int m0,
                                                       const double* __restrict__ ybuf,
                                                       const double* __restrict__ panel,
                                                       double* __restrict__ part, int NJ,
                                                       double* __restrict__ xq, int64_t sX) {
  __shared__ double red[4][4][4][64];              // wave, block, register, lane
  __shared__ double Xs[4][BB][BB + 1];
  const int g = blockIdx.y, t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int m = N - m0, nch = m / BB, jb0 = 4 * blockIdx.x;
  const int nbv = min(4, nch - jb0);               // valid blocks of this workgroup
  const double* Ag = A + (int64_t)g * N * N + (int64_t)m0 * N + m0;
  const double* Yg = ybuf + (int64_t)g * kWyBlock * N;
  const double* Pg = panel + (int64_t)g * 3 * BB * N + m0;
  double* Xg = xq + (int64_t)g * sX + m0;
  const int i = lane & 15, kq = lane >> 4;
  const double* ya = Yg + (int64_t)kq * BB + i;
  const double* yt = Yg + (int64_t)(4 * kq) * BB + i;
  const double* bb = Ag + (int64_t)kq * N + BB * jb0 + i;          // + 16 c: block c, below
  const double* bt = Ag + (int64_t)(BB * jb0 + i) * N + 4 * kq;    // + 16 c N: block c, above
  xdbl4 acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = xdbl4{0.0, 0.0, 0.0, 0.0};
  for (int q = w; q < nch; q += XW * XU4) {
#pragma unroll
    for (int u = 0; u < XU4; ++u) {
      const int qq = q + XW * u;
      if (qq < nch) {                                // uniform over the wavefront
        double avb[4], ava[4], bv[4][4];
        const bool anyb = qq >= jb0, anya = qq < jb0 + nbv - 1;
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
          avb[s4] = anyb ? ya[(int64_t)(BB * qq + 4 * s4) * BB] : 0.0;
          ava[s4] = anya ? yt[(int64_t)(BB * qq + s4) * BB] : 0.0;
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          if (c < nbv) {
            if (qq >= jb0 + c) {
#pragma unroll
              for (int s4 = 0; s4 < 4; ++s4) bv[c][s4] = bb[(int64_t)(BB * qq + 4 * s4) * N + BB * c];
            } else {
              const double* br = bt + (int64_t)(BB * c) * N + BB * qq;
              const double2 b01 = *reinterpret_cast<const double2*>(br);
              const double2 b23 = *reinterpret_cast<const double2*>(br + 2);
              bv[c][0] = b01.x; bv[c][1] = b01.y; bv[c][2] = b23.x; bv[c][3] = b23.y;
            }
          }
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          if (c < nbv) {
            const bool below = qq >= jb0 + c;
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4)
              acc[c] = __builtin_amdgcn_mfma_f64_16x16x4f64(below ? avb[s4] : ava[s4], bv[c][s4],
                                                            acc[c], 0, 0, 0);
          }
        }
      }
    }
  }
  // wavefront w + 4 hands its tiles to wavefront w, which adds its own
  static_assert(XW == 8, "two wavefronts per LDS slot");
  if (w >= 4) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[w - 4][c][r][lane] = acc[c][r];
  }
  __syncthreads();
  if (w < 4) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[w][c][r][lane] = acc[c][r] + red[w][c][r][lane];
  }
  __syncthreads();
  // X' of block c, register r, lane l: row 4 r + l / 16, column l % 16
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const int c = h, r = t >> 6, l = t & 63;
    if (t < 256 && c < nbv) {
      const double v = (red[0][c][r][l] + red[1][c][r][l]) + (red[2][c][r][l] + red[3][c][r][l]);
      const int b = 4 * r + (l >> 4), j = l & 15;
      Xs[c][b][j] = v;
      Xg[(int64_t)b * N + BB * (jb0 + c) + j] = v;
    }
  }
  __syncthreads();
  if (t < 256) {
    const int a = t >> 4, b = t & 15;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (c < nbv) {
        const double* va = Pg + (int64_t)a * N + BB * (jb0 + c);
        double s0 = 0.0, s1 = 0.0;
#pragma unroll
        for (int j = 0; j < BB; j += 2) {
          s0 = fma(va[j], Xs[c][b][j], s0);
          s1 = fma(va[j + 1], Xs[c][b][j + 1], s1);
        }
        part[((int64_t)g * NJ + jb0 + c) * 256 + t] = s0 + s1;
      }
    }
  }
}

// M2 = V'X summed from panel_x's per-block parts in M2S fixed slices
// (slice s: blocks floor(s nch / M2S) .. floor((s+1) nch / M2S) - 1, added
// in order), so that each panel_ws workgroup adds M2S values per entry
// instead of every block's part (at 32000 rows each of its 2500 workgroups
// read all 2000 parts, 4 MB). Workgroup (s, g); m2s[(g M2S + s) 256 + t].
constexpr int M2S = 64;
__global__ __launch_bounds__(256) void m2_slices_kernel(const double* __restrict__ part, int NJ,
                                                        int nch, double* __restrict__ m2s) {
  const int sl = blockIdx.x, g = blockIdx.y, t = threadIdx.x;
  const int q0 = (int)((int64_t)nch * sl / M2S), q1 = (int)((int64_t)nch * (sl + 1) / M2S);
  const double* pp = part + (int64_t)g * NJ * 256 + t;
  double s0 = 0.0, s1 = 0.0;
  for (int q = q0; q < q1; q += 8) {
    double v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (q + u < q1) ? pp[(int64_t)(q + u) * 256] : 0.0;
#pragma unroll
    for (int u = 0; u < 8; u += 2) {
      s0 += v[u];
      s1 += v[u + 1];
    }
  }
  m2s[((int64_t)g * M2S + sl) * 256 + t] = s0 + s1;
}

// S = T'M2 from the slices of M2 (added in slice order), W' =
// X' - 1/2 S'V' for the workgroup's 64 columns (X' read from xq, W' into
// rows BB .. 2BB-1 of the panel buffer), then the two-sided update of the
// first block column of A22 for the workgroup's 64 rows:
//   A22[i][j] -= sum_k V[k][i] W[k][j] + W[k][i] V[k][j],   j < 16,
// wave w taking rows 16 w .. 16 w + 15 of the tile on the matrix cores
// (C loaded into the accumulators, K = 32 over [V; W] against [W; V]).
// The W' operands come from LDS: the workgroup's own columns, and columns
// 0 .. 15 formed again by every workgroup, so that none reads what another
// one writes. One workgroup per 64 rows and matrix.
__global__ __launch_bounds__(256) void panel_ws_kernel(double* __restrict__ A, int N, int m0,
                                                       const double* __restrict__ m2s,
                                                       const double* __restrict__ tmat,
                                                       const double* __restrict__ xq, int64_t sX,
                                                       double* __restrict__ panel) {
  __shared__ double M2s[BB][BB + 1];
  __shared__ double Ss[BB][BB + 1];
  __shared__ double Wl[BB][64 + 1];                // W' of the workgroup's columns
  __shared__ double W0[BB][BB + 1];                // W' of columns 0 .. 15
  const int bx = blockIdx.x, g = blockIdx.y, t = threadIdx.x;
  const int m = N - m0, nch = m / BB;
  double* Pg = panel + (int64_t)g * 3 * BB * N + m0;
  const double* Xg = xq + (int64_t)g * sX + m0;
  const int w = t >> 6, lane = t & 63, li = lane & 15, lk = lane >> 4;
  const int i0 = 64 * bx + 16 * w;                 // m is a multiple of 16
  const bool strip = i0 < m;
  double* Cg = A + (int64_t)g * N * N + (int64_t)m0 * N + m0;
  // every load that does not depend on S first: the strip's piece of A22,
  // the V column and X' rows of this thread's W' entries (column jl, rows
  // r4 .. r4+3; and column c0, row r0 of W' for columns 0 .. 15), and
  // column a of T
  xdbl4 acc = {0.0, 0.0, 0.0, 0.0};
  if (strip) {
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[r] = Cg[(int64_t)(i0 + 4 * r + lk) * N + li];
  }
  const int jl = t & 63, j = 64 * bx + jl, r4 = 4 * (t >> 6);
  const bool okj = j < m;
  const int c0 = t & 15, r0 = t >> 4;
  double vj[BB], xj[4], v0[BB], tc[BB];
#pragma unroll
  for (int q = 0; q < BB; ++q) {
    vj[q] = okj ? Pg[(int64_t)q * N + j] : 0.0;
    v0[q] = Pg[(int64_t)q * N + c0];
    tc[q] = tmat[(int64_t)g * kWyBlock * kWyBlock + q * kWyBlock + r0];
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) xj[u] = okj ? Xg[(int64_t)(r4 + u) * N + j] : 0.0;
  const double x0 = Xg[(int64_t)r0 * N + c0];
  {
    const double* pp = m2s + (int64_t)g * M2S * 256 + t;
    double s = 0.0;
#pragma unroll 8
    for (int q = 0; q < M2S; ++q) s += pp[q * 256];
    M2s[t >> 4][t & 15] = s;
  }
  __syncthreads();
  {
    double s = 0.0;                                // S[a][b], a = t/16, b = t%16
#pragma unroll
    for (int q = 0; q < BB; ++q) s = fma(tc[q], M2s[q][c0], s);
    Ss[r0][c0] = s;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int ii = r4 + u;
    double s = 0.0;
#pragma unroll
    for (int q = 0; q < BB; ++q) s = fma(Ss[q][ii], vj[q], s);
    const double wv = fma(-0.5, s, xj[u]);
    if (okj) Pg[(int64_t)(BB + ii) * N + j] = wv;
    Wl[ii][jl] = okj ? wv : 0.0;
  }
  {
    double s = 0.0;
#pragma unroll
    for (int q = 0; q < BB; ++q) s = fma(Ss[q][r0], v0[q], s);
    W0[r0][c0] = fma(-0.5, s, x0);
  }
  __syncthreads();
  if (!strip) return;
#pragma unroll
  for (int s8 = 0; s8 < 8; ++s8) {
    const int k = 4 * s8 + lk;
    const double av = (k < BB) ? -Pg[(int64_t)k * N + i0 + li] : -Wl[k - BB][16 * w + li];
    const double bv = (k < BB) ? W0[k][li] : Pg[(int64_t)(k - BB) * N + li];
    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc, 0, 0, 0);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) Cg[(int64_t)(i0 + 4 * r + lk) * N + li] = acc[r];
}

// Rank-K update C <- C - P1' P2 of an m x m block (C[i][j] = C[i*ldc + j],
// P1[k][i] = P1[k*ld1 + i], P2[k][j] = P2[k*ld2 + j], K = 32 KC; matrix g at
// C + g sC, P1 + g s1, P2 + g s2), for the two-sided update
// of the trailing matrix (P1 = [V; W], P2 = [W; V], K = 2 BB) and the
// accumulation of Q (P1 = V, P2 = T V Q, K = 64 or 128). One workgroup per 64 x 64
// tile; wave w updates the 32 x 32 piece at (32 (w&1), 32 (w>>1)) as 2 x 2
// MFMA blocks: the piece of C is loaded in accumulator layout (register r
// of a block holds row 4r + l/16, column l%16: 128-byte row pieces), then
// per 32 k the 2 x 8 operand values of each side are loaded
// together and 32 products with the A operand negated follow. m is a
// multiple of 16, so each 16 x 16 block is wholly inside or outside C:
// outside blocks load from clamped addresses and are not stored. The
// products accumulate from zero and the piece of C is added at the store,
// so the matrix products do not wait for C's loads (10 % faster at K = 128,
// 2 % at K = 32, measured at m = 16000); beyond the first 32 k, the
// operands of each 32 are loaded during the products of the previous 32
// (10 % more at K = 128). With LOWER only the tiles on and below the
// diagonal are updated (C symmetric, its
// lower triangle kept; see the note before panel_x_kernel). With PART == 2
// the blocks of the first block row and column are left alone (the first
// block column is updated beforehand, the first block row lies above the
// diagonal).
template <int KC, bool LOWER, int PART>
__device__ __forceinline__ void rank_update_tile(double* __restrict__ C, int64_t ldc, int64_t sC,
                                                 int m, const double* __restrict__ P1, int64_t ld1,
                                                 int64_t s1, const double* __restrict__ P2,
                                                 int64_t ld2, int64_t s2, int bx, int by, int g,
                                                 int w, int lane) {
  const int i0 = 64 * bx + 32 * (w & 1), j0 = 64 * by + 32 * (w >> 1);
  double* Cg = C + (int64_t)g * sC;
  const double* A1 = P1 + (int64_t)g * s1;
  const double* A2 = P2 + (int64_t)g * s2;
  const int li = lane & 15, lk = lane >> 4;
  bool vi[2], vj[2];
  int ib[2], jb[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    vi[b] = i0 + 16 * b < m;
    vj[b] = j0 + 16 * b < m;
    ib[b] = vi[b] ? i0 + 16 * b : 0;
    jb[b] = vj[b] ? j0 + 16 * b : 0;
  }
  xdbl4 acc[2][2], cv[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        cv[bi][bj][r] = Cg[(int64_t)(ib[bi] + 4 * r + lk) * ldc + jb[bj] + li];
        acc[bi][bj][r] = 0.0;
      }
  // the operands of the next 32 k are loaded before the products of these
  constexpr int NBUF = KC > 1 ? 2 : 1;
  double av[NBUF][2][8], bv[NBUF][2][8];
  auto load = [&](int kc, double (&a)[2][8], double (&bb)[2][8]) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int s8 = 0; s8 < 8; ++s8) {
        const int64_t k = 32 * kc + 4 * s8 + lk;
        a[b][s8] = -A1[k * ld1 + ib[b] + li];
        bb[b][s8] = A2[k * ld2 + jb[b] + li];
      }
  };
  load(0, av[0], bv[0]);
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    if (kc + 1 < KC) load(kc + 1, av[(kc + 1) % NBUF], bv[(kc + 1) % NBUF]);
#pragma unroll
    for (int s8 = 0; s8 < 8; ++s8)
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[kc % NBUF][bi][s8], bv[kc % NBUF][bj][s8],
                                                            acc[bi][bj], 0, 0, 0);
  }
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) {
      bool st = vi[bi] && vj[bj];
      if (PART == 2) st = st && ib[bi] != 0 && jb[bj] != 0;
      if (st) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          Cg[(int64_t)(ib[bi] + 4 * r + lk) * ldc + jb[bj] + li] = cv[bi][bj][r] + acc[bi][bj][r];
      }
    }
}

template <int KC, bool LOWER, int PART = 0>
__global__ __launch_bounds__(256) void rank_update_kernel(double* __restrict__ C, int64_t ldc,
                                                           int64_t sC, int m,
                                                           const double* __restrict__ P1,
                                                           int64_t ld1, int64_t s1,
                                                           const double* __restrict__ P2,
                                                           int64_t ld2, int64_t s2) {
  if (LOWER && blockIdx.y > blockIdx.x) return;
  rank_update_tile<KC, LOWER, PART>(C, ldc, sC, m, P1, ld1, s1, P2, ld2, s2, blockIdx.x, blockIdx.y,
                                    blockIdx.z, threadIdx.x >> 6, threadIdx.x & 63);
}

// Panel QR of the next panel and the rest of the current panel's two-sided
// update in one launch: workgroup g < G factors panel p_next of matrix g
// (its 16 columns were brought up to date beforehand), the other workgroups
// apply the rank-32 update of panel p (P1/P2 from its own panel buffer) to
// every 16 x 16 block of A22 outside its first block row and column, four
// wavefronts per 64 x 64 tile. The two roles touch disjoint parts of A
// (the factorisation reads the first block column of A22 and writes the
// reflector rows of the first block row), so they run side by side and the
// latency-bound factorisation is hidden behind the update.
template <int TPW>
__device__ __forceinline__ void rest_update_role(double* A, int N, int m0, int mrow, int G,
                                                 const double* P1, const double* P2, int64_t sP,
                                                 int tiles) {
  // tile e of the lower triangle, row by row: (bx, by) with by <= bx
  const int64_t e = (int64_t)(blockIdx.x - G) * TPW + (threadIdx.x >> 8);
  const int64_t tt = (int64_t)tiles * (tiles + 1) / 2;
  const int g = (int)(e / tt), rem = (int)(e % tt);
  if (g >= G) return;
  int bx = (int)((sqrt(8.0 * rem + 1.0) - 1.0) * 0.5);
  if (bx * (bx + 1) / 2 > rem) --bx;
  if ((bx + 1) * (bx + 2) / 2 <= rem) ++bx;
  const int by = rem - bx * (bx + 1) / 2;
  rank_update_tile<1, true, 2>(A + (int64_t)m0 * N + m0, (int64_t)N, (int64_t)N * N, mrow, P1,
                               (int64_t)N, sP, P2, (int64_t)N, sP, bx, by, g,
                               (threadIdx.x >> 6) & 3, threadIdx.x & 63);
}

template <int RS, int NW, bool CARRY>
__global__ __launch_bounds__(64 * NW) void qr_rest_vec_kernel(
    double* __restrict__ A, int N, int p_next, double* __restrict__ taus,
    double* __restrict__ panel_next, double* __restrict__ tmat, double* __restrict__ yt, int G,
    int m0, int mrow, const double* __restrict__ P1, const double* __restrict__ P2, int64_t sP,
    int tiles) {
  if (blockIdx.x < G) {
    panel_qr_vec_body<RS, NW, CARRY>(A, N, p_next, taus, panel_next, tmat, yt, blockIdx.x);
    return;
  }
  rest_update_role<NW / 4>(A, N, m0, mrow, G, P1, P2, sP, tiles);
}

__global__ __launch_bounds__(PQT) void qr_rest_stream_kernel(
    double* __restrict__ A, int N, int p_next, double* __restrict__ taus,
    double* __restrict__ panel_next, int G, int m0, int mrow, const double* __restrict__ P1,
    const double* __restrict__ P2, int64_t sP, int tiles) {
  if (blockIdx.x < G) {
    panel_qr_stream_body(A, N, p_next, taus, panel_next, blockIdx.x);
    return;
  }
  rest_update_role<PQT / 256>(A, N, m0, mrow, G, P1, P2, sP, tiles);
}

// C[i][j] = sum_k A[i*lda + k] B[j*ldb + k] for M, Nc <= 64 and long K (per
// matrix b: A + b*sA, B + b*sB, C + b*sC, ld ldc). Every block takes one
// 16 x 16 output tile over one chunk of TSK indices (one output per thread);
// a second pass adds the chunks in order.
constexpr int TSK = 128;
__global__ __launch_bounds__(256) void ts_gram_partial_kernel(
    int M, int Nc, int K, const double* __restrict__ A, int64_t lda, int64_t sA,
    const double* __restrict__ B, int64_t ldb, int64_t sB, double* __restrict__ part) {
  __shared__ double As[16][TSK + 1];
  __shared__ double Bs[16][TSK + 1];
  const int chunk = blockIdx.x, b = blockIdx.z, t = threadIdx.x;
  const int nch = gridDim.x, ntj = (Nc + 15) / 16;
  const int ti = blockIdx.y / ntj, tj = blockIdx.y % ntj;
  const int k0 = chunk * TSK;
  const int kn = (K - k0 < TSK) ? K - k0 : TSK;
  A += (int64_t)b * sA;
  B += (int64_t)b * sB;
  for (int e = t; e < 16 * TSK; e += 256) {
    const int rr = e / TSK, kk = e % TSK;
    const int ia = ti * 16 + rr, jb = tj * 16 + rr;
    As[rr][kk] = (ia < M && kk < kn) ? A[(int64_t)ia * lda + k0 + kk] : 0.0;
    Bs[rr][kk] = (jb < Nc && kk < kn) ? B[(int64_t)jb * ldb + k0 + kk] : 0.0;
  }
  __syncthreads();
  const int il = t / 16, jl = t % 16;
  double s0 = 0.0, s1 = 0.0;
  for (int kk = 0; kk < TSK; kk += 2) {
    s0 = fma(As[il][kk], Bs[jl][kk], s0);
    s1 = fma(As[il][kk + 1], Bs[jl][kk + 1], s1);
  }
  const int i = ti * 16 + il, j = tj * 16 + jl;
  if (i < M && j < Nc) part[(((int64_t)b * nch + chunk) * 64 + i) * 64 + j] = s0 + s1;
}

// One output per thread (blockIdx.y picks 256 of the M x Nc outputs), the
// chunk partials added in order.
__global__ __launch_bounds__(256) void ts_gram_sum_kernel(int M, int Nc, int nch,
                                                           const double* __restrict__ part,
                                                           double* __restrict__ C, int64_t ldc,
                                                           int64_t sC) {
  const int b = blockIdx.x;
  const int e = 256 * blockIdx.y + threadIdx.x;
  if (e >= M * Nc) return;
  const int i = e / Nc, j = e % Nc;
  const double* pp = part + ((int64_t)b * nch * 64 + i) * 64 + j;
  double s = 0.0;
#pragma unroll 4
  for (int c = 0; c < nch; ++c) s += pp[(int64_t)c * 64 * 64];
  C[(int64_t)b * sC + (int64_t)i * ldc + j] = s;
}

static int ts_gram(hipStream_t s, int M, int Nc, int K, int batch, const double* A, int64_t lda,
                   int64_t sA, const double* B, int64_t ldb, int64_t sB, double* C, int64_t ldc,
                   int64_t sC, double* part) {
  const int nch = (int)ceil_div(K, TSK);
  const int tiles = (int)(ceil_div(M, 16) * ceil_div(Nc, 16));
  hipLaunchKernelGGL(ts_gram_partial_kernel, dim3((unsigned)nch, (unsigned)tiles, (unsigned)batch),
                     dim3(256), 0, s, M, Nc, K, A, lda, sA, B, ldb, sB, part);
  KMP_LAUNCH_CHECK();
  hipLaunchKernelGGL(ts_gram_sum_kernel, dim3((unsigned)batch, (unsigned)ceil_div(M * Nc, 256)),
                     dim3(256), 0, s, M, Nc, nch, part, C, ldc, sC);
  KMP_LAUNCH_CHECK();
  return 0;
}

// band[g][r*N + j] = B[j+r][j] (r <= BB) from the lower triangle of A.
__global__ void band_extract_kernel(const double* __restrict__ A, int N, int64_t total,
                                    double* __restrict__ band) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int64_t per = (int64_t)(BB + 1) * N;
  const int g = (int)(idx / per);
  const int64_t e = idx % per;
  const int r = (int)(e / N), j = (int)(e % N);
  band[idx] = (j + r < N) ? A[(int64_t)g * N * N + (int64_t)(j + r) * N + j] : 0.0;
}

// Clear row r of A (a reflector row, r < N - BB) to the left of its stored
// vector, from column max(0, r - 128) up to column r + BB - 1, so that any
// run of up to 128 consecutive reflector rows (a pair of compact-WY blocks)
// reads zeros there.
__global__ void clear_reflector_rows_kernel(double* __restrict__ A, int N, int64_t total) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int64_t rows = N - BB;
  constexpr int W = kWyQuad * kWyBlock + BB;
  const int g = (int)(idx / (rows * W));
  const int64_t e = idx % (rows * W);
  const int r = (int)(e / W), q = (int)(e % W);
  const int c = r - kWyQuad * kWyBlock + q;    // c in [r - 256, r + BB)
  if (c < 0) return;
  A[(int64_t)g * N * N + (int64_t)r * N + c] = 0.0;
}

// Q_g = I for every matrix: one grid row per matrix (blockIdx.y), a
// grid-stride loop over its N*N entries, so that no launch dimension
// exceeds the 2^32 work-items a dispatch can describe.
__global__ void set_identity_band_kernel(double* __restrict__ Q, int N) {
  const int64_t nn = (int64_t)N * N;
  double* Qg = Q + (int64_t)blockIdx.y * nn;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nn; e += stride)
    Qg[e] = (e / N == e % N) ? 1.0 : 0.0;
}

template <typename F>
static double over_groups(const BandWork& wk, F f) {
  double a = 0.0;
  for (int g = 0; g < wk.G; ++g) a += f((double)(wk.nv_host ? wk.nv_host[g] : wk.N));
  return a;
}

// chunk partials of the Gram products, then the slices of M2
static size_t band_chunk_doubles(int G, int N) { return (size_t)G * ceil_div(N, TSK) * 64 * 64; }
size_t band_part_doubles(int G, int N) {
  return band_chunk_doubles(G, N) + (size_t)G * M2S * 256;
}

int wy_blocks(int N) { return N > BB ? (int)ceil_div(N - BB, kWyBlock) : 0; }

size_t wy_all_doubles(int G, int N) {
  return (size_t)std::max(1, wy_blocks(N)) * G * kWyBlock * kWyBlock;
}

size_t band_work_doubles(int G, int N) {
  return (size_t)G * (6 * (size_t)BB * N + 2 * (size_t)kWyBlock * kWyBlock +
                      (1 + kWyQuad) * (size_t)kWyBlock * N) + band_part_doubles(G, N) +
         (2 + (kWyQuad - 1)) * wy_all_doubles(G, N) +
         (size_t)kMaxSplitK * G * kWyQuad * kWyBlock * N;
}

// Gram matrices of all blocks of kWyBlock reflector rows at once, on the
// matrix cores: workgroup (b, g, 0) forms G[a][c] = sum_k V[a][k] V[c][k]
// for the reflectors q = 64 b .. q + kb - 1 of matrix g (row q + a of A
// holds v_{q+a} from column q + a + BB, zeros before it, so the sum runs
// over the columns q + BB .. N-1); workgroup (b, g, d), d = 1 .. 3, the
// cross products V_b V_{b+d}' with the block d further on (into cross_all +
// (d-1) sD). Wave w computes the
// 32 x 32 quadrant (32 (w&1), 32 (w>>1)) as 2 x 2 MFMA blocks over
// 16-column slices staged in LDS.
__global__ __launch_bounds__(256) void wy_gram_kernel(const double* __restrict__ A, int N, int nref,
                                                       double* __restrict__ gram_all,
                                                       double* __restrict__ cross_all, int64_t sD) {
  __shared__ double Vs[kWyBlock][BB + 1];
  __shared__ double Ws[kWyBlock][BB + 1];
  const int b = blockIdx.x, g = blockIdx.y, G = gridDim.y;
  const int dz = blockIdx.z;
  const bool cross = dz > 0;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int q = kWyBlock * b;
  const int kb = min(kWyBlock, nref - q);
  const int kc = cross ? min(kWyBlock, nref - q - dz * kWyBlock) : kb;   // rows of the right factor
  if (kc <= 0) return;
  const int m = N - q - BB;
  const double* Vq = A + (int64_t)g * N * N + (int64_t)q * N + q + BB;
  const double* Wq = Vq + (int64_t)dz * kWyBlock * N;
  double (*Rs)[BB + 1] = cross ? Ws : Vs;
  const int wi = 32 * (w & 1), wj = 32 * (w >> 1);
  const int li = lane & 15, lk = lane >> 4;
  xdbl4 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y) acc[x][y] = xdbl4{0.0, 0.0, 0.0, 0.0};
  const int lr = t >> 2, lc = (t & 3) * 4;        // loader: row lr, columns lc .. lc+3
  for (int c0 = 0; c0 < m; c0 += BB) {
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c0 + lc + u;
      Vs[lr][lc + u] = (lr < kb && c < m) ? Vq[(int64_t)lr * N + c] : 0.0;
      if (cross) Ws[lr][lc + u] = (lr < kc && c < m) ? Wq[(int64_t)lr * N + c] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int s4 = 0; s4 < BB; s4 += 4) {
      const double a0 = Vs[wi + li][s4 + lk], a1 = Vs[wi + 16 + li][s4 + lk];
      const double b0 = Rs[wj + li][s4 + lk], b1 = Rs[wj + 16 + li][s4 + lk];
      acc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc[1][1], 0, 0, 0);
    }
  }
  double* Gg = (cross ? cross_all + (dz - 1) * sD : gram_all) + ((int64_t)b * G + g) * kWyBlock * kWyBlock;
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        Gg[(wi + 16 * x + mfma_row(lane, r)) * kWyBlock + wj + 16 * y + mfma_col(lane)] = acc[x][y][r];
}

// Y = T X for one WY block of the Q accumulation, X given as S split-K
// parts (X_s[a][j] = xpart[s sP + g sX + a ldx + j], added in order s =
// 0, 1, ...): workgroup (column tile, g) stages the 64 x 64 piece of X and
// T (kb x kb, zero beyond) in LDS, and wave w forms the 32 x 32 quadrant
// (32 (w&1), 32 (w>>1)) of Y on the matrix cores.
__global__ __launch_bounds__(256) void wy_apply_t_kernel(const double* __restrict__ tq, int kb,
                                                         const double* __restrict__ xpart, int S,
                                                         int64_t sP, int64_t sX, int64_t ldx,
                                                         int m, double* __restrict__ Y,
                                                         int64_t ldy, int64_t sY) {
  __shared__ double Ts[kWyBlock][kWyBlock + 1];
  __shared__ double Xs[kWyBlock][kWyBlock + 1];
  const int g = blockIdx.y, j0 = kWyBlock * blockIdx.x, t = threadIdx.x;
  const double* Tg = tq + (int64_t)g * kWyBlock * kWyBlock;
  const double* Xg = xpart + (int64_t)g * sX;
  {
    // thread t stages row a = t/4, columns 16 (t%4) .. +15 of both tiles;
    // every load is issued before the first sum
    const int a = t >> 2, jq = 16 * (t & 3);
    const bool ra = a < kb;
    double tv[16], xv[kMaxSplitK][16];
#pragma unroll
    for (int u = 0; u < 16; ++u) tv[u] = (ra && jq + u < kb) ? Tg[a * kWyBlock + jq + u] : 0.0;
#pragma unroll
    for (int q = 0; q < kMaxSplitK; ++q)
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int j = j0 + jq + u;
        xv[q][u] = (ra && q < S && j < m) ? Xg[(int64_t)q * sP + (int64_t)a * ldx + j] : 0.0;
      }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      double v = xv[0][u];
#pragma unroll
      for (int q = 1; q < kMaxSplitK; ++q) v += xv[q][u];   // zero past S: same sum
      Ts[a][jq + u] = tv[u];
      Xs[a][jq + u] = v;
    }
  }
  __syncthreads();
  const int w = t >> 6, lane = t & 63, li = lane & 15, lk = lane >> 4;
  const int i0 = 32 * (w & 1), jw = 32 * (w >> 1);
  xdbl4 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = xdbl4{0.0, 0.0, 0.0, 0.0};
  for (int k = 0; k < kb; k += 4) {
    double av[2], bv[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      av[b] = Ts[i0 + 16 * b + li][k + lk];
      bv[b] = Xs[k + lk][jw + 16 * b + li];
    }
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
        acc[bi][bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[bi], bv[bj], acc[bi][bj], 0, 0, 0);
  }
  double* Yg = Y + (int64_t)g * sY;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int a = i0 + 16 * bi + 4 * r + lk, j = jw + 16 * bj + li;
        if (a < kb && j0 + j < m) Yg[(int64_t)a * ldy + j0 + j] = acc[bi][bj][r];
      }
}

// Y for a pair of consecutive WY blocks a, b = a+1 applied in one pass
// (block b first): with X = [X_a; X_b] = [V_a; V_b] Q22 given as S split-K
// parts (rows 0..63: X_a, 64..127: X_b, row r of part s at xpart + s sP +
// g sX + r ldx), Y_b = T_b X_b and Y_a = T_a (X_a - G_ab Y_b), G_ab =
// V_a V_b', since V_a (Q22 - V_b' Y_b) = X_a - G_ab Y_b. Then
// Q22 - V_b' Y_b - V_a' Y_a = Q22 - [V_a; V_b]' [Y_a; Y_b]. Workgroup
// (32-column tile, g) stages both X tiles and one 64 x 64 factor at a time
// in LDS; wave w forms rows 16 w .. 16 w + 15 of each product on the
// matrix cores.
__global__ __launch_bounds__(256) void wy_apply_pair_kernel(
    const double* __restrict__ ta, const double* __restrict__ tb, const double* __restrict__ gab,
    const double* __restrict__ xpart, int S, int64_t sP, int64_t sX, int64_t ldx, int m,
    double* __restrict__ Y, int64_t ldy, int64_t sY) {
  constexpr int W = kWyBlock, CT = 32;
  __shared__ double Fs[W][W + 1];
  __shared__ double Xa[W][CT + 1];
  __shared__ double Xb[W][CT + 1];
  const int g = blockIdx.y, j0 = CT * blockIdx.x, t = threadIdx.x;
  const int w = t >> 6, lane = t & 63, li = lane & 15, lk = lane >> 4;
  const int64_t fo = (int64_t)g * W * W;
  const auto load_f = [&](const double* F) {
#pragma unroll
    for (int u = 0; u < W * W / 256; ++u) {
      const int e = t + 256 * u;
      Fs[e / W][e % W] = F[fo + e];
    }
  };
  load_f(tb);
  {
    // thread t stages row a = t/4, columns 8 (t%4) .. +7 of both tiles;
    // every load is issued before the first sum
    const int a = t >> 2, jq = 8 * (t & 3);
    const double* Xg = xpart + (int64_t)g * sX;
    double va[kMaxSplitK][8], vb[kMaxSplitK][8];
#pragma unroll
    for (int q = 0; q < kMaxSplitK; ++q)
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + jq + u;
        const bool ok = q < S && j < m;
        const double* xr = Xg + (int64_t)q * sP + (int64_t)a * ldx + j;
        va[q][u] = ok ? xr[0] : 0.0;
        vb[q][u] = ok ? xr[(int64_t)W * ldx] : 0.0;
      }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      double sa = va[0][u], sb = vb[0][u];
#pragma unroll
      for (int q = 1; q < kMaxSplitK; ++q) {   // zero past S: the same sums
        sa += va[q][u];
        sb += vb[q][u];
      }
      Xa[a][jq + u] = sa;
      Xb[a][jq + u] = sb;
    }
  }
  __syncthreads();
  // acc <- +/- F rows 16w.. times X (64 x 32), added to acc
  const auto mm = [&](double sgn, double (*X)[CT + 1], xdbl4 (&acc)[2]) {
#pragma unroll
    for (int k = 0; k < W; k += 4) {
      const double a = sgn * Fs[16 * w + li][k + lk];
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
        acc[bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, X[k + lk][16 * bj + li], acc[bj], 0, 0, 0);
    }
  };
  double* Yg = Y + (int64_t)g * sY;
  const auto put = [&](xdbl4 (&acc)[2], double (*X)[CT + 1], int row0) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int a = 16 * w + 4 * r + lk, j = 16 * bj + li;
        if (X) X[a][j] = acc[bj][r];
        if (j0 + j < m) Yg[(int64_t)(row0 + a) * ldy + j0 + j] = acc[bj][r];
      }
  };
  xdbl4 acc[2] = {xdbl4{0.0, 0.0, 0.0, 0.0}, xdbl4{0.0, 0.0, 0.0, 0.0}};
  mm(1.0, Xb, acc);                                   // Y_b = T_b X_b
  __syncthreads();
  put(acc, Xb, W);                                    // Y_b over X_b
  load_f(gab);
  __syncthreads();
#pragma unroll
  for (int bj = 0; bj < 2; ++bj)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[bj][r] = Xa[16 * w + 4 * r + lk][16 * bj + li];
  mm(-1.0, Xb, acc);                                  // X_a - G_ab Y_b
  __syncthreads();
#pragma unroll
  for (int bj = 0; bj < 2; ++bj)
#pragma unroll
    for (int r = 0; r < 4; ++r) Xa[16 * w + 4 * r + lk][16 * bj + li] = acc[bj][r];
  load_f(ta);
  __syncthreads();
  acc[0] = acc[1] = xdbl4{0.0, 0.0, 0.0, 0.0};
  mm(1.0, Xa, acc);                                   // Y_a = T_a (X_a - G_ab Y_b)
  put(acc, nullptr, 0);
}

// Y for four consecutive WY blocks a, b, c, d applied in one pass (d
// first), the same recurrence one block further: with X = [X_a; X_b; X_c;
// X_d] = [V_a; ..; V_d] Q22 as S split-K parts (rows 0..63: X_a, .., 192..255:
// X_d) and G_xy = V_x V_y',
//   Y_d = T_d X_d,  Y_c = T_c (X_c - G_cd Y_d),
//   Y_b = T_b (X_b - G_bc Y_c - G_bd Y_d),
//   Y_a = T_a (X_a - G_ab Y_b - G_ac Y_c - G_ad Y_d),
// since V_x applied to Q22 after the later blocks' reflectors is X_x minus
// the G_xy Y_y of those blocks. Then Q22 -= [V_a; ..; V_d]' [Y_a; ..; Y_d],
// one rank-256 update. tq: T of block a (those of b, c, d at + sW, 2 sW,
// 3 sW); c1, c2, c3: the cross products at distance 1, 2, 3 of block a
// (of the following blocks at + sW, ..). Workgroup (32-column tile, g)
// keeps the four X tiles and one 64 x 64 factor at a time in LDS; wave w
// forms rows 16 w .. 16 w + 15 of each product on the matrix cores.
__global__ __launch_bounds__(256) void wy_apply_quad_kernel(
    const double* __restrict__ tq, const double* __restrict__ c1, const double* __restrict__ c2,
    const double* __restrict__ c3, int64_t sW, const double* __restrict__ xpart, int S, int64_t sP,
    int64_t sX, int64_t ldx, int m, double* __restrict__ Y, int64_t ldy, int64_t sY) {
  constexpr int W = kWyBlock, CT = 32;
  __shared__ double Fs[W][W + 1];
  __shared__ double Xs[kWyQuad][W][CT + 1];
  const int g = blockIdx.y, j0 = CT * blockIdx.x, t = threadIdx.x;
  const int w = t >> 6, lane = t & 63, li = lane & 15, lk = lane >> 4;
  const int64_t fo = (int64_t)g * W * W;
  const auto load_f = [&](const double* F) {
#pragma unroll
    for (int u = 0; u < W * W / 256; ++u) {
      const int e = t + 256 * u;
      Fs[e / W][e % W] = F[fo + e];
    }
  };
  {
    // thread t stages row a = t/4, columns 8 (t%4) .. +7 of each tile; the
    // parts of one tile are loaded before they are added
    const int a = t >> 2, jq = 8 * (t & 3);
    const double* Xg = xpart + (int64_t)g * sX;
#pragma unroll 1
    for (int k = 0; k < kWyQuad; ++k) {
      double v[kMaxSplitK][8];
#pragma unroll
      for (int q = 0; q < kMaxSplitK; ++q)
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + jq + u;
          const bool ok = q < S && j < m;
          v[q][u] = ok ? Xg[(int64_t)q * sP + (int64_t)(k * W + a) * ldx + j] : 0.0;
        }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        double sum = v[0][u];
#pragma unroll
        for (int q = 1; q < kMaxSplitK; ++q) sum += v[q][u];   // zero past S: the same sum
        Xs[k][a][jq + u] = sum;
      }
    }
  }
  __syncthreads();                                    // the four tiles staged
  // acc <- acc +/- F rows 16w.. times X (64 x 32)
  const auto mm = [&](double sgn, double (*X)[CT + 1], xdbl4 (&acc)[2]) {
#pragma unroll
    for (int k = 0; k < W; k += 4) {
      const double f = sgn * Fs[16 * w + li][k + lk];
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
        acc[bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(f, X[k + lk][16 * bj + li], acc[bj], 0, 0, 0);
    }
  };
  double* Yg = Y + (int64_t)g * sY;
  // the wave's rows of acc into X (LDS, when given) and into rows row0 + .. of Y
  const auto put = [&](const xdbl4 (&acc)[2], double (*X)[CT + 1], int row0) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int a = 16 * w + 4 * r + lk, j = 16 * bj + li;
        if (X) X[a][j] = acc[bj][r];
        if (row0 >= 0 && j0 + j < m) Yg[(int64_t)(row0 + a) * ldy + j0 + j] = acc[bj][r];
      }
  };
  const auto own = [&](double (*X)[CT + 1], xdbl4 (&acc)[2]) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[bj][r] = X[16 * w + 4 * r + lk][16 * bj + li];
  };
  xdbl4 acc[2];
  // block k: X_k -= sum over the later blocks l of G_kl Y_l, then Y_k = T_k X_k
  for (int k = kWyQuad - 1; k >= 0; --k) {
    own(Xs[k], acc);
    for (int l = k + 1; l < kWyQuad; ++l) {
      const double* cd = (l - k == 1) ? c1 : (l - k == 2) ? c2 : c3;
      __syncthreads();                                // the previous factor read by all
      load_f(cd + (int64_t)k * sW);
      __syncthreads();
      mm(-1.0, Xs[l], acc);
    }
    __syncthreads();                                  // every read of Fs and of X_k done
    put(acc, Xs[k], -1);
    load_f(tq + (int64_t)k * sW);
    __syncthreads();
    acc[0] = acc[1] = xdbl4{0.0, 0.0, 0.0, 0.0};
    mm(1.0, Xs[k], acc);
    __syncthreads();                                  // X_k read by all before Y_k replaces it
    put(acc, Xs[k], k * W);
  }
}

int band_reduce(hipStream_t s, const BandWork& wk) {
  const int G = wk.G, N = wk.N;
  if (G <= 0) return 0;
  if (N % 64 != 0 || N < 64 || N > kMaxSharedOrder) {
    set_error("band_reduce: N must be a multiple of 64 in [64, " + std::to_string(kMaxSharedOrder) +
              "]");
    return KMP_EINVAL;
  }
  int rc;
  const int64_t sP = (int64_t)3 * BB * N;
  KMP_HIP_TRY(hipMemsetAsync(wk.tau, 0, sizeof(double) * (size_t)G * N, s));
  double* const pbuf[2] = {wk.panel, wk.panel2};
  double* const m2s = wk.part + band_chunk_doubles(G, N);   // the slices of M2
  const auto tiles_of = [](int m) { return (int)ceil_div(m, 64); };
  const auto dual_grid = [&](int m, int tpw) {
    const int64_t t = tiles_of(m);
    return (unsigned)(G + ceil_div(t * (t + 1) / 2 * G, (int64_t)tpw));
  };
  // Panel factorisation of panel p into buffer pb: alone (dual = false) or
  // in one launch with the rest of the previous panel's two-sided update
  // (dual = true; that panel's first block column is up to date already).
  // The register kernel is chosen by the number of rows: 8 wavefronts (32
  // rows per slot) up to 1280 rows, then 16 (64 rows per slot), so the
  // unrolled steps stay within the instruction cache and the slots within
  // the registers; the streaming kernel beyond 2048 rows.
  const auto factor_panel = [&](int p, double* pb, bool dual, const double* pprev) -> int {
    const int mrow = N - p - BB;
    const int mprev = mrow + BB, m0prev = p;
    const double* P1 = pprev ? pprev + m0prev : nullptr;
    const double* P2 = pprev ? pprev + (int64_t)BB * N + m0prev : nullptr;
    const int tp = tiles_of(mprev);
    const int rs = (int)ceil_div(mrow, 32), rs16 = (int)ceil_div(mrow, 64);
#define KMP_PQR(RSV, NWV, CV)                                                                     \
  do {                                                                                            \
    if (dual)                                                                                     \
      hipLaunchKernelGGL((qr_rest_vec_kernel<RSV, NWV, CV>), dim3(dual_grid(mprev, NWV / 4)),     \
                         dim3(64 * NWV), 0, s, wk.A, N, p, wk.tau, pb, wk.tmat, wk.xbuf, G,       \
                         m0prev, mprev, P1, P2, sP, tp);                                          \
    else                                                                                          \
      hipLaunchKernelGGL((panel_qr_vec_kernel<RSV, NWV, CV>), dim3(G), dim3(64 * NWV), 0, s,      \
                         wk.A, N, p, wk.tau, pb, wk.tmat, wk.xbuf);                               \
  } while (0)
    if (rs <= 8) KMP_PQR(8, 8, true);
    else if (rs <= 16) KMP_PQR(16, 8, true);
    else if (rs <= 24) KMP_PQR(24, 8, true);
    else if (rs <= 32) KMP_PQR(32, 8, true);
    else if (rs <= 40) KMP_PQR(40, 8, true);
    else if (rs16 <= 24) KMP_PQR(24, 16, false);
    else if (rs16 <= 32) KMP_PQR(32, 16, false);
#undef KMP_PQR
    else if (dual)
      hipLaunchKernelGGL(qr_rest_stream_kernel, dim3(dual_grid(mprev, PQT / 256)), dim3(PQT), 0, s,
                         wk.A, N, p, wk.tau, pb, G, m0prev, mprev, P1, P2, sP, tp);
    else
      hipLaunchKernelGGL(panel_qr_kernel, dim3(G), dim3(PQT), 0, s, wk.A, N, p, wk.tau, pb);
    KMP_LAUNCH_CHECK();
    return 0;
  };
  // T of panel p's block reflector and Y' = T'V' (BB x mrow, transposed
  // into xbuf): the register kernel forms T, and Y' up to kFusedYtRows
  // rows, else the product follows; after the streaming kernel, the Gram
  // of V, then dlarft, then the product
  const auto panel_wy = [&](int p, const double* pb) -> int {
    const int m0 = p + BB, mrow = N - m0;
    if (mrow <= kFusedYtRows) return 0;
    if (mrow > 2048) {
      if ((rc = ts_gram(s, BB, BB, mrow, G, pb + m0, N, sP, pb + m0, N, sP, wk.gram, kWyBlock,
                        (int64_t)kWyBlock * kWyBlock, wk.part)) != 0)
        return rc;
      if ((rc = wy_form_t(s, wk.gram, wk.tau, wk.tmat, G, N, BB, p)) != 0) return rc;
    }
    GemmArgs g1;
    g1.M = BB; g1.N = mrow; g1.K = BB; g1.batch = G;
    g1.A = wk.tmat; g1.lda = kWyBlock; g1.sA = (int64_t)kWyBlock * kWyBlock;
    g1.B = pb + m0; g1.ldb = N; g1.sB = sP;
    g1.C = wk.xbuf; g1.ldc = BB; g1.sC = (int64_t)kWyBlock * N;     // transposed, m x 16
    return gemm(s, g1, false, false, false);
  };
  // panel read twice per column step and written once (algorithmic: once)
  const auto qr_bytes = [&](int m0) {
    return over_groups(wk, [&](double n) { return 16.0 * std::max(0.0, n - m0) * BB; });
  };
  const auto qr_flops = [&](int m0) {
    return over_groups(wk, [&](double n) { return 4.0 * std::max(0.0, n - m0) * BB * BB; });
  };
  kc_begin(KMP_KC_PANEL, s);
  if ((rc = factor_panel(0, pbuf[0], false, nullptr)) != 0) return rc;
  kc_end(KMP_KC_PANEL, s, qr_bytes(BB), qr_flops(BB));
  kc_begin(KMP_KC_PANEL_WY, s);
  if ((rc = panel_wy(0, pbuf[0])) != 0) return rc;
  for (int p = 0; p + BB < N; p += BB) {
    const int m0 = p + BB, mrow = N - m0;
    double* const pb = pbuf[(p / BB) & 1];
    // X' = Y' A22 (into ybuf) and the block products of M2 = V'X
    const int NJ = (int)ceil_div(N, BB);
    const int64_t sXq = (int64_t)2 * kWyBlock * N;
    hipLaunchKernelGGL(panel_x_kernel, dim3((unsigned)ceil_div(mrow / BB, 4), (unsigned)G),
                       dim3(64 * XW), 0, s, wk.A, N, m0, wk.xbuf, (const double*)pb, wk.part, NJ,
                       wk.ybuf, sXq);
    KMP_LAUNCH_CHECK();
    kc_end(KMP_KC_PANEL_WY, s, over_groups(wk, [&](double n) {
             const double m = std::max(0.0, n - m0); return 8.0 * m * m; }),
           over_groups(wk, [&](double n) {
             const double m = std::max(0.0, n - m0); return 2.0 * BB * m * m; }));
    // A22 -= V W' + W V' (K = 2 BB over the [V; W; V] rows), W' = X' -
    // 1/2 (T'M2)' V': W' and the first block column in one launch; then,
    // with a next panel, its factorisation beside the rest of the update.
    const bool next = m0 + BB < N;
    kc_begin(KMP_KC_TRAIL, s);
    const double* P1 = pb + m0;
    const double* P2 = pb + (int64_t)BB * N + m0;
    const unsigned tl = (unsigned)tiles_of(mrow);
    hipLaunchKernelGGL(m2_slices_kernel, dim3((unsigned)M2S, (unsigned)G), dim3(256), 0, s,
                       (const double*)wk.part, NJ, mrow / BB, m2s);
    KMP_LAUNCH_CHECK();
    hipLaunchKernelGGL(panel_ws_kernel, dim3(tl, (unsigned)G), dim3(256), 0, s, wk.A, N, m0,
                       (const double*)m2s, (const double*)wk.tmat, (const double*)wk.ybuf, sXq,
                       pb);
    KMP_LAUNCH_CHECK();
    if (next) {
      if ((rc = factor_panel(m0, pbuf[((p / BB) & 1) ^ 1], true, pb)) != 0) return rc;
    } else {
      hipLaunchKernelGGL((rank_update_kernel<1, true, 2>), dim3(tl, tl, (unsigned)G), dim3(256), 0,
                         s, wk.A + (int64_t)m0 * N + m0, (int64_t)N, (int64_t)N * N, mrow, P1,
                         (int64_t)N, sP, P2, (int64_t)N, sP);
      KMP_LAUNCH_CHECK();
    }
    // the lower triangle of A22 read and written once, rank-2 BB products
    // on it; with a next panel, that panel's factorisation as well
    kc_end(KMP_KC_TRAIL, s,
           over_groups(wk, [&](double n) {
             const double m = std::max(0.0, n - m0); return 8.0 * m * m; }) +
               (next ? qr_bytes(m0 + BB) : 0.0),
           over_groups(wk, [&](double n) {
             const double m = std::max(0.0, n - m0); return 2.0 * BB * m * m; }) +
               (next ? qr_flops(m0 + BB) : 0.0));
    if (next) {
      kc_begin(KMP_KC_PANEL_WY, s);
      if ((rc = panel_wy(m0, pbuf[((p / BB) & 1) ^ 1])) != 0) return rc;
    }
  }
  // the band, then clean reflector rows for the accumulation of Q
  {
    const int64_t tot = (int64_t)G * (BB + 1) * N;
    hipLaunchKernelGGL(band_extract_kernel, dim3((unsigned)ceil_div(tot, 256)), dim3(256), 0, s,
                       wk.A, N, tot, wk.band);
    KMP_LAUNCH_CHECK();
    if (wk.band_ready) KMP_HIP_TRY(hipEventRecord(wk.band_ready, s));
    const int64_t tz = (int64_t)G * (N - BB) * (kWyQuad * kWyBlock + BB);
    hipLaunchKernelGGL(clear_reflector_rows_kernel, dim3((unsigned)ceil_div(tz, 256)), dim3(256), 0,
                       s, wk.A, N, tz);
    KMP_LAUNCH_CHECK();
    const int64_t bx = std::min<int64_t>(ceil_div((int64_t)N * N, 256), 1 << 20);
    hipLaunchKernelGGL(set_identity_band_kernel, dim3((unsigned)bx, (unsigned)G), dim3(256), 0, s,
                       wk.Q, N);
    KMP_LAUNCH_CHECK();
  }
  // Q = H_0 H_1 ... (reflector rows 0 .. N-BB-1), accumulated backwards in
  // blocks of kWyBlock rows: Q[q+BB:, q+BB:] -= V' (T (V Q[q+BB:, q+BB:])).
  // The Grams, cross products and T factors of all blocks depend on the
  // reflectors only and are formed first, two launches for all blocks.
  // The last (partial) block goes alone, then the others in fours, one
  // pass over Q22 and one rank-256 update per four blocks (see
  // wy_apply_quad_kernel), then a pair and a single block at the bottom if
  // they are left.
  const int nref = N - BB;
  const int nblk = wy_blocks(N);
  kc_begin(KMP_KC_QFORM, s);
  const int64_t sD = (int64_t)wy_all_doubles(G, N);        // between the cross-product distances
  hipLaunchKernelGGL(wy_gram_kernel, dim3((unsigned)nblk, (unsigned)G, (unsigned)kWyQuad), dim3(256), 0,
                     s, wk.A, N, nref, wk.gram_all, wk.cross_all, sD);
  KMP_LAUNCH_CHECK();
  if ((rc = wy_form_t_blocks(s, wk.gram_all, wk.tau, wk.tmat_all, G, N, nref, nblk)) != 0) return rc;
  // reflector rows of each block read for its Gram and, with those of the
  // three next blocks, for the cross products; 64 x 64 products over m
  // columns
  kc_end(KMP_KC_QFORM, s, over_groups(wk, [&](double n) {
           double a = 0.0;
           for (int b = 0; b < nblk; ++b)
             a += (2.0 * kWyQuad - 1.0) * 8.0 * kWyBlock * std::max(0.0, n - kWyBlock * b - BB);
           return a; }),
         over_groups(wk, [&](double n) {
           double a = 0.0;
           for (int b = 0; b < nblk; ++b)
             a += kWyQuad * 2.0 * kWyBlock * kWyBlock * std::max(0.0, n - kWyBlock * b - BB);
           return a; }));
  const int64_t sW = (int64_t)G * kWyBlock * kWyBlock;      // between blocks in tmat_all, cross_all
  const int64_t sY = (int64_t)kWyQuad * kWyBlock * N;       // per matrix in ybuf and xpart
  const int64_t sXP = (int64_t)G * sY;                      // between split-K parts of xpart
  // nb consecutive blocks from block b in one pass: 4 (full blocks), 2, or
  // 1 (the partial last block, or a single full one)
  const auto step = [&](int b, int nb) -> int {
    const bool pair = nb == 2, quad = nb == kWyQuad;
    const int q = kWyBlock * b;
    const int kb = nb > 1 ? nb * kWyBlock : std::min(kWyBlock, nref - q);
    const int m = N - q - BB;
    kc_begin(KMP_KC_QFORM, s);
    // X = V Q[q+BB:, q+BB:] (kb x m) as split-K parts, in the transposed
    // form X' = Q[q+BB:, q+BB:]' V' (m x kb: the A operand is Q22 read by
    // rows, B the reflector rows)
    GemmArgs h1;
    h1.M = m; h1.N = kb; h1.K = m; h1.batch = G;
    h1.A = wk.Q + (int64_t)(q + BB) * N + q + BB; h1.lda = N; h1.sA = (int64_t)N * N;
    h1.B = wk.A + (int64_t)q * N + q + BB; h1.ldb = N; h1.sB = (int64_t)N * N;
    h1.ldc = N; h1.sC = sY;
    const int S1 = splitk_parts(h1);
    if ((rc = gemm_partial(s, h1, false, S1, wk.xpart, sXP, nullptr, nullptr)) != 0) return rc;
    const double* tq = wk.tmat_all + (int64_t)b * sW;
    if (quad) {
      const double* c1 = wk.cross_all + (int64_t)b * sW;
      hipLaunchKernelGGL(wy_apply_quad_kernel, dim3((unsigned)ceil_div(m, 32), (unsigned)G),
                         dim3(256), 0, s, tq, c1, c1 + sD, c1 + 2 * sD, sW,
                         (const double*)wk.xpart, S1, sXP, sY, (int64_t)N, m, wk.ybuf, (int64_t)N,
                         sY);
    } else if (pair) {
      hipLaunchKernelGGL(wy_apply_pair_kernel, dim3((unsigned)ceil_div(m, 32), (unsigned)G), dim3(256),
                         0, s, tq, tq + sW, (const double*)(wk.cross_all + (int64_t)b * sW),
                         (const double*)wk.xpart, S1, sXP, sY, (int64_t)N, m, wk.ybuf, (int64_t)N,
                         sY);
    } else {
      hipLaunchKernelGGL(wy_apply_t_kernel, dim3((unsigned)ceil_div(m, kWyBlock), (unsigned)G),
                         dim3(256), 0, s, tq, kb, (const double*)wk.xpart, S1, sXP, sY, (int64_t)N,
                         m, wk.ybuf, (int64_t)N, sY);
    }
    KMP_LAUNCH_CHECK();
    // Q[q+BB:, q+BB:] -= V' Y  (K = kb: 256 for four blocks, 128 for a
    // pair, 64 for a full single block, else the generic product)
    const dim3 ug((unsigned)ceil_div(m, 64), (unsigned)ceil_div(m, 64), (unsigned)G);
    double* Q22 = wk.Q + (int64_t)(q + BB) * N + q + BB;
    const double* P1 = wk.A + (int64_t)q * N + q + BB;
    if (kb == kWyQuad * kWyBlock) {
      hipLaunchKernelGGL((rank_update_kernel<8, false>), ug, dim3(256), 0, s, Q22, (int64_t)N,
                         (int64_t)N * N, m, P1, (int64_t)N, (int64_t)N * N,
                         (const double*)wk.ybuf, (int64_t)N, sY);
      KMP_LAUNCH_CHECK();
    } else if (kb == 2 * kWyBlock) {
      hipLaunchKernelGGL((rank_update_kernel<4, false>), ug, dim3(256), 0, s, Q22, (int64_t)N,
                         (int64_t)N * N, m, P1, (int64_t)N, (int64_t)N * N,
                         (const double*)wk.ybuf, (int64_t)N, sY);
      KMP_LAUNCH_CHECK();
    } else if (kb == kWyBlock) {
      hipLaunchKernelGGL((rank_update_kernel<2, false>), ug, dim3(256), 0, s, Q22, (int64_t)N,
                         (int64_t)N * N, m, P1, (int64_t)N, (int64_t)N * N,
                         (const double*)wk.ybuf, (int64_t)N, sY);
      KMP_LAUNCH_CHECK();
    } else {
      GemmArgs h3;
      h3.M = m; h3.N = m; h3.K = kb; h3.batch = G;
      h3.A = P1; h3.lda = N; h3.sA = (int64_t)N * N;
      h3.B = wk.ybuf; h3.ldb = N; h3.sB = sY;
      h3.C = Q22; h3.ldc = N; h3.sC = (int64_t)N * N;
      h3.alpha = -1.0; h3.beta = 1.0;
      if ((rc = gemm(s, h3, false, false, true)) != 0) return rc;
    }
    // Q22 read twice, written once; flops of V Q22, T X (and G Y), V' Y
    kc_end(KMP_KC_QFORM, s, over_groups(wk, [&](double n) {
             const double mm = std::max(0.0, n - q - BB); return 24.0 * mm * mm; }),
           over_groups(wk, [&](double n) {
             const double mm = std::max(0.0, n - q - BB);
             const double tk = quad ? 10.0 * kWyBlock * kWyBlock
                                    : pair ? 3.0 * kWyBlock * kWyBlock : (double)kb * kb;
             return 4.0 * kb * mm * mm + 2.0 * tk * mm; }));
    return 0;
  };
  int b = nblk - 1;
  if (nref % kWyBlock != 0) {
    if ((rc = step(b, 1)) != 0) return rc;
    --b;
  }
  for (; b >= kWyQuad - 1; b -= kWyQuad)
    if ((rc = step(b - kWyQuad + 1, kWyQuad)) != 0) return rc;
  if (b >= 1) {
    if ((rc = step(b - 1, 2)) != 0) return rc;
    b -= 2;
  }
  if (b == 0 && (rc = step(0, 1)) != 0) return rc;
  return 0;
}

}  // namespace kmp
