// Shared device helpers and host-side error plumbing for the kmpath library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "kmpath.h"

namespace kmp {

// ---------------------------------------------------------------- errors
void set_error(const std::string& msg);
const char* last_error();

#define KMP_HIP_TRY(expr)                                                        \
  do {                                                                           \
    hipError_t _e = (expr);                                                      \
    if (_e != hipSuccess) {                                                      \
      ::kmp::set_error(std::string(#expr) + ": " + hipGetErrorString(_e));       \
      return KMP_EHIP;                                                           \
    }                                                                            \
  } while (0)

#define KMP_LAUNCH_CHECK()                                                       \
  do {                                                                           \
    hipError_t _e = hipGetLastError();                                           \
    if (_e != hipSuccess) {                                                      \
      ::kmp::set_error(std::string("kernel launch: ") + hipGetErrorString(_e));  \
      return KMP_EHIP;                                                           \
    }                                                                            \
  } while (0)

constexpr int kWave = 64;

// Optional per-class kernel timing with HIP events (see kmp_path_spec
// timing_mask). The driver installs a clock for the duration of a call;
// launchers bracket their launches with kc_begin / kc_end.
struct KernelClock;
KernelClock* current_clock();
void kc_begin(int cls, hipStream_t s);
void kc_end(int cls, hipStream_t s, double bytes, double flops);

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// ---------------------------------------------------- MFMA f64 16x16x4 layout
// v_mfma_f64_16x16x4_f64 on gfx950, per lane l of the wave: the A operand is
// element (i = l%16, k = l/16), the B operand element (k = l/16, j = l%16),
// and accumulator register r holds D(i = 4 r + l/16, j = l%16).
__device__ __forceinline__ int mfma_row(int lane, int r) { return 4 * r + (lane >> 4); }
__device__ __forceinline__ int mfma_col(int lane) { return lane & 15; }

// ------------------------------------------------------- device reductions
// Fixed-order butterfly within a 64-lane wavefront: every lane ends with the
// same value, and the association order does not depend on timing.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ double wave_max(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off, kWave));
  return v;
}

// Block-wide sum for a block of NW waves; `red` holds NW doubles of LDS.
// Result returned to every thread. Deterministic (wave butterflies, then the
// per-wave results added in wave order).
template <int NW>
__device__ __forceinline__ double block_sum(double v, double* red) {
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < NW; ++i) s += red[i];
  return s;
}

// ---------------------------------------------------------------- losses
// psi(y, f): derivative of the training loss with respect to f.
//   hinge:    y * L'_delta(y f)  with L'_delta = -1 | (u-1-delta)/(2 delta) | 0
//   logistic: -y / (1 + exp(y f))
//   check:    -rho'_{tau,delta}(y - f) with rho' = tau | (r + delta(2tau-1))/(2delta) | tau-1
__device__ __forceinline__ double loss_psi(int loss, double y, double f, double delta, double tau) {
  if (loss == 0) {
    const double u = y * f;
    double d = 0.0;
    if (u <= 1.0 - delta) d = -1.0;
    else if (u < 1.0 + delta) d = (u - 1.0 - delta) / (2.0 * delta);
    return y * d;
  } else if (loss == 1) {
    return -y / (1.0 + exp(y * f));
  } else {
    const double r = y - f;
    double d;
    if (r >= delta) d = tau;
    else if (r <= -delta) d = tau - 1.0;
    else d = (r + delta * (2.0 * tau - 1.0)) / (2.0 * delta);
    return -d;
  }
}

// Training (smoothed) loss value.
__device__ __forceinline__ double loss_value(int loss, double y, double f, double delta, double tau) {
  if (loss == 0) {
    const double u = y * f;
    if (u <= 1.0 - delta) return 1.0 - u;
    if (u >= 1.0 + delta) return 0.0;
    const double t = u - 1.0 - delta;
    return t * t / (4.0 * delta);
  } else if (loss == 1) {
    const double m = -y * f;               // log(1 + e^m), overflow-safe
    return m > 0.0 ? m + log1p(exp(-m)) : log1p(exp(m));
  } else {
    const double r = y - f;
    if (r >= delta) return tau * r;
    if (r <= -delta) return (tau - 1.0) * r;
    return (r * r + 2.0 * r * delta * (2.0 * tau - 1.0) + delta * delta) / (4.0 * delta);
  }
}

// Unsmoothed loss used for the held-out CV score.
__device__ __forceinline__ double loss_eval(int loss, double y, double f, double tau) {
  if (loss == 0) {
    const double u = 1.0 - y * f;
    return u > 0.0 ? u : 0.0;
  } else if (loss == 1) {
    const double m = -y * f;
    return m > 0.0 ? m + log1p(exp(-m)) : log1p(exp(m));
  } else {
    const double r = y - f;
    return r * (r < 0.0 ? tau - 1.0 : tau);
  }
}

// 1/x from the hardware estimate and two Newton-Raphson steps
// r <- r + r (1 - x r), which square the relative error each; for the
// positive, normal pivots of the LDL' sweep.
__device__ __forceinline__ double rcp_newton(double x) {
  double r = __builtin_amdgcn_rcp(x);
  double e = fma(-x, r, 1.0);
  r = fma(r, e, r);
  e = fma(-x, r, 1.0);
  return fma(r, e, r);
}

// sqrt(x) for normal x > 0 by Goldschmidt's iteration (Markstein, IA-64
// and Elementary Functions, 2000): y ~ sqrt(x) and h ~ 1/(2 sqrt(x)) from
// the hardware reciprocal square root, one coupled Newton-Raphson step on
// both, then y corrected by the residual x - y^2.
__device__ __forceinline__ double sqrt_newton(double x) {
  const double r = __builtin_amdgcn_rsq(x);
  double y = x * r, h = 0.5 * r;
  const double e = fma(-y, h, 0.5);
  y = fma(y, e, y);
  h = fma(h, e, h);
  return fma(fma(-y, y, x), h, y);
}

}  // namespace kmp
