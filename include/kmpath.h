/*
 * kmpath -- cross-validated regularisation paths of RBF kernel machines on
 * one AMD Instinct MI355X (gfx950), fp64 throughout.
 *
 * Problem (Appendix A.1, eq. (kernelsvm); Appendix A.2, fold-restricted
 * form). For every kernel bandwidth sigma_s, quantile level tau_q (check
 * loss only), fold v and penalty lambda_l, with T_v the training points of
 * fold v (fold id != v, increasing index order), n_v = |T_v| and
 * K_v = K[T_v, T_v], K(x, x') = exp(-||x - x'||^2 / (2 sigma^2)):
 *
 *   minimise over alpha in R^{n_v}, beta in R
 *     F = (1/n_v) sum_{i in T_v} loss(y_i, f_i) + lambda alpha' K_v alpha,
 *     f = K_v alpha + beta 1,
 *
 * where loss is the delta-smoothed hinge L_delta(y f) (Appendix A.1), the
 * logistic loss log(1 + exp(-y f)) or the smoothed check loss
 * rho_{tau,delta}(y - f) (kernel quantile regression). The method is the
 * paper's: one factorisation of each K_v reused for every lambda
 * (Appendix A.3), the majorise-minimise update of Appendix A.1 with
 * Nesterov acceleration (Algorithm 1), all (fold x lambda) problems advanced
 * together, and the finite-smoothing schedule delta <- eta * delta
 * (Algorithm 1, outer loop).
 *
 * Conventions for every entry point:
 *  - Pointers documented as DEVICE point to memory on the current HIP device
 *    (e.g. torch tensors); HOST pointers are ordinary host memory. All
 *    arrays are caller-owned; the library keeps no pointer after returning.
 *  - fp64 arrays are densely packed in the layouts stated; int arrays are
 *    int32 unless stated.
 *  - Work is enqueued on `stream` (0 = the null stream). Entry points that
 *    return host results synchronise that stream before returning.
 *  - Return 0 on success, a negative KMP_E* code on error (nothing is
 *    written to outputs after an argument error), +1 (KMP_WMAXITER) when the
 *    path finished but some cell hit max_iter. kmp_strerror explains codes.
 *  - Not thread-safe on one workspace; distinct workspaces may be used
 *    concurrently.
 */
#ifndef KMPATH_H
#define KMPATH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KMP_OK 0
#define KMP_WMAXITER 1     /* finished; some cells stopped at max_iter      */
#define KMP_WNOTEXACT 2    /* finished; with KMP_FLAG_EXACT_HINGE some cells
                              kept their smoothed solution (status 3)       */
#define KMP_EINVAL (-1)    /* bad shape, lambda <= 0, sigma <= 0, tau, loss  */
#define KMP_EFOLD (-2)     /* fold id out of range, empty fold, one class    */
#define KMP_EWORKSPACE (-3)/* workspace missing or too small                 */
#define KMP_EHIP (-4)      /* HIP runtime error (see kmp_strerror)           */
#define KMP_ENONFINITE (-5)/* NaN or Inf in X, y or the iteration            */

#define KMP_HINGE 0        /* smoothed hinge, y in {-1,+1}                   */
#define KMP_LOGISTIC 1     /* logistic, y in {-1,+1}; no smoothing stages    */
#define KMP_CHECK 2        /* smoothed check loss, any real y                */

#define KMP_FLAG_RESTART 1 /* adaptive (gradient) restart of the momentum    */
#define KMP_FLAG_REFIT 4   /* full-data refit: every (sigma, tau, lambda) is
                          fitted on all n points (the fold with an empty
                          held-out set; Algorithm 1's final refit). V must
                          be 1 and fold_id is ignored (may be NULL);
                          outputs keep their [S][Q][V][L] layout with V = 1,
                          cv_sum and cv_err are zero and selected is not
                          written. For the margin losses y must hold both
                          classes.                                         */
#define KMP_FLAG_SHARED_FACTOR 8 /* exact CV with one factorisation of the full
                          K per bandwidth (Appendix A.2, exact cross-validation
                          formula; Algorithm 1's single decomposition): the
                          problem of fold v is solved as the n-point problem
                          whose held-out points carry no loss (zero response
                          weight), with the loss normalised by n_v; its
                          minimiser is the fold solution with zero
                          coefficients on the held-out points (the paper's
                          Lemma 2). Every (tau, fold, lambda) is a column on
                          the one factor. Same outputs as the per-fold mode;
                          n <= 40960. With V = n and fold_id[i] = i this is
                          exact leave-one-out CV (Algorithm 1 as printed).  */
#define KMP_FLAG_EXACT_HINGE 16 /* finite smoothing to the exact hinge SVM
                          (Appendix A.1; Algorithm 1's outer loop ends when
                          the SVM's KKT conditions hold): after the smoothing
                          stages every cell's exact minimiser of eq.
                          (kernelsvm) on its fold is recovered from the point
                          sets of its smoothed solution (below / on / above
                          the margin: a linear system on the points on the
                          margin, solved on the GPU, sets corrected until the
                          KKT conditions hold to 1e-9, at most 128 rounds).
                          alpha, beta, the held-out sums are the exact
                          solution's and objective is the hinge objective of
                          eq. (kernelsvm). A cell with more margin points than
                          its system holds (min(N, 384), N its padded order)
                          or not settled keeps the smoothed solution, status
                          3, return KMP_WNOTEXACT. Hinge loss, per-fold
                          factors only; the workspace grows by about
                          (min(N, 384) + 1)^2 doubles per column.           */
#define KMP_FLAG_EAGER 32  /* launch every iteration directly. Otherwise, for
                          padded orders up to 2048 and poll_every <= 64, the
                          poll_every iterations between two convergence polls
                          are recorded once per smoothing stage as a HIP graph
                          and replayed (those orders are launch-bound); the
                          graph's split-K factor is the one for all columns,
                          so results agree with eager launches to rounding  */
#define KMP_FLAG_GLOBAL_SOLVE 2 /* keep the banded solve's working vector in
                          device memory at every order (it is there anyway
                          above the rows one workgroup's LDS holds: 20224
                          padded rows on gfx950); results agree to rounding */

/* Kernel classes timed with HIP events when their bit is set in
 * kmp_path_spec.timing_mask (1 << class). */
#define KMP_KC_GRAM 0         /* a1 Gram + fold gather                         */
#define KMP_KC_PANEL 1        /* a2 Householder QR of a band-reduction panel    */
#define KMP_KC_PANEL_WY 2     /* a2 panel products Y = VT, X = A22 Y, W         */
#define KMP_KC_TRAIL 3        /* a2 trailing update A22 -= V W' + W V' (MFMA)  */
#define KMP_KC_QFORM 4        /* a2 compact-WY accumulation of Q (MFMA)        */
#define KMP_KC_PRECOMPUTE 5   /* a3 per-stage column factors                   */
#define KMP_KC_GEMM_F 6       /* a4+a5 f = (Q B) abar with the loss epilogue   */
#define KMP_KC_GEMM_ZHAT 7    /* a6 zhat = Q' z                                */
#define KMP_KC_UPDATE 8       /* a7 banded solve, step, KKT, restart, momentum */
#define KMP_KC_FINALIZE 9     /* a10                                           */
#define KMP_NKC 10

/* Solver settings. kmp_default_spec fills the defaults named below. */
typedef struct {
  int32_t loss;        /* KMP_HINGE, KMP_LOGISTIC or KMP_CHECK              */
  double delta0;       /* first smoothing level (hinge/check), default 1    */
  double eta;          /* smoothing shrink factor, default 0.125            */
  int32_t n_stages;    /* smoothing levels delta0*eta^s, s < n_stages (3)   */
  double tol;          /* stop a cell when n_v*max(||Q'(z+2 lambda alpha)||_2,
                          |1'z|) <= tol at the extrapolated point (1e-9)    */
  int32_t max_iter;    /* iterations per stage per cell (100000)            */
  int32_t poll_every;  /* iterations between host convergence polls (8)     */
  int32_t flags;       /* KMP_FLAG_RESTART (default on), KMP_FLAG_GLOBAL_SOLVE,
                          KMP_FLAG_REFIT, KMP_FLAG_SHARED_FACTOR,
                          KMP_FLAG_EXACT_HINGE, KMP_FLAG_EAGER              */
  int32_t timing_mask; /* kernel classes to time with HIP events (default 0) */
  int32_t timing_every;/* bracket one launch in every timing_every launches
                          of a timed class (default 1: all)                 */
} kmp_path_spec;

/* Phase times in milliseconds, measured with HIP events on `stream`. */
typedef struct {
  double gram_ms;      /* a1: Gram + fold gather                            */
  double factor_ms;    /* a2: per-fold band factorisation and Q             */
  double precompute_ms;/* a3: per-stage per-column factors                  */
  double path_ms;      /* a4-a9: iterations                                 */
  double finalize_ms;  /* a10: alpha, objectives, CV sums                   */
  double total_ms;
  int64_t iterations;  /* iterations launched, summed over stages and batches */
  int64_t cell_iterations; /* sum over cells of iterations to convergence   */
  /* per kernel class (only classes in timing_mask are filled): summed event
   * time, launches, and algorithmic work of those launches (bytes that must
   * move to or from device memory, and flops), as defined per class in the
   * documentation of the kernels                                             */
  double kernel_ms[KMP_NKC];
  int64_t kernel_launches[KMP_NKC];  /* bracketed (sampled) launches         */
  int64_t kernel_seen[KMP_NKC];      /* all launches of the class            */
  double kernel_bytes[KMP_NKC];
  double kernel_flops[KMP_NKC];
  /* the part of the four sums above that comes from bracketed launches whose
   * algorithmic intensity (flops per byte) is above the ridge point of the
   * device, fp64 matrix peak over HBM peak (78.6e12 / 8e12 flop/B): those
   * launches are bound by the matrix cores, the others by memory bandwidth  */
  double kernel_ms_mb[KMP_NKC];
  int64_t kernel_launches_mb[KMP_NKC];
  double kernel_bytes_mb[KMP_NKC];
  double kernel_flops_mb[KMP_NKC];
} kmp_timings;

void kmp_default_spec(kmp_path_spec* spec);

/* Bytes of DEVICE workspace kmp_fit_path needs for this problem when the
 * bandwidths are processed `sigma_batch` at a time (1 <= sigma_batch <= S).
 * fold_id is HOST, n entries. Returns 0 if the arguments are invalid.     */
size_t kmp_workspace_bytes(const kmp_path_spec* spec, int64_t n, int64_t d,
                           int32_t L, const int32_t* fold_id, int32_t V,
                           int32_t S, int32_t Q, int32_t sigma_batch);

/* The whole CV path (Appendix A.2-A.4; Algorithm 1 in its V-fold form).
 *
 * Inputs
 *   X        DEVICE, n x d row-major, leading dimension ldx >= d (elements)
 *   y        DEVICE, n; +/-1 for hinge/logistic
 *   sigmas   HOST, S > 0 bandwidths (> 0)
 *   taus     HOST, Q levels in (0,1) for KMP_CHECK; ignored (Q must be 1)
 *            for the margin losses
 *   lambdas  HOST, L > 0 penalties (> 0), any order
 *   fold_id  HOST, n ids in [0, V); every fold non-empty; for hinge and
 *            logistic every training set must contain both classes
 *   workspace DEVICE, >= kmp_workspace_bytes(..., sigma_batch) for some
 *            sigma_batch; the largest batch that fits is used
 * Outputs (DEVICE unless stated; index order [s][q][v][l], s fastest-slowest
 * as written, i.e. cell (s,q,v,l) at ((s*Q + q)*V + v)*L + l):
 *   alpha    [S][Q][V][L][n]; zeros at the held-out indices of fold v
 *   beta     [S][Q][V][L]
 *   objective[S][Q][V][L]   F at the final delta, from K in observation space
 *   cv_sum   [S][Q][V][L]   sum over held-out j of the unsmoothed loss
 *   cv_err   [S][Q][V][L]   held-out y f <= 0 count (0 for KMP_CHECK); may be NULL
 *   iters    [S][Q][V][L]   iterations summed over stages; may be NULL
 *   status   [S][Q][V][L]   0 converged, 1 max_iter, 2 non-finite, 3 exact
 *                           hinge solution not reached (KMP_FLAG_EXACT_HINGE);
 *                           may be NULL
 *   selected HOST [S][Q]: argmin_l sum_v cv_sum/n, ties to larger lambda; may be NULL
 *   selected_joint HOST [Q][2]: the (s, l) minimising sum_v cv_sum/n over all
 *            bandwidths and penalties, ties to the larger lambda, then the
 *            larger sigma; may be NULL
 *   timings  HOST, may be NULL
 * The return code reports cells that stopped at max_iter (KMP_WMAXITER) or
 * went non-finite (KMP_ENONFINITE) whether or not `status` is given.
 * Synchronises `stream` before returning.                                   */
int kmp_fit_path(void* stream, const kmp_path_spec* spec,
                 const double* X, int64_t n, int64_t d, int64_t ldx,
                 const double* y,
                 const double* sigmas, int32_t S,
                 const double* taus, int32_t Q,
                 const double* lambdas, int32_t L,
                 const int32_t* fold_id, int32_t V,
                 void* workspace, size_t workspace_bytes,
                 double* alpha, double* beta, double* objective,
                 double* cv_sum, int32_t* cv_err, int32_t* iters,
                 int32_t* status, int32_t* selected, int32_t* selected_joint,
                 kmp_timings* timings);

/* Random V-fold assignment (HOST output fold_id, n entries): SplitMix64
 * (Steele, Lea & Flood 2014) seeded with `seed` drives a Fisher-Yates
 * shuffle from the top, j = high 64 bits of (draw * (i+1)); then
 * fold_id[perm[i]] = i mod V. Integer-only and reproducible.             */
int kmp_make_folds(int64_t n, int32_t V, uint64_t seed, int32_t* fold_id);

/* a1 on its own: the RBF kernel matrix of the paper's kernel="rbf" models
 * (Section 2's API; the kernel matrix K of eq. (kernelsvm), Appendix A.1),
 * parameterised as K(x, x') = exp(-||x - x'||^2 / (2 sigma^2)), in blocks
 * K_s[i][j] = exp(-max(0, |x_r|^2 + |x_c|^2 -
 * 2 x_r.x_c) / (2 sigma_s^2)) with r = rows[i], c = cols[j] (DEVICE int32
 * index lists into X), exactly 1 where r == c, and 0 where either index is
 * negative (padding). out DEVICE, S blocks of m x p row-major with leading
 * dimension ld_out >= p, block s at out + s*m*ld_out. sigmas HOST.        */
int kmp_rbf_gram(void* stream, const double* X, int64_t n, int64_t d, int64_t ldx,
                 const int32_t* rows, int64_t m, const int32_t* cols, int64_t p,
                 const double* sigmas, int32_t S, double* out, int64_t ld_out);

/* kmp_rbf_gram for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same arguments, layout, results and errors, but every temporary (the
 * squared row norms of X and the bandwidth factors) lives in a static device
 * array of 65536 doubles (512 KiB) that the library holds on each device
 * until the process ends, and the call allocates nothing. n must be at most
 * 65528 (KMP_EINVAL otherwise, before any device work). All calls on one
 * device share that array: calls that overlap on one device (different
 * streams or threads) race and must be serialised by the caller.            */
int kmp_rbf_gram_noalloc(void* stream, const double* X, int64_t n, int64_t d, int64_t ldx,
                         const int32_t* rows, int64_t m, const int32_t* cols, int64_t p,
                         const double* sigmas, int32_t S, double* out, int64_t ld_out);

/* One-stage alternative to a2 (kmp_fit_path uses kmp_band_reduce): G
 * symmetric N x N matrices A (DEVICE, row-major, packed,
 * matrix g at A + g*N*N; destroyed) are reduced to A_g = Q_g T_g Q_g' with
 * Q_g orthogonal (DEVICE out, same layout) and T_g symmetric tridiagonal
 * with diagonal diag[g*N + i] and off-diagonal off[g*N + i] = T[i+1][i]
 * (off[g*N + N-1] = 0). Householder reduction (Golub & Van Loan, Alg.
 * 8.3.1), blocked as in LAPACK's dsytrd, Q accumulated in compact-WY form.
 * Every matrix must have N valid rows (zero padding rows are allowed).     */
int kmp_tridiag(void* stream, double* A, int32_t G, int32_t N,
                double* Qout, double* diag, double* off);

/* a2 on its own, band form: G symmetric N x N matrices A (DEVICE, row-major,
 * packed, matrix g at A + g*N*N; destroyed) are reduced to A_g = Q_g B_g Q_g'
 * with Q_g orthogonal (DEVICE out, same layout) and B_g symmetric banded with
 * lower bandwidth KMP_BAND: band[g*(KMP_BAND+1)*N + r*N + j] = B_g[j+r][j]
 * (DEVICE out; entries with j + r >= N are 0). Blocked Householder reduction
 * (first stage of the successive band reduction, Bischof, Lang & Sun 2000):
 * panel QR, compact-WY two-sided trailing updates on matrix cores, Q
 * accumulated in compact-WY blocks. N must be a multiple of 64 in
 * [64, 40960]; zero padding rows are allowed.                             */
#define KMP_BAND 16
int kmp_band_reduce(void* stream, double* A, int32_t G, int32_t N, double* Qout, double* band);

/* a4-a7 on their own: one majorise-minimise step of the path from a
 * caller-given state, for C columns of one problem (Appendix A.1, the update
 * (beta, alpha) <- (beta, alpha) - H^{-1} (1'z ; K z + 2 lambda K alpha),
 * z_i = psi(y_i, f_i)/n, f = K alpha + beta; H applied through the block
 * form of its inverse of Appendix A.3, here in the band basis of K's
 * factorisation K = Q B Q'). Column c has penalty lambdas[c] (and level
 * taus[c] for KMP_CHECK); the curvature bound is 1/kappa with kappa = 2 delta
 * (hinge, check) or 4 (logistic, delta ignored). No extrapolation: the step
 * is taken from the given point itself.
 *   K         DEVICE, n x n row-major symmetric kernel matrix (not modified;
 *             it is factorised into library scratch, stream-ordered)
 *   y         DEVICE, n labels (+/-1 for hinge and logistic)
 *   lambdas   HOST, C penalties > 0; taus HOST, C levels in (0,1) (check
 *             loss only, else may be NULL)
 *   alpha_in  DEVICE [C][n], beta_in DEVICE [C]: the states
 *   alpha_out DEVICE [C][n], beta_out DEVICE [C]: the states after the step
 *   kkt_out   DEVICE [C] or NULL: n max(||Q'(z + 2 lambda alpha)||_2, |1'z|)
 *             at the given state
 * n <= 32768, C <= 65535. Synchronises `stream`; KMP_EINVAL on bad
 * arguments (nothing written), KMP_EHIP on runtime errors.                  */
int kmp_path_step(void* stream, int32_t loss, double delta, const double* K, int64_t n,
                  const double* y, const double* lambdas, const double* taus, int32_t C,
                  const double* alpha_in, const double* beta_in, double* alpha_out,
                  double* beta_out, double* kkt_out);

/* The path's dense products on their own (a4 f = (Q B) abar and a6
 * zhat = Q' z are such products, Appendix A.3: every iteration is O(n^2)
 * matrix products): C_g = A_g B_g for g < G, fp64 on the matrix cores.
 * A DEVICE, G blocks of M x K row-major at A + g*M*K; B DEVICE, K x N
 * row-major at B + g*K*N; C DEVICE, M x N row-major at C + g*M*N
 * (overwritten; zero when K = 0). G <= 65535. Synchronises `stream`.       */
int kmp_dgemm_grouped(void* stream, int32_t G, int32_t M, int32_t N, int32_t K,
                      const double* A, const double* B, double* C);

/* Message for a return code, or the last HIP error text for KMP_EHIP. */
const char* kmp_strerror(int code);

/* Name of kernel class `cls` (0 <= cls < KMP_NKC), or "" if out of range. */
const char* kmp_kernel_class_name(int cls);

/* Library version string. */
const char* kmp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KMPATH_H */
