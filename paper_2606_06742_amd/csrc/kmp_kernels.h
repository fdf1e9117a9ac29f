// Internal launcher interface between the host driver and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kmp {

// Batched tile GEMM on fp64 MFMA: for every batch b,
//   C_b = alpha * op(A_b) * op(B_b) + beta * C_b      (M x N, inner K)
// Element (i,k) of A is A[i*lda + k] when a_kcontig, else A[k*lda + i];
// element (k,j) of B is B[j*ldb + k] when b_kcontig, else B[k*ldb + j];
// element (i,j) of C is C[i*ldc + j] when c_rowmajor, else C[j*ldc + i].
// Batch b uses A + b*sA, B + b*sB, C + b*sC.
struct GemmArgs {
  int M = 0, N = 0, K = 0, batch = 1;
  const double* A = nullptr; int64_t lda = 0, sA = 0;
  const double* B = nullptr; int64_t ldb = 0, sB = 0;
  double* C = nullptr; int64_t ldc = 0, sC = 0;
  double alpha = 1.0, beta = 0.0;
};

// Loss epilogue of the first path GEMM (f = Q (T abar) then z): for row i of
// batch b and column c, with f = acc + bbar[c]:
//   Z[i][c] = psi(y[i], f)/cnv[c] if i < nv[b] and row i is a training row
//             of column c, else 0,
// and partial[b][tile][c] = sum of Z over the rows of the row tile. A row is
// a training row of every column unless fold ids are given (shared-factor
// exact CV): then row i is held out of column c when rfold[i] == cfold[c].
struct LossEpi {
  int loss = 0;
  double delta = 1.0;
  const double* y = nullptr; int64_t sy = 0;     // labels, per batch stride
  const int* nv = nullptr;                       // valid rows per batch
  const int* cnv = nullptr;                      // loss normaliser per column (stride sbb)
  const int32_t* rfold = nullptr;                // fold id per row (stride sy), or null
  const int32_t* cfold = nullptr;                // held-out fold per column (stride sbb)
  const double* bbar = nullptr; int64_t sbb = 0; // per column intercepts
  const double* tau = nullptr; int64_t stau = 0; // per column tau (check)
  double* partial = nullptr; int64_t spart = 0;  // [tiles][N] per batch
};

int gemm(hipStream_t s, const GemmArgs& g, bool a_kcontig, bool b_kcontig, bool c_rowmajor);
int gemm_loss(hipStream_t s, const GemmArgs& g, const LossEpi& e);
// Rows per output tile gemm_loss uses for g (the partial sums hold one row
// per tile): 32 or 64.
int gemm_loss_tile_rows(const GemmArgs& g);
constexpr int kMinTileRows = 32;
constexpr int kMaxSplitK = 4;
// Split-K: number of K parts for g (1..4), the partial products (column-
// major C layout per part, part stride sP), and the loss epilogue that adds
// the parts in order and writes Z plus 64-row column sums (see LossEpi).
// Both work on the active columns only: batch b has nact[b] of them, the
// k-th being column cmap[b*g.N + k] (B k-contiguous, C column-major).
// Tile of the partial products: 64 x 64 with the waves in a 2 x 2
// arrangement (every case), or, with active-column lists, whole-tile
// operands and M >= 128, the waves stacked by rows over 64 x 128 or
// 128 x 64 (three workgroups per compute unit instead of four: the split
// takes per_cu = 3 and the tile counts of the shape).
enum class PartTile { k64x64, k64x128, k128x64 };
// The tile for a launch over G batches of order M with na[g] active columns
// (host counts, C columns each if na is null) and its work tiles and
// resident workgroups per compute unit, for splitk_parts.
PartTile pick_part_tile(int M, int G, int C, const int* na, int64_t* tiles, int* per_cu);
int splitk_parts(const GemmArgs& g, int64_t tiles = 0, int per_cu = 4);
int gemm_partial(hipStream_t s, const GemmArgs& g, bool a_kcontig, int S, double* part, int64_t sP,
                 const int* cmap, const int* nact, PartTile tile = PartTile::k64x64);
int loss_epilogue(hipStream_t s, int M, int N, int batch, int S, const double* part, int64_t ldc,
                  int64_t sC, int64_t sP, double* Z, const LossEpi& e, const int* cmap,
                  const int* nact);

// ---------------------------------------------------------------- Gram
// out[0], out[1] = counts of non-finite entries of X (n x d, ldx) and y (n).
int count_nonfinite(hipStream_t s, const double* X, int64_t n, int64_t d, int64_t ldx,
                    const double* y, int* out);
// Squared row norms of X (n x d, ldx): nrm[i] = sum_k X[i][k]^2.
int row_norms(hipStream_t s, const double* X, int64_t n, int64_t d, int64_t ldx, double* nrm);

// Up to 8 doubles passed by value to a one-wavefront kernel that stores them
// at out (device).
struct Small8 {
  double v[8];
};
int store_small(hipStream_t s, const double* vals, int count, double* out);

// For each of `nb` index blocks (blockIdx.z = block q), rows idx_r + q*sr,
// cols idx_c + q*sc (m and p entries, negative = padding), write for each of
// S bandwidths: out + (s*sout_s + q*sout_q) + i*ld + j.
int rbf_blocks(hipStream_t s, const double* X, int64_t d, int64_t ldx, const double* nrm,
               const int32_t* idx_r, int64_t sr, int64_t m,
               const int32_t* idx_c, int64_t sc, int64_t p, int nb,
               const double* inv2s2, int S, double* out, int64_t sout_s, int64_t sout_q,
               int64_t ld);

// ------------------------------------------------------------ band form
constexpr int kBand = 16;      // lower bandwidth of B (= panel width of the reduction)
// Largest padded order per fold: N*N stays below 2^31 (32-bit row offsets
// r*N in the kernels) and the per-fold matrices of the largest workloads fit.
constexpr int kMaxOrder = 32768;
// Largest order of the one factor per bandwidth in the shared-factor mode
// (every kernel offset r*N + c still below 2^31).
constexpr int kMaxSharedOrder = 40960;
constexpr int kWyBlock = 64;   // reflectors per compact-WY block when forming Q
constexpr int kWyQuad = 4;     // compact-WY blocks applied to Q in one pass

// Reduction of G symmetric N x N matrices (row-major, packed, destroyed) to
// A_g = Q_g B_g Q_g' with B_g banded; band[g][r*N + j] = B_g[j+r][j], r <= kBand.
struct BandWork {
  int G = 0, N = 0;
  double* A = nullptr;      // G x N x N
  double* Q = nullptr;      // G x N x N, output
  double* band = nullptr;   // G x (kBand+1) x N, output
  double* tau = nullptr;    // G x N
  double* panel = nullptr;  // G x 3 kBand x N ([V; W; V] rows of the even panels)
  double* panel2 = nullptr; // G x 3 kBand x N (the same for the odd panels)
  double* tmat = nullptr;   // G x 64 x 64
  double* gram = nullptr;   // G x 64 x 64
  double* xbuf = nullptr;   // G x 64 x N
  double* ybuf = nullptr;   // G x 256 x N
  double* part = nullptr;   // band_part_doubles(G, N): chunk partials of the Gram products
  double* gram_all = nullptr;  // wy_blocks(N) x G x 64 x 64: Grams of the WY blocks of Q
  double* tmat_all = nullptr;  // same shape: their T factors
  double* cross_all = nullptr; // 3 x that shape: V_b V_{b+d}' at distance d = 1, 2, 3
  double* xpart = nullptr;     // kMaxSplitK x G x 256 x N: split-K parts of V Q in the Q accumulation
  const int* nv_host = nullptr;  // G valid orders (host), for the work counters; N if null
  hipEvent_t band_ready = nullptr;  // if set, recorded once the band is written
};
// Doubles of scratch band_reduce needs beyond A, Q, band and tau (the chunk
// partials included), and of the chunk partials alone.
size_t band_work_doubles(int G, int N);
size_t band_part_doubles(int G, int N);
// Number of kWyBlock-reflector blocks in which Q is accumulated, and the
// doubles of one of the gram_all / tmat_all buffers.
int wy_blocks(int N);
size_t wy_all_doubles(int G, int N);
int band_reduce(hipStream_t s, const BandWork& w);
// Compact-WY T factor (kb x kb, ld 64, per matrix) of reflectors p .. p+kb-1
// from their Gram matrix (ld 64) and tau[g*N + p + i].
int wy_form_t(hipStream_t s, const double* gram, const double* taus, double* tmat, int G, int N,
              int kb, int p);
// The same for all nblk blocks of kWyBlock reflectors 0 .., nref at once:
// block b's Gram and T at gram / tmat + b * G * 64 * 64 (+ g * 64 * 64).
int wy_form_t_blocks(hipStream_t s, const double* gram, const double* taus, double* tmat, int G,
                     int N, int nref, int nblk);

// --------------------------------------------------------- tridiagonal
struct TridiagWork {
  int G = 0, N = 0, nb = 32;
  double* A = nullptr;      // G x N x N, row-major; destroyed (holds reflectors)
  double* Q = nullptr;      // G x N x N, output
  double* diag = nullptr;   // G x N
  double* off = nullptr;    // G x N
  double* tau = nullptr;    // G x N (Householder scalars)
  double* panel = nullptr;  // G x 3nb x N  ([V; W; V] rows of the current panel)
  double* dots = nullptr;   // G x 2nb
  double* tmat = nullptr;   // G x 64 x 64 (compact-WY T factor of a block of Q)
  double* gram = nullptr;   // G x 64 x 64 (Gram of that block's reflectors)
  double* xbuf = nullptr;   // G x 64 x N
  double* ybuf = nullptr;   // G x 64 x N
  double* spart = nullptr;  // G x tridiag_parts(N) partial sums of w_raw'v
  double* pnext = nullptr;  // G x N next column, partially updated
  const int* nv_host = nullptr;  // G valid orders (host), for the work counters; N if null
  hipEvent_t band_ready = nullptr;  // if set, recorded once the band is written
};
// Per-matrix length of the spart buffer (partial sums of the products).
int tridiag_parts(int N);
// Doubles of scratch tridiagonalize needs beyond A, Q, diag, off, tau.
size_t tridiag_panel_doubles(int G, int N, int nb);
int tridiagonalize(hipStream_t s, const TridiagWork& w);
// nch independent parts, part k on stream ss[k] (launches interleaved).
int tridiagonalize_multi(const hipStream_t* ss, const TridiagWork* ws, int nch);

// ---------------------------------------------------------------- path
struct PathArrays {
  int G = 0;            // groups (sigma, fold)
  int N = 0;            // padded rows per group
  int C = 0;            // columns per group (tau x lambda)
  int loss = 0;
  bool global_solve = false;     // banded solve vector in device memory at every order
  const int* nv = nullptr;       // G valid rows
  const int* cnv = nullptr;      // G*C loss normaliser of each column (its n_v)
  const int32_t* rfold = nullptr;  // G x N fold id per row (shared-factor mode), else null
  const int32_t* cfold = nullptr;  // G*C held-out fold per column (shared-factor mode)
  const double* ylab = nullptr;  // G x N labels (0 at padding)
  const double* Q = nullptr;     // G x N x N
  const double* QB = nullptr;    // G x N x N: Q B, the A operand of the first GEMM
  const double* band = nullptr;  // G x (kBand+1) x N, band[g][r*N + j] = B[j+r][j]
  const double* cvec = nullptr;  // G x N, Q' 1 over valid rows
  const double* lam = nullptr;   // G*C
  const double* tau = nullptr;   // G*C
  // column-major per column N-vectors (column index gc = g*C + c)
  double* ahat = nullptr;
  double* abar = nullptr;
  double* zmat = nullptr;
  double* anew = nullptr;   // device-memory solve: forward results
  double* estep = nullptr;  // device-memory solve: w, then x, then a+
  double* ldl_l = nullptr;  // kBand x N per column: tiles of the banded LDL' factor
  double* ldl_d = nullptr;  // N per column: 1/D
  // the same factors of the matrix with rows and columns in reverse order,
  // and the twist block where the two meet (kBand^2 + kBand per column);
  // band_rev: the band of that reversed matrix (G x (kBand+1) x N)
  double* ldl_lr = nullptr;
  double* ldl_dr = nullptr;
  double* twist = nullptr;
  double* band_rev = nullptr;
  double* vhat = nullptr;
  double* uvec = nullptr;   // T vhat
  double* partial = nullptr;// G x tiles x C
  double* fpart = nullptr;  // kMaxSplitK x G x N x C split-K partials of f
  double* zpart = nullptr;  // kMaxSplitK x G x N x C split-K partials of zhat
  // per column scalars
  double* beta = nullptr;
  double* bbar = nullptr;
  double* rmom = nullptr;
  double* gcoef = nullptr;
  double* kkt = nullptr;
  int* flag = nullptr;      // 0 active, 1 converged, 2 max_iter, 3 non-finite
  int* iters = nullptr;     // per stage
  int* iters_total = nullptr;
  int* active_count = nullptr;  // 1 int
  int* cmap = nullptr;      // G x C: the active columns of each group, in order
  int* nact = nullptr;      // G: number of active columns of each group
  const int* nv_host = nullptr;  // G valid rows (host), for the work counters
  const int* nact_host = nullptr;  // G entries of nact as last read (host), same use
};

int path_init_columns(hipStream_t s, const PathArrays& p);
// A stage's setup: the LDL' factors of M = 2 lambda I + B/(n_v kappa) (they
// read the band, lambda and n_v only), then vhat, u and the momentum restart
// (these need c and the factors).
int path_stage_factor(hipStream_t s, const PathArrays& p, double kappa);
int path_stage_vectors(hipStream_t s, const PathArrays& p, double kappa);
int path_iteration(hipStream_t s, const PathArrays& p, double delta, double kappa, double tol,
                   int max_iter, int restart);
// Rebuilds cmap/nact from the column flags and writes the total number of
// active columns to active_count. The path GEMMs compute only the columns
// listed in cmap, so it runs after every change of the flags that should
// shrink the GEMMs (stage start, polls).
int path_compact(hipStream_t s, const PathArrays& p);
int group_ones_projection(hipStream_t s, const double* Q, const int* nv, int G, int N, double* cvec);
// QB = Q B for G groups (Q, QB: N x N row-major each; band as in PathArrays).
int form_qb(hipStream_t s, const double* Q, const double* band, int N, int G, double* QB);

// Exact hinge recovery after the smoothing stages (exact.hip): the buffers
// of one bandwidth batch (cols = G*C columns of N rows).
struct ExactArgs {
  int N = 0, C = 0;
  int64_t cols = 0;
  int emax = 0;                     // largest |E| solved (system (emax+1)^2)
  int64_t sys_stride = 0;           // doubles per column in sys
  double delta = 0.0, tol = 1e-9;
  const int* nv = nullptr;          // G valid rows
  const int* cnv = nullptr;         // per column loss normaliser
  const double* lam = nullptr;      // per column lambda
  const double* ylab = nullptr;     // G x N labels
  const double* K = nullptr;        // G x N x N observation-space Gram (row-major)
  const double* ftrain = nullptr;   // cols x N: K alpha of the smoothed solution
  const double* beta = nullptr;     // cols: smoothed intercepts
  int32_t* state = nullptr;         // cols x N: 0 L, 1 E, 2 R, 3 padding
  int32_t* elist = nullptr;         // cols x N: E rows in index order
  int* ne = nullptr;                // cols: |E|
  double* wl = nullptr;             // cols x N: y_j [j in L]
  double* fl = nullptr;             // cols x N: K wl
  double* sumyl = nullptr;          // cols: sum_L y_j
  double* sys = nullptr;            // cols x sys_stride
  double* alpha = nullptr;          // cols x N: candidate alpha
  double* fx = nullptr;             // cols x N: K alpha
  double* beta_x = nullptr;         // cols: candidate beta
  int* xflag = nullptr;             // cols: 0 open, 1 settled, -1 beyond emax, -2 singular
  int* pending = nullptr;           // 1 int: columns still open after a check
};
int exact_init(hipStream_t s, const ExactArgs& x);
int exact_sets(hipStream_t s, const ExactArgs& x);
int exact_solve(hipStream_t s, const ExactArgs& x);
int exact_check(hipStream_t s, const ExactArgs& x);
int exact_commit(hipStream_t s, const ExactArgs& x, double* alpha_loc, double* ftrain,
                 double* beta);

// Finalize: alpha_loc = Q ahat (zmat reused), training predictions
// f = K_v alpha + beta with K_v built again from X on the matrix cores (the
// objective is evaluated in observation space), held-out predictions
// K[H_v, T_v] alpha + beta likewise, objective/CV sums, scatter of alpha,
// counts of cells that hit max_iter or went non-finite.
struct FinalArgs {
  int n = 0, d = 0; int64_t ldx = 0;
  const double* X = nullptr; const double* nrm = nullptr; const double* y = nullptr;
  const int32_t* fold = nullptr;   // n fold ids (device)
  const int32_t* tidx = nullptr;   // V x N training indices (-1 pad)
  const int32_t* hidx = nullptr;   // V x Mh held-out indices (-1 pad)
  int Mh = 0;                      // padded held-out rows per fold (<= N)
  int V = 0, S_b = 0, Qt = 1, L = 0, s0 = 0, S = 0;
  const double* inv2s2 = nullptr;  // S_b bandwidth factors of this batch
  double delta = 1.0;
  double* kh = nullptr;            // G x N x N: training, then held-out kernel blocks (ld N)
  double* ftrain = nullptr;        // G x C x N training predictions (without beta)
  double* fbuf = nullptr;          // G x C x Mh held-out predictions (without beta)
  // outputs (full arrays, cell ((s*Q+q)*V+v)*L+l)
  double* alpha = nullptr; double* beta_out = nullptr; double* objective = nullptr;
  double* cv_sum = nullptr; int32_t* cv_err = nullptr; int32_t* iters = nullptr;
  int32_t* status = nullptr;
  int* stat_count = nullptr;       // 3 ints, accumulated: cells at max_iter, non-finite
                                   // cells, cells whose exact hinge solution was not reached
  bool shared = false;             // shared-factor mode (one group per bandwidth, all n rows)
  bool exact = false;              // recover the exact hinge SVM (objective: eq. (kernelsvm))
  ExactArgs ex;                    // its buffers (ex.cols > 0 when exact)
  int exact_rounds = 128;          // active-set rounds at most
  int* pending_host = nullptr;     // pinned int for the per-round count
};
int path_finalize(hipStream_t s, const PathArrays& p, const FinalArgs& f);

// Gather labels y[tidx] per fold into G groups (S_b copies over bandwidths).
int gather_labels(hipStream_t s, const double* y, const int32_t* tidx, int V, int S_b, int N,
                  double* ylab);

}  // namespace kmp
