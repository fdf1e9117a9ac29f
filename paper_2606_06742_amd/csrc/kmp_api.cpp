// Host driver and C ABI of the kmpath library (see include/kmpath.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "kmp_common.h"
#include "kmp_kernels.h"
#include "kmpath.h"

namespace kmp {

static thread_local std::string g_err;
void set_error(const std::string& msg) { g_err = msg; }
const char* last_error() { return g_err.c_str(); }

// Ridge point of the device: fp64 matrix peak over HBM peak (78.6 TFLOP/s,
// 8 TB/s). A launch whose algorithmic flops per byte exceed it is bound by
// the matrix cores, otherwise by memory bandwidth.
constexpr double kRidgeFlopPerByte = 78.6e12 / 8.0e12;

// Event brackets around selected launches; events come from a per-thread
// pool that lives as long as the thread and is reused by every call.
struct KernelClock {
  uint32_t mask = 0;
  int every = 1;
  int64_t seen[KMP_NKC] = {0};
  struct Rec {
    int cls;
    size_t ia, ib;
    double bytes, flops;
  };
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<Rec> recs;
  int open_cls = -1;
  size_t open_ev = 0;
  bool failed = false;
  hipEvent_t* next(size_t* idx) {
    if (used == pool.size()) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) {
        failed = true;
        return nullptr;
      }
      pool.push_back(e);
    }
    *idx = used;
    return &pool[used++];
  }
};
static thread_local KernelClock g_clock_obj;
static thread_local KernelClock* g_clock = nullptr;
KernelClock* current_clock() { return g_clock; }

void kc_begin(int cls, hipStream_t s) {
  KernelClock* c = g_clock;
  if (!c || !((c->mask >> cls) & 1u) || c->failed) return;
  if ((c->seen[cls]++) % c->every != 0) return;    // not sampled
  size_t ia;
  hipEvent_t* e = c->next(&ia);
  if (!e || hipEventRecord(*e, s) != hipSuccess) { c->failed = true; return; }
  c->open_cls = cls;
  c->open_ev = ia;
}

void kc_end(int cls, hipStream_t s, double bytes, double flops) {
  KernelClock* c = g_clock;
  if (!c || !((c->mask >> cls) & 1u) || c->failed || c->open_cls != cls) return;
  size_t ib;
  hipEvent_t* e = c->next(&ib);
  if (!e || hipEventRecord(*e, s) != hipSuccess) { c->failed = true; return; }
  c->recs.push_back({cls, c->open_ev, ib, bytes, flops});
  c->open_cls = -1;
}

// Iterations between two polls captured as one HIP graph. Orders up to
// kGraphMaxOrder are launch-bound (five launches of a few microseconds of
// work per iteration); their poll_every iterations are recorded once per
// smoothing stage and replayed. The recorded grids cover every column (the
// split-K factor too), since the kernels skip converged columns on the
// device; no timing events and no memory fills are recorded.
constexpr int kGraphMaxOrder = 2048;
constexpr int kGraphMaxIters = 64;

struct IterGraph {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  IterGraph() = default;
  IterGraph(const IterGraph&) = delete;
  IterGraph& operator=(const IterGraph&) = delete;
  ~IterGraph() {
    if (exec) (void)hipGraphExecDestroy(exec);
    if (graph) (void)hipGraphDestroy(graph);
  }
};

// The graph is recorded on a stream of its own (the caller's stream may be
// the null stream, which cannot record) and launched on the caller's; one
// per thread and device, created on first use, at the default priority.
static int capture_stream(hipStream_t* out) {
  int dev = 0;
  KMP_HIP_TRY(hipGetDevice(&dev));
  static thread_local std::map<int, hipStream_t> streams;
  auto it = streams.find(dev);
  if (it == streams.end()) {
    hipStream_t st = nullptr;
    KMP_HIP_TRY(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
    it = streams.emplace(dev, st).first;
  }
  *out = it->second;
  return 0;
}

static int capture_iterations(const PathArrays& pa, double delta, double kappa, double tol,
                              int max_iter, int restart, int count, IterGraph* out) {
  hipStream_t cs = nullptr;
  int rc = capture_stream(&cs);
  if (rc != 0) return rc;
  PathArrays pg = pa;
  pg.nact_host = nullptr;
  KernelClock* saved = g_clock;
  g_clock = nullptr;
  KMP_HIP_TRY(hipStreamBeginCapture(cs, hipStreamCaptureModeRelaxed));
  for (int k = 0; k < count && rc == 0; ++k)
    rc = path_iteration(cs, pg, delta, kappa, tol, max_iter, restart);
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(cs, &g);
  g_clock = saved;
  if (rc != 0 || e != hipSuccess) {
    if (g) (void)hipGraphDestroy(g);
    if (rc == 0) {
      set_error(std::string("hipStreamEndCapture: ") + hipGetErrorString(e));
      rc = KMP_EHIP;
    }
    return rc;
  }
  out->graph = g;
  KMP_HIP_TRY(hipGraphInstantiate(&out->exec, g, nullptr, nullptr, 0));
  return 0;
}

namespace {

// Device scratch of the allocation-free Gram entry point: the bandwidth
// factors (8 doubles) and the squared row norms of X (up to
// kStaticScratchDoubles - 8 rows). Each device holds its own copy for the
// life of the process; host code reaches it only through the address
// hipGetSymbolAddress returns on that device (static_scratch below).
constexpr size_t kStaticScratchDoubles = (size_t)1 << 16;   // 512 KiB
static __device__ __align__(256) double scratch[kStaticScratchDoubles];

int static_scratch(double** out) {
  int dev = 0;
  KMP_HIP_TRY(hipGetDevice(&dev));
  static std::mutex mu;
  static std::map<int, double*> ptrs;
  std::lock_guard<std::mutex> lk(mu);
  auto it = ptrs.find(dev);
  if (it == ptrs.end()) {
    void* p = nullptr;
    KMP_HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) {
      set_error("static scratch has no device address");
      return KMP_EHIP;
    }
    it = ptrs.emplace(dev, static_cast<double*>(p)).first;
  }
  *out = it->second;
  return 0;
}

// A second stream per device for work that can run beside the caller's
// stream (joined back through events); created on first use and kept for
// the life of the process, at the default priority.
int side_stream(hipStream_t* out) {
  int dev = 0;
  KMP_HIP_TRY(hipGetDevice(&dev));
  static std::mutex mu;
  static std::map<int, hipStream_t> streams;
  std::lock_guard<std::mutex> lk(mu);
  auto it = streams.find(dev);
  if (it == streams.end()) {
    hipStream_t st = nullptr;
    KMP_HIP_TRY(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
    it = streams.emplace(dev, st).first;
  }
  *out = it->second;
  return 0;
}

// Host-side resources every call on a device reuses: pinned staging memory
// for the small transfers (grown on demand) and events. Kept per thread and
// device for the life of the thread and never freed (the runtime may be
// gone when a thread ends). A call that returns before its stream has
// drained leaves the context dirty; the next call then waits for the device
// before it reuses the staging memory.
struct CallCtx {
  char* pin = nullptr;
  size_t pin_cap = 0;
  bool dirty = false;
  hipEvent_t ev_check = nullptr, ev_poll = nullptr, ev_band = nullptr, ev_fact = nullptr;
  std::vector<hipEvent_t> timing;    // pool of timing events (EventTimer)
};
int call_ctx(size_t pin_bytes, CallCtx** out) {
  int dev = 0;
  KMP_HIP_TRY(hipGetDevice(&dev));
  static thread_local std::map<int, CallCtx> ctxs;
  CallCtx& c = ctxs[dev];
  if (!c.ev_check) {
    for (hipEvent_t* e : {&c.ev_check, &c.ev_poll, &c.ev_band, &c.ev_fact})
      KMP_HIP_TRY(hipEventCreateWithFlags(e, hipEventDisableTiming));
  }
  if (c.dirty) {
    KMP_HIP_TRY(hipDeviceSynchronize());
    c.dirty = false;
  }
  if (pin_bytes > c.pin_cap) {
    if (c.pin) KMP_HIP_TRY(hipHostFree(c.pin));
    c.pin = nullptr;
    c.pin_cap = 0;
    const size_t cap = std::max<size_t>(pin_bytes, 1 << 20);
    KMP_HIP_TRY(hipHostMalloc((void**)&c.pin, cap, hipHostMallocDefault));
    c.pin_cap = cap;
  }
  *out = &c;
  return 0;
}

// Consecutive 64-byte aligned pieces of a staging buffer.
struct Bump {
  char* base = nullptr;
  size_t off = 0;
  static size_t round(size_t b) { return (b + 63) & ~(size_t)63; }
  template <typename T>
  T* take(size_t count) {
    T* r = reinterpret_cast<T*>(base + off);
    off += round(count * sizeof(T));
    return r;
  }
};

constexpr int kPanel = 32;       // Householder panel width
constexpr int64_t kMaxColumns = 65535;  // columns (groups x columns per group) per batch
// Exact hinge recovery: the largest margin set a column's system holds, and
// the doubles of that system (square matrix and right-hand side).
inline int exact_emax(int N) { return std::min(N, 384); }
inline int64_t exact_sys_doubles(int N) {
  const int64_t m = exact_emax(N) + 1;
  return m * m + m;
}
constexpr int kRowAlign = 64;    // padding of the per-fold matrix order
constexpr size_t kAlign = 256;

struct Plan {
  int64_t n = 0, d = 0;
  int V = 0, S = 0, Qt = 1, L = 0, Sb = 0;
  int N = 0, C = 0, G = 0, RT = 0;
  int Mh = 0;                    // held-out rows per fold, padded (max m_v rounded up to 64)
  bool shared = false;           // one factor of the full K per bandwidth (exact-CV form)
  bool exact = false;            // exact hinge recovery after the stages
  int nblk = 0;                  // row lists (groups per bandwidth): V, or 1 when shared
  std::vector<int> nv;           // per fold
  size_t bytes = 0;
};

struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + kAlign - 1) / kAlign * kAlign;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

// Workspace layout for one bandwidth batch (G = Sb * V groups). Used both to
// size and to carve, so the two can never disagree.
struct Layout {
  double *A, *Qm, *diag, *off, *tau, *cvec, *ylab, *panel, *dots, *tmat, *gram, *xbuf, *ybuf;
  double *spart, *pnext, *band, *bpart, *gram_all, *tmat_all, *cross_all, *xpart;
  double *ahat, *abar, *zmat, *anew, *estep, *ldl_l, *ldl_d, *vhat, *uvec, *partial, *fpart, *zpart;
  double *ldl_lr, *ldl_dr, *twist, *band_rev;
  double *beta, *bbar, *rmom, *gcoef, *kkt, *lam, *taucol, *fbuf, *nrm, *inv2s2;
  int *flag, *iters, *iters_total, *active, *nvg, *chk, *cmap, *nact, *stat_count, *cnv;
  int32_t *tidx, *hidx, *fold, *rfold, *cfold;
  // exact hinge recovery (only with KMP_FLAG_EXACT_HINGE)
  int32_t *ex_state, *ex_elist;
  int *ex_ne, *ex_flag, *ex_pending;
  double *ex_sumyl, *ex_beta, *ex_sys;
};

size_t carve(const Plan& p, void* ws, Layout* out) {
  Carver c(ws);
  Layout l{};
  const size_t G = (size_t)p.G, N = (size_t)p.N, C = (size_t)p.C, cols = G * C;
  l.A = c.take<double>(G * N * N);
  l.Qm = c.take<double>(G * N * N);
  l.diag = c.take<double>(G * N);
  l.off = c.take<double>(G * N);
  l.tau = c.take<double>(G * N);
  l.cvec = c.take<double>(G * N);
  l.ylab = c.take<double>(G * N);
  l.panel = c.take<double>(G * 3 * kPanel * N);
  l.dots = c.take<double>(G * 2 * kPanel);
  l.tmat = c.take<double>(G * kWyBlock * kWyBlock);
  l.gram = c.take<double>(G * kWyBlock * kWyBlock);
  l.xbuf = c.take<double>(G * kWyBlock * N);
  l.ybuf = c.take<double>(G * kWyQuad * kWyBlock * N);
  l.spart = c.take<double>(G * (size_t)tridiag_parts((int)N));
  l.pnext = c.take<double>(G * N);
  l.band = c.take<double>(G * (kBand + 1) * N);
  l.bpart = c.take<double>(band_part_doubles((int)G, (int)N));
  l.gram_all = c.take<double>(wy_all_doubles((int)G, (int)N));
  l.tmat_all = c.take<double>(wy_all_doubles((int)G, (int)N));
  l.cross_all = c.take<double>((kWyQuad - 1) * wy_all_doubles((int)G, (int)N));
  l.xpart = c.take<double>((size_t)kMaxSplitK * G * kWyQuad * kWyBlock * N);
  l.ahat = c.take<double>(cols * N);
  l.abar = c.take<double>(cols * N);
  l.zmat = c.take<double>(cols * N);
  l.anew = c.take<double>(cols * N);
  l.estep = c.take<double>(cols * N);
  l.ldl_l = c.take<double>(cols * kBand * N);
  l.ldl_d = c.take<double>(cols * N);
  l.ldl_lr = c.take<double>(cols * kBand * N);
  l.ldl_dr = c.take<double>(cols * N);
  l.twist = c.take<double>(cols * (kBand * kBand + kBand));
  l.band_rev = c.take<double>(G * (kBand + 1) * N);
  l.vhat = c.take<double>(cols * N);
  l.uvec = c.take<double>(cols * N);
  l.partial = c.take<double>(G * (size_t)p.RT * C);
  l.fpart = c.take<double>((size_t)kMaxSplitK * cols * N);
  l.zpart = c.take<double>((size_t)kMaxSplitK * cols * N);
  l.beta = c.take<double>(cols);
  l.bbar = c.take<double>(cols);
  l.rmom = c.take<double>(cols);
  l.gcoef = c.take<double>(cols);
  l.kkt = c.take<double>(cols);
  l.lam = c.take<double>(cols);
  l.taucol = c.take<double>(cols);
  l.fbuf = c.take<double>(cols * (size_t)p.Mh);
  l.nrm = c.take<double>((size_t)p.n);
  l.inv2s2 = c.take<double>((size_t)std::max(p.S, 1));
  l.flag = c.take<int>(cols);
  l.iters = c.take<int>(cols);
  l.iters_total = c.take<int>(cols);
  l.active = c.take<int>(1);
  l.cmap = c.take<int>(cols);
  l.nact = c.take<int>(G);
  l.chk = c.take<int>(2);
  l.stat_count = c.take<int>(3);
  l.nvg = c.take<int>(G);
  l.cnv = c.take<int>(cols);
  l.cfold = c.take<int32_t>(cols);
  l.rfold = c.take<int32_t>(p.shared ? G * N : 0);
  const size_t xc = p.exact ? cols : 0;
  l.ex_state = c.take<int32_t>(xc * N);
  l.ex_elist = c.take<int32_t>(xc * N);
  l.ex_ne = c.take<int>(xc);
  l.ex_flag = c.take<int>(xc);
  l.ex_pending = c.take<int>(p.exact ? 1 : 0);
  l.ex_sumyl = c.take<double>(xc);
  l.ex_beta = c.take<double>(xc);
  l.ex_sys = c.take<double>(xc * (size_t)exact_sys_doubles(p.N));
  l.tidx = c.take<int32_t>((size_t)p.nblk * N);
  l.hidx = c.take<int32_t>((size_t)p.V * p.Mh);
  l.fold = c.take<int32_t>((size_t)p.n);
  if (out) *out = l;
  return c.off + kAlign;
}

int make_plan(const kmp_path_spec* spec, int64_t n, int64_t d, int32_t L, const int32_t* fold,
              int32_t V, int32_t S, int32_t Qn, int32_t Sb, Plan* p) {
  // a refit is one "fold" whose held-out set is empty: V = 1, no fold ids
  const bool refit = spec && (spec->flags & KMP_FLAG_REFIT) != 0;
  const bool shared = spec && (spec->flags & KMP_FLAG_SHARED_FACTOR) != 0;
  if (!spec || n < 2 || d < 1 || L < 1 || S < 1 || Qn < 1 ||
      (refit ? V != 1 : (V < 2 || V > n || !fold))) {
    set_error(refit ? "invalid shape arguments (a full-data refit takes V = 1)"
                    : "invalid shape arguments");
    return KMP_EINVAL;
  }
  if (refit && shared) {
    set_error("a full-data refit has no folds to share a factor between");
    return KMP_EINVAL;
  }
  const bool exact = spec && (spec->flags & KMP_FLAG_EXACT_HINGE) != 0;
  if (exact && (spec->loss != KMP_HINGE || shared)) {
    set_error("the exact hinge recovery needs the hinge loss and per-fold factors");
    return KMP_EINVAL;
  }
  p->exact = exact;
  if (spec->loss != KMP_CHECK && Qn != 1) {
    set_error("Q must be 1 for the margin losses");
    return KMP_EINVAL;
  }
  p->n = n; p->d = d; p->V = V; p->S = S; p->Qt = Qn; p->L = L;
  p->nv.assign(V, 0);
  std::vector<int64_t> m(V, 0);
  for (int64_t i = 0; i < n && !refit; ++i) {
    const int32_t f = fold[i];
    if (f < 0 || f >= V) {
      set_error("fold id out of range at index " + std::to_string(i));
      return KMP_EFOLD;
    }
    m[f] += 1;
  }
  int maxnv = 0;
  int64_t maxm = 0;
  for (int v = 0; v < V; ++v) {
    if (m[v] == 0 && !refit) {
      set_error("fold " + std::to_string(v) + " is empty");
      return KMP_EFOLD;
    }
    p->nv[v] = (int)(n - m[v]);
    maxnv = std::max(maxnv, p->nv[v]);
    maxm = std::max(maxm, m[v]);
  }
  p->shared = shared;
  p->Sb = std::max(1, std::min<int>(Sb, S));
  if (shared) {
    // every point is a row of the one factor per bandwidth; a column is a
    // (tau, fold, lambda) problem whose held-out rows carry no loss
    p->N = (int)round_up(n, kRowAlign);
    p->Mh = 0;
    p->nblk = 1;
    p->C = Qn * V * L;
    p->G = p->Sb;
  } else {
    p->N = (int)round_up(maxnv, kRowAlign);
    // a fold's held-out set is no larger than any other fold's training
    // set, so the padded held-out block fits in the N x N factor buffer
    p->Mh = (int)round_up(maxm, kRowAlign);
    p->nblk = V;
    p->C = Qn * L;
    p->G = p->Sb * V;
  }
  if (p->N > (shared ? kMaxSharedOrder : kMaxOrder)) {
    set_error(shared ? "more than " + std::to_string(kMaxSharedOrder) +
                           " points for the shared factor"
                     : "more than " + std::to_string(kMaxOrder) + " training points per fold");
    return KMP_EINVAL;
  }
  // columns of a batch run along grid dimension y in some launches
  if ((int64_t)p->G * p->C > kMaxColumns) {
    set_error("more than " + std::to_string(kMaxColumns) +
              " (sigma, tau, fold, lambda) columns in one bandwidth batch");
    return KMP_EINVAL;
  }
  p->RT = (int)ceil_div(p->N, kMinTileRows);
  p->bytes = carve(*p, nullptr, nullptr);
  return 0;
}

// Phase times from HIP events: mark() records an event on the stream (a
// pool that grows as needed), span() notes a pair whose elapsed time is
// added to a total when sum() runs after the final synchronisation, so the
// host never waits on the device to read a phase time.
struct EventTimer {
  std::vector<hipEvent_t>& ev;    // pool, grown on demand and reused
  size_t used = 0;
  struct Span {
    double* acc;
    size_t a, b;
  };
  std::vector<Span> spans;
  explicit EventTimer(std::vector<hipEvent_t>& pool) : ev(pool) {}
  int mark(hipStream_t s, size_t* idx) {
    if (used == ev.size()) {
      hipEvent_t e;
      KMP_HIP_TRY(hipEventCreate(&e));
      ev.push_back(e);
    }
    *idx = used;
    KMP_HIP_TRY(hipEventRecord(ev[used++], s));
    return 0;
  }
  void span(double* acc, size_t a, size_t b) { spans.push_back({acc, a, b}); }
  void sum() {
    for (const auto& sp : spans) {
      float t = 0.f;
      if (hipEventElapsedTime(&t, ev[sp.a], ev[sp.b]) == hipSuccess) *sp.acc += t;
    }
    spans.clear();
  }
};

// The band reduction's buffers inside a carved workspace.
BandWork band_work_of(const Layout& lay, int G, int N, const int* nv_host) {
  BandWork bw;
  bw.G = G; bw.N = N; bw.A = lay.A; bw.Q = lay.Qm; bw.band = lay.band; bw.tau = lay.tau;
  static_assert(kPanel >= 2 * kBand, "two band panel buffers share the panel slot");
  bw.panel = lay.panel; bw.panel2 = lay.panel + (size_t)G * 3 * kBand * N;
  bw.tmat = lay.tmat; bw.gram = lay.gram; bw.xbuf = lay.xbuf;
  bw.ybuf = lay.ybuf; bw.part = lay.bpart; bw.nv_host = nv_host;
  bw.gram_all = lay.gram_all; bw.tmat_all = lay.tmat_all; bw.cross_all = lay.cross_all;
  bw.xpart = lay.xpart;
  return bw;
}

// The path solver's arrays inside a carved workspace.
PathArrays path_arrays_of(const Layout& lay, const Plan& plan, int loss, bool global_solve) {
  PathArrays pa;
  pa.N = plan.N; pa.C = plan.C; pa.loss = loss;
  pa.global_solve = global_solve;
  pa.nv = lay.nvg; pa.ylab = lay.ylab; pa.Q = lay.Qm; pa.band = lay.band;
  pa.cvec = lay.cvec; pa.lam = lay.lam; pa.tau = lay.taucol;
  pa.ahat = lay.ahat; pa.abar = lay.abar; pa.zmat = lay.zmat;
  pa.QB = lay.A;             // the factorisation's buffer, free once Q is formed
  pa.anew = lay.anew; pa.estep = lay.estep; pa.ldl_l = lay.ldl_l; pa.ldl_d = lay.ldl_d;
  pa.ldl_lr = lay.ldl_lr; pa.ldl_dr = lay.ldl_dr; pa.twist = lay.twist; pa.band_rev = lay.band_rev;
  pa.vhat = lay.vhat;
  pa.uvec = lay.uvec; pa.partial = lay.partial; pa.beta = lay.beta; pa.bbar = lay.bbar;
  pa.fpart = lay.fpart; pa.zpart = lay.zpart;
  pa.rmom = lay.rmom; pa.gcoef = lay.gcoef; pa.kkt = lay.kkt;
  pa.flag = lay.flag;
  pa.iters = lay.iters; pa.iters_total = lay.iters_total; pa.active_count = lay.active;
  pa.cmap = lay.cmap; pa.nact = lay.nact;
  pa.cnv = lay.cnv;
  pa.rfold = plan.shared ? lay.rfold : nullptr;
  pa.cfold = plan.shared ? lay.cfold : nullptr;
  return pa;
}

}  // namespace
}  // namespace kmp

using namespace kmp;

extern "C" {

void kmp_default_spec(kmp_path_spec* s) {
  if (!s) return;
  s->loss = KMP_HINGE;
  s->delta0 = 1.0;
  s->eta = 0.125;
  s->n_stages = 3;
  s->tol = 1e-9;
  s->max_iter = 100000;
  s->poll_every = 8;
  s->flags = KMP_FLAG_RESTART;
  s->timing_mask = 0;
  s->timing_every = 1;
}

const char* kmp_kernel_class_name(int cls) {
  static const char* names[KMP_NKC] = {"gram",        "panel",  "panel_wy", "trail_update",
                                       "q_form",      "precompute", "gemm_f", "gemm_zhat",
                                       "update",      "finalize"};
  return (cls >= 0 && cls < KMP_NKC) ? names[cls] : "";
}

const char* kmp_version(void) { return "kmpath 0.1 (gfx950, fp64)"; }

const char* kmp_strerror(int code) {
  switch (code) {
    case KMP_OK: return "ok";
    case KMP_WMAXITER: return "finished; some cells stopped at max_iter";
    case KMP_EINVAL: return g_err.empty() ? "invalid argument" : g_err.c_str();
    case KMP_EFOLD: return g_err.empty() ? "invalid fold assignment" : g_err.c_str();
    case KMP_EWORKSPACE: return g_err.empty() ? "workspace missing or too small" : g_err.c_str();
    case KMP_EHIP: return g_err.empty() ? "HIP runtime error" : g_err.c_str();
    case KMP_ENONFINITE: return g_err.empty() ? "non-finite input" : g_err.c_str();
    default: return "unknown code";
  }
}

int kmp_make_folds(int64_t n, int32_t V, uint64_t seed, int32_t* fold_id) {
  if (n <= 0 || V <= 0 || !fold_id) {
    set_error("kmp_make_folds: n, V must be positive and fold_id non-null");
    return KMP_EINVAL;
  }
  std::vector<int64_t> perm(n);
  for (int64_t i = 0; i < n; ++i) perm[i] = i;
  uint64_t st = seed;
  for (int64_t i = n - 1; i >= 1; --i) {
    st += 0x9E3779B97F4A7C15ULL;
    uint64_t z = st;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    z ^= z >> 31;
    const int64_t j = (int64_t)(((unsigned __int128)z * (unsigned __int128)(i + 1)) >> 64);
    std::swap(perm[i], perm[j]);
  }
  for (int64_t i = 0; i < n; ++i) fold_id[perm[i]] = (int32_t)(i % V);
  return KMP_OK;
}

size_t kmp_workspace_bytes(const kmp_path_spec* spec, int64_t n, int64_t d, int32_t L,
                           const int32_t* fold_id, int32_t V, int32_t S, int32_t Q,
                           int32_t sigma_batch) {
  Plan p;
  if (sigma_batch < 1 || sigma_batch > S) return 0;
  if (make_plan(spec, n, d, L, fold_id, V, S, Q, sigma_batch, &p) != 0) return 0;
  return p.bytes;
}

int kmp_rbf_gram(void* stream, const double* X, int64_t n, int64_t d, int64_t ldx,
                 const int32_t* rows, int64_t m, const int32_t* cols, int64_t p,
                 const double* sigmas, int32_t S, double* out, int64_t ld_out) {
  hipStream_t s = (hipStream_t)stream;
  if (!X || !rows || !cols || !sigmas || !out || n < 1 || d < 1 || ldx < d || m < 0 || p < 0 ||
      S < 1 || S > 8 || ld_out < p) {
    set_error("kmp_rbf_gram: invalid arguments");
    return KMP_EINVAL;
  }
  std::vector<double> f2(S);
  for (int i = 0; i < S; ++i) {
    if (!(sigmas[i] > 0.0) || !std::isfinite(sigmas[i])) {
      set_error("kmp_rbf_gram: sigma must be positive");
      return KMP_EINVAL;
    }
    f2[i] = 1.0 / (2.0 * sigmas[i] * sigmas[i]);
  }
  if (m == 0 || p == 0) return KMP_OK;
  double *nrm = nullptr, *dinv = nullptr;
  KMP_HIP_TRY(hipMallocAsync((void**)&nrm, sizeof(double) * n, s));
  KMP_HIP_TRY(hipMallocAsync((void**)&dinv, sizeof(double) * S, s));
  KMP_HIP_TRY(hipMemcpyAsync(dinv, f2.data(), sizeof(double) * S, hipMemcpyHostToDevice, s));
  int rc = row_norms(s, X, n, d, ldx, nrm);
  if (rc == 0)
    rc = rbf_blocks(s, X, d, ldx, nrm, rows, 0, m, cols, 0, p, 1, dinv, S, out, m * ld_out, 0,
                    ld_out);
  KMP_HIP_TRY(hipFreeAsync(nrm, s));
  KMP_HIP_TRY(hipFreeAsync(dinv, s));
  KMP_HIP_TRY(hipStreamSynchronize(s));
  return rc;
}

int kmp_rbf_gram_noalloc(void* stream, const double* X, int64_t n, int64_t d, int64_t ldx,
                         const int32_t* rows, int64_t m, const int32_t* cols, int64_t p,
                         const double* sigmas, int32_t S, double* out, int64_t ld_out) {
  hipStream_t s = (hipStream_t)stream;
  if (!X || !rows || !cols || !sigmas || !out || n < 1 || d < 1 || ldx < d || m < 0 || p < 0 ||
      S < 1 || S > 8 || ld_out < p) {
    set_error("kmp_rbf_gram_noalloc: invalid arguments");
    return KMP_EINVAL;
  }
  if ((size_t)n > kStaticScratchDoubles - 8) {
    set_error("kmp_rbf_gram_noalloc: n = " + std::to_string(n) + " above the " +
              std::to_string(kStaticScratchDoubles - 8) + " rows its static scratch holds");
    return KMP_EINVAL;
  }
  double f2[8];
  for (int i = 0; i < S; ++i) {
    if (!(sigmas[i] > 0.0) || !std::isfinite(sigmas[i])) {
      set_error("kmp_rbf_gram_noalloc: sigma must be positive");
      return KMP_EINVAL;
    }
    f2[i] = 1.0 / (2.0 * sigmas[i] * sigmas[i]);
  }
  if (m == 0 || p == 0) return KMP_OK;
  double* sc = nullptr;
  int rc = static_scratch(&sc);
  if (rc != 0) return rc;
  double* dinv = sc;          // S bandwidth factors
  double* nrm = sc + 8;       // n squared row norms
  if ((rc = store_small(s, f2, S, dinv)) != 0) return rc;
  if ((rc = row_norms(s, X, n, d, ldx, nrm)) != 0) return rc;
  if ((rc = rbf_blocks(s, X, d, ldx, nrm, rows, 0, m, cols, 0, p, 1, dinv, S, out, m * ld_out, 0,
                       ld_out)) != 0)
    return rc;
  KMP_HIP_TRY(hipStreamSynchronize(s));
  return KMP_OK;
}

int kmp_tridiag(void* stream, double* A, int32_t G, int32_t N, double* Qout, double* diag,
                double* off) {
  hipStream_t s = (hipStream_t)stream;
  if (!A || !Qout || !diag || !off || G < 1 || N < 1 || N % kPanel != 0) {
    set_error("kmp_tridiag: invalid arguments (N must be a positive multiple of 32)");
    return KMP_EINVAL;
  }
  TridiagWork w;
  w.G = G; w.N = N; w.nb = kPanel; w.A = A; w.Q = Qout; w.diag = diag; w.off = off;
  double* scratch = nullptr;
  const size_t extra = tridiag_panel_doubles(G, N, kPanel) + (size_t)G * N;
  KMP_HIP_TRY(hipMallocAsync((void**)&scratch, sizeof(double) * extra, s));
  double* q = scratch;
  w.tau = q; q += (size_t)G * N;
  w.panel = q; q += (size_t)G * 3 * kPanel * N;
  w.dots = q; q += (size_t)G * 2 * kPanel;
  w.tmat = q; q += (size_t)G * kWyBlock * kWyBlock;
  w.gram = q; q += (size_t)G * kWyBlock * kWyBlock;
  w.xbuf = q; q += (size_t)G * kWyBlock * N;
  w.ybuf = q; q += (size_t)G * kWyBlock * N;
  w.spart = q; q += (size_t)G * tridiag_parts(N);
  w.pnext = q;
  int rc = tridiagonalize(s, w);
  KMP_HIP_TRY(hipFreeAsync(scratch, s));
  KMP_HIP_TRY(hipStreamSynchronize(s));
  return rc;
}

int kmp_band_reduce(void* stream, double* A, int32_t G, int32_t N, double* Qout, double* band) {
  hipStream_t s = (hipStream_t)stream;
  static_assert(KMP_BAND == kBand, "band width of the header and the kernels differ");
  if (!A || !Qout || !band || G < 1 || N < 64 || N > kMaxOrder || N % 64 != 0) {
    set_error("kmp_band_reduce: invalid arguments (N must be a multiple of 64 in [64, " +
              std::to_string(kMaxOrder) + "])");
    return KMP_EINVAL;
  }
  BandWork w;
  w.G = G; w.N = N; w.A = A; w.Q = Qout; w.band = band;
  double* scratch = nullptr;
  const size_t extra = band_work_doubles(G, N) + (size_t)G * N;
  KMP_HIP_TRY(hipMallocAsync((void**)&scratch, sizeof(double) * extra, s));
  double* q = scratch;
  w.tau = q; q += (size_t)G * N;
  w.panel = q; q += (size_t)G * 3 * kBand * N;
  w.panel2 = q; q += (size_t)G * 3 * kBand * N;
  w.tmat = q; q += (size_t)G * kWyBlock * kWyBlock;
  w.gram = q; q += (size_t)G * kWyBlock * kWyBlock;
  w.xbuf = q; q += (size_t)G * kWyBlock * N;
  w.ybuf = q; q += (size_t)G * kWyQuad * kWyBlock * N;
  w.gram_all = q; q += wy_all_doubles(G, N);
  w.tmat_all = q; q += wy_all_doubles(G, N);
  w.cross_all = q; q += (kWyQuad - 1) * wy_all_doubles(G, N);
  w.xpart = q; q += (size_t)kMaxSplitK * G * kWyQuad * kWyBlock * N;
  w.part = q;
  int rc = band_reduce(s, w);
  KMP_HIP_TRY(hipFreeAsync(scratch, s));
  KMP_HIP_TRY(hipStreamSynchronize(s));
  return rc;
}

int kmp_fit_path(void* stream, const kmp_path_spec* spec, const double* X, int64_t n, int64_t d,
                 int64_t ldx, const double* y, const double* sigmas, int32_t S, const double* taus,
                 int32_t Qn, const double* lambdas, int32_t L, const int32_t* fold_id, int32_t V,
                 void* workspace, size_t workspace_bytes, double* alpha, double* beta,
                 double* objective, double* cv_sum, int32_t* cv_err, int32_t* iters,
                 int32_t* status, int32_t* selected, int32_t* selected_joint,
                 kmp_timings* timings) {
  hipStream_t s = (hipStream_t)stream;
  // ---------------------------------------------------------- validation
  const bool refit = spec && (spec->flags & KMP_FLAG_REFIT) != 0;
  if (!spec || !X || !y || !sigmas || !lambdas || (!fold_id && !refit) || !alpha || !beta ||
      !objective || !cv_sum) {
    set_error("null pointer argument");
    return KMP_EINVAL;
  }
  if (spec->loss < 0 || spec->loss > 2 || !(spec->tol > 0.0) || spec->max_iter < 1 ||
      spec->poll_every < 1 || (spec->loss != KMP_LOGISTIC &&
                               (!(spec->delta0 > 0.0) || !(spec->eta > 0.0 && spec->eta < 1.0) ||
                                spec->n_stages < 1))) {
    set_error("invalid solver settings");
    return KMP_EINVAL;
  }
  if (ldx < d) {
    set_error("ldx must be >= d");
    return KMP_EINVAL;
  }
  if (spec->loss == KMP_CHECK && (!taus || Qn < 1)) {
    set_error("check loss needs Q >= 1 tau values");
    return KMP_EINVAL;
  }
  for (int i = 0; i < S; ++i)
    if (!(sigmas[i] > 0.0) || !std::isfinite(sigmas[i])) {
      set_error("sigma must be positive and finite");
      return KMP_EINVAL;
    }
  for (int i = 0; i < L; ++i)
    if (!(lambdas[i] > 0.0) || !std::isfinite(lambdas[i])) {
      set_error("lambda must be positive and finite");
      return KMP_EINVAL;
    }
  if (spec->loss == KMP_CHECK)
    for (int i = 0; i < Qn; ++i)
      if (!(taus[i] > 0.0 && taus[i] < 1.0)) {
        set_error("tau must lie in (0, 1)");
        return KMP_EINVAL;
      }
  Plan plan;
  int rc = make_plan(spec, n, d, L, fold_id, V, S, Qn, 1, &plan);
  if (rc != 0) return rc;
  // largest bandwidth batch that fits the workspace
  int Sb = 0;
  for (int b = std::min(S, 8); b >= 1; --b) {   // the Gram epilogue takes <= 8 bandwidths
    Plan pb;
    if (make_plan(spec, n, d, L, fold_id, V, S, Qn, b, &pb) == 0 && pb.bytes <= workspace_bytes) {
      Sb = b;
      plan = pb;
      break;
    }
  }
  if (!workspace || Sb == 0) {
    set_error("workspace too small: need " +
              std::to_string(kmp_workspace_bytes(spec, n, d, L, fold_id, V, S, Qn, 1)) +
              " bytes for one bandwidth at a time");
    return KMP_EWORKSPACE;
  }
  Layout lay;
  carve(plan, workspace, &lay);
  const int N = plan.N, C = plan.C, G = plan.G;
  const size_t ncell = (size_t)S * Qn * V * L;
  // pinned staging for every host<->device transfer of the call
  const int nbatch = (S + Sb - 1) / Sb;
  const size_t pin_bytes =
      Bump::round(sizeof(double) * n) + Bump::round(2 * sizeof(int)) +
      Bump::round(sizeof(int32_t) * (size_t)plan.nblk * N) +
      Bump::round(sizeof(int32_t) * (size_t)V * plan.Mh) + Bump::round(sizeof(int32_t) * n) +
      Bump::round(sizeof(int) * ((size_t)G + 1)) +
      (size_t)nbatch * (Bump::round(sizeof(double) * Sb) +
                        2 * Bump::round(sizeof(double) * (size_t)G * C) +
                        2 * Bump::round(sizeof(int) * (size_t)G * C) +
                        Bump::round(sizeof(int) * (size_t)G)) +
      Bump::round(sizeof(int32_t) * (size_t)G * N) +
      Bump::round(sizeof(double) * ncell) + Bump::round(sizeof(int32_t) * ncell) +
      Bump::round(3 * sizeof(int)) + Bump::round(sizeof(int));
  CallCtx* ctx = nullptr;
  if ((rc = call_ctx(pin_bytes, &ctx)) != 0) return rc;
  Bump pin{ctx->pin, 0};
  // an early return leaves copies into the staging memory in flight
  struct DirtyGuard {
    CallCtx* c;
    bool clean = false;
    ~DirtyGuard() {
      if (!clean) c->dirty = true;
    }
  } dirty_guard{ctx};
  // Finiteness of X and y is counted on the device (two ints in the
  // workspace); y and the counts come back while the factorisation is
  // queued and are checked before anything is written to the outputs.
  if ((rc = count_nonfinite(s, X, n, d, ldx, y, lay.chk)) != 0) return rc;
  KMP_HIP_TRY(hipMemsetAsync(lay.stat_count, 0, 3 * sizeof(int), s));
  int* exact_pin = pin.take<int>(1);     // open columns after a recovery round
  double* hy = pin.take<double>(n);
  int* hchk = pin.take<int>(2);
  KMP_HIP_TRY(hipMemcpyAsync(hy, y, sizeof(double) * n, hipMemcpyDeviceToHost, s));
  KMP_HIP_TRY(hipMemcpyAsync(hchk, lay.chk, 2 * sizeof(int), hipMemcpyDeviceToHost, s));
  KMP_HIP_TRY(hipEventRecord(ctx->ev_check, s));
  const auto check_inputs = [&]() -> int {
    KMP_HIP_TRY(hipEventSynchronize(ctx->ev_check));
    if (hchk[0] != 0) {
      set_error(std::to_string(hchk[0]) + " non-finite entries in X");
      return KMP_ENONFINITE;
    }
    if (hchk[1] != 0) {
      set_error(std::to_string(hchk[1]) + " non-finite entries in y");
      return KMP_ENONFINITE;
    }
    if (spec->loss != KMP_CHECK) {
      std::vector<int64_t> pos(V, 0), neg(V, 0);   // held out per fold (none in a refit)
      int64_t tp = 0, tn = 0;
      for (int64_t i = 0; i < n; ++i) {
        if (hy[i] == 1.0) { if (!refit) pos[fold_id[i]]++; tp++; }
        else if (hy[i] == -1.0) { if (!refit) neg[fold_id[i]]++; tn++; }
        else {
          set_error("labels must be +1 or -1 for hinge and logistic losses");
          return KMP_EINVAL;
        }
      }
      for (int v = 0; v < V; ++v)
        if (tp - pos[v] == 0 || tn - neg[v] == 0) {
          set_error("training set of fold " + std::to_string(v) + " has a single class");
          return KMP_EFOLD;
        }
    }
    return 0;
  };

  const int nst = spec->loss == KMP_LOGISTIC ? 1 : spec->n_stages;
  // smoothing parameter and curvature bound of each stage
  const auto stage_delta = [&](int st) {
    return spec->loss == KMP_LOGISTIC ? 1.0 : spec->delta0 * std::pow(spec->eta, (double)st);
  };
  const auto stage_kappa = [&](int st) {
    return spec->loss == KMP_LOGISTIC ? 4.0 : 2.0 * stage_delta(st);
  };
  const double delta_final = stage_delta(nst - 1);

  // host-side index lists and per-column parameters
  // row lists: the training points of each fold, or (shared factor) every
  // point once
  const bool shared = plan.shared;
  const int NB = plan.nblk;
  int32_t* tidx = pin.take<int32_t>((size_t)NB * N);
  std::fill(tidx, tidx + (size_t)NB * N, -1);
  for (int v = 0; v < NB; ++v) {
    int k = 0;
    for (int64_t i = 0; i < n; ++i)
      if (shared || refit || fold_id[i] != v) tidx[(size_t)v * N + k++] = (int32_t)i;
  }
  KMP_HIP_TRY(hipMemcpyAsync(lay.tidx, tidx, sizeof(int32_t) * (size_t)NB * N,
                             hipMemcpyHostToDevice, s));
  int32_t* hidx = pin.take<int32_t>((size_t)V * plan.Mh);
  std::fill(hidx, hidx + (size_t)V * plan.Mh, -1);
  for (int v = 0; v < V; ++v) {
    int k = 0;
    for (int64_t i = 0; i < n; ++i)
      if (!refit && fold_id[i] == v) hidx[(size_t)v * plan.Mh + k++] = (int32_t)i;
  }
  KMP_HIP_TRY(hipMemcpyAsync(lay.hidx, hidx, sizeof(int32_t) * (size_t)V * plan.Mh,
                             hipMemcpyHostToDevice, s));
  int32_t* hfold = pin.take<int32_t>(n);
  if (refit)
    std::fill(hfold, hfold + n, -1);
  else
    std::copy(fold_id, fold_id + n, hfold);
  KMP_HIP_TRY(hipMemcpyAsync(lay.fold, hfold, sizeof(int32_t) * n, hipMemcpyHostToDevice, s));

  EventTimer tm(ctx->timing);
  double t_gram = 0, t_factor = 0, t_pre = 0, t_path = 0, t_fin = 0;
  struct ClockGuard {
    ClockGuard(uint32_t mask) {
      g_clock_obj.mask = mask;
      g_clock_obj.used = 0;
      for (auto& v : g_clock_obj.seen) v = 0;
      g_clock_obj.recs.clear();
      g_clock_obj.open_cls = -1;
      g_clock_obj.failed = false;
      g_clock = mask ? &g_clock_obj : nullptr;
    }
    ~ClockGuard() { g_clock = nullptr; }
  } clock_guard((uint32_t)spec->timing_mask);
  g_clock_obj.every = spec->timing_every > 0 ? spec->timing_every : 1;
  int64_t total_iters = 0;
  // pinned host buffer for the per-group and total active counts
  struct PollBuf {
    int* p;
    hipEvent_t ev;
  } poll{pin.take<int>((size_t)G + 1), ctx->ev_poll};
  // The first stage's factors need the band only: they are formed on a side
  // stream while the caller's stream accumulates Q, and the stage waits for
  // them. Leaving the call (also on an error) waits for the side stream.
  struct SideWork {
    hipStream_t st = nullptr;
    hipEvent_t band = nullptr, done = nullptr;
    bool queued = false;
    ~SideWork() {
      if (queued) (void)hipStreamSynchronize(st);
    }
  } side;
  if ((rc = side_stream(&side.st)) != 0) return rc;
  side.band = ctx->ev_band;
  side.done = ctx->ev_fact;
  size_t ev_start = 0, e1 = 0, e2 = 0, e3 = 0;
  if ((rc = tm.mark(s, &ev_start)) != 0) return rc;
  if ((rc = row_norms(s, X, n, d, ldx, lay.nrm)) != 0) return rc;

  PathArrays pa = path_arrays_of(lay, plan, spec->loss, (spec->flags & KMP_FLAG_GLOBAL_SOLVE) != 0);
  const bool use_graphs = (spec->flags & KMP_FLAG_EAGER) == 0 && N <= kGraphMaxOrder &&
                          spec->poll_every <= kGraphMaxIters;

  for (int s0 = 0; s0 < S; s0 += Sb) {
    const int sb = std::min(Sb, S - s0);
    const int Gb = sb * NB;
    pa.G = Gb;
    // per-batch parameters. Per fold: group g = (bandwidth, fold), column
    // c = (tau, lambda). Shared factor: group g = bandwidth, column
    // c = (tau, fold, lambda), rows held out of the column's fold carry no
    // loss, and each column keeps its fold's n_v as loss normaliser.
    double* f2 = pin.take<double>(Sb);
    double* lamc = pin.take<double>((size_t)G * C);
    double* tauc = pin.take<double>((size_t)G * C);
    int* nvg = pin.take<int>(G);
    int* cnvh = pin.take<int>((size_t)G * C);
    int32_t* cfh = pin.take<int32_t>((size_t)G * C);
    for (int i = 0; i < sb; ++i) f2[i] = 1.0 / (2.0 * sigmas[s0 + i] * sigmas[s0 + i]);
    const int cv_per_q = shared ? V * L : L;       // columns per tau level
    for (int g = 0; g < Gb; ++g) {
      nvg[g] = shared ? (int)n : plan.nv[g % V];
      for (int c = 0; c < C; ++c) {
        const int q = c / cv_per_q, r = c % cv_per_q, l = r % L;
        const int v = shared ? r / L : g % V;
        lamc[(size_t)g * C + c] = lambdas[l];
        tauc[(size_t)g * C + c] = spec->loss == KMP_CHECK ? taus[q] : 0.0;
        cnvh[(size_t)g * C + c] = plan.nv[v];
        cfh[(size_t)g * C + c] = shared ? v : -1;
      }
    }
    KMP_HIP_TRY(hipMemcpyAsync(lay.inv2s2, f2, sizeof(double) * sb, hipMemcpyHostToDevice, s));
    KMP_HIP_TRY(hipMemcpyAsync(lay.lam, lamc, sizeof(double) * (size_t)Gb * C,
                               hipMemcpyHostToDevice, s));
    KMP_HIP_TRY(hipMemcpyAsync(lay.taucol, tauc, sizeof(double) * (size_t)Gb * C,
                               hipMemcpyHostToDevice, s));
    KMP_HIP_TRY(hipMemcpyAsync(lay.nvg, nvg, sizeof(int) * Gb, hipMemcpyHostToDevice, s));
    KMP_HIP_TRY(hipMemcpyAsync(lay.cnv, cnvh, sizeof(int) * (size_t)Gb * C, hipMemcpyHostToDevice, s));
    KMP_HIP_TRY(hipMemcpyAsync(lay.cfold, cfh, sizeof(int32_t) * (size_t)Gb * C,
                               hipMemcpyHostToDevice, s));
    if (shared && s0 == 0) {
      // fold id of every row of every group (-1 at padding), the same for
      // every bandwidth; written once
      int32_t* rfh = pin.take<int32_t>((size_t)G * N);
      for (int g = 0; g < G; ++g)
        for (int i = 0; i < N; ++i) rfh[(size_t)g * N + i] = i < n ? fold_id[i] : -1;
      KMP_HIP_TRY(hipMemcpyAsync(lay.rfold, rfh, sizeof(int32_t) * (size_t)G * N,
                                 hipMemcpyHostToDevice, s));
    }
    pa.nv_host = nvg;
    // columns in each group's active list, as last read back (work counters)
    std::vector<int> nact_h(Gb, C);
    pa.nact_host = nact_h.data();

    // a1: Gram + fold gather into A (group g = s_local*V + v)
    if ((rc = tm.mark(s, &e1)) != 0) return rc;
    kc_begin(KMP_KC_GRAM, s);
    if ((rc = rbf_blocks(s, X, d, ldx, lay.nrm, lay.tidx, N, N, lay.tidx, N, N, NB, lay.inv2s2, sb,
                         lay.A, (int64_t)NB * N * N, (int64_t)N * N, N)) != 0)
      return rc;
    {
      // every kernel entry of every group is written once; the inner products
      // (2d flops each) are shared by the bandwidths of the batch
      double e2 = 0.0;
      for (int v = 0; v < NB; ++v) e2 += shared ? (double)n * n : (double)plan.nv[v] * plan.nv[v];
      kc_end(KMP_KC_GRAM, s, 8.0 * sb * e2, 2.0 * d * e2);
    }
    if ((rc = tm.mark(s, &e2)) != 0) return rc;
    // a2: factorisation
    BandWork bw = band_work_of(lay, Gb, N, nvg);
    bw.band_ready = side.band;
    if ((rc = band_reduce(s, bw)) != 0) return rc;
    if ((rc = form_qb(s, lay.Qm, lay.band, N, Gb, lay.A)) != 0) return rc;
    KMP_HIP_TRY(hipStreamWaitEvent(side.st, side.band, 0));
    side.queued = true;
    if ((rc = path_stage_factor(side.st, pa, stage_kappa(0))) != 0) return rc;
    KMP_HIP_TRY(hipEventRecord(side.done, side.st));
    if ((rc = group_ones_projection(s, lay.Qm, lay.nvg, Gb, N, lay.cvec)) != 0) return rc;
    if ((rc = gather_labels(s, y, lay.tidx, NB, sb, N, lay.ylab)) != 0) return rc;
    if ((rc = path_init_columns(s, pa)) != 0) return rc;
    if ((rc = tm.mark(s, &e3)) != 0) return rc;
    tm.span(&t_gram, e1, e2);
    tm.span(&t_factor, e2, e3);

    if (s0 == 0) {
      // the inputs' checks have long come back (the factorisation is
      // queued ahead of the device); on an error the queued work drains
      // into the workspace only
      if ((rc = check_inputs()) != 0) {
        (void)hipStreamSynchronize(s);
        return rc;
      }
      KMP_HIP_TRY(hipMemsetAsync(alpha, 0, sizeof(double) * ncell * n, s));
    }
    // a3-a9: smoothing stages
    for (int st = 0; st < nst; ++st) {
      const double delta = stage_delta(st);
      const double kappa = stage_kappa(st);
      size_t e4 = 0, e5 = 0, e6 = 0;
      if ((rc = tm.mark(s, &e4)) != 0) return rc;
      if (st == 0)
        KMP_HIP_TRY(hipStreamWaitEvent(s, side.done, 0));
      else if ((rc = path_stage_factor(s, pa, kappa)) != 0)
        return rc;
      if ((rc = path_stage_vectors(s, pa, kappa)) != 0) return rc;
      if ((rc = path_compact(s, pa)) != 0) return rc;
      if ((rc = tm.mark(s, &e5)) != 0) return rc;
      // The counts of active columns (per group and in total) come back to
      // pinned memory while the iterations go on: after a poll the next
      // iteration is queued before the host waits for the counts, so the
      // device never idles on the round trip (once every column has
      // converged, that iteration finds nothing to do and the stage ends).
      const auto post_poll = [&]() -> int {
        KMP_HIP_TRY(hipMemcpyAsync(poll.p, lay.nact, sizeof(int) * Gb, hipMemcpyDeviceToHost, s));
        KMP_HIP_TRY(hipMemcpyAsync(poll.p + Gb, lay.active, sizeof(int), hipMemcpyDeviceToHost, s));
        KMP_HIP_TRY(hipEventRecord(poll.ev, s));
        return 0;
      };
      const auto read_poll = [&](int* active) -> int {
        KMP_HIP_TRY(hipEventSynchronize(poll.ev));
        std::copy(poll.p, poll.p + Gb, nact_h.begin());
        *active = poll.p[Gb];
        return 0;
      };
      const int restart = (spec->flags & KMP_FLAG_RESTART) ? 1 : 0;
      IterGraph ig;
      if (use_graphs && (rc = capture_iterations(pa, delta, kappa, spec->tol, spec->max_iter,
                                                 restart, spec->poll_every, &ig)) != 0)
        return rc;
      if ((rc = post_poll()) != 0) return rc;
      bool pending = true;
      int it = 0;
      while (it < spec->max_iter) {
        if (ig.exec && it % spec->poll_every == 0 && it + spec->poll_every <= spec->max_iter) {
          KMP_HIP_TRY(hipGraphLaunch(ig.exec, s));
          it += spec->poll_every;
        } else {
          if ((rc = path_iteration(s, pa, delta, kappa, spec->tol, spec->max_iter, restart)) != 0)
            return rc;
          ++it;
          // the active lists follow every iteration (one small launch), so
          // the GEMMs drop a converged column at once; the counts still
          // come back at the polls only
          if (it % spec->poll_every != 0 && (rc = path_compact(s, pa)) != 0) return rc;
        }
        if (pending) {
          int active = 0;
          if ((rc = read_poll(&active)) != 0) return rc;
          pending = false;
          if (active == 0) break;
        }
        if (it % spec->poll_every == 0 || it >= spec->max_iter) {
          if ((rc = path_compact(s, pa)) != 0) return rc;
          if ((rc = post_poll()) != 0) return rc;
          pending = true;
        }
      }
      if (pending) {
        int active = 0;
        if ((rc = read_poll(&active)) != 0) return rc;
      }
      total_iters += it;
      if ((rc = tm.mark(s, &e6)) != 0) return rc;
      tm.span(&t_pre, e4, e5);
      tm.span(&t_path, e5, e6);
    }

    // a10: finalize
    FinalArgs fa;
    fa.n = (int)n; fa.d = (int)d; fa.ldx = ldx; fa.X = X; fa.nrm = lay.nrm; fa.y = y;
    fa.fold = lay.fold; fa.tidx = lay.tidx; fa.V = V; fa.S_b = sb; fa.Qt = Qn; fa.L = L;
    fa.s0 = s0; fa.S = S; fa.inv2s2 = lay.inv2s2; fa.delta = delta_final; fa.fbuf = lay.fbuf;
    fa.hidx = lay.hidx; fa.Mh = plan.Mh; fa.kh = lay.A; fa.ftrain = lay.fpart;
    fa.alpha = alpha; fa.beta_out = beta; fa.objective = objective; fa.cv_sum = cv_sum;
    fa.shared = shared;
    fa.cv_err = cv_err; fa.iters = iters; fa.status = status; fa.stat_count = lay.stat_count;
    if (plan.exact) {
      // the recovery's work vectors reuse column buffers the finalize no
      // longer needs
      ExactArgs& x = fa.ex;
      x.N = N; x.C = C; x.cols = (int64_t)Gb * C;
      x.emax = exact_emax(N);
      x.sys_stride = exact_sys_doubles(N);
      x.delta = delta_final; x.tol = 1e-9;
      x.nv = lay.nvg; x.cnv = lay.cnv; x.lam = lay.lam; x.ylab = lay.ylab; x.K = lay.A;
      x.state = lay.ex_state; x.elist = lay.ex_elist; x.ne = lay.ex_ne;
      x.wl = lay.abar; x.fl = lay.anew; x.alpha = lay.estep; x.fx = lay.uvec;
      x.sumyl = lay.ex_sumyl; x.sys = lay.ex_sys; x.beta_x = lay.ex_beta;
      x.xflag = lay.ex_flag; x.pending = lay.ex_pending;
      fa.exact = true;
      fa.delta = 0.0;            // the objective reported is the hinge objective
      fa.pending_host = exact_pin;
    }
    size_t f0 = 0, f1 = 0;
    if ((rc = tm.mark(s, &f0)) != 0) return rc;
    if ((rc = path_finalize(s, pa, fa)) != 0) return rc;
    if ((rc = tm.mark(s, &f1)) != 0) return rc;
    tm.span(&t_fin, f0, f1);
  }
  size_t ev_end = 0;
  if ((rc = tm.mark(s, &ev_end)) != 0) return rc;
  // host-side selection and status summary: the three arrays come back
  // with one wait
  double* hcv = pin.take<double>(ncell);
  int32_t* hit = pin.take<int32_t>(ncell);
  int* hstat = pin.take<int>(3);
  KMP_HIP_TRY(hipMemcpyAsync(hcv, cv_sum, sizeof(double) * ncell, hipMemcpyDeviceToHost, s));
  KMP_HIP_TRY(hipMemcpyAsync(hstat, lay.stat_count, 3 * sizeof(int), hipMemcpyDeviceToHost, s));
  if (iters)
    KMP_HIP_TRY(hipMemcpyAsync(hit, iters, sizeof(int32_t) * ncell, hipMemcpyDeviceToHost, s));
  KMP_HIP_TRY(hipStreamSynchronize(s));
  dirty_guard.clean = true;
  double t_total = 0.0;
  tm.span(&t_total, ev_start, ev_end);
  tm.sum();

  // the return code comes from the device's counts of cells that went
  // non-finite or stopped at max_iter, whether or not `status` was given
  if (hstat[1] > 0) {
    set_error(std::to_string(hstat[1]) + " cells with non-finite values in the iteration");
    return KMP_ENONFINITE;
  }
  const bool any_max = hstat[0] > 0;
  const bool any_inexact = hstat[2] > 0;
  int64_t cell_iters = 0;
  if (iters)
    for (size_t i = 0; i < ncell; ++i) cell_iters += hit[i];
  // selection (Appendix A.4: the fold-wise validation losses, pooled): the
  // CV score of (s, q, l) is sum_v cv_sum / n; per (s, q) the smallest
  // score wins with ties to the larger lambda, and jointly over (s, l) per q
  // with ties to the larger lambda, then the larger sigma
  const auto score = [&](int si, int q, int l) {
    double sc = 0.0;
    for (int v = 0; v < V; ++v) sc += hcv[(((size_t)si * Qn + q) * V + v) * L + l];
    return sc / (double)n;
  };
  if (selected && !refit) {
    for (int si = 0; si < S; ++si)
      for (int q = 0; q < Qn; ++q) {
        int best = -1;
        double bs = 0.0;
        for (int l = 0; l < L; ++l) {
          const double sc = score(si, q, l);
          if (best < 0 || sc < bs || (sc == bs && lambdas[l] > lambdas[best])) {
            best = l;
            bs = sc;
          }
        }
        selected[si * Qn + q] = best;
      }
  }
  if (selected_joint && !refit) {
    for (int q = 0; q < Qn; ++q) {
      int bsig = -1, bl = -1;
      double bs = 0.0;
      for (int si = 0; si < S; ++si)
        for (int l = 0; l < L; ++l) {
          const double sc = score(si, q, l);
          const bool better =
              bsig < 0 || sc < bs ||
              (sc == bs && (lambdas[l] > lambdas[bl] ||
                            (lambdas[l] == lambdas[bl] && sigmas[si] > sigmas[bsig])));
          if (better) {
            bsig = si;
            bl = l;
            bs = sc;
          }
        }
      selected_joint[2 * q] = bsig;
      selected_joint[2 * q + 1] = bl;
    }
  }
  if (timings) {
    for (int k = 0; k < KMP_NKC; ++k) {
      timings->kernel_ms[k] = 0.0;
      timings->kernel_launches[k] = 0;
      timings->kernel_seen[k] = g_clock ? g_clock->seen[k] : 0;
      timings->kernel_bytes[k] = 0.0;
      timings->kernel_flops[k] = 0.0;
      timings->kernel_ms_mb[k] = 0.0;
      timings->kernel_launches_mb[k] = 0;
      timings->kernel_bytes_mb[k] = 0.0;
      timings->kernel_flops_mb[k] = 0.0;
    }
    if (g_clock && !g_clock->failed) {
      for (const auto& r : g_clock->recs) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, g_clock->pool[r.ia], g_clock->pool[r.ib]) != hipSuccess) continue;
        timings->kernel_ms[r.cls] += ms;
        timings->kernel_launches[r.cls] += 1;
        timings->kernel_bytes[r.cls] += r.bytes;
        timings->kernel_flops[r.cls] += r.flops;
        if (r.flops > kRidgeFlopPerByte * r.bytes) {
          timings->kernel_ms_mb[r.cls] += ms;
          timings->kernel_launches_mb[r.cls] += 1;
          timings->kernel_bytes_mb[r.cls] += r.bytes;
          timings->kernel_flops_mb[r.cls] += r.flops;
        }
      }
    }
    timings->gram_ms = t_gram;
    timings->factor_ms = t_factor;
    timings->precompute_ms = t_pre;
    timings->path_ms = t_path;
    timings->finalize_ms = t_fin;
    timings->total_ms = t_total;
    timings->iterations = total_iters;
    timings->cell_iterations = cell_iters;
  }
  return any_max ? KMP_WMAXITER : (any_inexact ? KMP_WNOTEXACT : KMP_OK);
}

int kmp_dgemm_grouped(void* stream, int32_t G, int32_t M, int32_t N, int32_t K, const double* A,
                      const double* B, double* C) {
  hipStream_t s = (hipStream_t)stream;
  if (G < 0 || M < 0 || N < 0 || K < 0) {
    set_error("kmp_dgemm_grouped: negative size");
    return KMP_EINVAL;
  }
  if (G == 0 || M == 0 || N == 0) return KMP_OK;
  if (!C || (K > 0 && (!A || !B))) {
    set_error("kmp_dgemm_grouped: null pointer");
    return KMP_EINVAL;
  }
  if (G > 65535) {
    set_error("kmp_dgemm_grouped: at most 65535 groups per call");
    return KMP_EINVAL;
  }
  if (K == 0) {   // empty sum
    KMP_HIP_TRY(hipMemsetAsync(C, 0, sizeof(double) * (size_t)G * M * N, s));
    KMP_HIP_TRY(hipStreamSynchronize(s));
    return KMP_OK;
  }
  GemmArgs g;
  g.M = M; g.N = N; g.K = K; g.batch = G;
  g.A = A; g.lda = K; g.sA = (int64_t)M * K;
  g.B = B; g.ldb = N; g.sB = (int64_t)K * N;
  g.C = C; g.ldc = N; g.sC = (int64_t)M * N;
  g.alpha = 1.0; g.beta = 0.0;
  int rc = gemm(s, g, true, false, true);
  if (rc != 0) return rc;
  KMP_HIP_TRY(hipStreamSynchronize(s));
  return KMP_OK;
}

int kmp_path_step(void* stream, int32_t loss, double delta, const double* K, int64_t n,
                  const double* y, const double* lambdas, const double* taus, int32_t C,
                  const double* alpha_in, const double* beta_in, double* alpha_out,
                  double* beta_out, double* kkt_out) {
  hipStream_t s = (hipStream_t)stream;
  if (loss < 0 || loss > 2 || !K || !y || !lambdas || !alpha_in || !beta_in || !alpha_out ||
      !beta_out || n < 2 || C < 1 || (loss != KMP_LOGISTIC && !(delta > 0.0)) ||
      (loss == KMP_CHECK && !taus)) {
    set_error("kmp_path_step: invalid arguments");
    return KMP_EINVAL;
  }
  for (int c = 0; c < C; ++c) {
    if (!(lambdas[c] > 0.0) || !std::isfinite(lambdas[c])) {
      set_error("kmp_path_step: lambda must be positive and finite");
      return KMP_EINVAL;
    }
    if (loss == KMP_CHECK && !(taus[c] > 0.0 && taus[c] < 1.0)) {
      set_error("kmp_path_step: tau must lie in (0, 1)");
      return KMP_EINVAL;
    }
  }
  // one group of all n rows (the full-data layout), C columns
  kmp_path_spec spec;
  kmp_default_spec(&spec);
  spec.loss = loss;
  spec.flags = KMP_FLAG_REFIT;
  Plan plan;
  int rc = make_plan(&spec, n, 1, C, nullptr, 1, 1, 1, 1, &plan);
  if (rc != 0) return rc;
  if (n > kMaxOrder) {
    set_error("kmp_path_step: n above the largest factor order");
    return KMP_EINVAL;
  }
  // make_plan lays out C = Q L columns with Q = 1, L = C
  const int N = plan.N;
  const double kappa = loss == KMP_LOGISTIC ? 4.0 : 2.0 * delta;
  void* ws = nullptr;
  KMP_HIP_TRY(hipMallocAsync(&ws, plan.bytes, s));
  struct Free {
    void* p;
    hipStream_t s;
    ~Free() {
      if (p) (void)hipFreeAsync(p, s);
    }
  } free_ws{ws, s};
  Layout lay;
  carve(plan, ws, &lay);
  const size_t cols = (size_t)C;
  // host-side parameters (pageable: small, synchronous copies)
  std::vector<double> lam(lambdas, lambdas + C), tau(C, 0.0);
  if (loss == KMP_CHECK) tau.assign(taus, taus + C);
  std::vector<int> nvg(1, (int)n), cnv(C, (int)n);
  std::vector<int32_t> cf(C, -1);
  KMP_HIP_TRY(hipMemcpyAsync(lay.lam, lam.data(), sizeof(double) * cols, hipMemcpyHostToDevice, s));
  KMP_HIP_TRY(hipMemcpyAsync(lay.taucol, tau.data(), sizeof(double) * cols, hipMemcpyHostToDevice, s));
  KMP_HIP_TRY(hipMemcpyAsync(lay.nvg, nvg.data(), sizeof(int), hipMemcpyHostToDevice, s));
  KMP_HIP_TRY(hipMemcpyAsync(lay.cnv, cnv.data(), sizeof(int) * cols, hipMemcpyHostToDevice, s));
  KMP_HIP_TRY(hipMemcpyAsync(lay.cfold, cf.data(), sizeof(int32_t) * cols, hipMemcpyHostToDevice, s));
  // K into the padded factor buffer, y into the padded labels
  KMP_HIP_TRY(hipMemsetAsync(lay.A, 0, sizeof(double) * (size_t)N * N, s));
  KMP_HIP_TRY(hipMemcpy2DAsync(lay.A, sizeof(double) * N, K, sizeof(double) * n,
                               sizeof(double) * n, n, hipMemcpyDeviceToDevice, s));
  KMP_HIP_TRY(hipMemsetAsync(lay.ylab, 0, sizeof(double) * N, s));
  KMP_HIP_TRY(hipMemcpyAsync(lay.ylab, y, sizeof(double) * n, hipMemcpyDeviceToDevice, s));
  // a2 and the stage setup on this matrix
  BandWork bw = band_work_of(lay, 1, N, nvg.data());
  if ((rc = band_reduce(s, bw)) != 0) return rc;
  if ((rc = form_qb(s, lay.Qm, lay.band, N, 1, lay.A)) != 0) return rc;
  PathArrays pa = path_arrays_of(lay, plan, loss, false);
  pa.G = 1;
  pa.nv_host = nvg.data();
  std::vector<int> nact_h(1, C);
  pa.nact_host = nact_h.data();
  if ((rc = group_ones_projection(s, lay.Qm, lay.nvg, 1, N, lay.cvec)) != 0) return rc;
  if ((rc = path_init_columns(s, pa)) != 0) return rc;
  // the caller's state in the factor basis: ahat = Q' alpha, beta
  KMP_HIP_TRY(hipMemsetAsync(lay.zmat, 0, sizeof(double) * cols * N, s));
  KMP_HIP_TRY(hipMemcpy2DAsync(lay.zmat, sizeof(double) * N, alpha_in, sizeof(double) * n,
                               sizeof(double) * n, C, hipMemcpyDeviceToDevice, s));
  GemmArgs g;
  g.M = N; g.N = C; g.K = N; g.batch = 1;
  g.A = lay.Qm; g.lda = N; g.sA = (int64_t)N * N;
  g.B = lay.zmat; g.ldb = N; g.sB = (int64_t)N * C;
  g.C = lay.ahat; g.ldc = N; g.sC = (int64_t)N * C;
  if ((rc = gemm(s, g, false, true, false)) != 0) return rc;
  KMP_HIP_TRY(hipMemcpyAsync(lay.beta, beta_in, sizeof(double) * cols, hipMemcpyDeviceToDevice, s));
  // factors and vectors of the stage (momentum restarted: the step is taken
  // from the given point itself), then one iteration with tol = 0 so every
  // column steps
  if ((rc = path_stage_factor(s, pa, kappa)) != 0) return rc;
  if ((rc = path_stage_vectors(s, pa, kappa)) != 0) return rc;
  if ((rc = path_compact(s, pa)) != 0) return rc;
  if ((rc = path_iteration(s, pa, loss == KMP_LOGISTIC ? 1.0 : delta, kappa, 0.0, 1 << 30, 0)) != 0)
    return rc;
  // alpha = Q a+ back to the caller's layout
  g.A = lay.Qm;
  g.B = lay.ahat;
  g.C = lay.zmat;
  if ((rc = gemm(s, g, true, true, false)) != 0) return rc;
  KMP_HIP_TRY(hipMemcpy2DAsync(alpha_out, sizeof(double) * n, lay.zmat, sizeof(double) * N,
                               sizeof(double) * n, C, hipMemcpyDeviceToDevice, s));
  KMP_HIP_TRY(hipMemcpyAsync(beta_out, lay.beta, sizeof(double) * cols, hipMemcpyDeviceToDevice, s));
  if (kkt_out)
    KMP_HIP_TRY(hipMemcpyAsync(kkt_out, lay.kkt, sizeof(double) * cols, hipMemcpyDeviceToDevice, s));
  KMP_HIP_TRY(hipStreamSynchronize(s));
  return KMP_OK;
}

}  // extern "C"
