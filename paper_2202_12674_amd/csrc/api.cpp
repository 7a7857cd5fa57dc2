// Host runtime of the C ABI declared in include/lssvm.h: argument checks,
// workspace carve-up, the CG driver loop (Sec. III-B) and the bias step
// (Eq. (15)). Every numeric step runs in the gfx950 kernels of kernels.hip;
// this file only validates, sequences launches and reads back scalars.
#include "lssvm.h"
#include "lssvm_error.h"
#include "lssvm_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

namespace lssvm {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

void clear_error() { g_last_error.clear(); }

namespace {

#define LSSVM_HIP(call)                                                                  \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(LSSVM_EHIP, "%s failed: %s (%s:%d)", #call, hipGetErrorString(e_),     \
                  __FILE__, __LINE__);                                                   \
  } while (0)

#define LSSVM_TRY(expr)      \
  do {                       \
    int rc_ = (expr);        \
    if (rc_ != LSSVM_OK) return rc_; \
  } while (0)

constexpr size_t kAlign = 256;
// Supported sizes: the tile visit order takes n^2 / 8192 bytes (2 GiB at
// n = 2^22) and packs tile indices in 16 bits; a panel's buffer span stays
// below 4 GiB up to 2^21 features.
constexpr int64_t kMaxPoints = int64_t(1) << 22;
constexpr int64_t kMaxFeatures = int64_t(1) << 21;

// LSSVM_LOG=1 in the environment: one stderr line per batch of CG iterations
// and one per finished training (read once per process).
bool log_enabled() {
  static const bool on = [] {
    const char* v = std::getenv("LSSVM_LOG");
    return v && *v && std::strcmp(v, "0") != 0;
  }();
  return on;
}
constexpr int64_t kReplaceEvery = 50;  // residual recomputed every 50th iteration

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }
inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

using clock_t_ = std::chrono::steady_clock;
inline double ms_since(clock_t_::time_point t0) {
  return std::chrono::duration<double, std::milli>(clock_t_::now() - t0).count();
}

// Padded sizes for n points of d features (element type T).
struct Geometry {
  int64_t n, d, N;  // N = n - 1 unknowns of the reduced system
  int64_t tile, bk;
  int64_t ld;       // points per feature row of the layout (>= n, multiple of tile)
  int64_t d_pad;    // features, multiple of 2 bk
  int64_t nT;       // tiles per edge of the reduced system
  int64_t NP;       // nT * tile: padded length of every CG vector
  int64_t nb;       // blocks of the CG vector kernels over NP (block partials per reduction)
  int64_t ksplit;   // linear kernel: workgroups per tile, each over a share of the features
  int64_t lin_tail_q;      // linear kernel: tiles of the last partial round (or 0), run by
  int64_t lin_tail_split;  // the launch's trailing workgroups, split this many ways
  int64_t tail_q;   // other kernels: tiles of the last partial round that are split (or 0)
  int64_t tail_split;  // ... over this many workgroups each
};

#ifndef LSSVM_FUSED_SMALL
#define LSSVM_FUSED_SMALL 1
#endif
// Small problems run each CG iteration (except the residual recomputations)
// as one launch: the product's tiles and, in the last workgroup, the vector
// work (launch_tiles_cg). Their iterations are launch-bound: four dependent
// launches of a few microseconds each against a product of ~10 us. (At 4096
// points the same fusion cost more than it saved: the release and ticket of
// each of ~1000 workgroups made the launch ~50 us longer than the product.)
inline bool fused_iteration(const Geometry& g, int32_t kernel) {
  const bool one_launch = kernel == LSSVM_LINEAR ? g.lin_tail_q == 0 : g.tail_q == 0;
  return LSSVM_FUSED_SMALL && g.NP <= kFusedMaxNP && one_launch;
}

inline int64_t tri_count(int64_t nT) { return nT * (nT + 1) / 2; }

// Workgroups resident at once in a tile launch: two per CU on 256 CUs.
constexpr int64_t kResidentTiles = 512;
#ifndef LSSVM_LINEAR_SPLIT_MAX
#define LSSVM_LINEAR_SPLIT_MAX 16
#endif

#ifndef LSSVM_LINEAR_TAIL
#define LSSVM_LINEAR_TAIL 1
#endif
#ifndef LSSVM_LINEAR_TAIL_MAX
#define LSSVM_LINEAR_TAIL_MAX 64
#endif

// Finer split of the linear kernel's tiles in a last partial round that
// already runs S ways: the largest T (up to 64) with Q T within one round of
// resident workgroups and an even number of feature blocks per share.
inline int64_t linear_tail_split(int64_t Q, int64_t S, int64_t nkb) {
  int64_t T = S;
  while (LSSVM_LINEAR_TAIL && T < LSSVM_LINEAR_TAIL_MAX && Q * T * 2 <= kResidentTiles && nkb % (4 * T) == 0)
    T *= 2;
  return T;
}

// Feature split of the linear kernel's tiles. A product of W tiles split S
// ways runs in rounds of R resident workgroups, each as long as 1/S of a
// tile plus a fixed cost of about two feature blocks (the first block's load
// latency and the epilogue). The full rounds take floor(W S / R) of those;
// the Q tiles left for a last partial round run as the launch's trailing
// workgroups, split T >= S ways (the feature shares add into the row sums
// like any split's, so no fixup is needed), which takes 1/T of a tile plus
// the fixed cost. S (and T) halve the block count, which must stay even. A
// problem of one round or less keeps its tiles in one launch.
inline void linear_plan(int64_t nT, int64_t nkb, int64_t* split, int64_t* q, int64_t* tail_split) {
  const int64_t W = tri_count(nT);
  const double f = 2.0 / (double)nkb;
  auto plan = [&](int64_t S, int64_t* Q, int64_t* T) {
    *Q = 0;
    *T = S;
    if (W * S <= kResidentTiles) return 1.0 / (double)S + f;
    const int64_t full = W * S / kResidentTiles;
    const int64_t left = W - full * (kResidentTiles / S);
    double c = (double)full * (1.0 / (double)S + f);
    if (left > 0) {
      const int64_t t = linear_tail_split(left, S, nkb);
      c += 1.0 / (double)t + f;
      if (t > S) {
        *Q = left;
        *T = t;
      }
    }
    return c;
  };
  int64_t best = 1, bq, bt;
  double best_cost = plan(1, &bq, &bt);
  for (int64_t S = 2; S <= LSSVM_LINEAR_SPLIT_MAX && nkb % (2 * S) == 0; S *= 2) {
    int64_t Q, T;
    const double c = plan(S, &Q, &T);
    if (c < 0.95 * best_cost) {   // a clear gain only: each split adds workgroups and atomics
      best = S;
      best_cost = c;
      bq = Q;
      bt = T;
    }
  }
  *split = best;
  *q = bq;
  *tail_split = bt;
}

// The tiles beyond the last full round of resident workgroups run one per
// CU and take about as long as a whole round. When they are at most a
// quarter round, each is split over S (4..16) workgroups that park their
// partial inner products, and one more launch sums them per tile and
// finishes it: the tail then costs ~1/S of a round plus the fixup.
inline void tail_plan(int64_t nT, int64_t nkb, int64_t* q, int64_t* split) {
  const int64_t Q = tri_count(nT) % kResidentTiles;
  int64_t S = 1;
  while (S < 16 && Q * S * 2 <= kResidentTiles && nkb % (4 * S) == 0) S *= 2;
  *q = (Q > 0 && S >= 4) ? Q : 0;
  *split = *q > 0 ? S : 1;
}

template <typename T>
Geometry geometry(int64_t n, int64_t d) {
  Geometry g{};
  g.n = n;
  g.d = d;
  g.N = n - 1;
  g.tile = TileShape<T>::T;
  g.bk = TileShape<T>::BK;
  g.ld = round_up(n, g.tile);
  g.d_pad = round_up(d, 2 * g.bk);   // an even number of feature blocks (two LDS stages)
  g.nT = (g.N + g.tile - 1) / g.tile;
  g.NP = g.nT * g.tile;
  g.nb = cg_blocks(g.NP);
  linear_plan(g.nT, g.d_pad / g.bk, &g.ksplit, &g.lin_tail_q, &g.lin_tail_split);
  tail_plan(g.nT, g.d_pad / g.bk, &g.tail_q, &g.tail_split);
  return g;
}

// Carves aligned sub-buffers out of the caller's workspace (or only sizes them).
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <typename U>
  U* take(int64_t count) {
    U* p = base ? reinterpret_cast<U*>(base + off) : nullptr;
    off = align_up(off + (size_t)count * sizeof(U));
    return p;
  }
};

template <typename T>
struct TrainWs {
  T* Xt;
  T* norms;
  double* q64;
  int64_t* acc; // fixed-point row sums of a product (two words per row)
  T* gpart;     // parked inner products of split tail tiles
  double* pq;   // per tile panel: sum p_j, then sum q_j p_j (2 nT)
  double *rhs, *x, *r, *dir, *qv;
  double* xbest;   // iterate of the smallest recomputed residual (returned on a stall)
  double *bp0, *bp1, *bp2;
  double* scal;
  int* flags;
  uint32_t* order;
  double* hist;
  unsigned* ticket;   // workgroups done in a fused iteration's launch
  size_t bytes;
};


template <typename T>
TrainWs<T> carve_train(const Geometry& g, void* base) {
  Carver c(base);
  TrainWs<T> w{};
  w.Xt = c.take<T>(g.d_pad * g.ld);
  w.norms = c.take<T>(g.ld);
  w.q64 = c.take<double>(g.ld);
  // Row sums: two 64-bit words per row, however many tiles add to them; the
  // split tail's parked inner products (at most a quarter round of tiles).
  w.acc = c.take<int64_t>(2 * g.NP);
  w.gpart = c.take<T>(g.tail_q * g.tail_split * g.tile * g.tile);
  w.pq = c.take<double>(2 * g.nT);
  w.rhs = c.take<double>(g.NP);
  w.x = c.take<double>(g.NP);
  w.r = c.take<double>(g.NP);
  w.dir = c.take<double>(g.NP);
  w.qv = c.take<double>(g.NP);
  w.xbest = c.take<double>(g.NP);
  w.bp0 = c.take<double>(g.nb + 1);
  w.bp1 = c.take<double>(g.nb + 1);
  w.bp2 = c.take<double>(g.nb + 1);   // energy partials at residual recomputations
  w.scal = c.take<double>(S_COUNT);
  w.flags = c.take<int>(F_COUNT);
  w.order = c.take<uint32_t>(LSSVM_TILE_GROUP > 0 ? tri_count(g.nT) : 0);
  w.hist = c.take<double>(g.NP + 1);   // r^T r after each iteration (at most N of them)
  w.ticket = c.take<unsigned>(64);
  w.bytes = c.off;
  return w;
}

template <typename T>
struct PredictWs {
  T *Xtr, *ntr, *alpha;
  T *Xte, *nte;
  double* part;
  int* flags;
  double* lin_part;  // linear kernel: partial sums of w over point chunks
  double* lin_w;     // linear kernel: w = sum_i alpha_i x_i
  double* lin_f;     // linear kernel: <w, x> per test point
  int64_t ld_te, nTc, nTr;
  size_t bytes;
};

template <typename T>
PredictWs<T> carve_predict(const Geometry& g, int64_t n_test, void* base) {
  Carver c(base);
  PredictWs<T> w{};
  w.ld_te = round_up(n_test, g.tile);
  w.nTc = g.ld / g.tile;
  w.nTr = w.ld_te / g.tile;
  w.Xtr = c.take<T>(g.d_pad * g.ld);
  w.ntr = c.take<T>(g.ld);
  w.alpha = c.take<T>(g.ld);
  w.Xte = c.take<T>(g.d_pad * w.ld_te);
  w.nte = c.take<T>(w.ld_te);
  w.part = c.take<double>(w.nTc * w.ld_te);
  w.flags = c.take<int>(F_COUNT);
  w.lin_part = c.take<double>(linear_predict_part_elems(g.n, g.d));
  w.lin_w = c.take<double>(g.d);
  w.lin_f = c.take<double>(n_test);
  w.bytes = c.off;
  return w;
}

// Host-side state of one call in flight: a pinned buffer for the few
// scalars read back per batch of CG iterations, and timing events (creating
// a few hundred events costs more than a small training takes). Calls lease
// a context from a process-wide pool and return it when they end, so the
// pool holds as many contexts as calls ever ran at once, however many
// threads come and go; contexts live until the process ends.
struct HostCtx {
  double* p = nullptr;   // 64 doubles, pinned
  int* flags = nullptr;  // inside p
  int device = -1;       // device the events belong to
  std::vector<hipEvent_t> ev;
  hipError_t ensure() {
    if (p) return hipSuccess;
    void* v = nullptr;
    hipError_t e = hipHostMalloc(&v, 64 * sizeof(double), hipHostMallocDefault);
    if (e != hipSuccess) return e;
    p = static_cast<double*>(v);
    flags = reinterpret_cast<int*>(p + 32);
    return hipSuccess;
  }
};
std::mutex g_pool_mu;
std::vector<HostCtx*> g_pool_free;
std::atomic<int64_t> g_pool_size{0};
thread_local HostCtx* g_ctx = nullptr;   // the context of this thread's call in flight

struct CtxLease {
  HostCtx* prev;
  CtxLease() : prev(g_ctx) {
    std::lock_guard<std::mutex> lock(g_pool_mu);
    if (!g_pool_free.empty()) {
      g_ctx = g_pool_free.back();
      g_pool_free.pop_back();
    } else {
      g_ctx = new HostCtx();
      ++g_pool_size;
    }
  }
  ~CtxLease() {
    std::lock_guard<std::mutex> lock(g_pool_mu);
    g_pool_free.push_back(g_ctx);
    g_ctx = prev;
  }
  CtxLease(const CtxLease&) = delete;
  CtxLease& operator=(const CtxLease&) = delete;
};

// HIP events around each implicit product, recorded on the launch stream.
// Pairs carry the CG iteration they belong to, so products that ran after
// the stop (and returned at once) are left out.
struct MatvecTimer {
  static constexpr int kPairs = 2 * 64;   // up to two products per queued iteration
  bool on = false;
  hipEvent_t* ev = nullptr;   // 2 kPairs events of the thread's pool
  int64_t tag[kPairs] = {};
  int used = 0;          // event pairs recorded since the last harvest
  double total_ms = 0.0;
  int64_t count = 0;
  double* out = nullptr;   // caller's array of per-product times, or null
  int64_t cap = 0;
  hipError_t init(bool enable, double* times = nullptr, int64_t capacity = 0) {
    on = enable;
    out = times;
    cap = capacity;
    if (!on) return hipSuccess;
    int device = 0;
    hipError_t r = hipGetDevice(&device);
    if (r != hipSuccess) return r;
    HostCtx& c = *g_ctx;
    if (c.device != device) {
      for (hipEvent_t e : c.ev) (void)hipEventDestroy(e);
      c.ev.clear();
      c.device = device;
    }
    while (c.ev.size() < (size_t)(2 * kPairs)) {
      hipEvent_t e = nullptr;
      if ((r = hipEventCreate(&e)) != hipSuccess) return r;
      c.ev.push_back(e);
    }
    ev = c.ev.data();
    return hipSuccess;
  }
  // A batch queues at most 32 iterations of at most two products each, so the
  // pairs never run out; should they, the extra products are simply not timed.
  bool full() const { return used >= kPairs; }
  hipError_t start(hipStream_t s, int64_t iter) {
    if (!on || full()) return hipSuccess;
    tag[used] = iter;
    return hipEventRecord(ev[2 * used], s);
  }
  hipError_t stop(hipStream_t s) {
    if (!on || full()) return hipSuccess;
    hipError_t r = hipEventRecord(ev[2 * used + 1], s);
    ++used;
    return r;
  }
  // After the stream has been synchronised: add the pairs of iterations <= last.
  hipError_t harvest(int64_t last) {
    for (int i = 0; i < used; ++i) {
      if (tag[i] > last) continue;
      float ms = 0.f;
      hipError_t r = hipEventElapsedTime(&ms, ev[2 * i], ev[2 * i + 1]);
      if (r != hipSuccess) return r;
      total_ms += ms;
      if (out && count < cap) out[count] = ms;
      ++count;
    }
    used = 0;
    return hipSuccess;
  }
};

bool valid_dtype(int32_t dt) { return dt == LSSVM_F64 || dt == LSSVM_F32; }
bool valid_kernel(int32_t k) { return k == LSSVM_LINEAR || k == LSSVM_POLY || k == LSSVM_RBF; }

int check_kernel_params(int32_t kernel, const lssvm_params* kp) {
  if (!valid_kernel(kernel)) return fail(LSSVM_EINVAL, "unknown kernel %d", (int)kernel);
  if (kernel == LSSVM_LINEAR) return LSSVM_OK;
  if (!kp) return fail(LSSVM_EINVAL, "kernel parameters required for kernel %d", (int)kernel);
  if (!(kp->gamma > 0.0) || !std::isfinite(kp->gamma))
    return fail(LSSVM_EINVAL, "gamma must be finite and > 0 (got %g)", kp->gamma);
  if (kernel == LSSVM_POLY) {
    if (kp->degree < 1) return fail(LSSVM_EINVAL, "degree must be >= 1 (got %d)", kp->degree);
    if (!std::isfinite(kp->coef0)) return fail(LSSVM_EINVAL, "coef0 must be finite");
  }
  return LSSVM_OK;
}

int check_sizes(int64_t n, int64_t d, int64_t min_n) {
  if (n < min_n) return fail(LSSVM_EINVAL, "n must be >= %lld (got %lld)", (long long)min_n,
                             (long long)n);
  if (d < 1) return fail(LSSVM_EINVAL, "d must be >= 1 (got %lld)", (long long)d);
  if (n > kMaxPoints || d > kMaxFeatures)
    return fail(LSSVM_EINVAL, "problem too large (n=%lld, d=%lld)", (long long)n, (long long)d);
  return LSSVM_OK;
}

int check_workspace(const void* ws, size_t have, size_t need) {
  if (!ws) return fail(LSSVM_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
    return fail(LSSVM_EINVAL, "workspace must be %zu-byte aligned", kAlign);
  if (have < need)
    return fail(LSSVM_EINVAL, "workspace too small: %zu bytes given, %zu needed", have, need);
  return LSSVM_OK;
}

// Exponent scale of the RBF tile epilogue: fp32 evaluates exp(-gamma dist)
// as exp2(-(gamma log2 e) dist) on the hardware base-2 exponential.
template <typename T> T rbf_scale(double gamma);
template <> float rbf_scale<float>(double gamma) { return (float)(gamma * 1.4426950408889634); }
template <> double rbf_scale<double>(double gamma) { return gamma; }

// Workgroups per tile of every product of n points (a training's CG
// iterations, its residual recomputations, a warm start's and the true
// residual's products, lssvm_matvec). On a small problem, whose iterations
// are fused launches, the few tiles take one CU each and their matrix work
// is most of the launch, so the linear kernel's split goes as far as one
// round of workgroups allows, down to a single feature block per workgroup.
// All products of a problem take the same split: each split rounds the
// operator its own way (fp32 partial inner products), and a recomputed
// residual from a differently rounded operator than the iterations' stalls
// fp32 CG above its eps.
inline int64_t product_split(const Geometry& g, int32_t kernel) {
  if (kernel != LSSVM_LINEAR) return 1;
  int64_t S = g.ksplit;
  if (!fused_iteration(g, kernel)) return S;
  const int64_t nkb = g.d_pad / g.bk, W = tri_count(g.nT);
  // double while every workgroup keeps an even block count (the two-stage
  // loop) or gets exactly one (the single-block variant)
  while (S < LSSVM_LINEAR_SPLIT_MAX && W * 2 * S <= kResidentTiles &&
         (nkb % (4 * S) == 0 || nkb == 2 * S))
    S *= 2;
  return S;
}

template <typename T>
TileArgs<T> sym_args(const Geometry& g, const TrainWs<T>& w, const lssvm_params& kp,
                     int32_t kernel, const double* p) {
  TileArgs<T> a{};
  a.A = w.Xt;
  a.B = w.Xt;
  a.lda = g.ld;
  a.ldb = g.ld;
  a.nkb = g.d_pad / g.bk;
  a.nA = w.norms;
  a.nB = w.norms;
  a.pv = p;
  a.q64 = w.q64;
  a.pq = w.pq;
  a.gamma = (T)kp.gamma;
  a.coef0 = (T)kp.coef0;
  a.rbf_scale = rbf_scale<T>(kp.gamma);
  a.degree = kp.degree;
  a.nTc = g.nT;
  a.ksplit = product_split(g, kernel);
  a.order = LSSVM_TILE_GROUP > 0 ? w.order : nullptr;
  a.acc = w.acc;
  a.fx = w.scal + S_PMAX;      // [S_PMAX], [S_NMAX], [S_FIXSC]
  a.fx_bad = w.flags + F_PRODUCT;
  return a;
}

#ifndef LSSVM_DIAG_TAIL
#define LSSVM_DIAG_TAIL 1
#endif

// The tile visit order, written into the workspace on the device (once per
// call). The linear kernel's finer-split last round takes diagonal tiles
// where there are enough: each of its T splits then adds into one panel of
// row sums, where the last tiles of the grouped order share a few panels
// (up to a super-tile's worth of tiles times T atomic additions per word).
// The same launch zeroes the flags, the scalars and the row-sum words.
template <typename T>
int clear_and_order(const Geometry& g, const TrainWs<T>& w, int32_t kernel, hipStream_t s) {
  const bool ordered = LSSVM_TILE_GROUP > 0 && g.nT > 0;
  const int64_t nd = (LSSVM_DIAG_TAIL && kernel == LSSVM_LINEAR) ? std::min(g.lin_tail_q, g.nT) : 0;
  LSSVM_HIP(launch_setup_clear(g.nT, LSSVM_TILE_GROUP, nd, ordered ? w.order : nullptr, w.flags,
                               w.scal, w.acc, 2 * g.NP, w.ticket, s));
  return LSSVM_OK;
}

// a1 + a2: layout, norms, q and k_mm (left on the device). With check set,
// reads back the input flags and reports a non-finite X; otherwise the
// caller reads them back with its next result.
template <typename T>
int setup_points(const Geometry& g, const TrainWs<T>& w, const T* X, int32_t kernel,
                 const lssvm_params& kp, hipStream_t s, bool check = true) {
  LSSVM_TRY(clear_and_order<T>(g, w, kernel, s));
  LSSVM_HIP(launch_layout<T>(X, g.n, g.d, w.Xt, g.ld, g.d_pad, w.flags, s));
  LSSVM_HIP(launch_norms_q<T>(w.Xt, g.ld, g.d_pad, g.N, g.N, kernel, kp.gamma, kp.coef0,
                              kp.degree, w.norms, w.q64, w.scal, s));
  if (!check) return LSSVM_OK;
  LSSVM_HIP(hipMemcpyAsync(g_ctx->flags, w.flags, F_COUNT * sizeof(int), hipMemcpyDeviceToHost,
                           s));
  LSSVM_HIP(hipStreamSynchronize(s));
  if (g_ctx->flags[F_NONFINITE]) return fail(LSSVM_ENONFINITE, "X holds a NaN or an infinity");
  return LSSVM_OK;
}

// A finished product's row sums and the terms of Q~ p the tiles leave out.
template <typename T>
RankOne rank_one(const Geometry& g, const TrainWs<T>& w, int32_t kernel, double C,
                 const double* p) {
  (void)kernel;
  return RankOne{w.pq, g.nT, w.acc, w.q64, p, w.scal, w.flags, 1.0 / C};
}

// The tile launches of one product: all tiles whole (the linear kernel's
// split tiles included), or the full rounds whole and the tail split, parked
// and fixed up.
// The one launch of a linear product: its workgroup count, with a's fields
// for the finer-split last round set. Feature splits add up, so the last
// round only splits finer, as the launch's trailing workgroups: they start
// as the whole tiles finish, with no second launch to wait for.
template <typename T>
int64_t linear_launch(const Geometry& g, TileArgs<T>& a) {
  const int64_t F = tri_count(g.nT) - g.lin_tail_q;
  if (g.lin_tail_q == 0) return F * a.ksplit;
  a.tail_slot = F * a.ksplit;
  a.tail_split = g.lin_tail_split;
  a.tail_tile = F;
  return F * a.ksplit + g.lin_tail_q * g.lin_tail_split;
}

template <typename T>
hipError_t launch_product(const Geometry& g, TileArgs<T> a, int32_t kernel, T* gpart,
                          hipStream_t s) {
  const int64_t W = tri_count(g.nT);
  if (kernel == LSSVM_LINEAR) return launch_tiles_sym<T>(a, kernel, kWhole, linear_launch(g, a), s);
  if (g.tail_q == 0) return launch_tiles_sym<T>(a, kernel, kWhole, W, s);
  const int64_t F = W - g.tail_q;
  hipError_t e = launch_tiles_sym<T>(a, kernel, kWhole, F, s);
  if (e != hipSuccess) return e;
  a.tile_offset = F;
  a.ksplit = g.tail_split;
  a.gpart = gpart;
  e = launch_tiles_sym<T>(a, kernel, kPartial, g.tail_q * g.tail_split, s);
  if (e != hipSuccess) return e;
  return launch_tiles_sym<T>(a, kernel, kFixup, g.tail_q, s);
}

// One implicit product K p into the partial-sum buffer (plus the per-panel
// sums of the rank-one terms).
template <typename T>
int matvec_partials(const Geometry& g, const TrainWs<T>& w, const lssvm_params& kp,
                    int32_t kernel, const double* p, hipStream_t s) {
  LSSVM_HIP(launch_product<T>(g, sym_args<T>(g, w, kp, kernel, p), kernel, w.gpart, s));
  return LSSVM_OK;
}

template <typename T>
int timed_matvec(const Geometry& g, const TrainWs<T>& w, const lssvm_params& kp, int32_t kernel,
                 const double* p, hipStream_t s, MatvecTimer& tm, int64_t iter) {
  LSSVM_HIP(tm.start(s, iter));
  TileArgs<T> a = sym_args<T>(g, w, kp, kernel, p);
  a.stop = w.scal + S_STATUS + ST_DONE;   // skip the launches once CG has stopped
  LSSVM_HIP(launch_product<T>(g, a, kernel, w.gpart, s));
  LSSVM_HIP(tm.stop(s));
  return LSSVM_OK;
}


template <typename T>
int train_impl(const T* X, const T* y, int64_t n, int64_t d, int32_t kernel,
               const lssvm_params& kp, double C, double eps, int64_t max_iter, void* workspace,
               size_t ws_bytes, T* alpha_out, double* b_out, lssvm_info* info, hipStream_t s) {
  const auto t0 = clock_t_::now();
  const Geometry g = geometry<T>(n, d);
  TrainWs<T> w = carve_train<T>(g, nullptr);
  LSSVM_TRY(check_workspace(workspace, ws_bytes, w.bytes));
  w = carve_train<T>(g, workspace);
  LSSVM_HIP(g_ctx->ensure());

  if (info) {
    info->iterations = 0;
    info->n_matvec = 0;
    info->t_matvec_ms = 0.0;
    info->n_matvec_timed = 0;
    info->rel_residual = 0.0;
    info->true_rel_residual = -1.0;
    info->t_setup_ms = info->t_cg_ms = info->t_total_ms = 0.0;
    info->stop_reason = LSSVM_STOP_EPS;
  }

  if (n == 1) {  // alpha = [0], b = y_0
    LSSVM_HIP(hipMemsetAsync(w.flags, 0, F_COUNT * sizeof(int), s));
    LSSVM_HIP(launch_layout<T>(X, g.n, g.d, w.Xt, g.ld, g.d_pad, w.flags, s));
    LSSVM_HIP(launch_single_point<T>(y, alpha_out, w.scal, w.flags, s));
    LSSVM_HIP(hipMemcpyAsync(g_ctx->flags, w.flags, F_COUNT * sizeof(int),
                             hipMemcpyDeviceToHost, s));
    LSSVM_HIP(hipMemcpyAsync(g_ctx->p, w.scal + S_B, sizeof(double), hipMemcpyDeviceToHost, s));
    LSSVM_HIP(hipStreamSynchronize(s));
    if (g_ctx->flags[F_NONFINITE]) return fail(LSSVM_ENONFINITE, "X holds a NaN or an infinity");
    if (g_ctx->flags[F_BADLABEL]) return fail(LSSVM_EBADLABEL, "labels must be +1 or -1");
    *b_out = g_ctx->p[0];
    if (info) {
      info->rel_residual = 0.0;
      info->true_rel_residual = info->compute_true_residual ? 0.0 : -1.0;
      info->t_total_ms = ms_since(t0);
    }
    return LSSVM_OK;
  }

  // ---- setup: a1, a2, a3 (one read-back for the input flags and r0^T r0)
  LSSVM_TRY(setup_points<T>(g, w, X, kernel, kp, s, /*check=*/false));
  LSSVM_HIP(launch_rhs_init<T>(y, g.N, g.NP, w.rhs, w.x, w.xbest, w.r, w.dir, w.bp0, w.flags,
                               w.scal, s));
  LSSVM_HIP(launch_finish_delta0(w.bp0, g.nb, w.scal, eps * eps, w.flags, s));
  // one read-back: r0^T r0 and the input flags
  LSSVM_HIP(hipMemcpyAsync(g_ctx->p, w.scal + S_DELTA0, (S_INFLAGS - S_DELTA0 + 1) * sizeof(double),
                           hipMemcpyDeviceToHost, s));
  LSSVM_HIP(hipStreamSynchronize(s));
  const double inflags = g_ctx->p[S_INFLAGS - S_DELTA0];
  if (inflags == 1.0 || inflags == 3.0) return fail(LSSVM_ENONFINITE, "X holds a NaN or an infinity");
  if (inflags == 2.0) return fail(LSSVM_EBADLABEL, "labels must be +1 or -1");
  const double delta0 = g_ctx->p[0];
  const double t_setup = ms_since(t0);
  MatvecTimer tm;
  LSSVM_HIP(tm.init(info && info->time_matvec, info ? info->matvec_times : nullptr,
                    info ? info->matvec_times_capacity : 0));

  // ---- a4 + a5: conjugate gradients
  // Iterations are enqueued in batches (1, 2, 4, ... up to 32) and the status
  // is read once per batch; kernels queued after the stop return at once, so
  // the iterate is the one of the stopping iteration. CG stops on eps, on
  // curvature breakdown, or stalled: at a residual recomputation neither the
  // true residual nor the energy set a new minimum (the iterate is then the
  // one with the smallest recomputed residual).
  const auto t1 = clock_t_::now();
  if (max_iter <= 0) max_iter = g.N;
  int64_t queued = 0, it = 0;
  bool done = delta0 == 0.0;  // all labels equal: alpha~ = 0 solves the system
  bool broke = false, stalled = false;
  double delta = delta0;
  int status = LSSVM_OK;
  int64_t batch = 1;   // fused (small) problems start at 8, below
  double* st = g_ctx->p;
  int64_t warm_products = 0;
  if (info && info->warm_start && !done) {
    // x0 = the caller's alpha~, r0 = rhs - Q~ x0, dir = r0; the stop threshold
    // set from rhs^T rhs above is kept
    LSSVM_HIP(launch_pad_to_f64<T>(alpha_out, g.N, w.x, g.NP, w.scal, s));
    LSSVM_TRY(matvec_partials<T>(g, w, kp, kernel, w.x, s));
    LSSVM_HIP(launch_cg_residual(rank_one(g, w, kernel, C, w.x), g.NP, g.N, w.rhs,
                                 w.r, w.bp1, w.bp2, s));
    LSSVM_HIP(launch_warm_start(w.bp1, w.bp2, g.nb, w.scal, w.r, w.dir, w.x, w.xbest, g.NP, s));
    LSSVM_HIP(hipMemcpyAsync(st, w.scal + S_STATUS, ST_COUNT * sizeof(double),
                             hipMemcpyDeviceToHost, s));
    LSSVM_HIP(hipStreamSynchronize(s));
    delta = st[ST_DELTA];
    done = st[ST_DONE] != 0.0;
    warm_products = 1;
    if (!std::isfinite(delta))
      return fail(LSSVM_ENONFINITE, "the warm-start alpha gives a non-finite residual");
  }
  // Iterations queued after the stop return at once but still pay for their
  // launches, so once two status reads give a rate of decrease of r^T r, a
  // batch is also capped at the iterations that rate needs to reach the stop
  // threshold (with a quarter to spare).
  int64_t it_prev = 0, need = max_iter;
  double delta_prev = delta;
  const bool fused = fused_iteration(g, kernel);
  // A fused iteration takes ~15 us and a status read-back ~30 us: small
  // problems start with 8 iterations queued (those run past the stop return at
  // once, a few microseconds each)
  if (fused) batch = 8;
  while (!done && queued < max_iter) {
    const int64_t nq = std::min<int64_t>(std::min(batch, need), max_iter - queued);
    for (int64_t b = 0; b < nq; ++b) {
      const int64_t k = ++queued;
      const int par = (int)((k - 1) & 1);  // r^T r of the current iterate lives in S_DHIST + par
      const bool refresh = k % kReplaceEvery == 0;
      if (fused && !refresh) {   // product and vector work in one launch
        LSSVM_HIP(tm.start(s, k));
        TileArgs<T> a = sym_args<T>(g, w, kp, kernel, w.dir);
        a.stop = w.scal + S_STATUS + ST_DONE;
        FusedCg f{w.ticket, rank_one(g, w, kernel, C, w.dir), w.qv, w.x, w.r, w.dir, w.scal,
                  w.hist, g.NP, g.N, k, g.NP + 1, par};
        const int64_t nwg = kernel == LSSVM_LINEAR ? linear_launch(g, a) : tri_count(g.nT);
        LSSVM_HIP(launch_tiles_cg<T>(a, kernel, nwg, f, s));
        LSSVM_HIP(tm.stop(s));
        continue;
      }
      LSSVM_TRY(timed_matvec<T>(g, w, kp, kernel, w.dir, s, tm, k));
      LSSVM_HIP(launch_cg_gather(rank_one(g, w, kernel, C, w.dir), g.NP, g.N, w.qv, w.bp0, s));
      if (refresh) {
        LSSVM_HIP(launch_cg_update(1, w.bp0, g.nb, w.scal, par, w.dir, w.qv, w.x, w.r, w.bp1,
                                   g.NP, s));
        LSSVM_TRY(timed_matvec<T>(g, w, kp, kernel, w.x, s, tm, k));
        LSSVM_HIP(launch_cg_residual(rank_one(g, w, kernel, C, w.x), g.NP, g.N, w.rhs,
                                     w.r, w.bp1, w.bp2, s));
      } else {
        LSSVM_HIP(launch_cg_update(0, w.bp0, g.nb, w.scal, par, w.dir, w.qv, w.x, w.r, w.bp1,
                                   g.NP, s));
      }
      LSSVM_HIP(launch_cg_direction(w.bp1, g.nb, w.scal, par, k, w.r, w.dir, g.NP, w.hist,
                                    g.NP + 1, refresh ? k / kReplaceEvery : 0, w.bp2, w.x,
                                    w.xbest, s));
    }
    LSSVM_HIP(hipMemcpyAsync(st, w.scal + S_STATUS, ST_COUNT * sizeof(double),
                             hipMemcpyDeviceToHost, s));
    LSSVM_HIP(hipStreamSynchronize(s));
    it = (int64_t)st[ST_ITER];
    done = st[ST_DONE] != 0.0;
    broke = st[ST_BREAK] != 0.0;
    stalled = st[ST_STALL] != 0.0;
    LSSVM_HIP(tm.harvest(done ? it : queued));
    if (broke) {
      it += 1;   // the update of the next iteration found the curvature
      status = fail(LSSVM_EBREAKDOWN, "CG breakdown at iteration %lld (d^T Q d = %g)",
                    (long long)it, st[ST_CURV]);
      break;
    }
    delta = st[ST_DELTA];
    if (log_enabled())
      std::fprintf(stderr, "[lssvm] CG iteration %lld: relative residual %.3e (%.1f ms)\n",
                   (long long)it, delta0 > 0.0 ? std::sqrt(delta / delta0) : 0.0,
                   ms_since(t1));
    batch = std::min<int64_t>(2 * batch, 32);
    need = max_iter;
    if (it > it_prev && delta > 0.0 && delta < delta_prev && st[ST_STOP] < delta) {
      const double per_it = std::log(delta / delta_prev) / (double)(it - it_prev);   // < 0
      const double to_go = std::log(st[ST_STOP] / delta) / per_it;                    // > 0
      if (to_go < 1e9) need = std::max<int64_t>(1, (int64_t)std::ceil(1.25 * to_go));
    }
    it_prev = it;
    delta_prev = delta;
  }
  const bool converged = done && !broke && !stalled;
  // products: one per iteration plus each completed residual recomputation
  // (a breakdown stops before its iteration's recomputation)
  const int64_t nmv = it + (broke ? it - 1 : it) / kReplaceEvery + warm_products;
  const double t_cg = ms_since(t1);
  auto report = [&](double t_total) {
    if (!info) return;
    info->iterations = it;
    info->stop_reason = broke     ? LSSVM_STOP_BREAKDOWN
                        : stalled ? LSSVM_STOP_STALL
                        : converged ? LSSVM_STOP_EPS
                                    : LSSVM_STOP_MAX_ITER;
    info->rel_residual = delta0 > 0.0 ? std::sqrt(delta / delta0) : 0.0;
    info->n_matvec = nmv;
    info->t_matvec_ms = tm.total_ms;
    info->n_matvec_timed = tm.count;
    info->t_setup_ms = t_setup;
    info->t_cg_ms = t_cg;
    info->t_total_ms = t_total;
  };
  if (status < 0) {   // breakdown: outputs untouched, the report says how far CG got
    report(ms_since(t0));
    return status;
  }
  if (stalled) {
    // the iterate of the smallest recomputed residual, whose r^T r the status reported
    LSSVM_HIP(hipMemcpyAsync(w.x, w.xbest, g.NP * sizeof(double), hipMemcpyDeviceToDevice, s));
    status = LSSVM_NOT_CONVERGED;
    fail(LSSVM_NOT_CONVERGED,
         "CG stalled after %lld iterations: no new minimum of the true residual or the energy "
         "(best relative residual %g)", (long long)it, std::sqrt(delta / delta0));
  } else if (!converged) {
    status = LSSVM_NOT_CONVERGED;
    fail(LSSVM_NOT_CONVERGED, "CG stopped after %lld iterations at relative residual %g",
         (long long)it, std::sqrt(delta / delta0));
  }
  if (info && info->residual_history && it > 0) {
    const int64_t nh = std::min(std::min(it, info->history_capacity), g.NP + 1);
    if (nh > 0) {
      LSSVM_HIP(hipMemcpyAsync(info->residual_history, w.hist, nh * sizeof(double),
                               hipMemcpyDeviceToHost, s));
      LSSVM_HIP(hipStreamSynchronize(s));
      for (int64_t k = 0; k < nh; ++k) info->residual_history[k] /= delta0;
    }
  }

  // ---- a6: alpha_m and b
  LSSVM_HIP(launch_bias<T>(w.x, w.q64, g.N, y, w.scal, 1.0 / C, alpha_out, s));
  LSSVM_HIP(hipMemcpyAsync(g_ctx->p, w.scal + S_B, sizeof(double), hipMemcpyDeviceToHost, s));
  LSSVM_HIP(hipStreamSynchronize(s));
  *b_out = g_ctx->p[0];

  const double t_total = ms_since(t0);   // the optional true-residual product is not training
  if (log_enabled())
    std::fprintf(stderr,
                 "[lssvm] train n=%lld d=%lld: %lld iterations, relative residual %.3e, "
                 "setup %.2f ms, cg %.2f ms, total %.2f ms\n",
                 (long long)n, (long long)d, (long long)it,
                 delta0 > 0.0 ? std::sqrt(delta / delta0) : 0.0, t_setup, t_cg, t_total);
  report(t_total);
  if (info && info->compute_true_residual) {
    double tr = 0.0;
    if (delta0 > 0.0) {
      LSSVM_TRY(matvec_partials<T>(g, w, kp, kernel, w.x, s));
      LSSVM_HIP(launch_true_residual(rank_one(g, w, kernel, C, w.x), g.NP, g.N, w.rhs, w.bp1, s));
      LSSVM_HIP(launch_finish_sum(w.bp1, g.nb, w.scal, S_TRUE, s));
      LSSVM_HIP(hipMemcpyAsync(g_ctx->p, w.scal + S_TRUE, sizeof(double), hipMemcpyDeviceToHost,
                               s));
      LSSVM_HIP(hipStreamSynchronize(s));
      tr = std::sqrt(g_ctx->p[0] / delta0);
    }
    info->true_rel_residual = tr;
  }
  return status;
}

// Workspace of lssvm_cg_step: the scalar area and two block-partial arrays.
constexpr int64_t kMaxStepLen = int64_t(1) << 34;
struct StepWs {
  double *scal, *bp0, *bp1;
  size_t bytes;
};
StepWs carve_step(int64_t N, void* base) {
  Carver c(base);
  StepWs w{};
  const int64_t nb = vec_blocks(N);
  w.scal = c.take<double>(S_COUNT);
  w.bp0 = c.take<double>(nb + 1);
  w.bp1 = c.take<double>(nb + 1);
  w.bytes = c.off;
  return w;
}

bool overlaps(const void* a, const void* b, int64_t bytes) {
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  return pa < pb + bytes && pb < pa + bytes;
}

template <typename T>
int matvec_impl(const T* X, int64_t n, int64_t d, int32_t kernel, const lssvm_params& kp,
                double C, const T* p, T* out, void* workspace, size_t ws_bytes, hipStream_t s) {
  const Geometry g = geometry<T>(n, d);
  TrainWs<T> w = carve_train<T>(g, nullptr);
  LSSVM_TRY(check_workspace(workspace, ws_bytes, w.bytes));
  w = carve_train<T>(g, workspace);
  LSSVM_HIP(g_ctx->ensure());
  LSSVM_TRY(setup_points<T>(g, w, X, kernel, kp, s));
  LSSVM_HIP(launch_pad_to_f64<T>(p, g.N, w.dir, g.NP, w.scal, s));
  LSSVM_TRY(matvec_partials<T>(g, w, kp, kernel, w.dir, s));
  LSSVM_HIP(launch_mv_out<T>(rank_one(g, w, kernel, C, w.dir), g.NP, g.N, out, s));
  LSSVM_HIP(hipStreamSynchronize(s));
  return LSSVM_OK;
}

template <typename T>
int predict_impl(const T* Xtr, const T* alpha, double b, int64_t n, int64_t d, int32_t kernel,
                 const lssvm_params& kp, const T* Xte, int64_t n_test, void* workspace,
                 size_t ws_bytes, T* scores, int32_t* labels, hipStream_t s) {
  const Geometry g = geometry<T>(n, d);
  PredictWs<T> w = carve_predict<T>(g, n_test, nullptr);
  LSSVM_TRY(check_workspace(workspace, ws_bytes, w.bytes));
  w = carve_predict<T>(g, n_test, workspace);
  LSSVM_HIP(g_ctx->ensure());
  LSSVM_HIP(hipMemsetAsync(w.flags, 0, F_COUNT * sizeof(int), s));
  if (kernel == LSSVM_LINEAR) {  // Eq. (15): w = sum_i alpha_i x_i, f(x) = <w, x> + b
    LSSVM_HIP(launch_linear_predict<T>(Xtr, alpha, n, d, Xte, n_test, b, w.lin_part, w.lin_w,
                                       w.lin_f, scores, labels, w.flags, s));
    LSSVM_HIP(hipMemcpyAsync(g_ctx->flags, w.flags, F_COUNT * sizeof(int), hipMemcpyDeviceToHost,
                             s));
    LSSVM_HIP(hipStreamSynchronize(s));
    if (g_ctx->flags[F_NONFINITE])
      return fail(LSSVM_ENONFINITE, "X_train or X_test holds a NaN or an infinity");
    return LSSVM_OK;
  }
  LSSVM_HIP(launch_layout<T>(Xtr, n, d, w.Xtr, g.ld, g.d_pad, w.flags, s));
  LSSVM_HIP(launch_layout<T>(Xte, n_test, d, w.Xte, w.ld_te, g.d_pad, w.flags, s));
  if (kernel == LSSVM_RBF) {  // squared norms are only read by the radial kernel
    LSSVM_HIP(launch_norms_q<T>(w.Xtr, g.ld, g.d_pad, -1, 0, kernel, kp.gamma, kp.coef0,
                                kp.degree, w.ntr, nullptr, nullptr, s));
    LSSVM_HIP(launch_norms_q<T>(w.Xte, w.ld_te, g.d_pad, -1, 0, kernel, kp.gamma, kp.coef0,
                                kp.degree, w.nte, nullptr, nullptr, s));
  }
  LSSVM_HIP(launch_pad_vec<T>(alpha, n, w.alpha, g.ld, s));
  TileArgs<T> a{};
  a.A = w.Xte;
  a.B = w.Xtr;
  a.lda = w.ld_te;
  a.ldb = g.ld;
  a.nkb = g.d_pad / g.bk;
  a.nA = w.nte;
  a.nB = w.ntr;
  a.wB = w.alpha;
  a.gamma = (T)kp.gamma;
  a.coef0 = (T)kp.coef0;
  a.rbf_scale = rbf_scale<T>(kp.gamma);
  a.degree = kp.degree;
  a.nTc = w.nTc;
  a.ksplit = 1;
  a.part = w.part;
  a.part_ld = w.ld_te;
  LSSVM_HIP(launch_tiles_gen<T>(a, kernel, w.nTr, s));
  LSSVM_HIP(launch_predict_finish<T>(w.part, w.nTc, w.ld_te, n_test, b, scores, labels, w.flags,
                                     s));
  LSSVM_HIP(hipMemcpyAsync(g_ctx->flags, w.flags, F_COUNT * sizeof(int), hipMemcpyDeviceToHost,
                           s));
  LSSVM_HIP(hipStreamSynchronize(s));
  if (g_ctx->flags[F_NONFINITE])
    return fail(LSSVM_ENONFINITE, "X_train or X_test holds a NaN or an infinity");
  return LSSVM_OK;
}

template <typename T>
size_t train_bytes(int64_t n, int64_t d) {
  return carve_train<T>(geometry<T>(n, d), nullptr).bytes;
}

template <typename T>
size_t predict_bytes(int64_t n, int64_t n_test, int64_t d) {
  return carve_predict<T>(geometry<T>(n, d), n_test, nullptr).bytes;
}

lssvm_params params_or_default(const lssvm_params* kp) {
  lssvm_params p{1.0, 0.0, 1};
  if (kp) p = *kp;
  return p;
}

}  // namespace
}  // namespace lssvm

using namespace lssvm;

extern "C" {

size_t lssvm_cg_step_workspace_bytes(int64_t N) {
  if (N < 1 || N > kMaxStepLen) return 0;
  return carve_step(N, nullptr).bytes;
}

int lssvm_cg_step(int64_t N, double* x, double* r, double* d, const double* q, double* scalars,
                  void* workspace, size_t workspace_bytes, void* stream) {
  try {
    g_last_error.clear();
    if (!x || !r || !d || !q || !scalars) return fail(LSSVM_EINVAL, "NULL array argument");
    if (N < 1 || N > kMaxStepLen)
      return fail(LSSVM_EINVAL, "N must be in [1, 2^34] (got %lld)", (long long)N);
    const void* v[4] = {x, r, d, q};
    for (int i = 0; i < 4; ++i)
      for (int j = i + 1; j < 4; ++j)
        if (overlaps(v[i], v[j], N * (int64_t)sizeof(double)))
          return fail(LSSVM_EINVAL, "x, r, d and q must not overlap");
    StepWs w = carve_step(N, workspace);
    LSSVM_TRY(check_workspace(workspace, workspace_bytes, w.bytes));
    LSSVM_HIP(launch_cg_step(N, x, r, d, q, scalars, w.scal, w.bp0, w.bp1,
                             static_cast<hipStream_t>(stream)));
    return LSSVM_OK;
  } catch (...) {
    return fail(LSSVM_EHIP, "internal error");
  }
}

int lssvm_cg_step_noalloc(int64_t N, double* x, double* r, double* d, const double* q,
                          double* scalars, void* stream) {
  try {
    g_last_error.clear();
    if (!x || !r || !d || !q || !scalars) return fail(LSSVM_EINVAL, "NULL array argument");
    if (N < 1 || N > kMaxStepLen)
      return fail(LSSVM_EINVAL, "N must be in [1, 2^34] (got %lld)", (long long)N);
    const void* v[4] = {x, r, d, q};
    for (int i = 0; i < 4; ++i)
      for (int j = i + 1; j < 4; ++j)
        if (overlaps(v[i], v[j], N * (int64_t)sizeof(double)))
          return fail(LSSVM_EINVAL, "x, r, d and q must not overlap");
    double* base = nullptr;
    int64_t capacity = 0;
    LSSVM_HIP(static_scratch(&base, &capacity));
    const size_t need = carve_step(N, nullptr).bytes;
    if (need > (size_t)capacity * sizeof(double))
      return fail(LSSVM_EINVAL, "N = %lld needs %zu bytes of scratch, above the %lld held",
                  (long long)N, need, (long long)(capacity * (int64_t)sizeof(double)));
    StepWs w = carve_step(N, base);
    LSSVM_HIP(launch_cg_step(N, x, r, d, q, scalars, w.scal, w.bp0, w.bp1,
                             static_cast<hipStream_t>(stream)));
    return LSSVM_OK;
  } catch (...) {
    return fail(LSSVM_EHIP, "internal error");
  }
}

int64_t lssvm_host_contexts(void) { return g_pool_size.load(); }

size_t lssvm_workspace_bytes(int64_t n, int64_t d, int32_t dtype) {
  if (n < 1 || d < 1 || n > kMaxPoints || d > kMaxFeatures || !valid_dtype(dtype)) return 0;
  return dtype == LSSVM_F64 ? train_bytes<double>(n, d) : train_bytes<float>(n, d);
}

size_t lssvm_predict_workspace_bytes(int64_t n, int64_t n_test, int64_t d, int32_t dtype) {
  if (n < 1 || n_test < 1 || d < 1 || n > kMaxPoints || n_test > kMaxPoints ||
      d > kMaxFeatures || !valid_dtype(dtype))
    return 0;
  return dtype == LSSVM_F64 ? predict_bytes<double>(n, n_test, d)
                            : predict_bytes<float>(n, n_test, d);
}

int32_t lssvm_tile_size(int32_t dtype) {
  if (dtype == LSSVM_F64) return TileShape<double>::T;
  if (dtype == LSSVM_F32) return TileShape<float>::T;
  return 0;
}

int lssvm_tile_plan(int64_t n, int64_t d, int32_t dtype, int32_t kernel, int64_t* plan) {
  clear_error();
  if (n < 2 || d < 1 || n > kMaxPoints || d > kMaxFeatures)
    return fail(LSSVM_EINVAL, "tile_plan: need 2 <= n <= 2^22 and 1 <= d <= 2^21");
  if (kernel != LSSVM_LINEAR && kernel != LSSVM_POLY && kernel != LSSVM_RBF)
    return fail(LSSVM_EINVAL, "tile_plan: unknown kernel");
  if (dtype != LSSVM_F64 && dtype != LSSVM_F32) return fail(LSSVM_EINVAL, "tile_plan: unknown dtype");
  if (!plan) return fail(LSSVM_EINVAL, "tile_plan: null plan");
  const Geometry g = dtype == LSSVM_F64 ? geometry<double>(n, d) : geometry<float>(n, d);
  const bool lin = kernel == LSSVM_LINEAR;
  plan[0] = product_split(g, kernel);
  plan[1] = lin ? g.lin_tail_q : g.tail_q;
  plan[2] = lin ? g.lin_tail_split : g.tail_split;
  if (plan[1] == 0) plan[2] = plan[0];
  return LSSVM_OK;
}

const char* lssvm_last_error(void) { return g_last_error.c_str(); }

int lssvm_train(const void* X, const void* y, int64_t n, int64_t d, int32_t dtype,
                int32_t kernel, const lssvm_params* kp, double C, double eps, int64_t max_iter,
                void* workspace, size_t workspace_bytes, void* alpha_out, double* b_out,
                lssvm_info* info, void* stream) {
  try {
    g_last_error.clear();
    if (!X || !y || !alpha_out || !b_out) return fail(LSSVM_EINVAL, "NULL array argument");
    if (!valid_dtype(dtype)) return fail(LSSVM_EINVAL, "unknown dtype %d", (int)dtype);
    LSSVM_TRY(check_sizes(n, d, 1));
    LSSVM_TRY(check_kernel_params(kernel, kp));
    if (!(C > 0.0) || !std::isfinite(C)) return fail(LSSVM_EINVAL, "C must be finite and > 0");
    if (!(eps > 0.0 && eps < 1.0)) return fail(LSSVM_EINVAL, "eps must lie in (0, 1)");
    if (max_iter < 0) return fail(LSSVM_EINVAL, "max_iter must be >= 0");
    if (info && info->residual_history == nullptr && info->history_capacity != 0)
      return fail(LSSVM_EINVAL, "history_capacity without residual_history");
    if (info && info->matvec_times == nullptr && info->matvec_times_capacity != 0)
      return fail(LSSVM_EINVAL, "matvec_times_capacity without matvec_times");
    const lssvm_params p = params_or_default(kp);
    hipStream_t s = static_cast<hipStream_t>(stream);
    CtxLease lease;
    if (dtype == LSSVM_F64)
      return train_impl<double>(static_cast<const double*>(X), static_cast<const double*>(y), n, d,
                                kernel, p, C, eps, max_iter, workspace, workspace_bytes,
                                static_cast<double*>(alpha_out), b_out, info, s);
    return train_impl<float>(static_cast<const float*>(X), static_cast<const float*>(y), n, d,
                             kernel, p, C, eps, max_iter, workspace, workspace_bytes,
                             static_cast<float*>(alpha_out), b_out, info, s);
  } catch (...) {
    return fail(LSSVM_EHIP, "internal error");
  }
}

int lssvm_predict(const void* X_train, const void* alpha, double b, int64_t n, int64_t d,
                  int32_t dtype, int32_t kernel, const lssvm_params* kp, const void* X_test,
                  int64_t n_test, void* workspace, size_t workspace_bytes, void* scores_out,
                  int32_t* labels_out, void* stream) {
  try {
    g_last_error.clear();
    if (!X_train || !alpha || !X_test || !scores_out)
      return fail(LSSVM_EINVAL, "NULL array argument");
    if (!valid_dtype(dtype)) return fail(LSSVM_EINVAL, "unknown dtype %d", (int)dtype);
    LSSVM_TRY(check_sizes(n, d, 1));
    if (n_test < 1 || n_test > kMaxPoints)
      return fail(LSSVM_EINVAL, "n_test must be in [1, 2^22] (got %lld)", (long long)n_test);
    LSSVM_TRY(check_kernel_params(kernel, kp));
    if (!std::isfinite(b)) return fail(LSSVM_EINVAL, "b must be finite");
    const lssvm_params p = params_or_default(kp);
    hipStream_t s = static_cast<hipStream_t>(stream);
    CtxLease lease;
    if (dtype == LSSVM_F64)
      return predict_impl<double>(static_cast<const double*>(X_train),
                                  static_cast<const double*>(alpha), b, n, d, kernel, p,
                                  static_cast<const double*>(X_test), n_test, workspace,
                                  workspace_bytes, static_cast<double*>(scores_out), labels_out,
                                  s);
    return predict_impl<float>(static_cast<const float*>(X_train),
                               static_cast<const float*>(alpha), b, n, d, kernel, p,
                               static_cast<const float*>(X_test), n_test, workspace,
                               workspace_bytes, static_cast<float*>(scores_out), labels_out, s);
  } catch (...) {
    return fail(LSSVM_EHIP, "internal error");
  }
}

int lssvm_matvec(const void* X, int64_t n, int64_t d, int32_t dtype, int32_t kernel,
                 const lssvm_params* kp, double C, const void* p, void* out, void* workspace,
                 size_t workspace_bytes, void* stream) {
  try {
    g_last_error.clear();
    if (!X || !p || !out) return fail(LSSVM_EINVAL, "NULL array argument");
    if (!valid_dtype(dtype)) return fail(LSSVM_EINVAL, "unknown dtype %d", (int)dtype);
    LSSVM_TRY(check_sizes(n, d, 2));
    LSSVM_TRY(check_kernel_params(kernel, kp));
    if (!(C > 0.0) || !std::isfinite(C)) return fail(LSSVM_EINVAL, "C must be finite and > 0");
    const lssvm_params pr = params_or_default(kp);
    hipStream_t s = static_cast<hipStream_t>(stream);
    CtxLease lease;
    if (dtype == LSSVM_F64)
      return matvec_impl<double>(static_cast<const double*>(X), n, d, kernel, pr, C,
                                 static_cast<const double*>(p), static_cast<double*>(out),
                                 workspace, workspace_bytes, s);
    return matvec_impl<float>(static_cast<const float*>(X), n, d, kernel, pr, C,
                              static_cast<const float*>(p), static_cast<float*>(out), workspace,
                              workspace_bytes, s);
  } catch (...) {
    return fail(LSSVM_EHIP, "internal error");
  }
}

}  // extern "C"
