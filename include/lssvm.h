/*
 * lssvm.h - C ABI of the MI355X (gfx950) LS-SVM training hot path.
 *
 * Least-squares SVM training as in PLSSVM (arXiv 2202.12674): the bordered
 * system of Sec. II-F, Eq. (11), [Q 1; 1^T 0][alpha; b] = [y; 0] with
 * Q_ij = k(x_i, x_j) + delta_ij / C, is reduced around the last point
 * m = n - 1 (Eqs. (12)-(14)) to the SPD system
 *     Q~ alpha~ = ybar - y_m 1,      N = n - 1 unknowns,
 * which is solved by conjugate gradients (Sec. III-B). Q~ is never stored:
 * every product Q~ p recomputes its entries (Eq. (16))
 *     Q~_ij = k(x_i,x_j) + delta_ij/C - k(x_m,x_j) - k(x_i,x_m) + k(x_m,x_m) + 1/C
 * tile by tile on the matrix cores. alpha_m = -sum(alpha~) (last row of
 * Eq. (11)) and b follows Eq. (15).
 *
 * Conventions shared by every entry point:
 * - Array arguments are DEVICE pointers unless marked "host". The caller
 *   owns all memory; the library allocates no device memory. Scratch space
 *   comes from the caller's `workspace` (device, 256-byte aligned, at least
 *   the size reported by the matching *_workspace_bytes call).
 * - dtype is LSSVM_F64 or LSSVM_F32 and applies to every floating-point
 *   device array of the call. In LSSVM_F32 the point data, the matrix-core
 *   contraction and the kernel epilogue are fp32; CG vectors, dot products,
 *   CG scalars and b are fp64.
 * - Points are n x d, row-major (point i's d features contiguous).
 * - All work is enqueued on `stream` (a hipStream_t; NULL = default stream)
 *   and the call returns only after it has finished.
 * - Return value: LSSVM_OK (0), LSSVM_NOT_CONVERGED (1, the outputs hold the
 *   iterate CG stopped with) or a negative error code, described by
 *   lssvm_last_error(). On LSSVM_EINVAL, LSSVM_ENONFINITE, LSSVM_EBADLABEL and
 *   LSSVM_EBREAKDOWN the output arrays and b_out are left untouched (a report
 *   struct such as lssvm_info still records how far the call got); after
 *   LSSVM_EHIP, a failed HIP runtime call, their contents are unspecified.
 *   Argument checks run on the host before any GPU work. No C++ exception
 *   crosses this boundary.
 * - Calls on one stream are serialised by the caller; calls that share a
 *   workspace must not overlap.
 */
#ifndef LSSVM_H_
#define LSSVM_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of every floating-point device array of a call. */
enum { LSSVM_F64 = 0, LSSVM_F32 = 1 };

/* Kernel functions of Sec. II-E (kernel table). */
enum {
    LSSVM_LINEAR = 0, /* <x, z>                                  */
    LSSVM_POLY = 1,   /* (gamma <x, z> + coef0)^degree, gamma > 0 */
    LSSVM_RBF = 2     /* exp(-gamma ||x - z||^2),       gamma > 0 */
};

/* Status codes. */
enum {
    LSSVM_OK = 0,
    LSSVM_NOT_CONVERGED = 1, /* eps not met: max_iter reached (outputs = last iterate)
                                or CG stalled (outputs = best recomputed iterate)     */
    LSSVM_EINVAL = -1,       /* bad argument (checked on the host, no GPU work done)  */
    LSSVM_ENONFINITE = -2,   /* X (or X_test) holds a NaN or an infinity              */
    LSSVM_EBADLABEL = -3,    /* a label is not exactly +1 or -1                       */
    LSSVM_EBREAKDOWN = -4,   /* CG curvature d^T Q~ d <= 0 or not finite (an indefinite
                                Q~: polynomial kernel with coef0 < 0)                */
    LSSVM_EHIP = -5          /* a HIP runtime call failed                             */
};

/* Why CG ended (lssvm_info.stop_reason). */
enum {
    LSSVM_STOP_EPS = 0,       /* r^T r <= eps^2 rhs^T rhs (or nothing to solve)         */
    LSSVM_STOP_MAX_ITER = 1,  /* max_iter iterations without meeting eps               */
    LSSVM_STOP_STALL = 2,     /* no progress at a residual recomputation (eps too small) */
    LSSVM_STOP_BREAKDOWN = 3  /* d^T Q~ d <= 0: Q~ is not positive definite             */
};

/* Kernel parameters (Sec. II-E). gamma: poly and rbf (> 0). coef0: the
 * polynomial's additive constant r (>= 0 keeps Q~ positive definite).
 * degree: the polynomial's exponent (>= 1). Ignored where unused. */
typedef struct lssvm_params {
    double gamma;
    double coef0;
    int32_t degree;
} lssvm_params;

/* Training report (host struct). Fields marked "in" are read by the library,
 * all others are written by it. */
typedef struct lssvm_info {
    int64_t iterations;            /* CG iterations performed (on LSSVM_EBREAKDOWN: the
                                      iteration whose curvature was not positive)    */
    int64_t n_matvec;              /* implicit Q~ products (incl. residual refreshes) */
    double rel_residual;           /* sqrt(r^T r / rhs^T rhs) of the CG recurrence (of
                                      the returned iterate's true residual if CG
                                      stalled)                                        */
    double true_rel_residual;      /* ||rhs - Q~ x|| / ||rhs|| if requested, else -1  */
    double t_setup_ms;             /* layout, q-vector, right-hand side               */
    double t_cg_ms;                /* CG loop                                         */
    double t_total_ms;             /* whole training (without the optional true-
                                      residual product)                              */
    int32_t compute_true_residual; /* in: nonzero -> one extra product at the end     */
    int32_t warm_start;            /* in: nonzero -> CG starts from the first n-1
                                      entries of alpha_out (see lssvm_train)         */
    double* residual_history;      /* in: host array or NULL; receives r^T r / rhs^T rhs
                                      after each iteration                           */
    int64_t history_capacity;      /* in: length of residual_history                 */
    int32_t time_matvec;           /* in: nonzero -> time every Q~ product with HIP
                                      events recorded on `stream`                    */
    int32_t stop_reason;           /* why CG ended: LSSVM_STOP_*                     */
    double t_matvec_ms;            /* sum of the timed Q~ products (tile kernel only) */
    int64_t n_matvec_timed;        /* number of products in t_matvec_ms              */
    double* matvec_times;          /* in: host array or NULL; receives the duration in
                                      ms of each timed product, in order, up to
                                      matvec_times_capacity of them (time_matvec) */
    int64_t matvec_times_capacity; /* in: length of matvec_times                     */
} lssvm_info;

/* Device workspace needed by lssvm_train and lssvm_matvec for n points of
 * d features. Returns 0 if n or d is outside the supported range (below) or
 * dtype is unknown. */
size_t lssvm_workspace_bytes(int64_t n, int64_t d, int32_t dtype);

/* Device workspace needed by lssvm_predict. Returns 0 if a size is outside
 * the supported range or dtype is unknown. */
size_t lssvm_predict_workspace_bytes(int64_t n, int64_t n_test, int64_t d, int32_t dtype);

/*
 * Train an LS-SVM (Sec. II-F, Eqs. (11)-(15); CG of Sec. III-B).
 *
 * X         device, n x d row-major, dtype. Must be finite.
 * y         device, n labels, dtype, each exactly +1 or -1.
 * n, d      1 <= n <= 2^22 points, 1 <= d <= 2^21 features (the supported
 *           range of every entry point; LSSVM_EINVAL outside it).
 * kernel    LSSVM_LINEAR / LSSVM_POLY / LSSVM_RBF; kp its parameters (host, may
 *           be NULL for LSSVM_LINEAR).
 * C         regularisation, finite and > 0.
 * eps       relative-residual target, 0 < eps < 1: CG stops once
 *           r^T r <= eps^2 rhs^T rhs (rhs = ybar - y_m 1, the residual of x = 0).
 * max_iter  iteration cap; 0 means N = n - 1.
 * alpha_out device, n values, dtype: alpha~ followed by alpha_m = -sum(alpha~).
 *           With info->warm_start set it is also an input: CG starts at x0 =
 *           its first n - 1 entries (finite; a previous solution, or a saved
 *           iterate to resume from) instead of 0, with r0 = rhs - Q~ x0 (one
 *           more product, counted in n_matvec and t_cg_ms). The stop test stays
 *           relative to rhs, so a start that already meets it returns after 0
 *           iterations with alpha~ = x0 (alpha_m and b recomputed).
 * b_out     host, the bias of Eq. (15).
 * info      host, may be NULL.
 * CG details (Sec. III-B): the residual is recomputed as rhs - Q~ x every
 * 50th iteration. CG ends
 *   - converged, once r^T r <= eps^2 rhs^T rhs (LSSVM_OK);
 *   - at max_iter (LSSVM_NOT_CONVERGED, outputs from the last iterate);
 *   - stalled, when at a recomputation neither the true residual nor the CG
 *     energy x^T Q~ x / 2 - rhs^T x is below its smallest value at the start
 *     and at the earlier recomputations: eps lies below what the arithmetic
 *     attains (LSSVM_NOT_CONVERGED, outputs from the iterate with the
 *     smallest recomputed residual);
 *   - on curvature breakdown, d^T Q~ d <= 0 (LSSVM_EBREAKDOWN, outputs
 *     untouched; Q~ is positive definite for coef0 >= 0).
 * n = 1 or all labels equal give alpha = 0, b = y_m without iterating.
 */
int lssvm_train(const void* X, const void* y, int64_t n, int64_t d, int32_t dtype,
                int32_t kernel, const lssvm_params* kp, double C, double eps,
                int64_t max_iter, void* workspace, size_t workspace_bytes,
                void* alpha_out, double* b_out, lssvm_info* info, void* stream);

/*
 * Score points with a trained model: f(x) = sum_i alpha_i k(x_i, x) + b
 * (Eq. (10) with the sign carried by alpha), label +1 iff f(x) > 0 else -1.
 *
 * X_train    device, n x d row-major, dtype; alpha device, n values, dtype.
 * X_test     device, n_test x d row-major, dtype, 1 <= n_test <= 2^22. Must be
 *            finite.
 * scores_out device, n_test values, dtype.
 * labels_out device, n_test int32 values (+1/-1), may be NULL.
 * A NaN or an infinity in X_train or X_test returns LSSVM_ENONFINITE with
 * scores_out and labels_out untouched.
 */
int lssvm_predict(const void* X_train, const void* alpha, double b, int64_t n, int64_t d,
                  int32_t dtype, int32_t kernel, const lssvm_params* kp,
                  const void* X_test, int64_t n_test, void* workspace,
                  size_t workspace_bytes, void* scores_out, int32_t* labels_out,
                  void* stream);

/*
 * One implicit product out = Q~ p of the reduced system (Eqs. (13), (16)),
 * the unit of work of each CG iteration.
 *
 * X     device, n x d row-major, dtype, 2 <= n <= 2^22, 1 <= d <= 2^21.
 * p     device, N = n - 1 values, dtype. out device, N values, dtype.
 * Uses the lssvm_workspace_bytes(n, d, dtype) workspace.
 */
int lssvm_matvec(const void* X, int64_t n, int64_t d, int32_t dtype, int32_t kernel,
                 const lssvm_params* kp, double C, const void* p, void* out,
                 void* workspace, size_t workspace_bytes, void* stream);

/* Device workspace needed by lssvm_cg_step on vectors of length N (0 if N is
 * out of range). */
size_t lssvm_cg_step_workspace_bytes(int64_t N);

/*
 * One conjugate-gradient iteration (Sec. III-B) on caller-held fp64 device
 * vectors of length N, for callers that apply the symmetric positive definite
 * operator A themselves (for instance a product spread over several devices):
 * with q = A d already computed,
 *     gamma = d^T q,  a = rr / gamma,  x += a d,  r -= a q,
 *     rr' = r^T r,    beta = rr' / rr, d = r + beta d.
 * This is the vector work of one iteration of lssvm_train, in the same
 * kernels (three passes over the vectors: 8 reads and 3 writes of N doubles).
 *
 * x, r, d    device, N doubles each, updated in place; q device, N doubles,
 *            read. The four must not overlap.
 * scalars    device, 4 doubles: in [0] = rr (r^T r of the current iterate);
 *            out [0] = rr', [1] = gamma, [2] = a, [3] = beta. On curvature
 *            breakdown (gamma <= 0 or a not finite) x, r and d are left as
 *            they were, [0] keeps rr and [3] is 0. At an exact solution
 *            (rr = 0, so r = 0) beta is 0 and d becomes r.
 * workspace  device, lssvm_cg_step_workspace_bytes(N) bytes, 256-byte aligned;
 *            its contents need not survive between calls.
 * stream     HIP stream (NULL = default). Everything is enqueued; nothing is
 *            read back, so calls can follow each other without a host wait.
 *            Calls that share a workspace must not run concurrently.
 * Returns LSSVM_OK or LSSVM_EINVAL (NULL or aliased vectors, N < 1 or above
 * 2^34, workspace) before any GPU work, or LSSVM_EHIP.
 */
int lssvm_cg_step(int64_t N, double* x, double* r, double* d, const double* q, double* scalars,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * lssvm_cg_step without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation. The step works in a fixed array of 32 KiB
 * of device memory that the library holds on every device it runs on (until
 * the process ends), which covers every N the call accepts; the call
 * allocates nothing and writes no memset into the stream.
 *
 * Arguments, results and errors as lssvm_cg_step (N in [1, 2^34], else
 * LSSVM_EINVAL before any GPU work); `stream` must belong to the current
 * device. Every call on one device shares that device's array, so calls that
 * may overlap on one device (other streams, other host threads) race and
 * must be serialised by the caller; each call starts by writing the state it
 * needs, so nothing carries over from the previous call.
 */
int lssvm_cg_step_noalloc(int64_t N, double* x, double* r, double* d, const double* q,
                          double* scalars, void* stream);

/* Host contexts (a pinned buffer and timing events each) that the library
 * holds: calls lease one for their duration from a process-wide pool, so the
 * count is the largest number of calls that ever ran at once, not the number
 * of threads that ever called. Informational. */
int64_t lssvm_host_contexts(void);

/* Device workspace of lssvm_mfma_peak (a fixed size). */
size_t lssvm_mfma_peak_workspace_bytes(void);

/*
 * Sustained matrix-core rate in TFLOP/s of the instruction the tile kernel
 * uses for dtype (fp32: v_mfma_f32_32x32x2_f32, fp64: v_mfma_f64_16x16x4_f64),
 * measured by a kernel that issues only that instruction on every SIMD, with
 * HIP events on `stream` (one warm-up launch, median of three). A measurement
 * aid: it sets the tile kernel's rate against what the chip sustains, beside
 * the published peak. workspace: device, lssvm_mfma_peak_workspace_bytes()
 * bytes, 256-byte aligned (overwritten). Synchronizes `stream`.
 * Returns LSSVM_OK, LSSVM_EINVAL or LSSVM_EHIP.
 */
int lssvm_mfma_peak(int32_t dtype, void* workspace, size_t workspace_bytes, double* tflops_out,
                    void* stream);

/* Message for the last failing call on this thread ("" if none). The pointer
 * stays valid until the next call on this thread. */
const char* lssvm_last_error(void);

/* Tile edge (points per tile) that the matrix-core kernels use for dtype,
 * 0 for an unknown dtype. Informational: sizes need no padding by the caller. */
int32_t lssvm_tile_size(int32_t dtype);

/* How the implicit products of lssvm_train and lssvm_matvec lay out their
 * upper-triangle tiles over workgroups for n >= 2 points of d features.
 * On success writes plan[0..2] (host memory, caller-owned):
 *   plan[0]  workgroups per tile in the full rounds: 1, except for the
 *            linear kernel on problems with few tiles, whose features are
 *            split over 2..16 workgroups per tile (the partial sums add up
 *            because the linear kernel value is the inner product itself);
 *   plan[1]  tiles of a last partial round that run split finer (0 if none):
 *            the linear kernel runs them as the trailing workgroups of
 *            the same launch, split the same additive way; the other
 *            kernels park their partial inner products and sum them in a
 *            fix-up launch;
 *   plan[2]  workgroups per such tile (plan[0] when plan[1] is 0).
 * Every split leaves an even number of feature blocks per workgroup, except
 * on small problems (n <= 1025 without a split last round, whose CG
 * iterations are single launches): there the linear kernel's tiles split as
 * far as one round of workgroups allows, down to one feature block each.
 * Every product of a problem (CG iterations, residual recomputations,
 * lssvm_matvec) uses the same plan.
 * Returns LSSVM_EINVAL (plan untouched) for n, d, dtype or kernel out of
 * range or a null plan. Informational. */
int lssvm_tile_plan(int64_t n, int64_t d, int32_t dtype, int32_t kernel, int64_t* plan);

#ifdef __cplusplus
}
#endif

#endif /* LSSVM_H_ */
