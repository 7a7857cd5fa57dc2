// Internal interface between the host runtime (api.cpp) and the gfx950
// kernels (kernels.hip). Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "tile_args.h"

namespace lssvm {

// Symmetric tiles are visited in GROUP x GROUP super-tiles of the upper
// triangle, and each of the 8 XCDs takes a contiguous run of that order, so
// the workgroups resident on one XCD share few point panels in its L2.
// 0 = plain column-by-column triangle order, no remap.
#ifndef LSSVM_TILE_GROUP
#define LSSVM_TILE_GROUP 8
#endif

// Slots of the small fp64 scalar area in the workspace.
enum Scalar : int {
  S_KMM = 0,     // k(x_m, x_m)
  S_DHIST = 1,   // r^T r of the current iterate, double-buffered: [1], [2]
  S_DELTA0 = 3,  // r0^T r0
  S_B = 4,       // bias
  S_ALPHA = 5,   // CG step length of the last update
  S_GAMMA = 6,   // curvature d^T Q~ d of the last update
  S_TRUE = 7,    // ||rhs - Q~ x||^2 (final report)
  S_STATUS = 8,  // 8 doubles read by the host after each batch of iterations:
                 // [0] r^T r of the last iteration run (on a stall: that of the
                 // best recomputed residual), [1] its curvature, [2] its step
                 // length, [3] its number, [4] done (converged, broken down or
                 // stalled), [5] breakdown, [6] stop threshold eps^2 r0^T r0,
                 // [7] stalled
  S_BEST = 16,   // smallest true r^T r so far (start, residual recomputations),
                 // double-buffered by recomputation: [16], [17]
  S_PHI = 18,    // smallest CG energy -(rhs + r)^T x / 2 so far, likewise: [18], [19]
  // Fixed-point row sums of the symmetric products (tiles.h): [20] max |p_j| of
  // the vector the next product multiplies (raised with an integer atomic max
  // on its bits by the kernel that writes the vector, cleared by the kernel
  // that reads the product), [21] max ||x_i||^2, [22] the scale 2^s the last
  // product used
  S_PMAX = 20,
  S_NMAX = 21,
  S_FIXSC = 22,
  S_INFLAGS = 23,   // the input flags as read after the right-hand side: 1 non-finite
                    // X, 2 a label other than +-1 (one read-back with S_DELTA0)
  S_COUNT = 24
};
enum StatusField : int { ST_DELTA = 0, ST_CURV = 1, ST_STEP = 2, ST_ITER = 3, ST_DONE = 4,
                         ST_BREAK = 5, ST_STOP = 6, ST_STALL = 7, ST_COUNT = 8 };

// The CG vector kernels run at most this many blocks of 256 threads (4 per
// CU), each striding over the vector, so every block can re-sum the previous
// kernel's block partials cheaply at any vector length.
constexpr int64_t kVecBlocks = 1024;
inline int64_t vec_blocks(int64_t len) {
  const int64_t b = (len + 255) / 256;
  return b < kVecBlocks ? (b > 0 ? b : 1) : kVecBlocks;
}

// The training's CG vector kernels (the readers of a product included: each
// row's sum is two words) run one block per 256 rows of the padded vectors,
// at most kVecBlocks, striding beyond that.
inline int64_t cg_blocks(int64_t NP) { return vec_blocks(NP); }

// Flags raised by kernels (int32 each).
// F_PRODUCT: a symmetric product had a row sum that is not finite (its
// entries then come out as NaN, so CG reports a breakdown).
enum Flag : int { F_NONFINITE = 0, F_BADLABEL = 1, F_PRODUCT = 2, F_COUNT = 4 };


// One symmetric product as its readers see it: (K p)_i in the fixed-point
// accumulators of the tiles, and the rank-one and diagonal terms of Q~ p that
// the tiles leave out (Eq. (13)): (Q~ p)_i = (K p)_i + (Q_mm - q_i) S - T +
// p_i / C for i < N, with S = sum_j p_j, T = sum_j q_j p_j (summed from the
// diagonal tiles' per-panel partials in a fixed order) and
// Q_mm = k(x_m, x_m) + 1/C. A reader clears the accumulators it reads.
struct RankOne {
  const double* pq;    // 2 nT panel partials: S_I, then T_I
  int64_t nT;
  int64_t* acc;        // fixed-point row sums (two words per row)
  const double* q64;   // q_i, zero beyond N
  const double* p;     // the vector multiplied, zero beyond N
  double* scal;        // k(x_m, x_m) at S_KMM, the product's scale at S_FIXSC
  const int* flags;    // F_PRODUCT
  double invC;
};

// One fused CG iteration for small problems (see launch_tiles_cg): the
// product's tiles, then, in the workgroup that finishes last, the vector work
// of k_cg_gather, k_cg_update and k_cg_direction on the whole vectors.
struct FusedCg {
  unsigned* ticket;   // zero before every launch; the last workgroup resets it
  RankOne c;          // c.p = the CG direction
  double *qv, *x, *r, *dir, *scal, *hist;
  int64_t NP, N, iter, hist_cap;
  int par;            // r^T r of the current iterate lives in S_DHIST + par
};
// Largest padded length the fused iteration handles: one workgroup reads every
// row sum and keeps each thread's rows (NP / 256) in registers.
constexpr int64_t kFusedMaxNP = 1024;

// The symmetric tiles' visit order (GROUP x GROUP super-tiles), packed
// (I << 16) | J, nT (nT + 1) / 2 entries.
// The first kernel of a training: zeroes the flags (F_COUNT ints), the
// scalars (S_COUNT doubles), the row-sum words (nacc int64) and the fused
// iteration's ticket (if given), and writes the tile visit order (order may
// be null: then nothing but the zeroing).
hipError_t launch_setup_clear(int64_t nT, int64_t group, int64_t diag_last, uint32_t* order,
                              int* flags, double* scal, int64_t* acc, int64_t nacc,
                              unsigned* ticket, hipStream_t s);

template <typename T>
hipError_t launch_layout(const T* X, int64_t n, int64_t d, T* Xt, int64_t ld, int64_t d_pad,
                         int* flags, hipStream_t s);
template <typename T>
hipError_t launch_norms_q(const T* Xt, int64_t ld, int64_t d_pad, int64_t m, int64_t N,
                          int kernel, double gamma, double coef0, int degree, T* norms,
                          double* q64, double* scal, hipStream_t s);
template <typename T>
// Symmetric tile launch of nwg workgroups doing `part` (a TilePart; a fixup
// launch has one workgroup per tile).
hipError_t launch_tiles_sym(const TileArgs<T>& a, int kernel, int part, int64_t nwg,
                            hipStream_t s);
template <typename T>
hipError_t launch_tiles_gen(const TileArgs<T>& a, int kernel, int64_t nTr, hipStream_t s);
// A whole CG iteration in one launch for small problems (NP <= kFusedMaxNP,
// a single whole-tile launch per
// product): the symmetric tiles of q = Q~ d, then the workgroup that
// finishes last (an atomic ticket after a device-scope release fence) adds the
// rank-one terms and does the update and the new direction, with the same
// status, stop test and breakdown handling as the separate kernels. Nothing
// waits on another workgroup.
template <typename T>
hipError_t launch_tiles_cg(const TileArgs<T>& a, int kernel, int64_t nwg, const FusedCg& f,
                           hipStream_t s);
// rhs = ybar - y_m 1, x = xbest = 0, r = dir = rhs, the block partials of
// r^T r; raises scal[S_PMAX] to max |dir| (the first product multiplies it).
template <typename T>
hipError_t launch_rhs_init(const T* y, int64_t N, int64_t NP, double* rhs, double* x,
                           double* xbest, double* r, double* dir, double* bpart, int* flags,
                           double* scal, hipStream_t s);
// CG kernels: once the status says done, every later kernel of the queue
// returns at once, so the host may enqueue iterations ahead of the test.
hipError_t launch_finish_delta0(const double* bpart, int64_t nb, double* scal, double eps2,
                                const int* flags, hipStream_t s);
// q = Q~ dir (c.p = dir) and the block partials of dir^T q.
hipError_t launch_cg_gather(const RankOne& c, int64_t NP, int64_t N, double* qv, double* bpart,
                            hipStream_t s);
hipError_t launch_cg_update(int x_only, const double* bp_in, int64_t nb, double* scal, int par,
                            const double* dir, const double* qv, double* x, double* r,
                            double* bp_out, int64_t NP, hipStream_t s);
// r = rhs - Q~ x (c.p = x), the block partials of r^T r and those of
// (rhs + r)^T x (minus twice the CG energy of x).
hipError_t launch_cg_residual(const RankOne& c, int64_t NP, int64_t N, const double* rhs, double* r,
                              double* bp_out, double* bp_phi, hipStream_t s);
// Warm start: delta = r0^T r0 from the block partials, dir = r0, the start as
// the best iterate so far (its residual and energy), done if already below
// the stop threshold.
hipError_t launch_warm_start(const double* bp_in, const double* bp_phi, int64_t nb, double* scal,
                             const double* r, double* dir, const double* x, double* xbest,
                             int64_t NP, hipStream_t s);
// One CG iteration on caller vectors of length N given q = A d: the scalars
// (device, 4 doubles) carry r^T r in and r^T r, d^T q, step, beta out.
hipError_t launch_cg_step(int64_t N, double* x, double* r, double* d, const double* q,
                          double* scalars, double* scal, double* bp0, double* bp1,
                          hipStream_t s);
// beta and the new direction; stop on eps. refresh > 0 marks the refresh-th
// residual recomputation: then r is a true residual, bp_phi holds the
// partials of (rhs + r)^T x, and CG stops, stalled, unless the residual or
// the energy sets a new minimum (x is copied to xbest on a new residual
// minimum).
hipError_t launch_cg_direction(const double* bp_in, int64_t nb, double* scal, int par,
                               int64_t iter, const double* r, double* dir, int64_t NP,
                               double* hist, int64_t hist_cap, int64_t refresh,
                               const double* bp_phi, const double* x, double* xbest,
                               hipStream_t s);
template <typename T>
hipError_t launch_bias(const double* x, const double* q64, int64_t N, const T* y, double* scal,
                       double invC, T* alpha_out, hipStream_t s);
// n = 1: alpha = [0] and b = y_0, alpha written only if the point and its
// label passed the checks (flags set by the layout kernel before it).
template <typename T>
hipError_t launch_single_point(const T* y, T* alpha_out, double* scal, int* flags, hipStream_t s);
template <typename T>
hipError_t launch_pad_vec(const T* src, int64_t len, T* dst, int64_t len_pad, hipStream_t s);
template <typename T>
hipError_t launch_mv_out(const RankOne& c, int64_t NP, int64_t N, T* out, hipStream_t s);
// scores = b + the sum of nslots partial slots; nothing is written if the
// input flags report a non-finite point.
template <typename T>
hipError_t launch_predict_finish(const double* part, int64_t nslots, int64_t ld, int64_t n_test,
                                 double b, T* scores, int32_t* labels, const int* flags,
                                 hipStream_t s);
// dst = src zero-padded, in fp64; with scal, also raises scal[S_PMAX] to max |dst|.
template <typename T>
hipError_t launch_pad_to_f64(const T* src, int64_t len, double* dst, int64_t len_pad,
                             double* scal, hipStream_t s);
hipError_t launch_finish_sum(const double* bpart, int64_t nb, double* scal, int slot,
                             hipStream_t s);
hipError_t launch_true_residual(const RankOne& c, int64_t NP, int64_t N, const double* rhs,
                                double* bp_out, hipStream_t s);

// Linear-kernel decision values through w = sum_i alpha_i x_i (Eq. (15)).
// part: linear_predict_part_elems(n, d) doubles; w: d doubles; f: n_test
// doubles (the inner products before the bias).
template <typename T>
hipError_t launch_linear_predict(const T* Xtr, const T* alpha, int64_t n, int64_t d, const T* Xte,
                                 int64_t n_test, double b, double* part, double* w, double* f,
                                 T* scores, int32_t* labels, int* flags, hipStream_t s);
int64_t linear_predict_part_elems(int64_t n, int64_t d);

// The device array that lssvm_cg_step_noalloc works in, for the current
// device: its address (resolved once per device) and its size in doubles.
hipError_t static_scratch(double** ptr, int64_t* capacity);

}  // namespace lssvm
