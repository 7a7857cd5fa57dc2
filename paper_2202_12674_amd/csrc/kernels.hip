// gfx950 (MI355X, CDNA4) kernels of the LS-SVM training hot path.
//
// a1  k_layout        row-major points -> padded feature-blocked layout (Sec. III-A)
// a2  k_norms_q       squared norms, q_i = k(x_i, x_m) and k(x_m, x_m) (Sec. III-C2)
// a3  k_rhs_init      rhs = ybar - y_m 1 (Eq. (14)), CG start vectors
// a4  k_tiles         implicit K p on the matrix cores, one tile of the upper
//                     triangle per workgroup (Sec. III-C1), rows and columns
//                     accumulated from the same tile; k_cg_gather adds the
//                     rank-one and diagonal terms that make it Q~ p (Eqs. (13), (16))
// a5  k_cg_*          CG vector updates with fixed-order fp64 reductions (Sec. III-B)
// a6  k_bias          alpha_m and b (Eqs. (11), (15))
// a7  k_tiles<gen>    decision values sum_j alpha_j k(x_j, x) + b (Eq. (10))
//
// Every reduction sums in a fixed order (no floating-point atomics), so the
// results are bitwise reproducible run to run.
#include "lssvm_internal.h"
#include "tiles.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>

namespace lssvm {

namespace {

constexpr int NT = 256;  // threads per block of the vector kernels

// fp64 kernel value from a dot product and a directly summed squared distance.
template <int KER>
__device__ inline double kernel_value64(double dot, double dist, double gamma, double coef0,
                                        int degree) {
  if constexpr (KER == KLIN) {
    return dot;
  } else if constexpr (KER == KPOLY) {
    const double base = gamma * dot + coef0;
    double r = base;
    for (int e = 1; e < degree; ++e) r *= base;
    return r;
  } else {
    return exp(-gamma * dist);
  }
}

// A commutative operation over the 64 lanes of a wave, every lane receiving
// the result: the 8-lane half rows (DPP: half mirror, then the two quad
// exchanges), the 16-lane rows (DPP rotate by 8), then row pairs and wave
// halves (permlane swaps). Each step combines a lane's value with its
// partner's, and both partners combine the same two values, so all lanes end
// with the same bits. Cross-lane moves in registers: no LDS round trip per
// step, as a shuffle would take.
template <typename Op>
__device__ inline double wave_reduce(double v, Op op) {
  v = op(v, dpp_move<kDppRowHalfMirror>(v));
  v = op(v, dpp_move<kDppQuadXor1>(v));
  v = op(v, dpp_move<kDppQuadXor2>(v));
  v = op(v, dpp_move<kDppRowRor8>(v));
  {
    const uint64_t u = as_u64(v);
    const auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)u, (uint32_t)u, false, false);
    const auto hi =
        __builtin_amdgcn_permlane16_swap((uint32_t)(u >> 32), (uint32_t)(u >> 32), false, false);
    v = op(as_f64(lo[0], hi[0]), as_f64(lo[1], hi[1]));   // rows 2k and 2k + 1
  }
  {
    const uint64_t u = as_u64(v);
    const auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)u, (uint32_t)u, false, false);
    const auto hi =
        __builtin_amdgcn_permlane32_swap((uint32_t)(u >> 32), (uint32_t)(u >> 32), false, false);
    v = op(as_f64(lo[0], hi[0]), as_f64(lo[1], hi[1]));   // the two halves
  }
  return v;
}
struct AddOp {
  __device__ double operator()(double a, double b) const { return a + b; }
};
struct MaxOp {
  __device__ double operator()(double a, double b) const { return fmax(a, b); }
};
__device__ inline double wave_sum(double v) { return wave_reduce(v, AddOp{}); }

// Block-wide sum of one double per thread; every thread gets the result.
// Fixed reduction order, so every block that sums the same values agrees.
__device__ inline double block_sum(double v, double* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  double s = 0.0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += sh[i];
  return s;
}

// Sum of the nb per-block partials written by the previous kernel.
__device__ inline double sum_partials(const double* bp, int64_t nb, double* sh) {
  double v = 0.0;
  for (int64_t i = threadIdx.x; i < nb; i += blockDim.x) v += bp[i];
  return block_sum(v, sh);
}

// Block-wide S, T and Q_mm of the rank-one terms (every block sums the
// panel partials in the same order, so all blocks agree).
struct RankOneSums {
  double S, Tq, qmm;
};
__device__ inline RankOneSums rank_one_sums(const RankOne& c, double* sh) {
  RankOneSums r;
  r.S = sum_partials(c.pq, c.nT, sh);
  r.Tq = sum_partials(c.pq + c.nT, c.nT, sh);
  r.qmm = c.scal[S_KMM] + c.invC;
  return r;
}
// (Q~ p)_i from the tile sum (K p)_i, for i < N.
__device__ inline double qtilde_row(const RankOne& c, const RankOneSums& r, int64_t i, double kp) {
  return kp + (r.qmm - c.q64[i]) * r.S - r.Tq + c.p[i] * c.invC;
}

// Block-wide maximum of one non-negative double per thread; every thread
// gets it.
__device__ inline double block_max(double v, double* sh) {
  v = wave_reduce(v, MaxOp{});
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  double m = 0.0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) m = fmax(m, sh[i]);
  return m;
}

// Raise scal[S_PMAX], the bound on |p_j| that fixes the next product's
// fixed-point scale, to m >= 0: the bits of non-negative doubles order like
// their values, so an integer atomic max keeps the largest whatever the order.
__device__ inline void raise_pmax(double* scal, double m) {
  atomicMax(reinterpret_cast<unsigned long long*>(scal + S_PMAX),
            (unsigned long long)__double_as_longlong(m));
}

// Row i's sum over the product's tiles from its two fixed-point words (see
// fixed_add in tiles.h): the exact integer sum, rounded once to fp64 and
// unscaled. The words are cleared for the next product.
__device__ inline double fixed_take(int64_t* acc, int64_t i, double inv_scale) {
  const int64_t L = acc[2 * i], H = acc[2 * i + 1];
  acc[2 * i] = 0;
  acc[2 * i + 1] = 0;
  const int64_t H2 = H + (L >> 32);   // L >= 0: a sum of unsigned 32-bit limbs
  const int64_t L2 = L & 0xffffffffLL;
  return ((double)H2 * 4294967296.0 + (double)L2) * inv_scale;
}

// (K p)_i of a finished product, or NaN once any of its row sums was not finite.
__device__ inline double product_row(const RankOne& c, int64_t i, double inv_scale, bool bad) {
  const double t = fixed_take(c.acc, i, inv_scale);
  return bad ? __builtin_nan("") : t;
}

// ------------------------------------------------------------- a1 layout ----
// Panel-major, feature-blocked layout. Points are grouped in panels of TP
// (the tile edge) and features in blocks of BK; panel pb holds its nkb blocks
// one after the other, and inside a block each point's BK features are
// contiguous:
//   Xb[((pb * nkb + kb) * TP + (i % TP)) * BK + kk] = x_i[kb * BK + kk],  pb = i / TP.
// A tile therefore streams one contiguous run of memory per panel (few pages,
// coalesced), and each point's features in a block are contiguous (wide LDS
// reads). Zero fill beyond n points and d features.
//
// One workgroup moves one slab b = pb * nkb + kb (TP points x BK features,
// 16 KiB) as 16-byte chunks, PER per thread, all loads issued before the
// stores: chunk c of the slab is point c / CPR's features (c % CPR) VEC ..,
// a 16-byte piece of one input row, so the lanes of a load instruction read
// whole 128-byte row segments and the stores are one contiguous run. With
// vec_ok (d a multiple of VEC and X 16-byte aligned) a chunk is one vector
// load; otherwise each element is loaded on its own.
template <typename T, int BK, int TP>
__global__ __launch_bounds__(256) void k_layout(const T* __restrict__ X, int64_t n, int64_t d,
                                                T* __restrict__ Xb, int64_t nslab, int64_t nkb,
                                                int vec_ok, int* __restrict__ flags) {
  constexpr int VEC = 16 / (int)sizeof(T), CPR = BK / VEC, PER = TP * CPR / 256;
  static_assert(TP * CPR % 256 == 0, "a slab splits evenly over 256 threads");
  typedef T vec_t __attribute__((ext_vector_type(VEC)));
  for (int64_t b = blockIdx.x; b < nslab; b += gridDim.x) {
    const int64_t pb = b / nkb, kb = b - pb * nkb;
    vec_t v[PER];
    bool bad = false;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int c = u * 256 + (int)threadIdx.x;
      const int64_t i = pb * TP + c / CPR, k = kb * BK + (c % CPR) * VEC;
      if (vec_ok) {
        if (i < n && k < d) {
          v[u] = *reinterpret_cast<const vec_t*>(X + i * d + k);
        } else {
#pragma unroll
          for (int e = 0; e < VEC; ++e) v[u][e] = T(0);
        }
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[u][e] = (i < n && k + e < d) ? X[i * d + k + e] : T(0);
      }
#pragma unroll
      for (int e = 0; e < VEC; ++e) bad |= !__builtin_isfinite(v[u][e]);
    }
    T* dst = Xb + b * TP * BK;
#pragma unroll
    for (int u = 0; u < PER; ++u)
      *reinterpret_cast<vec_t*>(dst + (u * 256 + (int)threadIdx.x) * VEC) = v[u];
    if (bad) flags[F_NONFINITE] = 1;
  }
}

// ----------------------------------------------------------- a2 norms, q ----
// Threads per point of k_norms_q: two lane groups (even and odd feature
// blocks) of one thread per 16-byte chunk of a point's block row.
template <typename T>
constexpr int norms_threads_per_point() {
  return 2 * (TileShape<T>::BK * (int)sizeof(T) / 16);
}

// ||x_i||^2 and, if a pivot m is given, the cached q_i = k(x_i, x_m) for
// i < N (zero beyond) and k(x_m, x_m). fp64 sums. A workgroup takes PPB
// points, KSPL x CPR threads per point: each thread sums one 16-byte chunk of
// the point's row in every KSPL-th feature block (a wave reads whole 128-byte
// rows), and the point's partial sums are then combined over its lanes (xor
// 1, 2, 4, 8: a fixed order).
template <typename T, int BK, int TP, int KER>
__global__ __launch_bounds__(256) void k_norms_q(const T* __restrict__ Xb, int64_t ld,
                                                 int64_t nkb, int64_t m, int64_t N, double gamma,
                                                 double coef0, int degree, T* __restrict__ norms,
                                                 double* __restrict__ q64,
                                                 double* __restrict__ scal) {
  constexpr int VEC = 16 / (int)sizeof(T), CPR = BK / VEC, KSPL = 2, TPP = KSPL * CPR;
  static_assert(TPP == norms_threads_per_point<T>() && BK == TileShape<T>::BK, "launch shape");
  constexpr int PPB = 256 / TPP;
  static_assert(TP % PPB == 0, "a workgroup's points lie in one panel");
  typedef T vec_t __attribute__((ext_vector_type(VEC)));
  __shared__ double sh[NT / 64];
  const int q = (int)threadIdx.x % CPR, h = ((int)threadIdx.x / CPR) % KSPL;
  const int64_t i = (int64_t)blockIdx.x * PPB + (int64_t)threadIdx.x / TPP;   // < ld
  const int64_t bstride = (int64_t)TP * BK;   // elements between a point's feature blocks
  const T* pi = Xb + ((i / TP) * nkb * TP + i % TP) * BK + q * VEC;
  double nrm = 0.0, dot = 0.0, dist = 0.0;
  if (m >= 0) {
    const T* pm = Xb + ((m / TP) * nkb * TP + m % TP) * BK + q * VEC;
#pragma unroll 4
    for (int64_t kb = h; kb < nkb; kb += KSPL) {
      const vec_t xi = *reinterpret_cast<const vec_t*>(pi + kb * bstride);
      const vec_t xm = *reinterpret_cast<const vec_t*>(pm + kb * bstride);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const double xv = (double)xi[e], xw = (double)xm[e];
        nrm += xv * xv;
        dot += xv * xw;
        const double df = xv - xw;
        dist += df * df;
      }
    }
  } else {
#pragma unroll 4
    for (int64_t kb = h; kb < nkb; kb += KSPL) {
      const vec_t xi = *reinterpret_cast<const vec_t*>(pi + kb * bstride);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const double xv = (double)xi[e];
        nrm += xv * xv;
      }
    }
  }
#pragma unroll
  for (int off = 1; off < TPP; off <<= 1) {
    nrm += __shfl_xor(nrm, off);
    dot += __shfl_xor(dot, off);
    dist += __shfl_xor(dist, off);
  }
  if (q == 0 && h == 0) {
    norms[i] = (T)nrm;
    if (m >= 0) {
      const double kv = kernel_value64<KER>(dot, dist, gamma, coef0, degree);
      q64[i] = i < N ? kv : 0.0;
      if (i == m) scal[S_KMM] = kv;
    }
  }
  if (m >= 0) {   // the largest squared norm bounds the kernel values (fixed-point scale)
    const double mx = block_max(nrm, sh);
    if (threadIdx.x == 0)
      atomicMax(reinterpret_cast<unsigned long long*>(scal + S_NMAX),
                (unsigned long long)__double_as_longlong(mx));
  }
}

// ------------------------------------------------------------- a3 rhs -------
template <typename T>
__global__ __launch_bounds__(256) void k_rhs_init(const T* __restrict__ y, int64_t N, int64_t NP,
                                                  double* rhs, double* x, double* xbest, double* r,
                                                  double* dir, double* bpart, int* flags,
                                                  double* scal) {
  __shared__ double sh[NT / 64];
  const double ym = (double)y[N];
  if (blockIdx.x == 0 && threadIdx.x == 0 && !(ym == 1.0 || ym == -1.0)) flags[F_BADLABEL] = 1;
  double acc = 0.0, vmax = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    double v = 0.0;
    if (i < N) {
      const double yi = (double)y[i];
      if (!(yi == 1.0 || yi == -1.0)) flags[F_BADLABEL] = 1;
      v = yi - ym;
    }
    rhs[i] = v;
    x[i] = 0.0;
    xbest[i] = 0.0;
    r[i] = v;
    dir[i] = v;
    acc += v * v;
    vmax = fmax(vmax, fabs(v));
  }
  const double s = block_sum(acc, sh);
  const double mx = block_max(vmax, sh);
  if (threadIdx.x == 0) {
    bpart[blockIdx.x] = s;
    raise_pmax(scal, mx);   // the first product multiplies dir
  }
}

__global__ __launch_bounds__(256) void k_finish_delta0(const double* bpart, int64_t nb,
                                                       double* scal, double eps2,
                                                       const int* flags) {
  __shared__ double sh[NT / 64];
  const double s = sum_partials(bpart, nb, sh);
  if (threadIdx.x == 0) {
    scal[S_INFLAGS] = (flags[F_NONFINITE] ? 1.0 : 0.0) + (flags[F_BADLABEL] ? 2.0 : 0.0);
    scal[S_DELTA0] = s;
    scal[S_DHIST + 0] = s;
    double* st = scal + S_STATUS;
    st[ST_DELTA] = s;
    st[ST_CURV] = 0.0;
    st[ST_STEP] = 0.0;
    st[ST_ITER] = 0.0;
    st[ST_DONE] = s == 0.0 ? 1.0 : 0.0;   // all labels equal: alpha~ = 0 solves it
    st[ST_BREAK] = 0.0;
    st[ST_STOP] = eps2 * s;
    st[ST_STALL] = 0.0;
    scal[S_BEST] = s;     // x = 0: the residual is rhs, the energy 0
    scal[S_PHI] = 0.0;
  }
}

// ------------------------------------------------------------- a5 CG --------
// q = Q~ d from the product's row sums and the rank-one terms (zero beyond
// N), and the block partials of d^T q (c.p = d). Block 0 clears the bound on
// |p| for the next vector.
__global__ __launch_bounds__(256) void k_cg_gather(RankOne c, int64_t NP, int64_t N, double* qv,
                                                   double* bpart) {
  __shared__ double sh[NT / 64];
  if (c.scal[S_STATUS + ST_DONE] != 0.0) return;
  const RankOneSums ro = rank_one_sums(c, sh);
  const double inv = 1.0 / c.scal[S_FIXSC];
  const bool bad = c.flags[F_PRODUCT] != 0;
  double prod = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    const double t = product_row(c, i, inv, bad);
    const double q = i < N ? qtilde_row(c, ro, i, t) : 0.0;
    qv[i] = q;
    prod += c.p[i] * q;
  }
  const double t = block_sum(prod, sh);
  if (threadIdx.x == 0) {
    bpart[blockIdx.x] = t;
    if (blockIdx.x == 0) c.scal[S_PMAX] = 0.0;
  }
}

// x += a d and r -= a q (or only x += a d when the residual is about to be
// recomputed from x). On curvature breakdown (d^T q <= 0 or a step that is
// not finite) every block leaves the vectors as they are.
__global__ __launch_bounds__(256) void k_cg_update(int x_only, const double* __restrict__ bp_in,
                                                   int64_t nb, double* scal, int par,
                                                   const double* __restrict__ dir,
                                                   const double* __restrict__ qv, double* x,
                                                   double* r, double* bp_out, int64_t NP) {
  __shared__ double sh[NT / 64];
  if (scal[S_STATUS + ST_DONE] != 0.0) return;
  const double gam = sum_partials(bp_in, nb, sh);
  const double delta = scal[S_DHIST + par];
  const double alpha = delta / gam;
  const bool broke = !(gam > 0.0) || !__builtin_isfinite(alpha);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    scal[S_ALPHA] = alpha;
    scal[S_GAMMA] = gam;
    if (broke) {
      scal[S_STATUS + ST_CURV] = gam;
      scal[S_STATUS + ST_STEP] = alpha;
      scal[S_STATUS + ST_BREAK] = 1.0;
      scal[S_STATUS + ST_DONE] = 1.0;
    }
  }
  if (broke) return;
  double v = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    const double xi = x[i] + alpha * dir[i];
    x[i] = xi;
    if (!x_only) {
      const double ri = r[i] - alpha * qv[i];
      r[i] = ri;
      v += ri * ri;
    } else {
      v = fmax(v, fabs(xi));
    }
  }
  if (!x_only) {
    const double t = block_sum(v, sh);
    if (threadIdx.x == 0) bp_out[blockIdx.x] = t;
  } else {   // the residual recomputation multiplies x next
    const double mx = block_max(v, sh);
    if (threadIdx.x == 0) raise_pmax(scal, mx);
  }
}

// r = rhs - Q~ x from the product's row sums (c.p = x), and the block
// partials of r^T r and of (rhs + r)^T x. Block 0 clears the bound on |p|.
__global__ __launch_bounds__(256) void k_cg_residual(RankOne c, int64_t NP, int64_t N,
                                                     const double* __restrict__ rhs, double* r,
                                                     double* bp_out, double* bp_phi) {
  __shared__ double sh[NT / 64];
  if (c.scal[S_STATUS + ST_DONE] != 0.0) return;
  const RankOneSums ro = rank_one_sums(c, sh);
  const double inv = 1.0 / c.scal[S_FIXSC];
  const bool bad = c.flags[F_PRODUCT] != 0;
  double v = 0.0, e = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    const double t = product_row(c, i, inv, bad);
    const double ri = i < N ? rhs[i] - qtilde_row(c, ro, i, t) : 0.0;
    r[i] = ri;
    v += ri * ri;
    e += (rhs[i] + ri) * c.p[i];   // (rhs + r)^T x = -2 x (energy), zero beyond N
  }
  const double t = block_sum(v, sh);
  const double u = block_sum(e, sh);
  if (threadIdx.x == 0) {
    bp_out[blockIdx.x] = t;
    bp_phi[blockIdx.x] = u;
    if (blockIdx.x == 0) c.scal[S_PMAX] = 0.0;
  }
}

// ||rhs - Q~ x||^2 partials without touching r (final report only).
__global__ __launch_bounds__(256) void k_true_residual(RankOne c, int64_t NP, int64_t N,
                                                       const double* __restrict__ rhs,
                                                       double* bp_out) {
  __shared__ double sh[NT / 64];
  const RankOneSums ro = rank_one_sums(c, sh);
  const double inv = 1.0 / c.scal[S_FIXSC];
  const bool bad = c.flags[F_PRODUCT] != 0;
  double v = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    const double t = product_row(c, i, inv, bad);
    if (i >= N) continue;
    const double ri = rhs[i] - qtilde_row(c, ro, i, t);
    v += ri * ri;
  }
  const double t = block_sum(v, sh);
  if (threadIdx.x == 0) bp_out[blockIdx.x] = t;
}

// beta = r^T r (new) / r^T r (old); d = r + beta d (beta = 0 if the old
// r^T r is 0, an exact solution). Block 0 records the iteration in the
// status (and the history) and raises done once r^T r <= eps^2 r0^T r0.
//
// At the refresh-th residual recomputation (refresh > 0) r is a true
// residual. Unless it met eps, CG has progressed if r^T r or the energy
// -(rhs + r)^T x / 2 is below the smallest so far (start and earlier
// recomputations, kept in slot (refresh - 1) & 1 of S_BEST / S_PHI; the
// updated minima go to the other slot, so no block reads a slot that block 0
// writes). A new smallest r^T r copies x to xbest; no progress at all stops
// CG, stalled, and the status then reports the best r^T r, whose iterate is
// in xbest.
__global__ __launch_bounds__(256) void k_cg_direction(const double* __restrict__ bp_in, int64_t nb,
                                                      double* scal, int par, int64_t iter,
                                                      const double* __restrict__ r, double* dir,
                                                      int64_t NP, double* hist, int64_t hist_cap,
                                                      int64_t refresh,
                                                      const double* __restrict__ bp_phi,
                                                      const double* __restrict__ x,
                                                      double* __restrict__ xbest) {
  __shared__ double sh[NT / 64];
  double* st = scal + S_STATUS;
  if (st[ST_DONE] != 0.0) return;
  const double dnew = sum_partials(bp_in, nb, sh);
  const double dold = scal[S_DHIST + par];
  const bool conv = dnew <= st[ST_STOP];
  bool stall = false;
  double dbest = dnew;
  if (refresh > 0 && !conv) {   // uniform over the grid: every block sums the same partials
    const double phi = -0.5 * sum_partials(bp_phi, nb, sh);
    const int rd = (int)((refresh - 1) & 1), wr = rd ^ 1;
    const double bd = scal[S_BEST + rd], bphi = scal[S_PHI + rd];
    const bool lower_res = dnew < bd, lower_phi = phi < bphi;
    stall = !lower_res && !lower_phi;
    dbest = lower_res ? dnew : bd;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      scal[S_BEST + wr] = dbest;
      scal[S_PHI + wr] = lower_phi ? phi : bphi;
    }
    if (lower_res)
      for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP;
           i += (int64_t)gridDim.x * NT)
        xbest[i] = x[i];
  }
  const double beta = dold != 0.0 ? dnew / dold : 0.0;
  if (!stall) {
    double dmax = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP;
         i += (int64_t)gridDim.x * NT) {
      const double di = r[i] + beta * dir[i];
      dir[i] = di;
      dmax = fmax(dmax, fabs(di));
    }
    const double mx = block_max(dmax, sh);   // the next product multiplies dir
    if (threadIdx.x == 0) raise_pmax(scal, mx);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    scal[S_DHIST + (par ^ 1)] = dnew;
    st[ST_DELTA] = stall ? dbest : dnew;
    st[ST_CURV] = scal[S_GAMMA];
    st[ST_STEP] = scal[S_ALPHA];
    st[ST_ITER] = (double)iter;
    if (iter <= hist_cap) hist[iter - 1] = dnew;
    if (conv) st[ST_DONE] = 1.0;
    if (stall) {
      st[ST_STALL] = 1.0;
      st[ST_DONE] = 1.0;
    }
  }
}

// After r = rhs - Q~ x0 for a warm start: r^T r becomes the current delta
// (the stop threshold stays eps^2 rhs^T rhs), the direction starts at r, x0
// is the best iterate so far (with its residual and energy), and done is
// raised if x0 already meets the threshold.
__global__ __launch_bounds__(256) void k_warm_start(const double* __restrict__ bp_in,
                                                    const double* __restrict__ bp_phi, int64_t nb,
                                                    double* scal, const double* __restrict__ r,
                                                    double* dir, const double* __restrict__ x,
                                                    double* __restrict__ xbest, int64_t NP) {
  __shared__ double sh[NT / 64];
  const double dlt = sum_partials(bp_in, nb, sh);
  const double phi = -0.5 * sum_partials(bp_phi, nb, sh);
  double dmax = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    dir[i] = r[i];
    xbest[i] = x[i];
    dmax = fmax(dmax, fabs(r[i]));
  }
  const double mx = block_max(dmax, sh);
  if (threadIdx.x == 0) raise_pmax(scal, mx);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    double* st = scal + S_STATUS;
    scal[S_DHIST + 0] = dlt;
    scal[S_BEST] = dlt;
    scal[S_PHI] = phi;
    st[ST_DELTA] = dlt;
    if (dlt <= st[ST_STOP]) st[ST_DONE] = 1.0;
  }
}

// ------------------------------------------------- a5 on caller vectors -----
// One CG iteration on vectors the caller holds, with q = A d supplied: the
// caller's scalars[0] (r^T r) enters the double-buffered slot, the status is
// cleared with a stop threshold no r^T r reaches, and after the update and
// direction kernels the new r^T r, d^T q, step and beta go back to scalars.
__global__ void k_step_begin(const double* scalars, double* scal) {
  if (threadIdx.x == 0) {
    scal[S_DHIST + 0] = scalars[0];
    scal[S_DHIST + 1] = scalars[0];
    for (int k = 0; k < ST_COUNT; ++k) scal[S_STATUS + k] = 0.0;
    scal[S_STATUS + ST_STOP] = -1.0;
  }
}

__global__ __launch_bounds__(256) void k_dot_partials(const double* __restrict__ a,
                                                      const double* __restrict__ b, int64_t len,
                                                      double* bp_out) {
  __shared__ double sh[NT / 64];
  double v = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < len; i += (int64_t)gridDim.x * NT)
    v += a[i] * b[i];
  const double t = block_sum(v, sh);
  if (threadIdx.x == 0) bp_out[blockIdx.x] = t;
}

__global__ void k_step_end(const double* scal, double* scalars) {
  if (threadIdx.x == 0) {
    const bool broke = scal[S_STATUS + ST_BREAK] != 0.0;
    const double rr_old = scal[S_DHIST + 0], rr_new = scal[S_DHIST + 1];
    scalars[0] = broke ? rr_old : rr_new;
    scalars[1] = scal[S_GAMMA];
    scalars[2] = scal[S_ALPHA];
    scalars[3] = broke || rr_old == 0.0 ? 0.0 : rr_new / rr_old;   // rr_old = 0: r = 0, beta 0
  }
}

// ------------------------------------------------------------- a6 bias ------
// alpha = [x, -sum x] (last row of Eq. (11)); b = y_m + Q_mm sum x - q^T x (Eq. (15)).
template <typename T>
__global__ __launch_bounds__(1024) void k_bias(const double* __restrict__ x,
                                               const double* __restrict__ q64, int64_t N,
                                               const T* __restrict__ y, double* scal, double invC,
                                               T* __restrict__ alpha_out) {
  __shared__ double sh[1024 / 64];
  double sx = 0.0, sqx = 0.0, xmax = 0.0;
  for (int64_t i = threadIdx.x; i < N; i += blockDim.x) {
    const double xi = x[i];
    sx += xi;
    sqx += q64[i] * xi;
    xmax = fmax(xmax, fabs(xi));
    alpha_out[i] = (T)xi;
  }
  sx = block_sum(sx, sh);
  sqx = block_sum(sqx, sh);
  xmax = block_max(xmax, sh);
  if (threadIdx.x == 0) {
    scal[S_PMAX] = xmax;   // an optional true-residual product multiplies x next
    alpha_out[N] = (T)(-sx);
    const double qmm = scal[S_KMM] + invC;
    scal[S_B] = (double)y[N] + qmm * sx - sqx;
  }
}

template <typename T>
__global__ void k_single_point(const T* __restrict__ y, T* __restrict__ alpha_out, double* scal,
                               int* flags) {
  if (threadIdx.x == 0) {
    const double y0 = (double)y[0];
    const bool bad = !(y0 == 1.0 || y0 == -1.0);
    if (bad) flags[F_BADLABEL] = 1;
    if (!bad && flags[F_NONFINITE] == 0) alpha_out[0] = T(0);   // outputs untouched on error
    scal[S_B] = y0;
  }
}

// --------------------------------------------- a7 linear-kernel shortcut ----
// For the linear kernel Phi is the identity, so w = sum_i alpha_i x_i (Eq. (15))
// and f(x) = <w, x> + b: O((n + n_test) d) instead of a tile contraction.
// Partial sums of w over chunks of kLinRows points (coalesced over features),
// then a fixed-order sum of the chunks.
constexpr int kLinRows = 64;
constexpr int64_t kLinMaxChunks = 32768;   // stays inside the 65535 grid limit in y
inline int64_t lin_rows(int64_t n) {
  const int64_t r = (n + kLinMaxChunks - 1) / kLinMaxChunks;
  return r > kLinRows ? r : kLinRows;
}

template <typename T>
__global__ __launch_bounds__(256) void k_linear_w_part(const T* __restrict__ X,
                                                       const T* __restrict__ alpha, int64_t n,
                                                       int64_t d, int64_t rows,
                                                       double* __restrict__ part,
                                                       int* __restrict__ flags) {
  const int64_t k = (int64_t)blockIdx.x * NT + threadIdx.x;
  const int64_t i0 = (int64_t)blockIdx.y * rows;
  if (k >= d) return;
  double acc = 0.0;
  bool bad = false;
  const int64_t i1 = i0 + rows < n ? i0 + rows : n;
  for (int64_t i = i0; i < i1; ++i) {
    const T xv = X[i * d + k];
    bad |= !__builtin_isfinite(xv);
    acc += (double)alpha[i] * (double)xv;
  }
  part[(int64_t)blockIdx.y * d + k] = acc;
  if (bad) flags[F_NONFINITE] = 1;
}

__global__ __launch_bounds__(256) void k_linear_w_sum(const double* __restrict__ part,
                                                      int64_t nchunks, int64_t d,
                                                      double* __restrict__ w) {
  const int64_t k = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (k >= d) return;
  double s = 0.0;
  for (int64_t c = 0; c < nchunks; ++c) s += part[c * d + k];
  w[k] = s;
}

// One block per test point: f = <w, x> (fp64) into a workspace vector; the
// bias, the scores and the labels follow in k_predict_finish once every
// point has been checked.
template <typename T>
__global__ __launch_bounds__(256) void k_linear_scores(const T* __restrict__ Xte, int64_t d,
                                                       const double* __restrict__ w,
                                                       double* __restrict__ f,
                                                       int* __restrict__ flags) {
  __shared__ double sh[NT / 64];
  const int64_t t = blockIdx.x;
  const T* x = Xte + t * d;
  double acc = 0.0;
  bool bad = false;
  for (int64_t k = threadIdx.x; k < d; k += NT) {
    const T xv = x[k];
    bad |= !__builtin_isfinite(xv);
    acc += (double)xv * w[k];
  }
  if (bad) flags[F_NONFINITE] = 1;
  const double v = block_sum(acc, sh);
  if (threadIdx.x == 0) f[t] = v;
}

// ------------------------------------------------------------ tile order ----
// Visit order of the upper-triangle tiles: GROUP x GROUP super-tiles column by
// column (super-rows top down), and inside each super-tile column by column.
// Position of tile (i, j) in that order: the tiles of the super-columns to
// the left, the full super-tiles above it in its super-column, and the
// columns of its super-tile before it.
__device__ inline int64_t grouped_position(int64_t nT, int64_t G, int64_t i, int64_t j) {
  const int64_t c0 = (j / G) * G, r0 = (i / G) * G;
  const int64_t ncols = (nT < c0 + G ? nT : c0 + G) - c0;
  int64_t p = c0 * (c0 + 1) / 2 + r0 * ncols;
  for (int64_t c = c0; c < j; ++c) p += (c + 1 < r0 + G ? c + 1 : r0 + G) - r0;
  return p + (i - r0);
}

// Thread t takes tile (i, j) of the column-major triangle and writes it,
// packed (i << 16) | j, at its position. The last nd diagonal tiles
// (i = j >= nT - nd) move to the end of the order, the others close up:
// a split last round made of diagonal tiles adds into nd disjoint panels,
// one tile each, instead of into the few panels the order ends on.
// The same launch zeroes the flags, the scalars and the row-sum words.
__global__ __launch_bounds__(256) void k_setup_clear(int64_t nT, int64_t G, int64_t nd,
                                                     uint32_t* __restrict__ order,
                                                     int* __restrict__ flags,
                                                     double* __restrict__ scal,
                                                     int64_t* __restrict__ acc, int64_t nacc,
                                                     unsigned* __restrict__ ticket) {
  const int64_t t0 = (int64_t)blockIdx.x * NT + threadIdx.x, stride = (int64_t)gridDim.x * NT;
  if (t0 < F_COUNT) flags[t0] = 0;
  if (t0 == 0 && ticket) *ticket = 0u;
  if (t0 < S_COUNT) scal[t0] = 0.0;
  for (int64_t t = t0; t < nacc; t += stride) acc[t] = 0;
  if (!order) return;
  const int64_t W = nT * (nT + 1) / 2;
  for (int64_t t = t0; t < W; t += stride) {
    int64_t i, j;
    tri_index(t, i, j);
    int64_t p;
    if (i == j && i >= nT - nd) {
      p = W - nd + (i - (nT - nd));
    } else {
      // the moved tiles that came before it: diagonal positions grow with k
      p = grouped_position(nT, G, i, j);
      int64_t lo = nT - nd, hi = nT;   // first k in [lo, hi) placed after p
      while (lo < hi) {
        const int64_t mid = (lo + hi) / 2;
        if (grouped_position(nT, G, mid, mid) < p) lo = mid + 1;
        else hi = mid;
      }
      p -= lo - (nT - nd);
    }
    order[p] = (uint32_t)((i << 16) | j);
  }
}

// ---------------------------------------------------------- misc vectors ----
template <typename T>
__global__ __launch_bounds__(256) void k_pad_vec(const T* __restrict__ src, int64_t len,
                                                 T* __restrict__ dst, int64_t len_pad) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (i < len_pad) dst[i] = i < len ? src[i] : T(0);
}

template <typename T>
__global__ __launch_bounds__(256) void k_mv_out(RankOne c, int64_t NP, int64_t N,
                                                T* __restrict__ out) {
  __shared__ double sh[NT / 64];
  const RankOneSums ro = rank_one_sums(c, sh);
  const double inv = 1.0 / c.scal[S_FIXSC];
  const bool bad = c.flags[F_PRODUCT] != 0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    const double t = product_row(c, i, inv, bad);
    if (i < N) out[i] = (T)qtilde_row(c, ro, i, t);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_predict_finish(const double* __restrict__ part,
                                                        int64_t nslots, int64_t ld, int64_t n_test,
                                                        double b, T* __restrict__ scores,
                                                        int32_t* __restrict__ labels,
                                                        const int* __restrict__ flags) {
  if (flags[F_NONFINITE] != 0) return;   // outputs untouched on error
  // 64 test points per workgroup: wave w sums slots w, w + 4, ... (eight
  // loads in flight per lane), then the four wave sums are added in order.
  __shared__ double sh[NT / 64][64];
  const int w = (int)threadIdx.x >> 6, l = (int)threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 64 + l;
  double s = 0.0;
  if (i < n_test) {
#pragma unroll 8
    for (int64_t sl = w; sl < nslots; sl += NT / 64) s += part[sl * ld + i];
  }
  sh[w][l] = s;
  __syncthreads();
  if (w == 0 && i < n_test) {
    double f = b;
#pragma unroll
    for (int v = 0; v < NT / 64; ++v) f += sh[v][l];
    scores[i] = (T)f;
    if (labels) labels[i] = f > 0.0 ? 1 : -1;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_pad_to_f64(const T* __restrict__ src, int64_t len,
                                                    double* __restrict__ dst, int64_t len_pad,
                                                    double* scal) {
  __shared__ double sh[NT / 64];
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  const double v = i < len ? (double)src[i] : 0.0;
  if (i < len_pad) dst[i] = v;
  if (scal) {   // a product multiplies dst next
    const double mx = block_max(fabs(v), sh);
    if (threadIdx.x == 0) raise_pmax(scal, mx);
  }
}

__global__ __launch_bounds__(256) void k_finish_sum(const double* bpart, int64_t nb, double* scal,
                                                    int slot) {
  __shared__ double sh[NT / 64];
  const double s = sum_partials(bpart, nb, sh);
  if (threadIdx.x == 0) scal[slot] = s;
}

// ------------------------------------------------ fused small iteration ----
// One CG iteration in one launch (launch_tiles_cg): the tiles of q = K d as
// in k_tiles, then the workgroup that finishes last does what k_cg_gather,
// k_cg_update and k_cg_direction do, for all rows at once. Each workgroup
// fences its partial sums (device-scope release) before it takes a ticket;
// the one that draws the last ticket fences again (acquire) and reads them
// all. Rows r = tid + 256 k sit in registers (NP <= 1024 -> k < 4). ONE:
// linear tiles split into single feature blocks (see tile_body).
template <typename T, int KER, bool ONE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_tiles_cg(
    TileArgs<T> a, FusedCg f) {
  if (!tile_body<T, true, KER, kWhole, ONE>(a)) return;   // CG had already stopped
  __shared__ int last;
  __shared__ double sh[NT / 64];
  // Every wave releases its own writes (row sums, rank-one partials) at agent
  // scope, then thread 0 draws a relaxed ticket; the workgroup that draws the
  // last one acquires before it reads. Release and acquire each on one side
  // only: full fences on both sides, and an acquire-release ticket, cost
  // ~1.8 us more per iteration.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(f.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
           (unsigned)(a.ntiles - 1);
  __syncthreads();
  if (!last) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  constexpr int R = (int)(kFusedMaxNP / NT);
  // Every global load of the vector step is issued here, at once: placed
  // where it is used, each would wait for the barrier of the reduction before
  // it and then for its own round trip, one after the other.
  const int tid = threadIdx.x;
  const RankOne& c = f.c;
  const double pS = tid < c.nT ? c.pq[tid] : 0.0;
  const double pT = tid < c.nT ? c.pq[c.nT + tid] : 0.0;
  const double kmm = f.scal[S_KMM], fxsc = f.scal[S_FIXSC];
  const double delta = f.scal[S_DHIST + f.par];
  double* st = f.scal + S_STATUS;
  const double stop = st[ST_STOP];
  const bool bad = c.flags[F_PRODUCT] != 0;
  int64_t lo[R], hi[R];
  double qm[R], dr[R], xr[R], rk[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int64_t i = tid + (int64_t)k * NT;
    lo[k] = hi[k] = 0;
    qm[k] = dr[k] = xr[k] = rk[k] = 0.0;
    if (i < f.NP) {
      lo[k] = c.acc[2 * i];
      hi[k] = c.acc[2 * i + 1];
      qm[k] = i < f.N ? c.q64[i] : 0.0;
      dr[k] = f.dir[i];
      xr[k] = f.x[i];
      rk[k] = f.r[i];
    }
  }
  // S and T of the rank-one terms (one reduction for both, each summed in
  // the order of block_sum)
  double S = wave_sum(pS), Tq = wave_sum(pT);
  {
    __shared__ double sh2[2][NT / 64];
    const int w = tid >> 6;
    if ((tid & 63) == 0) {
      sh2[0][w] = S;
      sh2[1][w] = Tq;
    }
    __syncthreads();
    S = Tq = 0.0;
    for (int v = 0; v < NT / 64; ++v) {
      S += sh2[0][v];
      Tq += sh2[1][v];
    }
  }
  const double qmm = kmm + c.invC, inv = 1.0 / fxsc;
  double qr[R];
  double g = 0.0;
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int64_t i = tid + (int64_t)k * NT;
    qr[k] = 0.0;
    if (i < f.NP) {
      c.acc[2 * i] = 0;   // cleared for the next product
      c.acc[2 * i + 1] = 0;
      const int64_t H2 = hi[k] + (lo[k] >> 32);   // as fixed_take
      const double t = bad ? __builtin_nan("")
                           : ((double)H2 * 4294967296.0 + (double)(lo[k] & 0xffffffffLL)) * inv;
      const double q = i < f.N ? t + (qmm - qm[k]) * S - Tq + dr[k] * c.invC : 0.0;
      qr[k] = q;
      f.qv[i] = q;
      g += dr[k] * q;
    }
  }
  const double gam = block_sum(g, sh);
  const double alpha = delta / gam;
  if (!(gam > 0.0) || !__builtin_isfinite(alpha)) {   // curvature breakdown: nothing moves
    if (threadIdx.x == 0) {
      f.scal[S_ALPHA] = alpha;
      f.scal[S_GAMMA] = gam;
      st[ST_CURV] = gam;
      st[ST_STEP] = alpha;
      st[ST_BREAK] = 1.0;
      st[ST_DONE] = 1.0;
      *f.ticket = 0u;
    }
    return;
  }
  double rr = 0.0;
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int64_t i = tid + (int64_t)k * NT;
    if (i < f.NP) {
      f.x[i] = xr[k] + alpha * dr[k];
      rk[k] = rk[k] - alpha * qr[k];
      f.r[i] = rk[k];
      rr += rk[k] * rk[k];
    }
  }
  const double dnew = block_sum(rr, sh);
  const double beta = delta != 0.0 ? dnew / delta : 0.0;
  double dmax = 0.0;
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int64_t i = threadIdx.x + (int64_t)k * NT;
    if (i < f.NP) {
      const double di = rk[k] + beta * dr[k];
      f.dir[i] = di;
      dmax = fmax(dmax, fabs(di));
    }
  }
  dmax = block_max(dmax, sh);
  if (threadIdx.x == 0) {
    f.scal[S_PMAX] = dmax;   // the next launch multiplies dir
    f.scal[S_ALPHA] = alpha;
    f.scal[S_GAMMA] = gam;
    f.scal[S_DHIST + (f.par ^ 1)] = dnew;
    st[ST_DELTA] = dnew;
    st[ST_CURV] = gam;
    st[ST_STEP] = alpha;
    st[ST_ITER] = (double)f.iter;
    if (f.iter <= f.hist_cap) f.hist[f.iter - 1] = dnew;
    if (dnew <= stop) st[ST_DONE] = 1.0;
    *f.ticket = 0u;   // the next launch starts after this one ends
  }
}

inline unsigned blocks_for(int64_t n) { return (unsigned)((n + NT - 1) / NT); }

}  // namespace

// ------------------------------------------------------------- launchers ----

hipError_t launch_setup_clear(int64_t nT, int64_t group, int64_t diag_last, uint32_t* order,
                              int* flags, double* scal, int64_t* acc, int64_t nacc,
                              unsigned* ticket, hipStream_t s) {
  const int64_t W = order ? nT * (nT + 1) / 2 : 0;
  const int64_t n = std::max<int64_t>(std::max<int64_t>(W, nacc), S_COUNT);
  const int64_t blocks = std::min<int64_t>((n + NT - 1) / NT, kVecBlocks);
  hipLaunchKernelGGL(k_setup_clear, dim3((unsigned)std::max<int64_t>(1, blocks)), dim3(NT), 0, s,
                     nT, group, diag_last, order, flags, scal, acc, nacc, ticket);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_layout(const T* X, int64_t n, int64_t d, T* Xt, int64_t ld, int64_t d_pad,
                         int* flags, hipStream_t s) {
  constexpr int BK = TileShape<T>::BK, TP = TileShape<T>::T, VEC = 16 / (int)sizeof(T);
  const int64_t nkb = d_pad / BK, nslab = (ld / TP) * nkb;
  const int vec_ok = d % VEC == 0 && reinterpret_cast<uintptr_t>(X) % 16 == 0;
  // slab-stride: the slab count can exceed what one dispatch should hold
  const int64_t blocks = std::min<int64_t>(nslab, int64_t(1) << 20);
  hipLaunchKernelGGL((k_layout<T, BK, TP>), dim3((unsigned)blocks), dim3(256), 0, s, X, n, d, Xt,
                     nslab, nkb, vec_ok, flags);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_norms_q(const T* Xt, int64_t ld, int64_t d_pad, int64_t m, int64_t N,
                          int kernel, double gamma, double coef0, int degree, T* norms,
                          double* q64, double* scal, hipStream_t s) {
  constexpr int BK = TileShape<T>::BK, TP = TileShape<T>::T;
  const int64_t nkb = d_pad / BK;
  constexpr int PPB = 256 / norms_threads_per_point<T>();   // points per workgroup
  const unsigned g = (unsigned)(ld / PPB);                   // ld is a multiple of TP
  switch (kernel) {
    case KLIN:
      hipLaunchKernelGGL((k_norms_q<T, BK, TP, KLIN>), dim3(g), dim3(NT), 0, s, Xt, ld, nkb, m, N,
                         gamma, coef0, degree, norms, q64, scal);
      break;
    case KPOLY:
      hipLaunchKernelGGL((k_norms_q<T, BK, TP, KPOLY>), dim3(g), dim3(NT), 0, s, Xt, ld, nkb, m, N,
                         gamma, coef0, degree, norms, q64, scal);
      break;
    default:
      hipLaunchKernelGGL((k_norms_q<T, BK, TP, KRBF>), dim3(g), dim3(NT), 0, s, Xt, ld, nkb, m, N,
                         gamma, coef0, degree, norms, q64, scal);
      break;
  }
  return hipGetLastError();
}

// Workgroups per tile launch: 2^23 x 256 threads stays below the 2^32 work
// items one dispatch can count; a multiple of 8, so every chunk starts on XCD 0.
constexpr int64_t kMaxTileGrid = int64_t(1) << 23;

// Feature blocks per workgroup: even (the two-stage loop runs them in pairs)
// or exactly one (the single-block variant).
template <typename T>
inline bool blocks_ok(const TileArgs<T>& a, int64_t split) {
  if (split < 1 || a.nkb % split != 0) return false;
  const int64_t per = a.nkb / split;
  return per % 2 == 0 || per == 1;
}

template <typename T, bool SYM, int PART>
hipError_t launch_tiles(TileArgs<T> a, int kernel, int64_t nwg, hipStream_t s) {
  if (SYM && PART != kFixup && !blocks_ok(a, a.ksplit)) return hipErrorInvalidValue;
  a.ntiles = nwg;
  for (int64_t base = 0; base < nwg; base += kMaxTileGrid) {
    a.tile_base = base;
    const dim3 grid((unsigned)std::min(kMaxTileGrid, nwg - base));
    switch (kernel) {
      case KLIN:
        if (SYM && PART == kWhole && a.nkb == a.ksplit)   // a single feature block each
          hipLaunchKernelGGL((k_tiles_one<T>), grid, dim3(256), 0, s, a);
        else
          hipLaunchKernelGGL((k_tiles<T, SYM, KLIN, PART>), grid, dim3(256), 0, s, a);
        break;
      case KPOLY:
        hipLaunchKernelGGL((k_tiles<T, SYM, KPOLY, PART>), grid, dim3(256), 0, s, a);
        break;
      default:
        hipLaunchKernelGGL((k_tiles<T, SYM, KRBF, PART>), grid, dim3(256), 0, s, a);
        break;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename T>
hipError_t launch_tiles_sym(const TileArgs<T>& a, int kernel, int part, int64_t nwg,
                            hipStream_t s) {
  switch (part) {
    case kPartial: return launch_tiles<T, true, kPartial>(a, kernel, nwg, s);
    case kFixup: return launch_tiles<T, true, kFixup>(a, kernel, nwg, s);
    default: return launch_tiles<T, true, kWhole>(a, kernel, nwg, s);
  }
}

template <typename T>
hipError_t launch_tiles_gen(const TileArgs<T>& a, int kernel, int64_t nTr, hipStream_t s) {
  return launch_tiles<T, false, kWhole>(a, kernel, nTr * a.nTc, s);
}

template <typename T>
hipError_t launch_tiles_cg(const TileArgs<T>& a0, int kernel, int64_t nwg, const FusedCg& f,
                           hipStream_t s) {
  if (nwg > kMaxTileGrid) return hipErrorInvalidValue;   // small problems only: one chunk
  TileArgs<T> a = a0;
  a.ntiles = nwg;
  a.tile_base = 0;
  const bool one = kernel == KLIN && a.nkb == a.ksplit;   // a single feature block each
  if ((kernel != KLIN && a.ksplit != 1) || !blocks_ok(a, a.ksplit)) return hipErrorInvalidValue;
  switch (kernel) {
    case KLIN:
      if (one)
        hipLaunchKernelGGL((k_tiles_cg<T, KLIN, true>), dim3((unsigned)nwg), dim3(256), 0, s, a, f);
      else
        hipLaunchKernelGGL((k_tiles_cg<T, KLIN, false>), dim3((unsigned)nwg), dim3(256), 0, s, a,
                           f);
      break;
    case KPOLY:
      hipLaunchKernelGGL((k_tiles_cg<T, KPOLY, false>), dim3((unsigned)nwg), dim3(256), 0, s, a, f);
      break;
    default:
      hipLaunchKernelGGL((k_tiles_cg<T, KRBF, false>), dim3((unsigned)nwg), dim3(256), 0, s, a, f);
      break;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_rhs_init(const T* y, int64_t N, int64_t NP, double* rhs, double* x,
                           double* xbest, double* r, double* dir, double* bpart, int* flags,
                           double* scal, hipStream_t s) {
  hipLaunchKernelGGL(k_rhs_init<T>, dim3((unsigned)cg_blocks(NP)), dim3(NT), 0, s, y, N, NP, rhs,
                     x, xbest, r, dir, bpart, flags, scal);
  return hipGetLastError();
}

hipError_t launch_finish_delta0(const double* bpart, int64_t nb, double* scal, double eps2,
                                const int* flags, hipStream_t s) {
  hipLaunchKernelGGL(k_finish_delta0, dim3(1), dim3(NT), 0, s, bpart, nb, scal, eps2, flags);
  return hipGetLastError();
}

hipError_t launch_cg_gather(const RankOne& c, int64_t NP, int64_t N, double* qv, double* bpart,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_cg_gather, dim3((unsigned)cg_blocks(NP)), dim3(NT), 0, s, c, NP, N, qv,
                     bpart);
  return hipGetLastError();
}

hipError_t launch_cg_update(int x_only, const double* bp_in, int64_t nb, double* scal, int par,
                            const double* dir, const double* qv, double* x, double* r,
                            double* bp_out, int64_t NP, hipStream_t s) {
  hipLaunchKernelGGL(k_cg_update, dim3((unsigned)cg_blocks(NP)), dim3(NT), 0, s, x_only, bp_in,
                     nb, scal, par, dir, qv, x, r, bp_out, NP);
  return hipGetLastError();
}

hipError_t launch_cg_residual(const RankOne& c, int64_t NP, int64_t N, const double* rhs, double* r,
                              double* bp_out, double* bp_phi, hipStream_t s) {
  hipLaunchKernelGGL(k_cg_residual, dim3((unsigned)cg_blocks(NP)), dim3(NT), 0, s, c, NP, N, rhs,
                     r, bp_out, bp_phi);
  return hipGetLastError();
}

hipError_t launch_true_residual(const RankOne& c, int64_t NP, int64_t N, const double* rhs,
                                double* bp_out, hipStream_t s) {
  hipLaunchKernelGGL(k_true_residual, dim3((unsigned)cg_blocks(NP)), dim3(NT), 0, s, c, NP, N,
                     rhs, bp_out);
  return hipGetLastError();
}

hipError_t launch_cg_direction(const double* bp_in, int64_t nb, double* scal, int par,
                               int64_t iter, const double* r, double* dir, int64_t NP,
                               double* hist, int64_t hist_cap, int64_t refresh,
                               const double* bp_phi, const double* x, double* xbest,
                               hipStream_t s) {
  hipLaunchKernelGGL(k_cg_direction, dim3((unsigned)cg_blocks(NP)), dim3(NT), 0, s, bp_in, nb,
                     scal, par, iter, r, dir, NP, hist, hist_cap, refresh, bp_phi, x, xbest);
  return hipGetLastError();
}

hipError_t launch_warm_start(const double* bp_in, const double* bp_phi, int64_t nb, double* scal,
                             const double* r, double* dir, const double* x, double* xbest,
                             int64_t NP, hipStream_t s) {
  hipLaunchKernelGGL(k_warm_start, dim3((unsigned)cg_blocks(NP)), dim3(NT), 0, s, bp_in, bp_phi,
                     nb, scal, r, dir, x, xbest, NP);
  return hipGetLastError();
}

hipError_t launch_cg_step(int64_t N, double* x, double* r, double* d, const double* q,
                          double* scalars, double* scal, double* bp0, double* bp1,
                          hipStream_t s) {
  const int64_t nb = vec_blocks(N);
  hipLaunchKernelGGL(k_step_begin, dim3(1), dim3(64), 0, s, scalars, scal);
  hipLaunchKernelGGL(k_dot_partials, dim3((unsigned)nb), dim3(NT), 0, s, d, q, N, bp0);
  hipLaunchKernelGGL(k_cg_update, dim3((unsigned)nb), dim3(NT), 0, s, 0, bp0, nb, scal, 0, d, q,
                     x, r, bp1, N);
  hipLaunchKernelGGL(k_cg_direction, dim3((unsigned)nb), dim3(NT), 0, s, bp1, nb, scal, 0,
                     (int64_t)1, r, d, N, (double*)nullptr, (int64_t)0, (int64_t)0,
                     (const double*)nullptr, (const double*)nullptr, (double*)nullptr);
  hipLaunchKernelGGL(k_step_end, dim3(1), dim3(64), 0, s, scal, scalars);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_bias(const double* x, const double* q64, int64_t N, const T* y, double* scal,
                       double invC, T* alpha_out, hipStream_t s) {
  hipLaunchKernelGGL(k_bias<T>, dim3(1), dim3(1024), 0, s, x, q64, N, y, scal, invC, alpha_out);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_single_point(const T* y, T* alpha_out, double* scal, int* flags,
                               hipStream_t s) {
  hipLaunchKernelGGL(k_single_point<T>, dim3(1), dim3(64), 0, s, y, alpha_out, scal, flags);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_pad_vec(const T* src, int64_t len, T* dst, int64_t len_pad, hipStream_t s) {
  hipLaunchKernelGGL(k_pad_vec<T>, dim3(blocks_for(len_pad)), dim3(NT), 0, s, src, len, dst,
                     len_pad);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_mv_out(const RankOne& c, int64_t NP, int64_t N, T* out, hipStream_t s) {
  hipLaunchKernelGGL(k_mv_out<T>, dim3((unsigned)cg_blocks(NP)), dim3(NT), 0, s, c, NP, N, out);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_predict_finish(const double* part, int64_t nslots, int64_t ld, int64_t n_test,
                                 double b, T* scores, int32_t* labels, const int* flags,
                                 hipStream_t s) {
  hipLaunchKernelGGL(k_predict_finish<T>, dim3((unsigned)((n_test + 63) / 64)), dim3(NT), 0, s,
                     part, nslots, ld, n_test, b, scores, labels, flags);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_pad_to_f64(const T* src, int64_t len, double* dst, int64_t len_pad,
                             double* scal, hipStream_t s) {
  hipLaunchKernelGGL(k_pad_to_f64<T>, dim3(blocks_for(len_pad)), dim3(NT), 0, s, src, len, dst,
                     len_pad, scal);
  return hipGetLastError();
}

hipError_t launch_finish_sum(const double* bpart, int64_t nb, double* scal, int slot,
                             hipStream_t s) {
  hipLaunchKernelGGL(k_finish_sum, dim3(1), dim3(NT), 0, s, bpart, nb, scal, slot);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_linear_predict(const T* Xtr, const T* alpha, int64_t n, int64_t d, const T* Xte,
                                 int64_t n_test, double b, double* part, double* w, double* f,
                                 T* scores, int32_t* labels, int* flags, hipStream_t s) {
  const int64_t rows = lin_rows(n);
  const int64_t nchunks = (n + rows - 1) / rows;
  const unsigned gx = (unsigned)((d + NT - 1) / NT);
  hipLaunchKernelGGL(k_linear_w_part<T>, dim3(gx, (unsigned)nchunks), dim3(NT), 0, s, Xtr, alpha,
                     n, d, rows, part, flags);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_linear_w_sum, dim3(gx), dim3(NT), 0, s, part, nchunks, d, w);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_linear_scores<T>, dim3((unsigned)n_test), dim3(NT), 0, s, Xte, d, w, f,
                     flags);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_predict_finish<T>(f, 1, n_test, n_test, b, scores, labels, flags, s);
}

// ------------------------------------------------- static device scratch ----
// The working memory of lssvm_cg_step_noalloc: the scalar area and the two
// block-partial arrays of one CG vector step, at most S_COUNT + 2 (1024 + 1)
// doubles whatever the vector length (the vector kernels run at most
// kVecBlocks blocks). Every device the library runs on holds one copy until
// the process ends; calls on one device share it.
constexpr int64_t kStaticScratchDoubles = 4096;   // 32 KiB
static_assert(S_COUNT + 2 * (kVecBlocks + 1) + 64 <= kStaticScratchDoubles,
              "static scratch holds the vector step's scalars and block partials");
static __device__ __align__(256) double scratch[kStaticScratchDoubles];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch_ptr[kMaxDevices] = {};   // device address of `scratch`, per device
}  // namespace

// In host code `scratch` names a host-side stand-in, not device memory: the
// device address is looked up once per device (with that device current) and
// only that address is handed to kernels.
hipError_t static_scratch(double** ptr, int64_t* capacity) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = static_cast<double*>(p);
  }
  *ptr = g_scratch_ptr[dev];
  *capacity = kStaticScratchDoubles;
  return hipSuccess;
}

int64_t linear_predict_part_elems(int64_t n, int64_t d) {
  const int64_t rows = lin_rows(n);
  return (n + rows - 1) / rows * d;
}

#define LSSVM_INSTANTIATE(T)                                                                      \
  template hipError_t launch_layout<T>(const T*, int64_t, int64_t, T*, int64_t, int64_t, int*,    \
                                       hipStream_t);                                              \
  template hipError_t launch_norms_q<T>(const T*, int64_t, int64_t, int64_t, int64_t, int,        \
                                        double, double, int, T*, double*, double*,                \
                                        hipStream_t);                                             \
  template hipError_t launch_tiles_sym<T>(const TileArgs<T>&, int, int, int64_t, hipStream_t);    \
  template hipError_t launch_tiles_gen<T>(const TileArgs<T>&, int, int64_t, hipStream_t);         \
  template hipError_t launch_tiles_cg<T>(const TileArgs<T>&, int, int64_t, const FusedCg&,        \
                                         hipStream_t);                                            \
  template hipError_t launch_rhs_init<T>(const T*, int64_t, int64_t, double*, double*, double*,   \
                                         double*, double*, double*, int*, double*, hipStream_t);  \
  template hipError_t launch_bias<T>(const double*, const double*, int64_t, const T*, double*,    \
                                     double, T*, hipStream_t);                                    \
  template hipError_t launch_single_point<T>(const T*, T*, double*, int*, hipStream_t);           \
  template hipError_t launch_pad_vec<T>(const T*, int64_t, T*, int64_t, hipStream_t);             \
  template hipError_t launch_mv_out<T>(const RankOne&, int64_t, int64_t, T*, hipStream_t);       \
  template hipError_t launch_predict_finish<T>(const double*, int64_t, int64_t, int64_t, double,  \
                                               T*, int32_t*, const int*, hipStream_t);            \
  template hipError_t launch_pad_to_f64<T>(const T*, int64_t, double*, int64_t, double*,          \
                                           hipStream_t);                                          \
  template hipError_t launch_linear_predict<T>(const T*, const T*, int64_t, int64_t, const T*,    \
                                               int64_t, double, double*, double*, double*, T*,    \
                                               int32_t*, int*, hipStream_t);

LSSVM_INSTANTIATE(float)
LSSVM_INSTANTIATE(double)

}  // namespace lssvm
