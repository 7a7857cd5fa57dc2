// gfx950 (MI355X, CDNA4) kernels of the LS-SVM training hot path.
//
// a1  k_layout        row-major points -> padded feature-blocked layout (Sec. III-A)
// a2  k_norms_q       squared norms, q_i = k(x_i, x_m) and k(x_m, x_m) (Sec. III-C2)
// a3  k_rhs_init      rhs = ybar - y_m 1 (Eq. (14)), CG start vectors
// a4  k_tiles         implicit Q~ p (Eq. (16)) on the matrix cores, one tile of the
//                     upper triangle per workgroup (Sec. III-C1), rows and columns
//                     accumulated from the same tile
// a5  k_cg_*          CG vector updates with fixed-order fp64 reductions (Sec. III-B)
// a6  k_bias          alpha_m and b (Eqs. (11), (15))
// a7  k_tiles<gen>    decision values sum_j alpha_j k(x_j, x) + b (Eq. (10))
//
// Every reduction sums in a fixed order (no floating-point atomics), so the
// results are bitwise reproducible run to run.
#include "lssvm_internal.h"

#include <hip/hip_runtime.h>

#include <cmath>

namespace lssvm {

namespace {

constexpr int NT = 256;  // threads per block of the vector kernels

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef double doublex4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- MFMA ------
// One matrix-core instruction computes an M x M block D += A B with a
// contraction depth K. Lane l supplies A[l % M][l / M] and B[l / M][l % M];
// accumulator element v of lane l is D[row(v, l)][l % M].
template <typename T> struct Mfma;

template <> struct Mfma<float> {  // v_mfma_f32_32x32x2_f32
  static constexpr int M = 32, K = 2, NACC = 16;
  using acc_t = floatx16;
  __device__ static inline acc_t zero() {
    acc_t z;
#pragma unroll
    for (int i = 0; i < NACC; ++i) z[i] = 0.f;
    return z;
  }
  __device__ static inline acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static inline int row(int v, int lane) {
    return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
  }
};

template <> struct Mfma<double> {  // v_mfma_f64_16x16x4_f64
  static constexpr int M = 16, K = 4, NACC = 4;
  using acc_t = doublex4;
  __device__ static inline acc_t zero() {
    acc_t z;
#pragma unroll
    for (int i = 0; i < NACC; ++i) z[i] = 0.0;
    return z;
  }
  __device__ static inline acc_t mma(double a, double b, acc_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
  __device__ static inline int row(int v, int lane) { return (lane >> 4) + 4 * v; }
};

// Workgroup tiling of the contraction: a T x T tile, four waves in a 2 x 2
// grid, each wave owning a (T/2) x (T/2) block of MFMA accumulators.
template <typename T> struct TileCfg {
  static constexpr int BM = TileShape<T>::T;
  static constexpr int BK = TileShape<T>::BK;
  static constexpr int WM = BM / 2, WN = BM / 2;
};

template <typename T> __device__ inline T texp(T x);
template <> __device__ inline float texp<float>(float x) { return expf(x); }
template <> __device__ inline double texp<double>(double x) { return exp(x); }

// Kernel value from the inner product g = <x_i, x_j> (and squared norms for RBF).
template <int KER, typename T>
__device__ inline T kernel_value(T g, T ni, T nj, T gamma, T coef0, int degree) {
  if constexpr (KER == KLIN) {
    return g;
  } else if constexpr (KER == KPOLY) {
    const T base = gamma * g + coef0;
    T r = base;
    for (int e = 1; e < degree; ++e) r *= base;
    return r;
  } else {
    T dist = ni + nj - T(2) * g;
    dist = dist > T(0) ? dist : T(0);
    return texp<T>(-gamma * dist);
  }
}

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

// t = J (J + 1) / 2 + I with 0 <= I <= J: enumerates the upper triangle of
// tiles column by column, so consecutive workgroups share the column panel.
__device__ inline void tri_index(int64_t t, int64_t& I, int64_t& J) {
  int64_t j = (int64_t)((sqrt(8.0 * (double)t + 1.0) - 1.0) * 0.5);
  while ((j + 1) * (j + 2) / 2 <= t) ++j;
  while (j * (j + 1) / 2 > t) --j;
  J = j;
  I = t - j * (j + 1) / 2;
}

// Wait until all of this wave's vector memory operations (including direct
// global -> LDS loads) have completed: s_waitcnt vmcnt(0), other counters free.
__device__ inline void vm_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Block-wide sum of one double per thread; every thread gets the result.
// Fixed reduction order, so every block that sums the same values agrees.
__device__ inline double block_sum(double v, double* sh) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
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

// ------------------------------------------------------------- a1 layout ----
// Panel-major, feature-blocked layout. Points are grouped in panels of TP
// (the tile edge) and features in blocks of BK; panel pb holds its nkb blocks
// one after the other, and inside a block each point's BK features are
// contiguous:
//   Xb[((pb * nkb + kb) * TP + (i % TP)) * BK + kk] = x_i[kb * BK + kk],  pb = i / TP.
// A tile therefore streams one contiguous run of memory per panel (few pages,
// coalesced), and each point's features in a block are contiguous (wide LDS
// reads). Zero fill beyond n points and d features.
template <typename T, int BK, int TP>
__global__ __launch_bounds__(256) void k_layout(const T* __restrict__ X, int64_t n, int64_t d,
                                                T* __restrict__ Xb, int64_t ld, int64_t nkb,
                                                int* __restrict__ flags) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= nkb * ld * BK) return;
  const int64_t kk = idx % BK;
  const int64_t r = (idx / BK) % TP;
  const int64_t kb = (idx / ((int64_t)BK * TP)) % nkb;
  const int64_t pb = idx / ((int64_t)BK * TP * nkb);
  const int64_t i = pb * TP + r, k = kb * BK + kk;
  T v = T(0);
  if (i < n && k < d) {
    v = X[i * d + k];
    if (!__builtin_isfinite(v)) flags[F_NONFINITE] = 1;
  }
  Xb[idx] = v;
}

// ----------------------------------------------------------- a2 norms, q ----
// One thread per point: ||x_i||^2 and, if a pivot m is given, the cached
// q_i = k(x_i, x_m) for i < N (zero beyond) and k(x_m, x_m). fp64 sums.
template <typename T, int BK, int TP, int KER>
__global__ __launch_bounds__(256) void k_norms_q(const T* __restrict__ Xb, int64_t ld,
                                                 int64_t nkb, int64_t m, int64_t N, double gamma,
                                                 double coef0, int degree, T* __restrict__ norms,
                                                 T* __restrict__ qT, double* __restrict__ q64,
                                                 double* __restrict__ scal) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (i >= ld) return;
  double nrm = 0.0, dot = 0.0, dist = 0.0;
  const T* pi = Xb + ((i / TP) * nkb * TP + i % TP) * BK;   // point i, block 0
  const T* pm = m >= 0 ? Xb + ((m / TP) * nkb * TP + m % TP) * BK : pi;   // pivot, block 0
  for (int64_t kb = 0; kb < nkb; ++kb) {
    const T* xi = pi + kb * TP * BK;            // this point's BK features (padding is 0)
    if (m >= 0) {
      const T* xm = pm + kb * TP * BK;
#pragma unroll
      for (int kk = 0; kk < BK; ++kk) {
        const double xv = (double)xi[kk], xw = (double)xm[kk];
        nrm += xv * xv;
        dot += xv * xw;
        const double df = xv - xw;
        dist += df * df;
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < BK; ++kk) {
        const double xv = (double)xi[kk];
        nrm += xv * xv;
      }
    }
  }
  norms[i] = (T)nrm;
  if (m >= 0) {
    const double kv = kernel_value64<KER>(dot, dist, gamma, coef0, degree);
    const double qv = i < N ? kv : 0.0;
    q64[i] = qv;
    qT[i] = (T)qv;
    if (i == m) scal[S_KMM] = kv;
  }
}

// ---------------------------------------------------------- a4 tiles --------
// One T x T tile of the pairwise contraction G = X_I X_J^T per workgroup,
// feature blocks of BK staged global -> registers -> LDS (double-buffered)
// and fed to the matrix cores. The epilogue turns G into kernel values and
// then into Q~ entries (symmetric mode) and folds them into row sums
// (times p_j) and, off the diagonal, column sums (times p_i), so that each
// off-diagonal tile serves both triangles. Row and column sums are reduced
// across lanes and waves in a fixed order and written as fp64 partials,
// one slot per tile column (rows of block I) or tile row (rows of block J).
template <typename T, bool SYM, int KER>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_tiles(
    TileArgs<T> a) {
  using MF = Mfma<T>;
  using C = TileCfg<T>;
  constexpr int BM = C::BM, BK = C::BK;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int CPR = BK / VEC;             // 16-byte chunks per point row of a block
  static_assert(CPR == 8, "rows of 128 bytes: the XOR swizzle below spans 8 chunks");
  constexpr int CHUNKS = BM * CPR;          // chunks per panel slice
  constexpr int LOADS = CHUNKS / 256;       // direct loads per thread per panel
  static_assert(CHUNKS % 256 == 0, "panel must split evenly over 256 threads");
  constexpr int RB = C::WM / MF::M, CB = C::WN / MF::M;
  constexpr int WAVES_N = BM / C::WN, WAVES_M = BM / C::WM;
  static_assert(WAVES_M * WAVES_N == 4, "four waves per workgroup");
  // Lane group g = lane / M contracts the features [g * FPG, (g + 1) * FPG) of
  // each block, one per MFMA step; A and B use the same feature order.
  constexpr int FPG = BK / MF::K;           // features per lane group and block
  constexpr int CPG = FPG / VEC;            // chunks per lane group
  static_assert(FPG % VEC == 0, "lane operands are read in 16-byte chunks");
  typedef T vec_t __attribute__((ext_vector_type(VEC)));
  typedef __attribute__((address_space(1))) const void* gptr_t;
  typedef __attribute__((address_space(3))) void* lptr_t;

  // LDS: per stage and panel, BM rows of 128 bytes; chunk c of point p sits at
  // physical chunk p * 8 + (c ^ ((p >> 1) & 7)). A 16-byte read serves 16
  // lanes (16 consecutive points, one logical chunk) per cycle: rows of even
  // and odd p fall in opposite bank halves, and (p >> 1) & 7 spreads each
  // half over its 8 four-bank groups, so the reads are conflict-free; the
  // lane-linear direct loads are conflict-free by construction.
  // one array per stage and panel: with fixed names the compiler can tell the
  // stage being filled from the stage being read and need not wait in between
  __shared__ __attribute__((aligned(16))) T As0[CHUNKS * VEC];
  __shared__ __attribute__((aligned(16))) T As1[CHUNKS * VEC];
  __shared__ __attribute__((aligned(16))) T Bs0[CHUNKS * VEC];
  __shared__ __attribute__((aligned(16))) T Bs1[CHUNKS * VEC];
  __shared__ double red_r[WAVES_N][BM];
  __shared__ double red_c[WAVES_M][BM];

  if constexpr (SYM) {
    if (a.status && a.status[ST_DONE] != 0.0) return;   // CG already stopped
  }
  int64_t I, J;
  if constexpr (SYM) {
    if (a.order) {
      // workgroup w runs on XCD w % 8: give each XCD a contiguous run of the order
      const uint32_t G = gridDim.x, w = blockIdx.x;
      const uint32_t x = w % kNumXcd, per = G / kNumXcd, extra = G % kNumXcd;
      const uint32_t slot = x * per + (x < extra ? x : extra) + w / kNumXcd;
      const uint32_t packed = a.order[slot];
      I = packed >> 16;
      J = packed & 0xFFFFu;
    } else {
      tri_index((int64_t)blockIdx.x, I, J);
    }
  } else {
    I = (int64_t)blockIdx.x / a.nTc;
    J = (int64_t)blockIdx.x % a.nTc;
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  // panel I is nkb consecutive blocks of BM * BK elements
  const T* __restrict__ Ap = a.A + I * a.nkb * BM * BK;
  const T* __restrict__ Bp = a.B + J * a.nkb * BM * BK;
  constexpr int64_t astride = (int64_t)BM * BK, bstride = (int64_t)BM * BK;

  // Direct global -> LDS loads of block kb into stage buf: instruction u of
  // wave w fills physical chunks [(4u + w) * 64, +64) lane by lane; each lane
  // fetches the logical chunk that belongs at its physical slot.
  int goff[LOADS];   // element offset of this lane's logical chunk inside a slice
#pragma unroll
  for (int u = 0; u < LOADS; ++u) {
    const int P = (u * 4 + wave) * 64 + lane;
    const int p = P / CPR, c = (P % CPR) ^ ((p >> 1) & 7);
    goff[u] = (p * CPR + c) * VEC;
  }
  auto dload = [&](int64_t kb, T (&sa)[CHUNKS * VEC], T (&sb)[CHUNKS * VEC]) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int base = (u * 4 + wave) * 64 * VEC;   // wave-uniform LDS element offset
      __builtin_amdgcn_global_load_lds((gptr_t)(Ap + kb * astride + goff[u]),
                                       (lptr_t)(&sa[base]), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((gptr_t)(Bp + kb * bstride + goff[u]),
                                       (lptr_t)(&sb[base]), 16, 0, 0);
    }
  };

  typename MF::acc_t acc[RB][CB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int j = 0; j < CB; ++j) acc[i][j] = MF::zero();

  const int cl = lane % MF::M;   // point of this lane inside an MFMA block
  const int kl = lane / MF::M;   // lane group: which features of the block it contracts

  auto compute = [&](const T (&sa)[CHUNKS * VEC], const T (&sb)[CHUNKS * VEC]) {
    vec_t av[RB][CPG], bv[CB][CPG];
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int p = wm * C::WM + i * MF::M + cl;
#pragma unroll
      for (int q = 0; q < CPG; ++q)
        av[i][q] = *reinterpret_cast<const vec_t*>(
            &sa[(p * CPR + ((kl * CPG + q) ^ ((p >> 1) & 7))) * VEC]);
    }
#pragma unroll
    for (int j = 0; j < CB; ++j) {
      const int p = wn * C::WN + j * MF::M + cl;
#pragma unroll
      for (int q = 0; q < CPG; ++q)
        bv[j][q] = *reinterpret_cast<const vec_t*>(
            &sb[(p * CPR + ((kl * CPG + q) ^ ((p >> 1) & 7))) * VEC]);
    }
#pragma unroll
    for (int kk = 0; kk < FPG; ++kk)
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < CB; ++j)
          acc[i][j] = MF::mma(av[i][kk / VEC][kk % VEC], bv[j][kk / VEC][kk % VEC], acc[i][j]);
  };

  // Two stages: while block kb is multiplied out of one stage, block kb + 1
  // streams into the other. A stage is refilled only after the barrier that
  // ends the iteration which last read it. The host pads the features to an
  // even number of blocks, so both halves of the loop body always run.
  //
  // Scheduling fences, chosen by measurement per element type: left alone,
  // the compiler sinks the fp32 block loads into the last quarter of the
  // compute (less time to hide them) and hoists the fp64 wait and barrier
  // above the last MFMAs of the block (the wave then stalls with work
  // unissued). Pinning the loads above the compute gains ~0.5% for fp32;
  // keeping the wait behind every MFMA gains ~5% for fp64 (the other fence
  // costs each type a little).
  constexpr bool kPinLoads = sizeof(T) == 4, kPinWait = sizeof(T) == 8;
  const int64_t nkb = a.nkb;
  dload(0, As0, Bs0);
  vm_wait_all();
  __syncthreads();
  for (int64_t kb = 0; kb < nkb; kb += 2) {
    dload(kb + 1, As1, Bs1);
    if constexpr (kPinLoads) __builtin_amdgcn_sched_barrier(0);
    compute(As0, Bs0);
    if constexpr (kPinWait) __builtin_amdgcn_sched_barrier(0);
    vm_wait_all();     // this wave's part of block kb + 1 has landed
    __syncthreads();   // every wave's part has landed; stage 0 is free
    if (kb + 2 < nkb) dload(kb + 2, As0, Bs0);
    if constexpr (kPinLoads) __builtin_amdgcn_sched_barrier(0);
    compute(As1, Bs1);
    if constexpr (kPinWait) __builtin_amdgcn_sched_barrier(0);
    vm_wait_all();
    __syncthreads();
  }

  // ---- epilogue: kernel values, Q~ entries, row and column sums
  // Kernel values and Q~ entries are formed in T; products with the vector
  // and the sums are fp64, so an fp32 product uses the fp64 CG direction as it
  // is instead of a rounded copy.
  const bool diag = SYM && (I == J);
  int64_t gj[CB];
  T nBj[CB], qBj[CB];
  double pBj[CB];
#pragma unroll
  for (int j = 0; j < CB; ++j) {
    gj[j] = J * BM + wn * C::WN + j * MF::M + cl;
    nBj[j] = (KER == KRBF) ? a.nB[gj[j]] : T(0);
    qBj[j] = SYM ? a.qB[gj[j]] : T(0);
    if constexpr (SYM) pBj[j] = a.pv[gj[j]];
    else pBj[j] = (double)a.wB[gj[j]];
  }
  double cs[CB];
#pragma unroll
  for (int j = 0; j < CB; ++j) cs[j] = 0.0;
  // one row block at a time: its row sums are reduced and parked in LDS at
  // once, which keeps few values live next to the accumulators
  constexpr int VH = MF::NACC > 8 ? 8 : MF::NACC;   // accumulator elements per pass
#pragma unroll
  for (int i = 0; i < RB; ++i) {
#pragma unroll
  for (int v0 = 0; v0 < MF::NACC; v0 += VH) {
    double rs[VH];
#pragma unroll
    for (int vv = 0; vv < VH; ++vv) {
      const int v = v0 + vv;
      const int lr = wm * C::WM + i * MF::M + MF::row(v, lane);
      const int64_t gi = I * BM + lr;
      const T nAi = (KER == KRBF) ? a.nA[gi] : T(0);
      const T qAi = SYM ? a.qA[gi] : T(0);
      const double pAi = SYM ? a.pv[gi] : 0.0;
      double rsum = 0.0;
#pragma unroll
      for (int j = 0; j < CB; ++j) {
        const T kv = kernel_value<KER, T>(acc[i][j][v], nAi, nBj[j], a.gamma, a.coef0, a.degree);
        if constexpr (SYM) {
          T qt = kv - qAi - qBj[j] + a.qmm;
          if (gi == gj[j]) qt += a.invC;
          rsum += (double)qt * pBj[j];
          cs[j] += (double)qt * pAi;
        } else {
          rsum += (double)kv * pBj[j];
        }
      }
      rs[vv] = rsum;
    }
    // lanes that share a row differ only in the bits of cl
#pragma unroll
    for (int vv = 0; vv < VH; ++vv)
#pragma unroll
      for (int off = 1; off < MF::M; off <<= 1) rs[vv] += __shfl_xor(rs[vv], off);
    if (cl == 0) {
#pragma unroll
      for (int vv = 0; vv < VH; ++vv)
        red_r[wn][wm * C::WM + i * MF::M + MF::row(v0 + vv, lane)] = rs[vv];
    }
  }
  }
  // lanes that share a column differ only in the bits above cl
#pragma unroll
  for (int j = 0; j < CB; ++j)
#pragma unroll
    for (int off = MF::M; off < 64; off <<= 1) cs[j] += __shfl_xor(cs[j], off);

  if (SYM && kl == 0) {
#pragma unroll
    for (int j = 0; j < CB; ++j) red_c[wm][wn * C::WN + j * MF::M + cl] = cs[j];
  }
  __syncthreads();
  if (tid < BM) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < WAVES_N; ++w) s += red_r[w][tid];
    a.part[J * a.part_ld + I * BM + tid] = s;
  } else if (SYM && !diag && tid < 2 * BM) {
    const int c = tid - BM;
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < WAVES_M; ++w) s += red_c[w][c];
    a.part[I * a.part_ld + J * BM + c] = s;
  }
}

// ------------------------------------------------------------- a3 rhs -------
template <typename T>
__global__ __launch_bounds__(256) void k_rhs_init(const T* __restrict__ y, int64_t N, int64_t NP,
                                                  double* rhs, double* x, double* r, double* dir,
                                                  double* bpart, int* flags) {
  __shared__ double sh[NT / 64];
  const double ym = (double)y[N];
  if (blockIdx.x == 0 && threadIdx.x == 0 && !(ym == 1.0 || ym == -1.0)) flags[F_BADLABEL] = 1;
  double acc = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    double v = 0.0;
    if (i < N) {
      const double yi = (double)y[i];
      if (!(yi == 1.0 || yi == -1.0)) flags[F_BADLABEL] = 1;
      v = yi - ym;
    }
    rhs[i] = v;
    x[i] = 0.0;
    r[i] = v;
    dir[i] = v;
    acc += v * v;
  }
  const double s = block_sum(acc, sh);
  if (threadIdx.x == 0) bpart[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_finish_delta0(const double* bpart, int64_t nb,
                                                       double* scal, double eps2) {
  __shared__ double sh[NT / 64];
  const double s = sum_partials(bpart, nb, sh);
  if (threadIdx.x == 0) {
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
  }
}

// ------------------------------------------------------------- a5 CG --------
// q = Q~ d from the tile partials (masked beyond N) and the block partials of d^T q.
__global__ __launch_bounds__(256) void k_cg_gather(const double* __restrict__ part, int64_t nslots,
                                                   int64_t NP, int64_t N,
                                                   const double* __restrict__ dir, double* qv,
                                                   double* bpart, const double* scal) {
  __shared__ double sh[NT / 64];
  if (scal[S_STATUS + ST_DONE] != 0.0) return;
  double prod = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    double s = 0.0;
    for (int64_t sl = 0; sl < nslots; ++sl) s += part[sl * NP + i];
    if (i >= N) s = 0.0;
    qv[i] = s;
    prod += dir[i] * s;
  }
  const double t = block_sum(prod, sh);
  if (threadIdx.x == 0) bpart[blockIdx.x] = t;
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
    x[i] += alpha * dir[i];
    if (!x_only) {
      const double ri = r[i] - alpha * qv[i];
      r[i] = ri;
      v += ri * ri;
    }
  }
  if (!x_only) {
    const double t = block_sum(v, sh);
    if (threadIdx.x == 0) bp_out[blockIdx.x] = t;
  }
}

// r = rhs - Q~ x from the tile partials, and the block partials of r^T r.
__global__ __launch_bounds__(256) void k_cg_residual(const double* __restrict__ part,
                                                     int64_t nslots, int64_t NP, int64_t N,
                                                     const double* __restrict__ rhs, double* r,
                                                     double* bp_out, const double* scal) {
  __shared__ double sh[NT / 64];
  if (scal[S_STATUS + ST_DONE] != 0.0) return;
  double v = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT) {
    double s = 0.0;
    for (int64_t sl = 0; sl < nslots; ++sl) s += part[sl * NP + i];
    const double ri = i < N ? rhs[i] - s : 0.0;
    r[i] = ri;
    v += ri * ri;
  }
  const double t = block_sum(v, sh);
  if (threadIdx.x == 0) bp_out[blockIdx.x] = t;
}

// ||rhs - Q~ x||^2 partials without touching r (final report only).
__global__ __launch_bounds__(256) void k_true_residual(const double* __restrict__ part,
                                                       int64_t nslots, int64_t NP, int64_t N,
                                                       const double* __restrict__ rhs,
                                                       double* bp_out) {
  __shared__ double sh[NT / 64];
  double v = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < N; i += (int64_t)gridDim.x * NT) {
    double s = 0.0;
    for (int64_t sl = 0; sl < nslots; ++sl) s += part[sl * NP + i];
    const double ri = rhs[i] - s;
    v += ri * ri;
  }
  const double t = block_sum(v, sh);
  if (threadIdx.x == 0) bp_out[blockIdx.x] = t;
}

// beta = r^T r (new) / r^T r (old); d = r + beta d. Block 0 records the
// iteration in the status (and the history) and raises done once
// r^T r <= eps^2 r0^T r0.
__global__ __launch_bounds__(256) void k_cg_direction(const double* __restrict__ bp_in, int64_t nb,
                                                      double* scal, int par, int64_t iter,
                                                      const double* __restrict__ r, double* dir,
                                                      int64_t NP, double* hist, int64_t hist_cap) {
  __shared__ double sh[NT / 64];
  double* st = scal + S_STATUS;
  if (st[ST_DONE] != 0.0) return;
  const double dnew = sum_partials(bp_in, nb, sh);
  const double dold = scal[S_DHIST + par];
  const double beta = dnew / dold;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT)
    dir[i] = r[i] + beta * dir[i];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    scal[S_DHIST + (par ^ 1)] = dnew;
    st[ST_DELTA] = dnew;
    st[ST_CURV] = scal[S_GAMMA];
    st[ST_STEP] = scal[S_ALPHA];
    st[ST_ITER] = (double)iter;
    if (iter <= hist_cap) hist[iter - 1] = dnew;
    if (dnew <= st[ST_STOP]) st[ST_DONE] = 1.0;
  }
}

// After r = rhs - Q~ x0 for a warm start: r^T r becomes the current delta
// (the stop threshold stays eps^2 rhs^T rhs), the direction starts at r, and
// done is raised if x0 already meets the threshold.
__global__ __launch_bounds__(256) void k_warm_start(const double* __restrict__ bp_in, int64_t nb,
                                                    double* scal, const double* __restrict__ r,
                                                    double* dir, int64_t NP) {
  __shared__ double sh[NT / 64];
  const double dlt = sum_partials(bp_in, nb, sh);
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < NP; i += (int64_t)gridDim.x * NT)
    dir[i] = r[i];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    double* st = scal + S_STATUS;
    scal[S_DHIST + 0] = dlt;
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
    scalars[3] = broke ? 0.0 : rr_new / rr_old;
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
  double sx = 0.0, sqx = 0.0;
  for (int64_t i = threadIdx.x; i < N; i += blockDim.x) {
    const double xi = x[i];
    sx += xi;
    sqx += q64[i] * xi;
    alpha_out[i] = (T)xi;
  }
  sx = block_sum(sx, sh);
  sqx = block_sum(sqx, sh);
  if (threadIdx.x == 0) {
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
    if (!(y0 == 1.0 || y0 == -1.0)) flags[F_BADLABEL] = 1;
    alpha_out[0] = T(0);
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

// One block per test point: f = <w, x> + b (fp64), label +1 iff f > 0.
template <typename T>
__global__ __launch_bounds__(256) void k_linear_scores(const T* __restrict__ Xte, int64_t n_test,
                                                       int64_t d, const double* __restrict__ w,
                                                       double b, T* __restrict__ scores,
                                                       int32_t* __restrict__ labels,
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
  const double f = block_sum(acc, sh) + b;
  if (threadIdx.x == 0) {
    scores[t] = (T)f;
    if (labels) labels[t] = f > 0.0 ? 1 : -1;
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
__global__ __launch_bounds__(256) void k_mv_out(const double* __restrict__ part, int64_t nslots,
                                                int64_t NP, int64_t N, T* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (i < N) {
    double s = 0.0;
    for (int64_t sl = 0; sl < nslots; ++sl) s += part[sl * NP + i];
    out[i] = (T)s;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_predict_finish(const double* __restrict__ part,
                                                        int64_t nslots, int64_t ld, int64_t n_test,
                                                        double b, T* __restrict__ scores,
                                                        int32_t* __restrict__ labels) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (i < n_test) {
    double s = b;
    for (int64_t sl = 0; sl < nslots; ++sl) s += part[sl * ld + i];
    scores[i] = (T)s;
    if (labels) labels[i] = s > 0.0 ? 1 : -1;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_pad_to_f64(const T* __restrict__ src, int64_t len,
                                                    double* __restrict__ dst, int64_t len_pad) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (i < len_pad) dst[i] = i < len ? (double)src[i] : 0.0;
}

__global__ __launch_bounds__(256) void k_finish_sum(const double* bpart, int64_t nb, double* scal,
                                                    int slot) {
  __shared__ double sh[NT / 64];
  const double s = sum_partials(bpart, nb, sh);
  if (threadIdx.x == 0) scal[slot] = s;
}

inline unsigned blocks_for(int64_t n) { return (unsigned)((n + NT - 1) / NT); }

}  // namespace

// ------------------------------------------------------------- launchers ----

template <typename T>
hipError_t launch_layout(const T* X, int64_t n, int64_t d, T* Xt, int64_t ld, int64_t d_pad,
                         int* flags, hipStream_t s) {
  constexpr int BK = TileShape<T>::BK, TP = TileShape<T>::T;
  const int64_t total = d_pad * ld;
  hipLaunchKernelGGL((k_layout<T, BK, TP>), dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                     s, X, n, d, Xt, ld, d_pad / BK, flags);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_norms_q(const T* Xt, int64_t ld, int64_t d_pad, int64_t m, int64_t N,
                          int kernel, double gamma, double coef0, int degree, T* norms, T* qT,
                          double* q64, double* scal, hipStream_t s) {
  constexpr int BK = TileShape<T>::BK, TP = TileShape<T>::T;
  const int64_t nkb = d_pad / BK;
  const unsigned g = blocks_for(ld);
  switch (kernel) {
    case KLIN:
      hipLaunchKernelGGL((k_norms_q<T, BK, TP, KLIN>), dim3(g), dim3(NT), 0, s, Xt, ld, nkb, m, N,
                         gamma, coef0, degree, norms, qT, q64, scal);
      break;
    case KPOLY:
      hipLaunchKernelGGL((k_norms_q<T, BK, TP, KPOLY>), dim3(g), dim3(NT), 0, s, Xt, ld, nkb, m, N,
                         gamma, coef0, degree, norms, qT, q64, scal);
      break;
    default:
      hipLaunchKernelGGL((k_norms_q<T, BK, TP, KRBF>), dim3(g), dim3(NT), 0, s, Xt, ld, nkb, m, N,
                         gamma, coef0, degree, norms, qT, q64, scal);
      break;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_tiles_sym(const TileArgs<T>& a, int kernel, int64_t ntiles_1d, hipStream_t s) {
  dim3 grid((unsigned)ntiles_1d);
  switch (kernel) {
    case KLIN: hipLaunchKernelGGL((k_tiles<T, true, KLIN>), grid, dim3(256), 0, s, a); break;
    case KPOLY: hipLaunchKernelGGL((k_tiles<T, true, KPOLY>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_tiles<T, true, KRBF>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_tiles_gen(const TileArgs<T>& a, int kernel, int64_t nTr, hipStream_t s) {
  dim3 grid((unsigned)(nTr * a.nTc));
  switch (kernel) {
    case KLIN: hipLaunchKernelGGL((k_tiles<T, false, KLIN>), grid, dim3(256), 0, s, a); break;
    case KPOLY: hipLaunchKernelGGL((k_tiles<T, false, KPOLY>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_tiles<T, false, KRBF>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_rhs_init(const T* y, int64_t N, int64_t NP, double* rhs, double* x, double* r,
                           double* dir, double* bpart, int* flags, hipStream_t s) {
  hipLaunchKernelGGL(k_rhs_init<T>, dim3((unsigned)vec_blocks(NP)), dim3(NT), 0, s, y, N, NP, rhs, x, r,
                     dir, bpart, flags);
  return hipGetLastError();
}

hipError_t launch_finish_delta0(const double* bpart, int64_t nb, double* scal, double eps2,
                                hipStream_t s) {
  hipLaunchKernelGGL(k_finish_delta0, dim3(1), dim3(NT), 0, s, bpart, nb, scal, eps2);
  return hipGetLastError();
}

hipError_t launch_cg_gather(const double* part, int64_t nslots, int64_t NP, int64_t N,
                            const double* dir, double* qv, double* bpart, const double* scal,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_cg_gather, dim3((unsigned)vec_blocks(NP)), dim3(NT), 0, s, part, nslots, NP, N, dir,
                     qv, bpart, scal);
  return hipGetLastError();
}

hipError_t launch_cg_update(int x_only, const double* bp_in, int64_t nb, double* scal, int par,
                            const double* dir, const double* qv, double* x, double* r,
                            double* bp_out, int64_t NP, hipStream_t s) {
  hipLaunchKernelGGL(k_cg_update, dim3((unsigned)vec_blocks(NP)), dim3(NT), 0, s, x_only, bp_in, nb, scal,
                     par, dir, qv, x, r, bp_out, NP);
  return hipGetLastError();
}

hipError_t launch_cg_residual(const double* part, int64_t nslots, int64_t NP, int64_t N,
                              const double* rhs, double* r, double* bp_out, const double* scal,
                              hipStream_t s) {
  hipLaunchKernelGGL(k_cg_residual, dim3((unsigned)vec_blocks(NP)), dim3(NT), 0, s, part, nslots, NP, N,
                     rhs, r, bp_out, scal);
  return hipGetLastError();
}

hipError_t launch_true_residual(const double* part, int64_t nslots, int64_t NP, int64_t N,
                                const double* rhs, double* bp_out, hipStream_t s) {
  hipLaunchKernelGGL(k_true_residual, dim3((unsigned)vec_blocks(NP)), dim3(NT), 0, s, part, nslots, NP, N,
                     rhs, bp_out);
  return hipGetLastError();
}

hipError_t launch_cg_direction(const double* bp_in, int64_t nb, double* scal, int par,
                               int64_t iter, const double* r, double* dir, int64_t NP,
                               double* hist, int64_t hist_cap, hipStream_t s) {
  hipLaunchKernelGGL(k_cg_direction, dim3((unsigned)vec_blocks(NP)), dim3(NT), 0, s, bp_in, nb, scal, par,
                     iter, r, dir, NP, hist, hist_cap);
  return hipGetLastError();
}

hipError_t launch_warm_start(const double* bp_in, int64_t nb, double* scal, const double* r,
                             double* dir, int64_t NP, hipStream_t s) {
  hipLaunchKernelGGL(k_warm_start, dim3((unsigned)vec_blocks(NP)), dim3(NT), 0, s, bp_in, nb, scal,
                     r, dir, NP);
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
                     (int64_t)1, r, d, N, (double*)nullptr, (int64_t)0);
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
hipError_t launch_mv_out(const double* part, int64_t nslots, int64_t NP, int64_t N, T* out,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_mv_out<T>, dim3(blocks_for(N)), dim3(NT), 0, s, part, nslots, NP, N, out);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_predict_finish(const double* part, int64_t nslots, int64_t ld, int64_t n_test,
                                 double b, T* scores, int32_t* labels, hipStream_t s) {
  hipLaunchKernelGGL(k_predict_finish<T>, dim3(blocks_for(n_test)), dim3(NT), 0, s, part, nslots,
                     ld, n_test, b, scores, labels);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_pad_to_f64(const T* src, int64_t len, double* dst, int64_t len_pad,
                             hipStream_t s) {
  hipLaunchKernelGGL(k_pad_to_f64<T>, dim3(blocks_for(len_pad)), dim3(NT), 0, s, src, len, dst,
                     len_pad);
  return hipGetLastError();
}

hipError_t launch_finish_sum(const double* bpart, int64_t nb, double* scal, int slot,
                             hipStream_t s) {
  hipLaunchKernelGGL(k_finish_sum, dim3(1), dim3(NT), 0, s, bpart, nb, scal, slot);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_linear_predict(const T* Xtr, const T* alpha, int64_t n, int64_t d, const T* Xte,
                                 int64_t n_test, double b, double* part, double* w, T* scores,
                                 int32_t* labels, int* flags, hipStream_t s) {
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
  hipLaunchKernelGGL(k_linear_scores<T>, dim3((unsigned)n_test), dim3(NT), 0, s, Xte, n_test, d,
                     w, b, scores, labels, flags);
  return hipGetLastError();
}

int64_t linear_predict_part_elems(int64_t n, int64_t d) {
  const int64_t rows = lin_rows(n);
  return (n + rows - 1) / rows * d;
}

#define LSSVM_INSTANTIATE(T)                                                                      \
  template hipError_t launch_layout<T>(const T*, int64_t, int64_t, T*, int64_t, int64_t, int*,    \
                                       hipStream_t);                                              \
  template hipError_t launch_norms_q<T>(const T*, int64_t, int64_t, int64_t, int64_t, int,        \
                                        double, double, int, T*, T*, double*, double*,            \
                                        hipStream_t);                                             \
  template hipError_t launch_tiles_sym<T>(const TileArgs<T>&, int, int64_t, hipStream_t);         \
  template hipError_t launch_tiles_gen<T>(const TileArgs<T>&, int, int64_t, hipStream_t);         \
  template hipError_t launch_rhs_init<T>(const T*, int64_t, int64_t, double*, double*, double*,   \
                                         double*, double*, int*, hipStream_t);                    \
  template hipError_t launch_bias<T>(const double*, const double*, int64_t, const T*, double*,    \
                                     double, T*, hipStream_t);                                    \
  template hipError_t launch_single_point<T>(const T*, T*, double*, int*, hipStream_t);           \
  template hipError_t launch_pad_vec<T>(const T*, int64_t, T*, int64_t, hipStream_t);             \
  template hipError_t launch_mv_out<T>(const double*, int64_t, int64_t, int64_t, T*,              \
                                       hipStream_t);                                              \
  template hipError_t launch_predict_finish<T>(const double*, int64_t, int64_t, int64_t, double,  \
                                               T*, int32_t*, hipStream_t);                        \
  template hipError_t launch_pad_to_f64<T>(const T*, int64_t, double*, int64_t, hipStream_t);   \
  template hipError_t launch_linear_predict<T>(const T*, const T*, int64_t, int64_t, const T*,    \
                                               int64_t, double, double*, double*, T*, int32_t*,   \
                                               int*, hipStream_t);

LSSVM_INSTANTIATE(float)
LSSVM_INSTANTIATE(double)

}  // namespace lssvm
