// The a4 / a7 tile kernel: the implicit Q~ product (Eq. (16)) and the
// decision values on the gfx950 matrix cores, one 128 x 128 tile of points per
// workgroup. Included by kernels.hip (one translation unit); kept on its own
// so that the tile kernel's source can be identified apart from the rest.
#pragma once

#include "lssvm_internal.h"

#include <hip/hip_runtime.h>

#include <cmath>

namespace lssvm {
namespace {


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
  const int64_t t = a.tile_base + (int64_t)blockIdx.x;   // this workgroup's tile slot
  if constexpr (SYM) {
    if (a.order) {
      // workgroup w runs on XCD w % 8 (chunks start at multiples of 8, so this
      // holds for the slot t too): give each XCD a contiguous run of the order
      const int64_t G = a.ntiles;
      const int64_t x = t % kNumXcd, per = G / kNumXcd, extra = G % kNumXcd;
      const int64_t slot = x * per + (x < extra ? x : extra) + t / kNumXcd;
      const uint32_t packed = a.order[slot];
      I = packed >> 16;
      J = packed & 0xFFFFu;
    } else {
      tri_index(t, I, J);
    }
  } else {
    I = t / a.nTc;
    J = t % a.nTc;
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


}  // namespace
}  // namespace lssvm
