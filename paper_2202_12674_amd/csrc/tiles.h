// The a4 / a7 tile kernel: the kernel-matrix part K p of the implicit Q~
// product (Eqs. (13), (16)) and the decision values on the gfx950 matrix
// cores, one 128 x 128 tile of points per workgroup. Included by kernels.hip
// (one translation unit); kept on its own, with its interface in
// tile_args.h, so that the tile kernel's code can be identified apart from
// the rest.
#pragma once

#include "tile_args.h"

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

// Exponential of the RBF kernel. fp32 uses the hardware base-2 exponential
// (v_exp_f32) on an exponent pre-scaled by log2(e) on the host; fp64 the
// full-precision exp.
template <typename T> __device__ inline T rbf_exp(T x);
template <> __device__ inline float rbf_exp<float>(float x) { return __builtin_amdgcn_exp2f(x); }
template <> __device__ inline double rbf_exp<double>(double x) { return exp(x); }

// Kernel value from the inner product g = <x_i, x_j> (and squared norms for
// RBF, with rbf_scale = gamma, times log2(e) in fp32). For the polynomial
// kernel this returns the base gamma g + coef0; poly_power raises a whole
// batch of bases to the degree with one uniform loop.
template <int KER, typename T>
__device__ inline T kernel_value(T g, T ni, T nj, T gamma, T coef0, T rbf_scale) {
  if constexpr (KER == KLIN) {
    return g;
  } else if constexpr (KER == KPOLY) {
    return gamma * g + coef0;
  } else {
    T dist = ni + nj - T(2) * g;
    dist = dist > T(0) ? dist : T(0);
    return rbf_exp<T>(-rbf_scale * dist);
  }
}

template <typename T, int R, int C>
__device__ inline void poly_power(T (&v)[R][C], int degree) {
  T base[R][C];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int c = 0; c < C; ++c) base[r][c] = v[r][c];
  for (int e = 1; e < degree; ++e)
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int c = 0; c < C; ++c) v[r][c] *= base[r][c];
}

// ------------------------------------------------------ cross-lane sums -----
// fp64 value of another lane: a DPP permutation (gfx9 encodings) applied to
// both 32-bit halves.
constexpr int kDppQuadXor1 = 0xB1;       // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4E;       // quad_perm [2, 3, 0, 1]
constexpr int kDppRowRor8 = 0x128;       // lane l <- lane l ^ 8 within 16-lane rows
constexpr int kDppRowHalfMirror = 0x141; // lane l <- lane 7 - l within 8-lane halves

__device__ inline uint64_t as_u64(double v) { return __builtin_bit_cast(uint64_t, v); }
__device__ inline double as_f64(uint32_t lo, uint32_t hi) {
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

template <int CTRL>
__device__ inline double dpp_move(double v) {
  const uint64_t u = as_u64(v);
  const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, false);
  return as_f64((uint32_t)lo, (uint32_t)hi);
}

// Sum over the 8 lanes of a half-row (lane bits 0..2), every lane receiving
// it: the half-mirror pairs l with 7 - l, then the two quad exchanges join
// the four pairs.
__device__ inline double sum8(double v) {
  v += dpp_move<kDppRowHalfMirror>(v);
  v += dpp_move<kDppQuadXor1>(v);
  v += dpp_move<kDppQuadXor2>(v);
  return v;
}

// Reduce-scatter steps: from a pair (a, b) in every lane, lanes with the
// given lane bit clear end up with a + a', lanes with it set with b + b',
// where ' is the partner lane across that bit. Each halves the values a lane
// carries with one exchange per pair instead of one per value.
__device__ inline double scatter_bit3(double a, double b, bool bit3) {
  const double keep = bit3 ? b : a, send = bit3 ? a : b;
  return keep + dpp_move<kDppRowRor8>(send);
}
// bit 4: v_permlane16_swap exchanges the odd 16-lane rows of its first
// operand with the even rows of its second
__device__ inline double scatter_bit4(double a, double b) {
  const uint64_t ua = as_u64(a), ub = as_u64(b);
  const auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)ua, (uint32_t)ub, false, false);
  const auto hi =
      __builtin_amdgcn_permlane16_swap((uint32_t)(ua >> 32), (uint32_t)(ub >> 32), false, false);
  return as_f64(lo[0], hi[0]) + as_f64(lo[1], hi[1]);
}
// bit 5: v_permlane32_swap exchanges the upper 32 lanes of its first operand
// with the lower 32 lanes of its second
__device__ inline double scatter_bit5(double a, double b) {
  const uint64_t ua = as_u64(a), ub = as_u64(b);
  const auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)ua, (uint32_t)ub, false, false);
  const auto hi =
      __builtin_amdgcn_permlane32_swap((uint32_t)(ua >> 32), (uint32_t)(ub >> 32), false, false);
  return as_f64(lo[0], hi[0]) + as_f64(lo[1], hi[1]);
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

// ------------------------------------------------ fixed-point row sums ----
// The symmetric tiles add their row and column sums into one accumulator per
// row with integer atomics, which makes the total independent of the order
// the tiles finish in (fp64 atomics would not be) and keeps the memory at two
// 64-bit words per row. A product's scale 2^s is fixed before it starts from
// bounds on |k(x_i, x_j)| and |p_j|: one tile's sum for a row is below
// 128 kmax pmax, so with s = 61 - e, 2^e > 256 kmax pmax, every scaled sum
// |v 2^s| < 2^60. It is rounded to an integer X once (a spacing 2^-s of about
// 2^-54 kmax pmax, far finer than the fp64 rounding of the sum itself) and
// added as two limbs, X mod 2^32 (unsigned) and floor(X / 2^32) (signed), so
// neither 64-bit word can overflow for any number of tiles below 2^31. The
// kernel that reads a row (fixed_take) restores X's sum exactly and rounds it
// once to fp64.
template <int KER, typename T>
__device__ inline double fixed_scale(const TileArgs<T>& a, double pmax, double nmax) {
  double km = 1.0;   // bound on |k(x_i, x_j)|: RBF values are at most 1
  if constexpr (KER == KLIN) {
    km = nmax;       // |<x, z>| <= ||x|| ||z||
  } else if constexpr (KER == KPOLY) {
    const double base = fabs((double)a.gamma) * nmax + fabs((double)a.coef0);
    for (int e = 0; e < a.degree; ++e) km *= base;
  }
  const double bound = 256.0 * km * pmax;
  if (!(bound > 0.0) || !(bound < 1e300)) return 1.0;   // p = 0 (sums 0) or no usable bound
  int e = 0;
  (void)frexp(bound, &e);   // bound < 2^e
  return ldexp(1.0, 61 - e);
}

__device__ inline void fixed_add(int64_t* acc, int* bad, int64_t row, double v, double scale) {
  const double t = v * scale;
  if (!(fabs(t) < 0x1p62)) {   // not finite, or beyond the bound: the product is unusable
    *bad = 1;
    return;
  }
  const int64_t X = __double2ll_rn(t);
  const unsigned long long lo = (unsigned long long)X & 0xffffffffull;
  const unsigned long long hi = (unsigned long long)(X >> 32);   // two's complement bits
  atomicAdd(reinterpret_cast<unsigned long long*>(acc + 2 * row), lo);
  atomicAdd(reinterpret_cast<unsigned long long*>(acc + 2 * row + 1), hi);
}

// XOR swizzle of the 16-byte chunk index inside a point's 128-byte LDS row.
// LDS has 64 four-byte banks, and a 16-byte read serves 16 lanes per cycle,
// so the 16 lanes served together must cover the 16 chunk positions of a
// 256-byte bank line. Those 16 lanes are not 16 consecutive lanes: measured
// with the bank-conflict counter, patterns that keep lanes 16 apart on one
// position run conflict-free, and the grouping that fits every pattern tried
// sets lane bit 5 and a parity of lane bits 2..4 apart. A point's row fixes
// the half-line (p & 1); the swizzle must spread the rest.
// fp32 (32 x 32 x 2 blocks): lanes l and l + 32 read chunks 4 apart of the
// same 32 points; (p >> 1) & 7 is conflict-free. fp64 (16 x 16 x 4 blocks):
// the four 16-lane groups read chunks 2 apart of the same 16 points, where
// (p >> 1) & 7 doubles every read (8 cycles instead of 4: half the fp64
// kernel's LDS time was conflict); ((p >> 1) & 1) | (p & 4) is conflict-free
// (measured, both chunk parities).
template <typename T> __device__ inline int chunk_swizzle(int p);
template <> __device__ inline int chunk_swizzle<float>(int p) { return (p >> 1) & 7; }
template <> __device__ inline int chunk_swizzle<double>(int p) { return ((p >> 1) & 1) | (p & 4); }

// Tile rows per band of the general-mode visit order.
constexpr int64_t kBandRows = 8;

// Third word of a raw buffer resource on gfx9-family targets (32-bit data
// format, no swizzle, no stride).
constexpr int kBufferWord3 = 0x00020000;

// Wait until all of this wave's vector memory operations (including direct
// global -> LDS loads) have completed: s_waitcnt vmcnt(0), other counters free.
__device__ inline void vm_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// The stop flag of launches that have none (a product outside CG).
__device__ const double kNeverStop = 0.0;

// ---------------------------------------------------------- a4 tiles --------
// One T x T tile of the pairwise contraction G = X_I X_J^T per workgroup,
// feature blocks of BK staged global -> LDS (double-buffered) and fed to the
// matrix cores. The epilogue turns G into kernel values and folds them into
// row sums (times p_j) and, off the diagonal, column sums (times p_i), so
// that each off-diagonal tile serves both triangles. Row and column sums are
// reduced across lanes and waves in a fixed order and added, in fixed point,
// to the rows' accumulators (symmetric mode: fixed_add), or written as fp64
// partials, one slot per tile column (general mode).
//
// PART splits a symmetric tile's features over a.ksplit workgroups for the
// kernels whose value needs the whole inner product: kPartial workgroups park
// their raw inner products G (the accumulators) in a.gpart and stop; a kFixup
// launch, one workgroup per tile, sums the parked splits in split order and
// runs the epilogue.
//
// ONE: every workgroup of the launch contracts exactly one feature block
// (a small problem's linear tiles split into single blocks), so the block
// the prologue loads is the only one and the two-stage loop is left out.
//
// The body returns false when the launch found CG already stopped (nothing
// done), true otherwise.
template <typename T, bool SYM, int KER, int PART, bool ONE = false>
__device__ __forceinline__ bool tile_body(const TileArgs<T>& a) {
  static_assert(!ONE || (SYM && KER == KLIN && PART == kWhole),
                "single-block workgroups: split linear tiles only");
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
  // physical chunk p * 8 + (c ^ chunk_swizzle<T>(p)) (see there: the swizzle
  // makes the operand reads conflict-free); the lane-linear direct loads are
  // conflict-free by construction.
  // one array per stage and panel: with fixed names the compiler can tell the
  // stage being filled from the stage being read and need not wait in between
  __shared__ __attribute__((aligned(16))) T As0[CHUNKS * VEC];
  __shared__ __attribute__((aligned(16))) T As1[CHUNKS * VEC];
  __shared__ __attribute__((aligned(16))) T Bs0[CHUNKS * VEC];
  __shared__ __attribute__((aligned(16))) T Bs1[CHUNKS * VEC];
  __shared__ double red_r[WAVES_N][BM];
  __shared__ double red_c[WAVES_M][BM];
  // The tile's panel vectors are staged with its first feature block, so the
  // epilogue reads no global memory (its loads of p and the norms otherwise
  // cost several L2 round trips per tile: up to 10% of the product at 64
  // features, 0.5% at 4096 in fp32; in fp64 ~1% at 1024 and 2048 features).
  // p over rows I and over columns J (symmetric mode) go to vp, q over panel
  // I to vq (diagonal tiles); the squared norms of both panels (radial
  // kernel) and the column weights (general mode) to vt[0], vt[1], vt[2].
  __shared__ __attribute__((aligned(16))) double vp[SYM ? 2 : 1][BM];
  __shared__ __attribute__((aligned(16))) double vq[SYM ? BM : 1];   // q over panel I (diagonal)
  __shared__ __attribute__((aligned(16))) T vt[3][BM];

  // CG already stopped? A whole or partial tile reads the flag with its
  // first loads in flight: waiting for it first would add a round trip to
  // every product of a small problem.
  double stop_v = 0.0;
  if constexpr (SYM) {
    stop_v = *(a.stop ? a.stop : &kNeverStop);
    if (PART == kFixup && stop_v != 0.0) return false;
  }
  int64_t I, J;
  // Symmetric tiles may have their features split over KS workgroups. For
  // the linear kernel each split sums K p over its share into slots of its
  // own (the sums add up because the kernel value is the inner product
  // itself); otherwise the splits meet in the kFixup launch. Workgroup slot v
  // takes split v % KS of tile v / KS of this launch, which starts at
  // a.tile_offset of the visit order; a linear launch's trailing slots run
  // its last round split finer (a.tail_slot).
  int64_t KS = (SYM && (KER == KLIN || PART != kWhole)) ? a.ksplit : 1;
  int64_t ks = 0, trel = 0, first = a.tile_offset;
  const int64_t t = a.tile_base + (int64_t)blockIdx.x;   // this workgroup's slot
  if constexpr (SYM) {
    int64_t v = t, G = a.ntiles;
    if (KER == KLIN && PART == kWhole && a.tail_split > 0) {
      if (t >= a.tail_slot) {
        KS = a.tail_split;
        first = a.tail_tile;
        v = t - a.tail_slot;
        G = 0;   // no XCD runs: each tail tile adds into a panel of its own
      } else {
        G = a.tail_slot;
      }
    }
    if (a.order && PART != kFixup && G > 0) {
      // workgroup w runs on XCD w % 8 (chunks start at multiples of 8, so this
      // holds for the slot t too): give each XCD a contiguous run of the order
      const int64_t x = t % kNumXcd, per = G / kNumXcd, extra = G % kNumXcd;
      v = x * per + (x < extra ? x : extra) + t / kNumXcd;
    }
    trel = v;
    if (PART != kFixup && KS > 1) {
      trel = v / KS;
      ks = v - trel * KS;
    }
    const int64_t tile = first + trel;
    if (a.order) {
      const uint32_t packed = a.order[tile];
      I = packed >> 16;
      J = packed & 0xFFFFu;
    } else {
      tri_index(tile, I, J);
    }
  } else {
    // Each XCD takes a contiguous run of slots (as above), and the slots walk
    // bands of up to 8 tile rows column by column, so the ~64 workgroups
    // resident on one XCD cover about 8 row panels x 8 column panels and
    // share both in its L2.
    const int64_t G = a.ntiles, nTr = G / a.nTc;
    const int64_t x = t % kNumXcd, per = G / kNumXcd, extra = G % kNumXcd;
    const int64_t v = x * per + (x < extra ? x : extra) + t / kNumXcd;
    const int64_t band = v / (kBandRows * a.nTc), r = v - band * kBandRows * a.nTc;
    const int64_t rows = nTr - band * kBandRows < kBandRows ? nTr - band * kBandRows : kBandRows;
    J = r / rows;
    I = band * kBandRows + (r - J * rows);
  }
  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index is uniform: kept in a scalar register, so the LDS address
  // of each direct load (M0) needs no per-load read-back from a vector register
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  // the bounds behind the fixed-point scale, read now: in the epilogue the
  // read would add a round trip after the last block
  double fx_pmax = 0.0, fx_nmax = 0.0;
  if constexpr (SYM) {
    fx_pmax = a.fx[0];
    fx_nmax = a.fx[1];
  }

  // panel I is a.nkb consecutive blocks of BM * BK elements; this workgroup
  // contracts blocks [ks nkb, (ks + 1) nkb) of it
  const int64_t nkb = a.nkb / KS;
  const T* __restrict__ Ap = a.A + (I * a.nkb + ks * nkb) * BM * BK;
  const T* __restrict__ Bp = a.B + (J * a.nkb + ks * nkb) * BM * BK;
  constexpr int64_t astride = (int64_t)BM * BK;   // elements per block of a panel

  // Direct loads of block kb into a stage, memory -> LDS with no registers in
  // between: instruction u of wave w fills physical chunks [(4u + w) * 64, +64)
  // lane by lane; each lane fetches the logical chunk that belongs at its
  // physical slot. They are buffer loads: one buffer resource per panel (scalar
  // registers, sized to this workgroup's span of the panel, so every load is
  // in range), the lane's chunk offset as the 32-bit vector offset and the
  // block's offset as the scalar offset, so a block's loads need no vector
  // instruction for their addresses. (Global loads into LDS took two 64-bit
  // vector adds and a readfirstlane per load; at 32768 x 4096 fp32 the tile
  // kernel ran at 88% of the matrix-core peak with them and 94.5% without,
  // bit-identical.) The spans stay below 4 GiB (at most 2^21 features: 1 GiB
  // fp32, 2 GiB fp64 per panel).
  uint32_t goff[LOADS];
#pragma unroll
  for (int u = 0; u < LOADS; ++u) {
    const int P = (u * 4 + wave) * 64 + lane;
    const int p = P / CPR, c = (P % CPR) ^ chunk_swizzle<T>(p);
    goff[u] = (uint32_t)((p * CPR + c) * VEC * (int)sizeof(T));
  }
  const int span = (int)(uint32_t)((uint64_t)nkb * astride * sizeof(T));
  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(Ap), (short)0, span, kBufferWord3);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(Bp), (short)0, span, kBufferWord3);
  auto dload = [&](int64_t kb, T (&sa)[CHUNKS * VEC], T (&sb)[CHUNKS * VEC]) {
    const int so = (int)(uint32_t)((uint64_t)kb * astride * sizeof(T));   // uniform
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int base = (u * 4 + wave) * 64 * VEC;   // wave-uniform LDS element offset
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lptr_t)(&sa[base]), 16, (int)goff[u], so,
                                               0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lptr_t)(&sb[base]), 16, (int)goff[u], so,
                                               0, 0);
    }
  };

  // One 16-byte piece per lane: a wave moves a 1 KiB vector (128 doubles) or
  // a T vector of 128 entries with lanes beyond it idle. Every vector is
  // padded to whole panels, so the pieces stay inside it.
  auto dvec = [&]() {
    constexpr int TL = BM * (int)sizeof(T) / 16;   // lanes per T vector
    constexpr int TE = 16 / (int)sizeof(T);        // T entries per lane
    if constexpr (SYM) {
      if (wave == 0) {
        __builtin_amdgcn_global_load_lds((gptr_t)(a.pv + I * BM + 2 * lane), (lptr_t)&vp[0][0],
                                         16, 0, 0);
        if (I == J && ks == 0)   // the diagonal tile's rank-one share needs q as well
          __builtin_amdgcn_global_load_lds((gptr_t)(a.q64 + I * BM + 2 * lane), (lptr_t)&vq[0],
                                           16, 0, 0);
      } else if (wave == 1)
        __builtin_amdgcn_global_load_lds((gptr_t)(a.pv + J * BM + 2 * lane), (lptr_t)&vp[1][0],
                                         16, 0, 0);
    } else {
      if (wave == 0 && lane < TL)
        __builtin_amdgcn_global_load_lds((gptr_t)(a.wB + J * BM + TE * lane), (lptr_t)&vt[2][0],
                                         16, 0, 0);
    }
    if constexpr (KER == KRBF) {
      if (wave == 2 && lane < TL)
        __builtin_amdgcn_global_load_lds((gptr_t)(a.nA + I * BM + TE * lane), (lptr_t)&vt[0][0],
                                         16, 0, 0);
      else if (wave == 3 && lane < TL)
        __builtin_amdgcn_global_load_lds((gptr_t)(a.nB + J * BM + TE * lane), (lptr_t)&vt[1][0],
                                         16, 0, 0);
    }
  };

  typename MF::acc_t acc[RB][CB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int j = 0; j < CB; ++j) acc[i][j] = MF::zero();

  const int cl = lane % MF::M;   // point of this lane inside an MFMA block
  const int kl = lane / MF::M;   // lane group: which features of the block it contracts

  // A block's operands are CPG groups of 16-byte LDS reads (chunk q of every
  // row and column block). fp64 reads group q + 1 into registers of its own
  // before group q's MFMAs issue, so a group's LDS latency hides behind the
  // MFMAs of the one before it (A/B: 4096 x 1024 linear 83.7% -> 85.3% of the
  // fp64 peak, 16384 x 2048 RBF 93.3% -> 93.6%). fp32, where the compiler
  // reuses one group's registers and the two workgroups of a CU cover each
  // other's waits, measured the same either way and keeps the plain loop.
  // Both issue the MFMAs in the order of a plain loop over the features.
  auto read_group = [&](const T (&sa)[CHUNKS * VEC], const T (&sb)[CHUNKS * VEC], int q,
                        vec_t (&a)[RB], vec_t (&b)[CB]) {
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int p = wm * C::WM + i * MF::M + cl;
      a[i] = *reinterpret_cast<const vec_t*>(
          &sa[(p * CPR + ((kl * CPG + q) ^ chunk_swizzle<T>(p))) * VEC]);
    }
#pragma unroll
    for (int j = 0; j < CB; ++j) {
      const int p = wn * C::WN + j * MF::M + cl;
      b[j] = *reinterpret_cast<const vec_t*>(
          &sb[(p * CPR + ((kl * CPG + q) ^ chunk_swizzle<T>(p))) * VEC]);
    }
  };
  auto compute = [&](const T (&sa)[CHUNKS * VEC], const T (&sb)[CHUNKS * VEC]) {
    if constexpr (sizeof(T) == 8) {
      vec_t av[2][RB], bv[2][CB];
      read_group(sa, sb, 0, av[0], bv[0]);
#pragma unroll
      for (int q = 0; q < CPG; ++q) {
        if (q + 1 < CPG) read_group(sa, sb, q + 1, av[(q + 1) & 1], bv[(q + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < VEC; ++e)
#pragma unroll
          for (int i = 0; i < RB; ++i)
#pragma unroll
            for (int j = 0; j < CB; ++j)
              acc[i][j] = MF::mma(av[q & 1][i][e], bv[q & 1][j][e], acc[i][j]);
      }
    } else {
      vec_t av[RB][CPG], bv[CB][CPG];
#pragma unroll
      for (int i = 0; i < RB; ++i) {
        const int p = wm * C::WM + i * MF::M + cl;
#pragma unroll
        for (int q = 0; q < CPG; ++q)
          av[i][q] = *reinterpret_cast<const vec_t*>(
              &sa[(p * CPR + ((kl * CPG + q) ^ chunk_swizzle<T>(p))) * VEC]);
      }
#pragma unroll
      for (int j = 0; j < CB; ++j) {
        const int p = wn * C::WN + j * MF::M + cl;
#pragma unroll
        for (int q = 0; q < CPG; ++q)
          bv[j][q] = *reinterpret_cast<const vec_t*>(
              &sb[(p * CPR + ((kl * CPG + q) ^ chunk_swizzle<T>(p))) * VEC]);
      }
#pragma unroll
      for (int kk = 0; kk < FPG; ++kk)
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
          for (int j = 0; j < CB; ++j)
            acc[i][j] = MF::mma(av[i][kk / VEC][kk % VEC], bv[j][kk / VEC][kk % VEC], acc[i][j]);
    }
  };

  // Two stages: while block kb is multiplied out of one stage, block kb + 1
  // streams into the other. A stage is refilled only after the barrier that
  // ends the iteration which last read it. The host pads the features to an
  // even number of blocks, so both halves of the loop body always run.
  //
  // Scheduling fence, chosen by measurement: left alone, the compiler sinks
  // the block loads into the compute (fp32: into its last quarter; fp64: it
  // waits for them, and holds the barrier, after the first four MFMAs, so the
  // load latency is hidden only by the other workgroup's waves). Pinned above
  // the compute, a wave's own 64 MFMAs cover it: fp32 +0.5%; fp64, with its
  // conflict-free LDS reads (chunk_swizzle), 16384 x 2048 RBF 90.9% -> 93.2%
  // of the fp64 peak, 16384 x 4096 linear 90.9% -> 95.5%, 16384 x 1024 cubic
  // 90.8% -> 92.3%, 4096 x 1024 linear 82.7% -> 84.0% (with the conflicting
  // reads pinning had cost fp64 ~1%).
  if constexpr (PART != kFixup) {
  dload(0, As0, Bs0);
  if constexpr (PART == kWhole) dvec();
  __builtin_amdgcn_sched_barrier(0);   // the flag is tested only behind the loads
  if (stop_v != 0.0) {   // uniform: the loads land in LDS before the workgroup ends
    vm_wait_all();
    return false;
  }
  vm_wait_all();
  __syncthreads();
  if constexpr (ONE) {
    compute(As0, Bs0);   // the epilogue touches none of the stages
  } else {
  for (int64_t kb = 0; kb < nkb; kb += 2) {
    dload(kb + 1, As1, Bs1);
    __builtin_amdgcn_sched_barrier(0);
    compute(As0, Bs0);
    vm_wait_all();     // this wave's part of block kb + 1 has landed
    __syncthreads();   // every wave's part has landed; stage 0 is free
    if (kb + 2 < nkb) dload(kb + 2, As0, Bs0);
    __builtin_amdgcn_sched_barrier(0);
    compute(As1, Bs1);
    vm_wait_all();
    __syncthreads();
  }
  }
  }

  // Split tiles: park this split's inner products, or sum all splits of the
  // tile in split order (the same sum whichever split finished last). Thread
  // tid's accumulators go to 16-byte units ((trel KS + s) NU + u) 256 + tid,
  // so every store and load instruction covers 4 KiB contiguously.
  if constexpr (PART != kWhole) {
    constexpr int PER = 16 / (int)sizeof(T);            // elements per 16-byte unit
    constexpr int UPB = MF::NACC / PER;                 // units per accumulator block
    constexpr int NU = RB * CB * UPB;                   // units per thread
    typedef T unit_t __attribute__((ext_vector_type(PER)));
    auto unit_ptr = [&](int64_t s, int u) {
      return reinterpret_cast<unit_t*>(a.gpart) + ((trel * KS + s) * NU + u) * 256 + tid;
    };
    if constexpr (PART == kPartial) {
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < CB; ++j)
#pragma unroll
          for (int w = 0; w < UPB; ++w) {
            unit_t x;
#pragma unroll
            for (int e = 0; e < PER; ++e) x[e] = acc[i][j][w * PER + e];
            *unit_ptr(ks, (i * CB + j) * UPB + w) = x;
          }
      return true;
    } else {
      dvec();
      vm_wait_all();
      __syncthreads();
      for (int64_t s2 = 0; s2 < KS; ++s2) {
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
          for (int j = 0; j < CB; ++j)
#pragma unroll
            for (int w = 0; w < UPB; ++w) {
              const unit_t x = *unit_ptr(s2, (i * CB + j) * UPB + w);
#pragma unroll
              for (int e = 0; e < PER; ++e) acc[i][j][w * PER + e] += x[e];
            }
      }
    }
  }

  // ---- epilogue: kernel values, row and column sums
  // Symmetric mode accumulates K_IJ p_J by rows and K_IJ^T p_I by columns;
  // the rank-one and diagonal terms that turn K into Q~ (Eq. (13)) are added
  // by the kernels that gather the partials. Kernel values are formed in T,
  // their products with the vector and all sums in fp64, so an fp32 product
  // uses the fp64 CG direction as it is instead of a rounded copy.
  const bool diag = SYM && (I == J);
  double fxs = 1.0;   // fixed-point scale of the row sums (symmetric mode)
  if constexpr (SYM) {
    fxs = fixed_scale<KER>(a, fx_pmax, fx_nmax);
    if (blockIdx.x == 0 && tid == 0) a.fx[2] = fxs;   // every workgroup finds the same
  }
  T nBj[CB];
  double pBj[CB];
#pragma unroll
  for (int j = 0; j < CB; ++j) {
    const int lj = wn * C::WN + j * MF::M + cl;
    nBj[j] = (KER == KRBF) ? vt[1][lj] : T(0);
    if constexpr (SYM) pBj[j] = vp[1][lj];
    else pBj[j] = (double)vt[2][lj];
  }
  double cs[CB];
#pragma unroll
  for (int j = 0; j < CB; ++j) cs[j] = 0.0;
  const bool bit3 = (lane >> 3) & 1;
  const int bit4 = (lane >> 4) & 1;
  // one row block and VH accumulator elements at a time: their row sums are
  // reduced and parked in LDS at once, which keeps few values live next to
  // the accumulators
  constexpr int VH = MF::NACC > 8 ? 8 : MF::NACC;
  static_assert(MF::M == 32 ? VH == 8 : (MF::M == 16 && VH == 4), "row-sum reduction layout");
  constexpr int NTOT = MF::M == 32 ? VH / 4 : VH / 2;   // row totals per lane and pass
#pragma unroll
  for (int i = 0; i < RB; ++i) {
#pragma unroll
  for (int v0 = 0; v0 < MF::NACC; v0 += VH) {
    T kv[VH][CB];
    double pAi[VH];
#pragma unroll
    for (int vv = 0; vv < VH; ++vv) {
      const int li = wm * C::WM + i * MF::M + MF::row(v0 + vv, lane);
      const T nAi = (KER == KRBF) ? vt[0][li] : T(0);
      pAi[vv] = SYM ? vp[0][li] : 0.0;
#pragma unroll
      for (int j = 0; j < CB; ++j)
        kv[vv][j] = kernel_value<KER, T>(acc[i][j][v0 + vv], nAi, nBj[j], a.gamma, a.coef0,
                                         a.rbf_scale);
    }
    if constexpr (KER == KPOLY) poly_power(kv, a.degree);
    double rs[VH];
#pragma unroll
    for (int vv = 0; vv < VH; ++vv) {
      double rsum = 0.0;
#pragma unroll
      for (int j = 0; j < CB; ++j) {
        const double k = (double)kv[vv][j];
        rsum += k * pBj[j];
        if constexpr (SYM) cs[j] += k * pAi[vv];
      }
      rs[vv] = rsum;
    }
    // Row totals: the M lanes of a row differ in the bits of cl. Reduce-
    // scatter over the high bits of cl, then a full sum over its low 3 bits;
    // lane cl then holds the totals of elements v0 + 4s + 2 bit3 + bit4 (fp32,
    // M = 32) or v0 + 2s + bit3 (fp64, M = 16).
    double tot[NTOT];
    int ve[NTOT];
    if constexpr (MF::M == 32) {
      double u[VH / 2];
#pragma unroll
      for (int t = 0; t < VH / 2; ++t) u[t] = scatter_bit4(rs[2 * t], rs[2 * t + 1]);
#pragma unroll
      for (int t = 0; t < VH / 4; ++t) {
        tot[t] = sum8(scatter_bit3(u[2 * t], u[2 * t + 1], bit3));
        ve[t] = v0 + 4 * t + 2 * (int)bit3 + bit4;
      }
    } else {
#pragma unroll
      for (int t = 0; t < VH / 2; ++t) {
        tot[t] = sum8(scatter_bit3(rs[2 * t], rs[2 * t + 1], bit3));
        ve[t] = v0 + 2 * t + (int)bit3;
      }
    }
    if ((cl & 7) == 0) {
#pragma unroll
      for (int t = 0; t < NTOT; ++t)
        red_r[wn][wm * C::WM + i * MF::M + MF::row(ve[t], lane)] = tot[t];
    }
  }
  }
  if constexpr (SYM) {
    // Column totals: the lanes of a column differ in the bits above cl
    // (bit 5 for fp32, bits 4 and 5 for fp64); after the reduce-scatter every
    // lane holds the total of one of the wave's columns.
    double ct;
    int jc;
    if constexpr (MF::M == 32) {
      static_assert(CB == 2, "fp32 column layout");
      ct = scatter_bit5(cs[0], cs[1]);
      jc = lane >> 5;
    } else {
      static_assert(CB == 4, "fp64 column layout");
      ct = scatter_bit4(scatter_bit5(cs[0], cs[1]), scatter_bit5(cs[2], cs[3]));
      jc = 2 * bit4 + (lane >> 5);
    }
    red_c[wm][wn * C::WN + jc * MF::M + cl] = ct;
  }
  __syncthreads();
  if (tid < BM) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < WAVES_N; ++w) s += red_r[w][tid];
    if constexpr (SYM) fixed_add(a.acc, a.fx_bad, I * BM + tid, s, fxs);
    else a.part[J * a.part_ld + I * BM + tid] = s;
  } else if (SYM && !diag && tid < 2 * BM) {
    const int c = tid - BM;
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < WAVES_M; ++w) s += red_c[w][c];
    fixed_add(a.acc, a.fx_bad, J * BM + c, s, fxs);
  }
  if constexpr (SYM) {
    // A diagonal tile also leaves its panel's share of the rank-one terms:
    // S_I = sum p_j and T_I = sum q_j p_j over the points j of panel I.
    if (diag && ks == 0) {
      constexpr int PW = BM / 64;   // waves holding one point each per lane
      __shared__ double red_d[PW][2];
      double sp = 0.0, sq = 0.0;
      if (tid < BM) {
        sp = vp[0][tid];
        sq = vq[tid] * sp;
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        sp += __shfl_xor(sp, off);
        sq += __shfl_xor(sq, off);
      }
      if (lane == 0 && wave < PW) {
        red_d[wave][0] = sp;
        red_d[wave][1] = sq;
      }
      __syncthreads();
      if (tid == 0) {
        double s0 = 0.0, s1 = 0.0;
#pragma unroll
        for (int w = 0; w < PW; ++w) {
          s0 += red_d[w][0];
          s1 += red_d[w][1];
        }
        a.pq[I] = s0;
        a.pq[a.nTc + I] = s1;
      }
    }
  }
  return true;
}

template <typename T, bool SYM, int KER, int PART>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_tiles(
    TileArgs<T> a) {
  tile_body<T, SYM, KER, PART>(a);
}

// Symmetric linear tiles split into single feature blocks (small problems:
// the products outside the fused iteration use its split, so every product
// of a training applies the same rounded operator).
template <typename T>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_tiles_one(
    TileArgs<T> a) {
  tile_body<T, true, KLIN, kWhole, true>(a);
}


}  // namespace
}  // namespace lssvm
