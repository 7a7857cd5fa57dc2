// The tile kernel's interface: the kernel functions, the tile shapes, the
// XCD count and the arguments of one launch. Shared by the tile kernel
// (tiles.h) and the host runtime; measurements of the tile kernel are tied to
// this header and tiles.h.
#pragma once

#include <cstdint>

namespace lssvm {

enum Kern : int { KLIN = 0, KPOLY = 1, KRBF = 2 };

// Points per tile edge and features per staged block, per element type
// (compile-time, like the block sizes of Sec. III-C4). The symmetric schedule
// needs square tiles.
#ifndef LSSVM_F32_BK
#define LSSVM_F32_BK 32
#endif
#ifndef LSSVM_F64_BK
#define LSSVM_F64_BK 16
#endif
constexpr int kNumXcd = 8;

template <typename T> struct TileShape;
template <> struct TileShape<float> { static constexpr int T = 128, BK = LSSVM_F32_BK; };
template <> struct TileShape<double> { static constexpr int T = 128, BK = LSSVM_F64_BK; };

// What a symmetric tile launch computes: whole tiles, parked feature splits
// of tiles (their raw inner products), or the fixup that sums a tile's parked
// splits and finishes it.
enum TilePart : int { kWhole = 0, kPartial = 1, kFixup = 2 };

template <typename T>
struct TileArgs {
  const T* A;    // panel-major feature-blocked row points (see k_layout)
  const T* B;    // panel-major feature-blocked column points
  int64_t lda, ldb;
  int64_t nkb;   // feature blocks of BK (even)
  const T* nA;   // squared norms of row points (RBF)
  const T* nB;   // squared norms of column points (RBF)
  const double* pv;   // symmetric mode: the vector multiplied (fp64), zero beyond N
  const double* q64;  // symmetric mode: q_i = k(x_i, x_m), zero beyond N
  double* pq;         // symmetric mode: per panel I, sum p_j at [I], sum q_j p_j at [nTc + I]
  const T* wB;        // general mode: per-column weights (alpha)
  T gamma, coef0;
  T rbf_scale;   // RBF exponent scale: gamma (fp64, exp) or gamma log2(e) (fp32, exp2)
  int degree;
  int64_t nTc;   // column tiles (general mode); tiles per side (symmetric mode)
  int64_t ksplit;  // symmetric mode: workgroups per tile, each over nkb / ksplit feature
                   // blocks (an even count). Linear kernel, whole tiles: every split
                   // adds its share of the row and column sums (the kernel value is
                   // the inner product itself). Split launches park inner products in
                   // gpart instead and a fixup launch finishes each tile.
  int64_t tile_offset;  // symmetric mode: first tile of the launch in the visit order
  // Linear kernel, whole tiles: with tail_split > 0, the workgroup slots from
  // tail_slot on run the last round split finer in the same launch: slot
  // tail_slot + u takes split u % tail_split of tile tail_tile + u / tail_split
  // of the visit order (its share of the features adds into the row sums like
  // any split's). tail_split = 0: no such slots.
  int64_t tail_slot, tail_split, tail_tile;
  T* gpart;             // split launches: parked inner products, ksplit 128^2 per tile
  const uint32_t* order;  // symmetric mode: (I << 16) | J per visit slot, or null
  double* part;  // general mode: partial sums, part[slot * part_ld + row]
  // symmetric mode: each row's sum over tiles, in fixed point (see fixed_add):
  // acc[2 row] the low 32-bit limbs, acc[2 row + 1] the signed high limbs
  int64_t* acc;
  // symmetric mode: fx[0] = max |p_j|, fx[1] = max ||x_i||^2 (the bounds of the
  // fixed-point scale); fx[2] receives the scale 2^s the launch used
  double* fx;
  int* fx_bad;          // symmetric mode: raised when a row sum is not finite
  const double* stop;   // symmetric mode: nonzero once CG has stopped (the launch then
                        // returns at once), or null
  int64_t part_ld;
  // A product's tiles may outnumber one launch (the dispatch grid counts work
  // items in 32 bits), so the launcher splits them into chunks: workgroup b of
  // a chunk takes tile slot tile_base + b of ntiles.
  int64_t tile_base, ntiles;
};

}  // namespace lssvm
