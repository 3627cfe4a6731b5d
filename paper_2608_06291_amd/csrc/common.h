// Internal definitions shared by the HIP sources of libbakron.so.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bk {

// Solver tile edge.  The matrix is cut into TS x TS tiles; all tiles on one
// tile anti-diagonal are mutually independent (App. B: no entry affects an
// entry on the same or an earlier anti-diagonal), so each leaf launch solves
// one tile anti-diagonal, one workgroup per tile.
constexpr int TS = 32;
constexpr int TILE_ELEMS = TS * TS;
// Node products use MACRO x MACRO solver tiles per workgroup (128 x 128).
constexpr int MACRO = 4;

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Packed lower-triangular tile storage of a normalised factor:
// tile (I, J), J <= I, lives at ((I * (I + 1)) / 2 + J) * TILE_ELEMS floats,
// row-major inside the tile.
__host__ __device__ inline int64_t packed_tile_offset(int64_t I, int64_t J) {
    return ((I * (I + 1)) / 2 + J) * (int64_t)TILE_ELEMS;
}

// Tile-major workspace: tile (I, J) of an mt x nt tile grid lives at
// (I * nt + J) * TILE_ELEMS floats, row-major inside the tile.
__host__ __device__ inline int64_t ws_tile_offset(int64_t I, int64_t J, int64_t nt) {
    return (I * nt + J) * (int64_t)TILE_ELEMS;
}

// One kernel launch of a solve, in stream order.  flops = algorithmic work
// (2 * TS^3 per (source, target) tile pair, plus the in-tile pairs of a
// leaf); mfma_flops = what the MFMA units execute including zero-masked
// operand tiles.
struct SolveOp {
    int kind;          // 0 = leaf, 1 = node
    int D, I_lo, ntiles;
    int K, Mid, L;
    int macro;         // node: solver tiles per workgroup edge (4 or 2)
    int item_off, item_cnt;  // node: slice of the work list
    double flops;
    double mfma_flops;
};

// Node work-list item (int4): x = first tile row I0, y = first tile column
// J0 of the MT x MT macro tile, z = (first source tile << 1) | push kind
// (0 column push, 1 row push), w = end of the source tile range.

}  // namespace bk
