// Internal definitions shared by the HIP sources of libbakron.so.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

namespace bk {

// Solver tile edge.  The matrix is cut into TS x TS tiles; all tiles on one
// tile anti-diagonal are mutually independent (App. B: no entry affects an
// entry on the same or an earlier anti-diagonal), and tile (I, J) depends
// only on tiles (I', J') with I' <= I, J' <= J.
constexpr int TS = 32;
constexpr int TILE_ELEMS = TS * TS;
// Node products use MACRO x MACRO solver tiles per workgroup (128 x 128).
constexpr int MACRO = 4;
// Largest supported near-field distance (tiles pulled by the target).
constexpr int KNEAR_MAX = 8;

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

// Launch plan of one solve shape (Alg. 6 on tile anti-diagonals).  Main ops
// run on the caller's stream, in order:
//   segment : a divide-and-conquer subtree [K, L) no wider than KNEAR + 1
//             tile anti-diagonals, solved by one persistent launch; each tile
//             pulls the errors of the tiles at distance 1..KNEAR above it and
//             to its left itself (Eq. (1)), so every (source, target) pair
//             closer than KNEAR + 1 is applied by the target;
//   node    : the push of a wider node [K, Mid, L), restricted to (source,
//             target) pairs farther apart than KNEAR, as dense MFMA products
//             into the targets on [tlo, thi).
// A node's push into its first right segment is a main op placed right after
// its left subtree.  Its pushes into the later segments of its right subtree
// may instead be side ops: they run on a second stream restricted to the CUs
// the segment launches leave free, in deadline order, each after its node's
// left subtree (main op `rel`), and every main op that touches a segment
// first waits for the side ops targeting it (`need_side`: all side ops with
// index below it).
// flops = algorithmic work (2 * TS^3 per (source, target) tile pair, plus the
// in-tile pairs of a solved tile); mfma_flops = executed on the matrix cores,
// zero-masked tiles included.
struct PlanOp {
    int kind;            // 0 segment, 1 node
    int K, Mid, L;       // segment: diagonals [K, L); node: sources [K, Mid)
    int tlo, thi;        // node: targets [tlo, thi)
    int strip_lo;        // segment: first tile column (strip) with a tile in [K, L)
    int nstrips;         // segment: number of such strips
    int counter;         // segment: index of its ticket counter
    int macro;           // node: solver tiles per workgroup edge (4 or 2)
    int item_off, item_cnt;
    int rel;             // side op: main op after which it may start
    int rec_rel;         // main op: some side op waits for it (record its event)
    int need_side;       // main op: side ops [0, need_side) must be complete first
    double flops, mfma_flops;
};
struct Plan {
    std::vector<PlanOp> ops;    // main stream
    std::vector<PlanOp> side;   // side stream (empty when not deferring)
    // host enqueue order: (0, main op index) or (1, side op index); side ops
    // are enqueued as soon as the main op they wait for has been enqueued
    std::vector<std::pair<int, int>> order;
    int side_cu_lo = 0;         // side stream runs on CUs [side_cu_lo, #CUs)
    int nseg = 0;
};

// Solve workspace: X, Y are mt*nt tile arrays of fp32; flags one int per
// tile; counters one ticket counter per segment; status one int (set when a
// wait gave up; cleared only by the host); scale_bad one int (debug scale
// validation).  status and scale_bad are the last two words.
struct Workspace {
    float* X;
    float* Y;
    int* flags;
    int* counters;
    int* status;
    int* scale_bad;
};

// Polls of a tile ready flag before the wait gives up (never reached in a
// correct run).
constexpr int SPIN_LIMIT = 1 << 22;

// Persistent segment launches use at most this many workgroups (one per CU).
constexpr int SEG_GRID = 256;

// Node work-list item (int4): x = first tile row I0, y = first tile column
// J0 of the MT x MT macro tile, z = (first source tile << 1) | push kind
// (0 column push, 1 row push), w = end of the source tile range.

// Quantiser of a solve (Sec. 3.1): alphabet {qlo..qhi}; scale of entry (i, j)
// = (gsize > 0 ? scale[i * ngroups + j / gsize] : scale[i]) * col_scale[j]
// (col_scale null: 1), one fp32 product.  Entries outside the m x n matrix
// (tile padding) get scale 0: their alphabet is {0} and, since W is zero
// padded and no feedback reaches them, their error is 0.
struct QuantArgs {
    const float* scale;
    const float* col_scale;
    int gsize, ngroups;
    float qlo, qhi;
};

__device__ inline float entry_scale(const QuantArgs& q, int64_t row, int64_t col, int64_t m,
                                    int64_t n) {
    if (row >= m || col >= n) return 0.0f;
    const float base = q.gsize > 0 ? q.scale[row * q.ngroups + col / q.gsize] : q.scale[row];
    return q.col_scale ? base * q.col_scale[col] : base;
}

// The column part of entry_scale for a fixed column: scale index
// row * rstride + goff, times cf (0 for a padding column).
struct ColScale {
    int goff;
    float cf;
};
__device__ inline ColScale col_scale_of(const QuantArgs& q, int64_t col, int64_t n) {
    ColScale c;
    c.goff = q.gsize > 0 && col < n ? (int)(col / q.gsize) : 0;
    c.cf = col >= n ? 0.0f : (q.col_scale ? q.col_scale[col] : 1.0f);
    return c;
}
template <bool GQ>
__device__ inline float row_scale_of(const QuantArgs& q, int64_t row, const ColScale& c,
                                     int64_t m) {
    if (row >= m) return 0.0f;
    if (!GQ) return q.scale[row];   // per-row scales: c is {0, 1}
    return q.scale[row * (q.gsize > 0 ? q.ngroups : 1) + c.goff] * c.cf;
}

// Fills n 32-bit words at p with v on stream st (debug poisoning).
hipError_t fill_words(hipStream_t st, void* p, int64_t n, uint32_t v);

// Sets *bad to 1 on stream st if any of `count` scales is negative, NaN or
// infinite (*bad is not cleared here).
hipError_t check_scales(hipStream_t st, const float* s, int64_t count, int* bad);

// Records the message returned by bakron_last_error() for this thread.
void set_last_error(const char* msg);

}  // namespace bk
