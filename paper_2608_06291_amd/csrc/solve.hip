// Solver kernels for BaKron (Alg. 6) on gfx950.
//
// Notation.  W~ is the workspace, E = V - W~ the committed errors, L^A / L^B
// the unit-lower normalised factors.  By Eq. (1) the value at which entry
// (p,q) is quantised is
//     W~_pq = W0_pq + sum_{(i,j) < (p,q)} L^B_pi E_ij L^A_qj ,
// the sum running over entries above-left of (p,q).  Split the sum by the
// first column index (App. B, proof of Thm 3.2, and Sec. 3.4's column/row
// splits):
//     W~_pq = W0_pq + sum_{j<q} F_pj L^A_qj + G_pq,
//     G_pq  = sum_{i<p} L^B_pi E_iq,        F_pj = G_pj + E_pj = (L^B E)_pj .
// G carries errors down a column through L^B, F carries them right along a
// row through L^A.  Every elementary update of Alg. 2 is applied exactly once
// this way, with mn(m+n)/2 multiply-adds in total (no band-masking overhead).
//
// Tiling.  TS x TS tiles; tile (I,J) depends only on tiles (I',J') with
// I'<=I, J'<=J, and tiles on one tile anti-diagonal D = I+J are independent.
// Two workspace arrays per tile:
//     X = W0 + (row pushes F L^A^T received so far)  -> after the tile is
//         solved it holds E of the tile;
//     Y = (column pushes L^B E received so far)       -> after the tile is
//         solved it holds F of the tile.
// The divide-and-conquer of Alg. 6 runs over ranges of tile anti-diagonals:
// solve the first half, push all errors of the first half into the second
// half, solve the second half.  The push of a node is two dense products:
//     Y[I,J] += sum_{I'} L^B[I,I'] E[I',J]       (same column, I' in S1)
//     X[I,J] += sum_{J'} F[I,J'] L^A[J,J']^T     (same row,    J' in S1)
// Products between tiles closer than KNEAR + 1 anti-diagonals are pulled by
// the target tile itself just before it is solved (a persistent "segment"
// launch covers a subtree of at most KNEAR + 1 anti-diagonals and orders its
// tiles with per-tile ready flags); node products take only pairs farther
// apart than KNEAR, so each (source, target) tile pair is applied exactly
// once.
#include <algorithm>

#include "common.h"

#include <vector>

namespace bk {


struct SegArgs {
    int K, L;         // tile anti-diagonals [K, L) of this launch
    int J_lo;         // first tile column (strip) with a tile in [K, L)
    int nstrips;      // strips J_lo .. J_lo + nstrips - 1
    int mt, nt;       // tile grid
    int64_t m, n;     // real sizes
    float* X;         // W0 + node row pushes; E once the tile is solved (column-major tiles)
    float* Y;         // node column pushes; F once the tile is solved (row-major tiles)
    const float* LA;  // packed factor tiles
    const float* LB;
    int b_ident;      // B = I (no column feedback)
    QuantArgs q;
    int8_t* codes;
    float* V;
    float* pre;       // may be null
    int knear;        // pull distances 1..knear (<= KNEAR_MAX)
    int* flags;       // per tile: 1 once F of the tile is published
    int* counter;     // strip ticket counter of this launch, 0 at entry
    int* status;      // set to 1 if a wait gave up (never in a correct run); sticky
    int spin_limit;   // polls before a wait gives up
};

// Bounded wait for a tile's ready flag, executed by a whole wave (uniform
// address).  A strip only ever waits for strips with smaller tickets, and
// tickets are handed out only to running workgroups, so the flag is set by a
// running workgroup; the bound only turns a logic error into a reported
// failure instead of a hang.  Once a wait has given up, the status word stays
// set (until the host reads and clears it) and every later wait returns at
// once, so a failed solve, and every solve after it, ends quickly with its
// output marked invalid.  The data behind the flag is read with
// device-coherent (sc1) loads, so no cache invalidation is needed here.
__device__ inline void wait_ready(const int* flag, int* status, int spin_limit) {
    int it = 0;
    while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
        __builtin_amdgcn_s_sleep(1);
        if (++it >= spin_limit ||
            __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
            __hip_atomic_store(status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
        }
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);   // keep the data loads after the wait
}

// Raw buffer descriptor over one 32 x 32 fp32 tile (16-byte loads).
__device__ inline __amdgpu_buffer_rsrc_t tile_rsrc(const float* t) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(t), (short)0, TILE_ELEMS * 4,
                                             0x00020000);
}
constexpr int CPOL_SC1 = 16;   // device-coherent load / store

// Near-field pulls on fp32 MFMA (v_mfma_f32_16x16x4f32).  The pulled sums of
// a tile are two 32 x 32 products per source distance k:
//   row kind    (into X): C[q][p] += sum_j L^A[J, J-k][q][j] F[I, J-k][p][j]
//   column kind (into Y): C[p][q] += sum_i L^B[I, I-k][p][i] E[I-k, J][i][q]
// Waves 0-3 own one 16 x 16 block of the row-kind C each, waves 4-7 one block
// of the column-kind C, so no partial sums have to be combined.  Every
// operand is read as contiguous 16-byte chunks of a row: lane (i, s) of a
// 16 x 16 x 4 step supplies A[i][k] and B[k][i] with k = 8s + 4c + t at step
// (c, t), i.e. chunks 2s and 2s + 1 of row i of both operand tiles.
//
// Factor tiles and the left strips' F tiles are staged in LDS with direct
// global -> LDS loads (no registers in flight), 16-byte chunk c of row r at
// chunk c ^ (r & 7) so that the row-per-lane reads above spread over the banks.
__device__ inline f32x4 lds_chunk(const float* t, int r, int c) {
    return *reinterpret_cast<const f32x4*>(t + r * TS + ((c ^ (r & 7)) << 2));
}
__device__ inline void mfma_8(f32x4 a0, f32x4 a1, f32x4 b0, f32x4 b1, f32x4& acc) {
#pragma unroll
    for (int t = 0; t < 4; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[t], b0[t], acc, 0, 0, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[t], b1[t], acc, 0, 0, 0);
}
// One wave copies rows 8 rb .. 8 rb + 7 of a row-major tile into a swizzled
// LDS tile: lane l fills physical chunk l & 7 of row 8 rb + (l >> 3).
template <int CPOL>
__device__ inline void stage_rows(const float* src, float* dst, int rb, int l) {
    const int r = 8 * rb + (l >> 3), c = (l & 7) ^ (r & 7);
    __builtin_amdgcn_global_load_lds(src + r * TS + 4 * c,
                                     (__attribute__((address_space(3))) void*)(dst + rb * 256), 16,
                                     0, CPOL);
}

constexpr int RING = KNEAR_MAX;   // E tiles of the strip kept in LDS
constexpr int RSTR = TS + 4;      // ring row stride: 16-byte rows, conflict-free b128 reads
constexpr int PULL_T0 = 2;        // first loop turn whose idle waves may consume staged operands

// Persistent solve of the tiles on anti-diagonals [K, L) by tile-column
// strips.  Each workgroup (512 threads, one per CU) repeatedly takes a strip
// ticket and solves the strip's tiles in [K, L) top to bottom; strip J waits
// only for strips J-1 .. J-2, which hold smaller tickets.  Inside a strip the
// column dependencies are local: the last RING errors E of the strip stay in
// LDS, and so do L^A[J, J-k] for k = 1..knear.  Per tile I:
//  1. pull.  The sources at distance k >= 2 of tile I are complete while
//     tile I-1 is being rounded (tile (I, J-2) finished before tile (I-1, J)
//     started, and every tile waits for its left neighbour, so one flag
//     stands for the whole row to its left).  Their operands are staged in
//     LDS at the start of tile I-1's rounding loop and the waves multiply them
//     in the loop turns in which they are idle; what remains (the first tile
//     of a strip, or a left strip that was late) is done here, followed by
//     distance 1: the row source (I, J-1) after its ready flag (device-
//     coherent loads) and the column source E(I-1) from the ring.  The 16 x 16
//     blocks meet in LDS;
//  2. in-tile rounding of the 63 element anti-diagonals (below);
//  3. publish F -> Y: the tile is gathered in LDS and written as whole
//     128-byte rows with device-coherent (sc1) 16-byte stores, which the
//     memory system acknowledges much sooner than scattered 4-byte ones; wait
//     for them, set the tile's flag.  E goes to the ring and to X (read by the
//     node launches after this one);
//  4. codes, V and pre, gathered in LDS and written as row segments.
//
// In-tile rounding: each thread owns two entries of one row p: slot 0 at
// column q0 and slot 1 at column q1 = q0 + 1 (mod 32), so p + q1 = p + q0 + 1.
// Half-wave h of wave w owns the rows' entries whose anti-diagonal index is
// {4w + 2h, 4w + 2h + 1} mod 32: two consecutive element anti-diagonals d
// (slot 0) and d + 1 (slot 1) are handled by the same half-wave, one barrier
// per pair.  Within a pair, the only feedback from diagonal d into d + 1 is
// the error of the entry just above (row p - 1, same column: one lane down,
// DPP wave_shr:1) through L^B[p][p-1], and the F of the entry just to the
// left (the thread's own slot 0) through L^A[q1][q0] (Eq. (1) restricted to
// the two diagonals).  After the barrier every thread adds the column pushes
// L^B[p][i] * E[i][q] and row pushes F[p][j] * L^A[q][j] of both diagonals to
// both of its entries.  Coefficients are register-resident, each factor row
// rotated so that step d reads register (d mod 32).
// GQ: scales per column group and/or per column (else one scale per row, the
// same for both entries of a thread).  ASYM: alphabet {qlo..qhi} (else the
// symmetric {-qhi..qhi}, clamped with one scalar operand).
template <bool GQ, bool ASYM>
__global__ __launch_bounds__(512) void k_seg(SegArgs a) {
    __shared__ float LBt[TS][TS];            // unpadded: the rotated reads below are conflict-free
    __shared__ float LAt[TS][TS];
    __shared__ float Ecs[2][2][2][2 * TS];   // [turn parity][round][diagonal of the pair][column (+ dummies)]
    __shared__ float2 Frs[2][2][2 * TS];     // [turn parity][round][row (+ dummies)] = (F on d, F on d + 1)
    __shared__ float HR[TS][TS + 1];         // pulled row-kind sum, [q][p]
    __shared__ float GC[TS][TS + 1];         // pulled column-kind sum, [p][q]
    __shared__ __attribute__((aligned(16))) float Ering[RING][TS][RSTR];   // E^T[q][i] per tile
    __shared__ __attribute__((aligned(16))) float LAs[KNEAR_MAX][TILE_ELEMS];      // L^A[J, J-k-1]
    __shared__ __attribute__((aligned(16))) float LBn[KNEAR_MAX][TILE_ELEMS];      // L^B[I', I'-k-1]
    __shared__ __attribute__((aligned(16))) float Yn[KNEAR_MAX - 1][TILE_ELEMS];   // F[I', J-k-2]
    __shared__ __attribute__((aligned(16))) float Fst[TS][RSTR];   // F of the tile, row-major
    __shared__ float So[GQ ? TS : 1][TS + 1];   // scales of the tile's entries (per row without GQ)
    __shared__ int tk, ynext;

    const int tid = threadIdx.x;
    const int w = tid >> 6, l = tid & 63;
    const int hf = l >> 5;
    const int p = l & 31;
    const int c0 = 4 * w + 2 * hf;
    const int q0 = (c0 - p) & 31;
    const int q1 = (q0 + 1) & 31;
    const float qhi = a.q.qhi, qlo = ASYM ? a.q.qlo : -qhi;
    const int knear = a.knear;
    const bool roww = w < 4;   // wave-uniform: row-kind or column-kind pull blocks

    for (;;) {
        if (tid == 0) tk = atomicAdd(a.counter, 1);
        __syncthreads();
        const int sidx = tk;
        if (sidx >= a.nstrips) break;   // uniform
        const int J = a.J_lo + sidx;
        const int I_first = a.K - J > 0 ? a.K - J : 0;
        const int I_last = a.L - 1 - J < a.mt - 1 ? a.L - 1 - J : a.mt - 1;
        const int kr = knear < J ? knear : J;   // row sources k = 1..kr of every tile of the strip
        const bool need_y = kr >= 2;

        // strip set-up: L^A[J, J] and L^A[J, J-k], the ring with the errors of
        // the tiles above that were solved by earlier launches, the first
        // tile's inputs and its staged pull operands.  Every load is issued
        // before any is waited for: one memory round trip per strip.
        const int npre = a.b_ident ? 0 : (knear < I_first ? knear : I_first);
        float2 rg[KNEAR_MAX];
#pragma unroll
        for (int k = 0; k < KNEAR_MAX; ++k)
            if (k < npre)   // uniform
                rg[k] = *reinterpret_cast<const float2*>(a.X + ws_tile_offset(I_first - 1 - k, J, a.nt) +
                                                          2 * tid);   // E^T, column-major E
        const float lat0 = a.LA[packed_tile_offset(J, J) + tid];
        const float lat1 = a.LA[packed_tile_offset(J, J) + tid + 512];
        for (int g = w; g < 4 * kr; g += 8)
            stage_rows<0>(a.LA + packed_tile_offset(J, J - 1 - (g >> 2)), LAs[g >> 2], g & 3, l);

        // inputs of the first tile; later tiles' inputs are prefetched during
        // the previous tile's rounding loop
        float pf_lb0, pf_lb1, pf_h0, pf_h1, pf_g0, pf_g1, pf_s0, pf_s1;
        // the column part of the scales of the thread's two columns (fixed per strip)
        const ColScale cs0 = GQ ? col_scale_of(a.q, (int64_t)J * TS + q0, a.n) : ColScale{0, 1.0f};
        const ColScale cs1 = GQ ? col_scale_of(a.q, (int64_t)J * TS + q1, a.n) : cs0;
        {
            const int64_t tb = ws_tile_offset(I_first, J, a.nt);
            const float* lbp = a.LB + packed_tile_offset(I_first, I_first);
            pf_lb0 = a.b_ident ? 0.0f : lbp[tid];
            pf_lb1 = a.b_ident ? 0.0f : lbp[tid + 512];
            pf_h0 = a.X[tb + q0 * TS + p];
            pf_h1 = a.X[tb + q1 * TS + p];
            pf_g0 = a.Y[tb + p * TS + q0];
            pf_g1 = a.Y[tb + p * TS + q1];
            const int row = I_first * TS + p;
            pf_s0 = row_scale_of<GQ>(a.q, row, cs0, a.m);
            pf_s1 = GQ ? row_scale_of<GQ>(a.q, row, cs1, a.m) : 0.0f;
        }
        // the first tile's pull operands: L^B[I_first, I_first - k] and the
        // left strips' F[I_first, J - k], k >= 2 (after the flag of
        // (I_first, J - 2), which stands for the whole row to its left)
        {
            const int nlb = npre;
            if (need_y) wait_ready(a.flags + I_first * a.nt + (J - 2), a.status, a.spin_limit);
            const int lim = 4 * (nlb + (need_y ? kr - 1 : 0));
            const int wu = __builtin_amdgcn_readfirstlane(w);
            __atomic_signal_fence(__ATOMIC_SEQ_CST);   // the F loads stay after the flag test
#pragma unroll
            for (int i = 0; i < (4 * (2 * KNEAR_MAX - 1) + 7) / 8; ++i) {
                const int g = wu + 8 * i;
                if (g < lim) {
                    const int ti = g >> 2;
                    if (ti < nlb)
                        stage_rows<0>(a.LB + packed_tile_offset(I_first, I_first - 1 - ti), LBn[ti], g & 3, l);
                    else
                        stage_rows<CPOL_SC1>(a.Y + ws_tile_offset(I_first, J - 2 - (ti - nlb), a.nt),
                                             Yn[ti - nlb], g & 3, l);
                }
            }
        }
        LAt[tid >> 5][tid & 31] = lat0;
        LAt[(tid + 512) >> 5][tid & 31] = lat1;
#pragma unroll
        for (int k = 0; k < KNEAR_MAX; ++k)
            if (k < npre)
                *reinterpret_cast<float2*>(&Ering[(I_first - 1 - k) % RING][(2 * tid) >> 5][(2 * tid) & 31]) = rg[k];
        __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's direct loads landed
        __syncthreads();

        // pull state of the next tile (uniform): which operands are staged,
        // and per wave the next source distance to multiply
        bool lb_staged = true, y_staged = true;   // the first tile's, above
        int nk = 2;
        f32x4 pacc = {0.0f, 0.0f, 0.0f, 0.0f};

        for (int I = I_first; I <= I_last; ++I) {
            // lane constants are recomputed per tile from an opaque copy of the
            // thread index, so the compiler does not keep every derived LDS
            // address of the unrolled loop below live across tiles
            int tid = threadIdx.x;
            asm volatile("" : "+v"(tid));
            const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), l = tid & 63;   // w: wave-uniform
            const int hf = l >> 5;
            const int p = l & 31;
            const int c0 = 4 * w + 2 * hf;
            const int q0 = (c0 - p) & 31;
            const int q1 = (q0 + 1) & 31;
            const int i16 = l & 15, ks = l >> 4;
            // pull block of this wave: A-operand rows ra0 + i16, B-operand rows rb
            const int ra0 = roww ? 16 * (w >> 1) : 16 * ((w - 4) >> 1);
            const int rb = (roww ? 16 * (w & 1) : 16 * ((w - 4) & 1)) + i16;
            const int ra = ra0 + i16;
            const int64_t tbase = ws_tile_offset(I, J, a.nt);
            float* const Xg = a.X + tbase;   // X tile: column-major
            float* const Yg = a.Y + tbase;   // Y tile: row-major
            {
                const int e0 = tid, e1 = tid + 512;   // LBt rows e >> 5, columns e & 31
                LBt[e0 >> 5][e0 & 31] = a.b_ident ? ((e0 >> 5) == (e0 & 31) ? 1.0f : 0.0f) : pf_lb0;
                LBt[e1 >> 5][e1 & 31] = a.b_ident ? ((e1 >> 5) == (e1 & 31) ? 1.0f : 0.0f) : pf_lb1;
            }
            float h0 = pf_h0, h1 = pf_h1;
            float g0 = pf_g0, g1 = pf_g1;
            // scales of the thread's two entries (one per row without GQ)
            const float s0 = pf_s0, s1 = GQ ? pf_s1 : s0;
            const float inv_s0 = (s0 > 0.0f) ? 1.0f / s0 : 0.0f;
            const float inv_s1 = GQ ? ((s1 > 0.0f) ? 1.0f / s1 : 0.0f) : inv_s0;
            const int kc = a.b_ident ? 0 : (knear < I ? knear : I);   // column sources k = 1..kc

            // multiplies source distance k of tile It into pacc (row or column kind)
            auto pull_src = [&](int It, int k) {
                f32x4 a0, a1, b0, b1;
                if (roww) {
                    a0 = lds_chunk(LAs[k - 1], ra, 2 * ks);
                    a1 = lds_chunk(LAs[k - 1], ra, 2 * ks + 1);
                    b0 = lds_chunk(Yn[k - 2], rb, 2 * ks);
                    b1 = lds_chunk(Yn[k - 2], rb, 2 * ks + 1);
                } else {
                    const float* e = &Ering[(It - k) % RING][rb][8 * ks];
                    a0 = lds_chunk(LBn[k - 1], ra, 2 * ks);
                    a1 = lds_chunk(LBn[k - 1], ra, 2 * ks + 1);
                    b0 = *reinterpret_cast<const f32x4*>(e);
                    b1 = *reinterpret_cast<const f32x4*>(e + 4);
                }
                mfma_8(a0, a1, b0, b1, pacc);
            };
            // issues the direct loads of tile It's operands: L^B[It, It-k],
            // k = 1..min(knear, It), and F[It, J-k], k = 2..kr
            auto stage = [&](int It, bool lb, bool y) {
                const int nlb = lb ? (knear < It ? knear : It) : 0;
                const int lim = 4 * (nlb + (y ? kr - 1 : 0));
                // wave w issues row groups g = w, w + 8, ... (uniform control flow)
#pragma unroll
                for (int i = 0; i < (4 * (2 * KNEAR_MAX - 1) + 7) / 8; ++i) {
                    const int g = w + 8 * i;
                    if (g < lim) {
                        const int ti = g >> 2;
                        if (ti < nlb)
                            stage_rows<0>(a.LB + packed_tile_offset(It, It - 1 - ti), LBn[ti], g & 3, l);
                        else
                            stage_rows<CPOL_SC1>(a.Y + ws_tile_offset(It, J - 2 - (ti - nlb), a.nt),
                                                 Yn[ti - nlb], g & 3, l);
                    }
                }
            };

            // 1. pull.  Operands not staged during the previous tile's loop
            // (first tile of the strip, or a left strip that was late) are
            // staged now.
            const bool lb_need = !a.b_ident && kc >= 1;
            if ((lb_need && !lb_staged) || (need_y && !y_staged)) {   // uniform
                if (need_y && !y_staged) wait_ready(a.flags + I * a.nt + (J - 2), a.status, a.spin_limit);
                stage(I, lb_need && !lb_staged, need_y && !y_staged);
                __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's direct loads landed
                __syncthreads();
            }
            {
                const int kmax = roww ? kr : kc;
                for (; nk <= kmax; ++nk) pull_src(I, nk);
                if (roww) {
                    if (kr >= 1) {   // distance 1: F[I, J-1] straight from memory after its flag
                        wait_ready(a.flags + I * a.nt + (J - 1), a.status, a.spin_limit);
                        const __amdgpu_buffer_rsrc_t r1 = tile_rsrc(a.Y + ws_tile_offset(I, J - 1, a.nt));
                        const f32x4 b0 = __builtin_amdgcn_raw_buffer_load_b128(r1, (rb * TS + 8 * ks) * 4, 0, CPOL_SC1);
                        const f32x4 b1 = __builtin_amdgcn_raw_buffer_load_b128(r1, (rb * TS + 8 * ks + 4) * 4, 0, CPOL_SC1);
                        mfma_8(lds_chunk(LAs[0], ra, 2 * ks), lds_chunk(LAs[0], ra, 2 * ks + 1), b0, b1, pacc);
                    }
                } else if (kc >= 1) {   // distance 1: E[I-1, J] from the ring
                    const float* e = &Ering[(I - 1) % RING][rb][8 * ks];
                    mfma_8(lds_chunk(LBn[0], ra, 2 * ks), lds_chunk(LBn[0], ra, 2 * ks + 1),
                           *reinterpret_cast<const f32x4*>(e), *reinterpret_cast<const f32x4*>(e + 4), pacc);
                }
                float (*out)[TS + 1] = roww ? HR : GC;
#pragma unroll
                for (int r = 0; r < 4; ++r) out[ra0 + 4 * ks + r][rb] = pacc[r];
            }
            if (tid == 0)   // can the next tile's row operands be staged during this tile's loop?
                ynext = (need_y && I < I_last)
                            ? __hip_atomic_load(a.flags + (I + 1) * a.nt + (J - 2), __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT)
                            : 0;
            __syncthreads();
            h0 += HR[q0][p];
            h1 += HR[q1][p];
            g0 += GC[p][q0];
            g1 += GC[p][q1];
            pacc = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            nk = 2;
            const bool has_next = I < I_last;
            const int kc_next = a.b_ident ? 0 : (knear < I + 1 ? knear : I + 1);
            lb_staged = has_next;
            y_staged = has_next && ynext != 0;
            if (has_next) {
                __atomic_signal_fence(__ATOMIC_SEQ_CST);   // the F loads stay after the flag test
                stage(I + 1, !a.b_ident && kc_next >= 1, y_staged);
            }
            const int kmax_next = roww ? (y_staged ? kr : 1) : kc_next;

            if (has_next) {   // prefetch the next tile's inputs (consumed after the loop)
                const int In = I + 1;
                const int64_t tb = ws_tile_offset(In, J, a.nt);
                const float* lbp = a.LB + packed_tile_offset(In, In);
                if (!a.b_ident) {
                    pf_lb0 = lbp[tid];
                    pf_lb1 = lbp[tid + 512];
                }
                pf_h0 = a.X[tb + q0 * TS + p];
                pf_h1 = a.X[tb + q1 * TS + p];
                pf_g0 = a.Y[tb + p * TS + q0];
                pf_g1 = a.Y[tb + p * TS + q1];
                const int rn = In * TS + p;
                pf_s0 = row_scale_of<GQ>(a.q, rn, cs0, a.m);
                if (GQ) pf_s1 = row_scale_of<GQ>(a.q, rn, cs1, a.m);
            }

            float lbr[TS], lar0[TS], lar1[TS];
#pragma unroll
            for (int k = 0; k < TS; ++k) { lbr[k] = LBt[p][(k - q0) & 31]; lar0[k] = LAt[q0][(k - p) & 31]; lar1[k] = LAt[q1][(k - p) & 31]; }

            // 2. in-tile rounding.  Quantisation without branches: a zero scale
            // gives inv_s = 0, so x = 0, code 0, V = 0 and E = -W~ (the entry's
            // alphabet is {0}).  Each thread keeps E, F and x of its own two
            // entries when it processes them.
            float eo0 = 0.0f, eo1 = 0.0f, fo0 = 0.0f, fo1 = 0.0f, xv0 = 0.0f, xv1 = 0.0f;
            // one round: the active half-wave quantises anti-diagonals d and d + 1
            // and broadcasts their E (per column) and F (per row) through LDS
            auto round = [&](int kp, int d, int tp, int rb) {
                const bool act = hf == ((kp >> 1) & 1);
                // slot 0: anti-diagonal d
                const bool v0 = act && (p + q0 == d);
                const float acc0 = g0 + h0;
                const float x0 = acc0 * inv_s0;
                const float r0 = __builtin_amdgcn_fmed3f(rintf(x0), qlo, qhi);
                const float ew0 = fmaf(r0, s0, -acc0);
                const float e0 = v0 ? ew0 : 0.0f;
                const float f0 = v0 ? g0 + ew0 : 0.0f;
                // slot 1: anti-diagonal d + 1, plus the two pushes from d
                const float eup = __int_as_float(
                    __builtin_amdgcn_update_dpp(0, __float_as_int(e0), 0x138, 0xf, 0xf, true));
                const float g1n = fmaf(lbr[(kp - 1) & 31], eup, g1);
                const float h1n = fmaf(f0, lar1[kp & 31], h1);
                const bool v1 = act && (p + q1 == d + 1);
                const float acc1 = g1n + h1n;
                const float x1 = acc1 * inv_s1;
                const float r1 = __builtin_amdgcn_fmed3f(rintf(x1), qlo, qhi);
                const float ew1 = fmaf(r1, s1, -acc1);
                const float e1 = v1 ? ew1 : 0.0f;
                const float f1 = v1 ? g1n + ew1 : 0.0f;
                // broadcast (the inactive half writes the dummy slots)
                Ecs[tp][rb][0][act ? q0 : TS + p] = e0;
                Ecs[tp][rb][1][act ? q1 : TS + p] = e1;
                Frs[tp][rb][act ? p : TS + p] = make_float2(f0, f1);
                // keep the processed entries' outputs
                eo0 = v0 ? e0 : eo0;
                fo0 = v0 ? f0 : fo0;
                xv0 = v0 ? x0 : xv0;
                eo1 = v1 ? e1 : eo1;
                fo1 = v1 ? f1 : fo1;
                xv1 = v1 ? x1 : xv1;
            };
            // every thread adds the pushes of one round to both of its entries
            auto update = [&](int kp, int tp, int rb) {
                const float ea0 = Ecs[tp][rb][0][q0], ea1 = Ecs[tp][rb][0][q1];
                const float eb0 = Ecs[tp][rb][1][q0], eb1 = Ecs[tp][rb][1][q1];
                const float2 fr = Frs[tp][rb][p];
                g0 = fmaf(lbr[kp & 31], ea0, g0);
                g0 = fmaf(lbr[(kp + 1) & 31], eb0, g0);
                g1 = fmaf(lbr[(kp - 1) & 31], ea1, g1);
                g1 = fmaf(lbr[kp & 31], eb1, g1);
                h0 = fmaf(fr.x, lar0[kp & 31], h0);
                h0 = fmaf(fr.y, lar0[(kp + 1) & 31], h0);
                h1 = fmaf(fr.x, lar1[kp & 31], h1);
                h1 = fmaf(fr.y, lar1[(kp + 1) & 31], h1);
            };
            // Wave kq owns anti-diagonals 4kq .. 4kq + 3 (mod 32): two rounds in a
            // row (its half 0, then its half 1).  Between them only that wave
            // needs the first round's values, so it reads them back itself (LDS
            // operations of one wave complete in order) and the workgroup
            // barrier comes once per turn of two rounds.  Buffers alternate
            // with the turn's parity, so a turn never overwrites values that a
            // slower wave may still be reading from the previous turn.
            // After the barrier of a turn, every wave except the one that is
            // active in the next turn multiplies one staged pull source of the
            // next tile (from turn PULL_T0 on, once the direct loads issued
            // before the loop have landed).
            for (int d0 = 0; d0 < 2 * TS; d0 += TS) {
#pragma unroll
                for (int kq = 0; kq < 8; ++kq) {
                    const int tp = kq & 1, kpa = 4 * kq, kpb = 4 * kq + 2;
                    const int turn = (d0 >> 2) + kq;
                    if (w == kq) {                       // wave-uniform
                        round(kpa, d0 + kpa, tp, 0);
                        __builtin_amdgcn_wave_barrier();
                        update(kpa, tp, 0);
                        round(kpb, d0 + kpb, tp, 1);
                    }
                    __syncthreads();
                    if (w != kq) update(kpa, tp, 0);
                    update(kpb, tp, 1);
                    if (turn == PULL_T0 - 1) __builtin_amdgcn_s_waitcnt(0x0F70);   // staged operands landed
                    if (turn >= PULL_T0 && w != ((kq + 1) & 7) && nk <= kmax_next) {
                        pull_src(I + 1, nk);
                        ++nk;
                    }
                }
            }

            // 3. publish F (device-coherent, whole rows), then the flag; E to the ring and X
            Fst[p][q0] = fo0;
            Fst[p][q1] = fo1;
            Xg[q0 * TS + p] = eo0;
            Xg[q1 * TS + p] = eo1;
            Ering[I % RING][q0][p] = eo0;
            Ering[I % RING][q1][p] = eo1;
            __syncthreads();
            if (w < 4) {   // wave w stores rows 8w .. 8w + 7, 16 bytes per lane
                const int r = 8 * w + (l >> 3), c = l & 7;
                const f32x4 v = *reinterpret_cast<const f32x4*>(&Fst[r][4 * c]);
                __builtin_amdgcn_raw_buffer_store_b128(v, tile_rsrc(Yg), (r * TS + 4 * c) * 4, 0, CPOL_SC1);
            }
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's stores are complete
            __syncthreads();
            if (tid == 0)
                __hip_atomic_store(a.flags + I * a.nt + J, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

            // 4. outputs, as whole row segments: every thread leaves x and the
            // scale of its entries in LDS (F is stored, Fst is free), then 256
            // threads write 4 consecutive entries of one row each (one 4-byte
            // code store and 16-byte V and pre stores instead of 64 scattered
            // rows per instruction)
            Fst[p][q0] = xv0;
            Fst[p][q1] = xv1;
            if (GQ) {
                So[p][q0] = s0;
                So[p][q1] = s1;
            } else {
                So[0][p] = s0;
            }
            __syncthreads();
            if (tid < 256) {
                const float nan = __builtin_nanf("");
                const int r = tid >> 3, cb = 4 * (tid & 7);
                const int64_t orow = (int64_t)I * TS + r, ocol = (int64_t)J * TS + cb;
                const f32x4 xq = *reinterpret_cast<const f32x4*>(&Fst[r][cb]);
                float cv[4], vv[4], pv[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const float sk = GQ ? So[r][cb + k] : So[0][r];
                    cv[k] = __builtin_amdgcn_fmed3f(rintf(xq[k]), qlo, qhi);
                    vv[k] = cv[k] * sk;
                    pv[k] = sk > 0.0f ? xq[k] : nan;
                }
                if (orow < a.m) {
                    const int64_t o = orow * a.n + ocol;
                    if ((a.n & 3) == 0 && ocol + 3 < a.n) {   // aligned, inside the matrix
                        uint32_t packed = 0;
#pragma unroll
                        for (int k = 0; k < 4; ++k) packed |= (uint32_t)(uint8_t)(int8_t)(int)cv[k] << (8 * k);
                        *reinterpret_cast<uint32_t*>(a.codes + o) = packed;
                        *reinterpret_cast<f32x4*>(a.V + o) = f32x4{vv[0], vv[1], vv[2], vv[3]};
                        if (a.pre) *reinterpret_cast<f32x4*>(a.pre + o) = f32x4{pv[0], pv[1], pv[2], pv[3]};
                    } else {
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            if (ocol + k < a.n) {
                                a.codes[o + k] = (int8_t)(int)cv[k];
                                a.V[o + k] = vv[k];
                                if (a.pre) a.pre[o + k] = pv[k];
                            }
                        }
                    }
                }
            }
        }
    }
}

// Fills n 32-bit words with v (a debug aid: poisoning the workspace before a
// solve shows that every word the solve reads was written by it first).
__global__ __launch_bounds__(256) void k_fill_u32(uint32_t* __restrict__ p, int64_t n, uint32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
        p[i] = v;
}

// *bad <- 1 if any of the `count` scales at s is negative, NaN or infinite
// (the quantiser needs finite scales >= 0).  *bad is cleared by the caller.
__global__ __launch_bounds__(256) void k_check_scales(const float* __restrict__ s, int64_t count,
                                                       int* __restrict__ bad) {
    bool ok = true;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) {
        const float v = s[i];
        ok = ok && v >= 0.0f && v <= 3.402823466e38f;
    }
    if (!ok) __hip_atomic_store(bad, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

hipError_t check_scales(hipStream_t st, const float* s, int64_t count, int* bad) {
    if (count <= 0) return hipSuccess;
    const int64_t g = std::min<int64_t>((count + 255) / 256, 1024);
    hipLaunchKernelGGL(k_check_scales, dim3((unsigned)g), dim3(256), 0, st, s, count, bad);
    return hipGetLastError();
}

hipError_t fill_words(hipStream_t st, void* p, int64_t n, uint32_t v) {
    if (n <= 0) return hipSuccess;
    const int64_t g = std::min<int64_t>((n + 255) / 256, 65536);
    hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)g), dim3(256), 0, st, static_cast<uint32_t*>(p), n, v);
    return hipGetLastError();
}

struct NodeArgs {
    int K, Mid;       // sources on tile anti-diagonals [K, Mid)
    int tlo, thi;     // targets on tile anti-diagonals [tlo, thi)
    int knear;
    int mt, nt;
    float* X;
    float* Y;
    const float* LA;
    const float* LB;
    const int4* items;  // work list of this launch (see NodeItem in common.h)
};

// Band push of one divide-and-conquer node on fp32 MFMA.
//
// Both pushes are computed as C[M][N] += sum_k A[M][k] * B[N][k] over source
// tiles kt (K chunks of TS), with every operand tile stored [row][k]:
//   column push: C = Y[I, J] (row-major), A = L^B[I, kt], B = E[kt, J] read
//                from X, whose tiles are column-major (= E^T);
//   row push:    C = X[I, J] stored column-major, i.e. C^T[J][I]
//                = sum L^A[J, kt] * F[I, kt]^T, A = L^A[J, kt], B = F[I, kt]
//                read from Y (row-major).
// So every global -> LDS copy is a straight 16-byte copy and every output
// write is coalesced.  A workgroup computes MT x MT solver tiles with 4 waves
// in a 2 x 2 arrangement (each wave MT/2 x MT/2 blocks of
// v_mfma_f32_32x32x2f32).  Inside a K chunk the 32 k's are split between the
// two lane halves (half h takes k = 16h + s at step s), so each lane reads 16
// consecutive floats per operand with four 16-byte LDS loads.  LDS is double
// buffered and the chunks two ahead are prefetched into registers while the
// current one is multiplied.  The (source, target) validity masks are separable, so
// invalid source tiles are staged as zeros and the sums stay exact.
//
// One workgroup per work-list item: the host lists only items with a
// non-empty source range, longest first, so the long K loops start early.
constexpr int LDS_STRIDE = TS + 4;   // 36 floats: 16-byte rows, no b128 bank conflicts
template <int MT>
__global__ __launch_bounds__(256, (MT == 4 ? 2 : 4)) void k_node(NodeArgs a) {
    constexpr int WB = MT / 2;       // 32x32 blocks per wave per dimension
    __shared__ __attribute__((aligned(16))) float As[2][MT * TS][LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) float Bs[2][MT * TS][LDS_STRIDE];
    const int4 it = a.items[blockIdx.x];
    const int I0 = it.x, J0 = it.y;
    const bool colpush = (it.z & 1) == 0;
    const int klo = it.z >> 1, khi = it.w;

    const int tid = threadIdx.x;
    const int wv = tid >> 6, l = tid & 63;
    const int wm = wv >> 1, wn = wv & 1;
    const int lr = l & 31, lk = l >> 5;
    const int srow = tid >> 3, sk = (tid & 7) * 4;   // staging: one float4 of each tile

    // Operand tile t of K chunk kt as a buffer resource: a valid tile covers
    // its 4 KB, an invalid one (outside the matrix, outside the (source,
    // target) masks or past the item's range) has no records, so its loads
    // return zeros without touching memory.  Every chunk therefore issues the
    // same loads unconditionally, which lets the compiler wait only for the
    // chunk it stores (the two-ahead prefetch stays in flight).  Per operand
    // tile the valid chunks form one range [lo, hi) and consecutive chunks sit
    // a fixed stride apart, so the per-item set-up below leaves two compares
    // and an address per tile per chunk.
    //   column push: A = L^B[I0 + t, kt] (kt <= I - knear - 1), B = E[kt, J0 + t]
    //                (kt + J in [K, Mid)), read from X;
    //   row push:    A = L^A[J0 + t, kt] (kt <= J - knear - 1), B = F[I0 + t, kt]
    //                (I + kt in [K, Mid)), read from Y.
    const float* abase[MT];
    const float* bbase[MT];
    int alo[MT], ahi[MT], blo[MT], bhi[MT];
    const int64_t bstride = colpush ? (int64_t)a.nt * TILE_ELEMS : TILE_ELEMS;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const int Ia = colpush ? I0 + t : J0 + t;   // factor tile row
        const bool arow = colpush ? Ia < a.mt : Ia < a.nt;
        abase[t] = arow ? (colpush ? a.LB : a.LA) + packed_tile_offset(Ia, 0) : a.LA;
        alo[t] = 0;
        ahi[t] = arow ? min(khi, Ia - a.knear) : 0;
        const int Ib = colpush ? J0 + t : I0 + t;   // fixed coordinate of the source tile
        const bool brow = colpush ? Ib < a.nt : Ib < a.mt;
        bbase[t] = brow ? (colpush ? a.X + ws_tile_offset(0, Ib, a.nt) : a.Y + ws_tile_offset(Ib, 0, a.nt))
                        : a.LA;
        blo[t] = max(a.K - Ib, 0);
        bhi[t] = brow ? min(khi, a.Mid - Ib) : 0;
    }
    // (an invalid tile's address may lie outside every allocation: with no
    // records nothing is read)
    auto rsrc = [](const float* base, int64_t stride, int kt, int lo, int hi) {
        const int nrec = (kt >= lo && kt < hi) ? TILE_ELEMS * 4 : 0;
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base + kt * stride), (short)0, nrec,
                                                 0x00020000);
    };
    // two register sets: while chunk kt is multiplied from LDS, chunk kt + 1
    // (loaded one iteration earlier) waits in one set and chunk kt + 2 is in
    // flight into the other, so each global load has two chunks of MFMA work
    // to hide behind
    f32x4 ra[2][MT], rb[2][MT];
    auto load = [&](int kt, int r) {
#pragma unroll
        for (int t = 0; t < MT; ++t) {
            ra[r][t] = __builtin_amdgcn_raw_buffer_load_b128(
                rsrc(abase[t], TILE_ELEMS, kt, alo[t], ahi[t]), tid * 16, 0, 0);
            rb[r][t] = __builtin_amdgcn_raw_buffer_load_b128(
                rsrc(bbase[t], bstride, kt, blo[t], bhi[t]), tid * 16, 0, 0);
        }
    };
    auto store = [&](int s, int r) {
#pragma unroll
        for (int t = 0; t < MT; ++t) {
            *reinterpret_cast<f32x4*>(&As[s][t * TS + srow][sk]) = ra[r][t];
            *reinterpret_cast<f32x4*>(&Bs[s][t * TS + srow][sk]) = rb[r][t];
        }
    };

    f32x16 acc[WB][WB];
#pragma unroll
    for (int x = 0; x < WB; ++x)
#pragma unroll
        for (int y = 0; y < WB; ++y) acc[x][y] = f32x16{0};

    // one K chunk: multiply LDS buffer s; issue the load of chunk kt + 2 into
    // register set r, then move chunk kt + 1 (set r ^ 1) into buffer s ^ 1
    auto chunk = [&](int kt, int s, int r) {
        load(kt + 2, r);   // past the range: no records, zeros
        f32x4 fa[WB][4], fb[WB][4];
#pragma unroll
        for (int x = 0; x < WB; ++x)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                fa[x][v] = *reinterpret_cast<const f32x4*>(
                    &As[s][(wm * WB + x) * TS + lr][lk * 16 + v * 4]);
#pragma unroll
        for (int y = 0; y < WB; ++y)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                fb[y][v] = *reinterpret_cast<const f32x4*>(
                    &Bs[s][(wn * WB + y) * TS + lr][lk * 16 + v * 4]);
#pragma unroll
        for (int st = 0; st < 16; ++st) {
#pragma unroll
            for (int x = 0; x < WB; ++x)
#pragma unroll
                for (int y = 0; y < WB; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[x][st >> 2][st & 3],
                                                                    fb[y][st >> 2][st & 3],
                                                                    acc[x][y], 0, 0, 0);
        }
        if (kt + 1 < khi) store(s ^ 1, r ^ 1);
        __syncthreads();
    };

    load(klo, 0);
    load(klo + 1, 1);
    store(0, 0);
    __syncthreads();
    // chunk klo + 2i uses buffer 0 and register set 0 for its prefetch,
    // chunk klo + 2i + 1 buffer 1 and set 1
    for (int kt = klo; kt < khi; kt += 2) {
        chunk(kt, 0, 0);
        if (kt + 1 < khi) chunk(kt + 1, 1, 1);
    }

    // epilogue: block (x, y) of wave (wm, wn) is output solver tile
    // (M tile wm*WB+x, N tile wn*WB+y); C[M][N] row-major inside the tile.
#pragma unroll
    for (int x = 0; x < WB; ++x)
#pragma unroll
        for (int y = 0; y < WB; ++y) {
            const int tm = wm * WB + x, tn = wn * WB + y;
            const int I = colpush ? I0 + tm : I0 + tn;
            const int J = colpush ? J0 + tn : J0 + tm;
            if (I >= a.mt || J >= a.nt || I + J < a.tlo || I + J >= a.thi) continue;
            float* out = (colpush ? a.Y : a.X) + ws_tile_offset(I, J, a.nt);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rr = (r >> 2) * 8 + lk * 4 + (r & 3);
                out[rr * TS + lr] += acc[x][y][r];
            }
        }
}

// X <- W (tile-major, column-major inside each tile, zero padding), Y <- 0,
// ready flags <- 0 and ticket counters <- 0 (the give-up status word is left
// as it is: it is cleared only when the host reads it).  One workgroup per tile; the
// transpose goes through LDS so that both the read of W and the write of X
// are coalesced.
template <bool VEC>
__global__ __launch_bounds__(256) void k_prep(const float* __restrict__ W, int64_t m, int64_t n,
                                              int mt, int nt, float* __restrict__ X,
                                              float* __restrict__ Y, int* __restrict__ flags,
                                              int* __restrict__ counters, int ncounters) {
    __shared__ float T[TS][TS + 1];
    const int64_t tile = blockIdx.x;
    const int64_t I = tile / nt, J = tile - (tile / nt) * nt;
    const int tid = threadIdx.x;
    const int64_t base = tile * TILE_ELEMS;
    if (VEC) {
        // W rows as 16-byte chunks (n % 4 == 0, W 16-byte aligned), one per
        // thread; X (the tile transposed) and Y as contiguous 16-byte stores
        const int r = tid >> 3, c4 = (tid & 7) * 4;
        const int64_t gr = I * TS + r, gc = J * TS + c4;
        float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (gr < m && gc < n) v = *reinterpret_cast<const float4*>(W + gr * n + gc);
        T[r][c4] = v.x;
        T[r][c4 + 1] = v.y;
        T[r][c4 + 2] = v.z;
        T[r][c4 + 3] = v.w;
        __syncthreads();
        const int c = tid >> 3, r4 = (tid & 7) * 4;
        *reinterpret_cast<float4*>(X + base + 4 * tid) =
            make_float4(T[r4][c], T[r4 + 1][c], T[r4 + 2][c], T[r4 + 3][c]);
        *reinterpret_cast<float4*>(Y + base + 4 * tid) = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    } else {
#pragma unroll
        for (int k = 0; k < TILE_ELEMS / 256; ++k) {
            const int e = k * 256 + tid;
            const int r = e >> 5, c = e & 31;
            const int64_t gr = I * TS + r, gc = J * TS + c;
            T[r][c] = (gr < m && gc < n) ? W[gr * n + gc] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < TILE_ELEMS / 256; ++k) {
            const int e = k * 256 + tid;
            const int c = e >> 5, r = e & 31;
            X[base + e] = T[r][c];
            Y[base + e] = 0.0f;
        }
    }
    if (tid == 0) flags[tile] = 0;
    if (tile == 0)
        for (int i = tid; i < ncounters; i += 256) counters[i] = 0;
}

// ---------------------------------------------------------------------------
// host launch driver

// Launches the plan: main ops on `st`, side ops on `side` (see Plan).
// ev_rel[i] is recorded on st after main op i when a side op waits for it;
// ev_side[c] on `side` after side op c.  tim (optional, profiling): an event
// pair around every launch, in enqueue order (prep first).
hipError_t run_plan(hipStream_t st, hipStream_t side, const Plan& plan, const float* W, int64_t m,
                    int64_t n, int mt, int nt, const Workspace& ws, const float* LA, const float* LB,
                    int b_ident, const QuantArgs& q, int8_t* codes, float* V, float* pre,
                    int knear, int spin_limit, const int4* items, hipEvent_t* tim,
                    hipEvent_t* ev_rel, hipEvent_t* ev_side) {
    int ti = 0;
    auto t_begin = [&](hipStream_t s) { if (tim) (void)hipEventRecord(tim[2 * ti], s); };
    auto t_end = [&](hipStream_t s) { if (tim) (void)hipEventRecord(tim[2 * ti + 1], s); ++ti; };
    hipError_t e;
    t_begin(st);
    if (n % 4 == 0 && reinterpret_cast<uintptr_t>(W) % 16 == 0)
        hipLaunchKernelGGL(k_prep<true>, dim3((unsigned)((int64_t)mt * nt)), dim3(256), 0, st, W, m,
                           n, mt, nt, ws.X, ws.Y, ws.flags, ws.counters, plan.nseg);
    else
        hipLaunchKernelGGL(k_prep<false>, dim3((unsigned)((int64_t)mt * nt)), dim3(256), 0, st, W, m,
                           n, mt, nt, ws.X, ws.Y, ws.flags, ws.counters, plan.nseg);
    t_end(st);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    SegArgs sa{};
    sa.mt = mt; sa.nt = nt; sa.m = m; sa.n = n; sa.X = ws.X; sa.Y = ws.Y;
    sa.LA = LA; sa.LB = LB; sa.b_ident = b_ident; sa.q = q;
    sa.codes = codes; sa.V = V; sa.pre = pre; sa.knear = knear; sa.flags = ws.flags;
    sa.status = ws.status;
    sa.spin_limit = spin_limit;
    NodeArgs nd{};
    nd.knear = knear; nd.mt = mt; nd.nt = nt; nd.X = ws.X; nd.Y = ws.Y; nd.LA = LA; nd.LB = LB;
    auto node = [&](const PlanOp& op, hipStream_t s) {
        nd.K = op.K;
        nd.Mid = op.Mid;
        nd.tlo = op.tlo;
        nd.thi = op.thi;
        nd.items = items + op.item_off;
        if (op.macro == 4)
            hipLaunchKernelGGL(k_node<4>, dim3((unsigned)op.item_cnt), dim3(256), 0, s, nd);
        else
            hipLaunchKernelGGL(k_node<2>, dim3((unsigned)op.item_cnt), dim3(256), 0, s, nd);
    };
    int waited_side = 0, waited_rel = -1;
    for (const std::pair<int, int>& o : plan.order) {
        if (o.first == 0) {
            const PlanOp& op = plan.ops[o.second];
            if (op.need_side > waited_side) {
                if ((e = hipStreamWaitEvent(st, ev_side[op.need_side - 1], 0)) != hipSuccess) return e;
                waited_side = op.need_side;
            }
            t_begin(st);
            if (op.kind == 0) {
                sa.K = op.K;
                sa.L = op.L;
                sa.J_lo = op.strip_lo;
                sa.nstrips = op.nstrips;
                sa.counter = ws.counters + op.counter;
                const int grid = op.nstrips < SEG_GRID ? op.nstrips : SEG_GRID;
                const bool gq = q.gsize > 0 || q.col_scale, asym = q.qlo != -q.qhi;
                if (gq && asym)
                    hipLaunchKernelGGL((k_seg<true, true>), dim3((unsigned)grid), dim3(512), 0, st, sa);
                else if (gq)
                    hipLaunchKernelGGL((k_seg<true, false>), dim3((unsigned)grid), dim3(512), 0, st, sa);
                else if (asym)
                    hipLaunchKernelGGL((k_seg<false, true>), dim3((unsigned)grid), dim3(512), 0, st, sa);
                else
                    hipLaunchKernelGGL((k_seg<false, false>), dim3((unsigned)grid), dim3(512), 0, st, sa);
            } else {
                node(op, st);
            }
            t_end(st);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            if (op.rec_rel && (e = hipEventRecord(ev_rel[o.second], st)) != hipSuccess) return e;
        } else {
            const PlanOp& op = plan.side[o.second];
            if (op.rel > waited_rel) {
                if ((e = hipStreamWaitEvent(side, ev_rel[op.rel], 0)) != hipSuccess) return e;
                waited_rel = op.rel;
            }
            t_begin(side);
            node(op, side);
            t_end(side);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            if ((e = hipEventRecord(ev_side[o.second], side)) != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

int plan_timed_launches(const Plan& plan) { return 1 + (int)plan.ops.size() + (int)plan.side.size(); }

}  // namespace bk
