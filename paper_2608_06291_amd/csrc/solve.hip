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
// A leaf solves the tiles of one anti-diagonal and immediately pushes to the
// KNEAR next tiles below and to the right; node products take only sources
// farther than KNEAR tiles, so each (source, target) tile pair is applied
// exactly once.
#include "common.h"

#include <vector>

namespace bk {

struct LeafArgs {
    int D;            // tile anti-diagonal
    int I_lo;         // first tile row on it
    int mt, nt;       // tile grid
    int64_t m, n;     // real sizes
    float* X;
    float* Y;
    const float* LA;  // packed factor tiles
    const float* LB;
    int b_ident;      // B = I (no column feedback)
    const float* scale;
    float qmax;
    int8_t* codes;
    float* V;
    float* pre;       // may be null
    int knear;
};

// One workgroup (1024 threads) per tile.  Thread <-> entry (p, q); wave w
// holds the entries with (p + q) mod 32 in {2w, 2w+1}, so the entries of one
// element anti-diagonal d are all in one wave (half of it).
//
// Per step d: the owners of diagonal d quantise and publish the error E of
// their column and the F of their row; every thread then adds one column
// push (L^B[p][d-q] * E[d-q][q]) and one row push (F[p][d-p] * L^A[q][d-p]).
// The coefficients are held in registers, each thread's factor row rotated so
// that step d reads register (d mod 32): no dynamic register indexing.
__global__ __launch_bounds__(1024) void k_leaf(LeafArgs a) {
    __shared__ float LBt[TS][TS];            // unpadded: the rotated reads below are conflict-free
    __shared__ float LAt[TS][TS];
    __shared__ float Et[TS][TS + 1];
    __shared__ float Ft[TS][TS + 1];
    __shared__ float Pw[16][TS][TS + 1];     // per-wave push factor tile (prefetched)
    __shared__ float Ow[16][TILE_ELEMS];     // per-wave push target tile, fragment order (prefetched)
    __shared__ float Ecol[2][TS];
    __shared__ float Frow[2][TS];

    const int I = a.I_lo + (int)blockIdx.x;
    const int J = a.D - I;
    const int tid = threadIdx.x;
    const int w = tid >> 6, l = tid & 63;
    const int c = 2 * w + (l >> 5);
    const int p = l & 31;
    const int q = (c - p) & 31;
    const int lr = l & 31, lk = l >> 5;

    // Near push of this wave: target kk = w/2 + 1 tiles below (even w, column
    // push into Y) or to the right (odd w, row push into X).  The factor tile
    // and the target tile do not change during this launch, so both are
    // fetched now and the push at the end touches no global memory before its
    // final store.
    const int kk = (w >> 1) + 1;
    const bool colpush = (w & 1) == 0;
    int TI = I, TJ = J;
    bool active = kk <= a.knear;
    const float* fac = nullptr;
    if (colpush) {
        TI = I + kk;
        active = active && !a.b_ident && TI < a.mt;
        if (active) fac = a.LB + packed_tile_offset(TI, I);
    } else {
        TJ = J + kk;
        active = active && TJ < a.nt;
        if (active) fac = a.LA + packed_tile_offset(TJ, J);
    }
    float* out = colpush ? a.Y : a.X;
    const int64_t to = ws_tile_offset(TI, TJ, a.nt);
    if (active) {
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            const int e0 = (s4 * 64 + l) * 4;
            const f32x4 v = *reinterpret_cast<const f32x4*>(fac + e0);
            const int r = e0 >> 5, cc = e0 & 31;
            Pw[w][r][cc] = v[0];
            Pw[w][r][cc + 1] = v[1];
            Pw[w][r][cc + 2] = v[2];
            Pw[w][r][cc + 3] = v[3];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int rr = (r >> 2) * 8 + lk * 4 + (r & 3);
            Ow[w][r * 64 + l] = out[to + rr * TS + lr];
        }
    }

    {   // diagonal factor tiles
        const int r = tid >> 5, cc = tid & 31;
        LAt[r][cc] = a.LA[packed_tile_offset(J, J) + tid];
        LBt[r][cc] = a.b_ident ? (r == cc ? 1.0f : 0.0f) : a.LB[packed_tile_offset(I, I) + tid];
    }
    const int64_t tbase = ws_tile_offset(I, J, a.nt);
    const int64_t xo = tbase + q * TS + p;     // X tiles are column-major
    const int64_t yo = tbase + p * TS + q;     // Y tiles are row-major
    float h = a.X[xo];
    float g = a.Y[yo];
    const int64_t row = (int64_t)I * TS + p, col = (int64_t)J * TS + q;
    const float s = (row < a.m) ? a.scale[row] : 0.0f;
    const float inv_s = (s > 0.0f) ? 1.0f / s : 0.0f;
    __syncthreads();

    float lbr[TS], lar[TS];
#pragma unroll
    for (int k = 0; k < TS; ++k) {
        lbr[k] = LBt[p][(k - q) & 31];
        lar[k] = LAt[q][(k - p) & 31];
    }

    float e_out = 0.0f, f_out = 0.0f, x_out = __builtin_nanf("");
    int c_out = 0;
    for (int d0 = 0; d0 < 2 * TS; d0 += TS) {
#pragma unroll
        for (int k = 0; k < TS; ++k) {
            if (w == (k >> 1) && (l >> 5) == (k & 1)) {
                const bool valid = (p + q == d0 + k);
                const float acc = g + h;
                float e = 0.0f, f = 0.0f;
                if (valid) {
                    float x, v;
                    int cc;
                    if (s > 0.0f) {
                        x = acc * inv_s;
                        float r = rintf(x);
                        r = fminf(fmaxf(r, -a.qmax), a.qmax);
                        cc = (int)r;
                        v = r * s;
                    } else {
                        x = __builtin_nanf("");
                        cc = 0;
                        v = 0.0f;
                    }
                    e = v - acc;
                    f = g + e;
                    e_out = e;
                    f_out = f;
                    x_out = x;
                    c_out = cc;
                }
                Ecol[k & 1][q] = e;
                Frow[k & 1][p] = f;
            }
            __syncthreads();
            const float ein = Ecol[k & 1][q];
            const float fin = Frow[k & 1][p];
            g = fmaf(lbr[k], ein, g);
            h = fmaf(fin, lar[k], h);
        }
    }

    a.X[xo] = e_out;
    a.Y[yo] = f_out;
    if (row < a.m && col < a.n) {
        const int64_t o = row * a.n + col;
        a.codes[o] = (int8_t)c_out;
        a.V[o] = (float)c_out * s;
        if (a.pre) a.pre[o] = x_out;
    }
    Et[p][q] = e_out;
    Ft[p][q] = f_out;
    __syncthreads();

    if (!active) return;   // wave-uniform; no barrier follows
    f32x16 acc = {0};
#pragma unroll
    for (int k0 = 0; k0 < TS; k0 += 2) {
        float av, bv;
        if (colpush) {            // Y[TI, J] += L^B[TI, I] (32x32) * E (32x32)
            av = Pw[w][lr][k0 + lk];
            bv = Et[k0 + lk][lr];
        } else {                  // X[I, TJ]^T += L^A[TJ, J] * F^T (X is column-major)
            av = Pw[w][lr][k0 + lk];
            bv = Ft[lr][k0 + lk];
        }
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int rr = (r >> 2) * 8 + lk * 4 + (r & 3);
        out[to + rr * TS + lr] = Ow[w][r * 64 + l] + acc[r];
    }
}

struct NodeArgs {
    int K, Mid, L;    // tile anti-diagonal range [K, L), split at Mid
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
// buffered and the next chunk is prefetched into registers while the current
// one is multiplied.  The (source, target) validity masks are separable, so
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

    auto a_tile = [&](int t, int kt) -> const float* {
        if (colpush) {
            const int I = I0 + t;
            return (I < a.mt && kt <= I - a.knear - 1) ? a.LB + packed_tile_offset(I, kt) : nullptr;
        }
        const int J = J0 + t;
        return (J < a.nt && kt <= J - a.knear - 1) ? a.LA + packed_tile_offset(J, kt) : nullptr;
    };
    auto b_tile = [&](int t, int kt) -> const float* {
        if (colpush) {
            const int J = J0 + t;
            return (J < a.nt && kt + J >= a.K && kt + J < a.Mid) ? a.X + ws_tile_offset(kt, J, a.nt)
                                                                 : nullptr;
        }
        const int I = I0 + t;
        return (I < a.mt && I + kt >= a.K && I + kt < a.Mid) ? a.Y + ws_tile_offset(I, kt, a.nt)
                                                             : nullptr;
    };
    f32x4 ra[MT], rb[MT];
    auto load = [&](int kt) {
#pragma unroll
        for (int t = 0; t < MT; ++t) {
            const float* pa = a_tile(t, kt);
            const float* pb = b_tile(t, kt);
            ra[t] = pa ? *reinterpret_cast<const f32x4*>(pa + tid * 4) : f32x4{0.f, 0.f, 0.f, 0.f};
            rb[t] = pb ? *reinterpret_cast<const f32x4*>(pb + tid * 4) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };
    auto store = [&](int s) {
#pragma unroll
        for (int t = 0; t < MT; ++t) {
            *reinterpret_cast<f32x4*>(&As[s][t * TS + srow][sk]) = ra[t];
            *reinterpret_cast<f32x4*>(&Bs[s][t * TS + srow][sk]) = rb[t];
        }
    };

    f32x16 acc[WB][WB];
#pragma unroll
    for (int x = 0; x < WB; ++x)
#pragma unroll
        for (int y = 0; y < WB; ++y) acc[x][y] = f32x16{0};

    load(klo);
    store(0);
    __syncthreads();
    for (int kt = klo; kt < khi; ++kt) {
        const int s = (kt - klo) & 1;
        const bool more = kt + 1 < khi;
        if (more) load(kt + 1);
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
        if (more) store(s ^ 1);
        __syncthreads();
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
            if (I >= a.mt || J >= a.nt || I + J < a.Mid || I + J >= a.L) continue;
            float* out = (colpush ? a.Y : a.X) + ws_tile_offset(I, J, a.nt);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rr = (r >> 2) * 8 + lk * 4 + (r & 3);
                out[rr * TS + lr] += acc[x][y][r];
            }
        }
}

// X <- W (tile-major, column-major inside each tile, zero padding), Y <- 0.
// One workgroup per tile; the transpose goes through LDS so that both the
// read of W and the write of X are coalesced.
__global__ __launch_bounds__(256) void k_prep(const float* __restrict__ W, int64_t m, int64_t n,
                                              int mt, int nt, float* __restrict__ X,
                                              float* __restrict__ Y) {
    __shared__ float T[TS][TS + 1];
    const int64_t tile = blockIdx.x;
    const int64_t I = tile / nt, J = tile - (tile / nt) * nt;
    const int tid = threadIdx.x;
#pragma unroll
    for (int k = 0; k < TILE_ELEMS / 256; ++k) {
        const int e = k * 256 + tid;
        const int r = e >> 5, c = e & 31;
        const int64_t gr = I * TS + r, gc = J * TS + c;
        T[r][c] = (gr < m && gc < n) ? W[gr * n + gc] : 0.0f;
    }
    __syncthreads();
    float* x = X + tile * TILE_ELEMS;
    float* y = Y + tile * TILE_ELEMS;
#pragma unroll
    for (int k = 0; k < TILE_ELEMS / 256; ++k) {
        const int e = k * 256 + tid;
        const int c = e >> 5, r = e & 31;
        x[e] = T[r][c];
        y[e] = 0.0f;
    }
}

// ---------------------------------------------------------------------------
// host launchers

hipError_t launch_prep(hipStream_t s, const float* W, int64_t m, int64_t n, int mt, int nt,
                       float* X, float* Y) {
    hipLaunchKernelGGL(k_prep, dim3((unsigned)((int64_t)mt * nt)), dim3(256), 0, s, W, m, n, mt, nt,
                       X, Y);
    return hipGetLastError();
}

hipError_t launch_leaf(hipStream_t s, const LeafArgs& a, int ntiles) {
    hipLaunchKernelGGL(k_leaf, dim3((unsigned)ntiles), dim3(1024), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_node(hipStream_t s, const NodeArgs& a, int nitems, int macro) {
    if (macro == 4)
        hipLaunchKernelGGL(k_node<4>, dim3((unsigned)nitems), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(k_node<2>, dim3((unsigned)nitems), dim3(256), 0, s, a);
    return hipGetLastError();
}

// Enqueue a whole solve.  evs (optional): 2 * (ops.size() + 1) events; a pair
// is recorded around the prep launch and around every schedule launch.
hipError_t run_schedule(hipStream_t s, const std::vector<SolveOp>& ops, const float* W, int64_t m,
                        int64_t n, int mt, int nt, float* X, float* Y, const float* LA,
                        const float* LB, int b_ident, const float* scale, float qmax,
                        int8_t* codes, float* V, float* pre, int knear, const int4* items,
                        hipEvent_t* evs) {
    if (evs) hipEventRecord(evs[0], s);
    hipError_t e = launch_prep(s, W, m, n, mt, nt, X, Y);
    if (evs) hipEventRecord(evs[1], s);
    if (e != hipSuccess) return e;
    LeafArgs la{};
    la.mt = mt;
    la.nt = nt;
    la.m = m;
    la.n = n;
    la.X = X;
    la.Y = Y;
    la.LA = LA;
    la.LB = LB;
    la.b_ident = b_ident;
    la.scale = scale;
    la.qmax = qmax;
    la.codes = codes;
    la.V = V;
    la.pre = pre;
    la.knear = knear;
    NodeArgs na{};
    na.knear = knear;
    na.mt = mt;
    na.nt = nt;
    na.X = X;
    na.Y = Y;
    na.LA = LA;
    na.LB = LB;
    size_t i = 1;
    for (const SolveOp& op : ops) {
        if (evs) hipEventRecord(evs[2 * i], s);
        if (op.kind == 0) {
            la.D = op.D;
            la.I_lo = op.I_lo;
            e = launch_leaf(s, la, op.ntiles);
        } else {
            na.K = op.K;
            na.Mid = op.Mid;
            na.L = op.L;
            na.items = items + op.item_off;
            e = launch_node(s, na, op.item_cnt, op.macro);
        }
        if (evs) hipEventRecord(evs[2 * i + 1], s);
        ++i;
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace bk
