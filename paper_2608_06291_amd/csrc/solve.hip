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
    __shared__ float LBt[TS][TS + 1];
    __shared__ float LAt[TS][TS + 1];
    __shared__ float Et[TS][TS + 1];
    __shared__ float Ft[TS][TS + 1];
    __shared__ float Pw[16][TS][TS + 1];   // per-wave factor tile for pushes
    __shared__ float Ecol[2][TS];
    __shared__ float Frow[2][TS];

    const int I = a.I_lo + (int)blockIdx.x;
    const int J = a.D - I;
    const int tid = threadIdx.x;
    const int w = tid >> 6, l = tid & 63;
    const int c = 2 * w + (l >> 5);
    const int p = l & 31;
    const int q = (c - p) & 31;

    {   // diagonal factor tiles
        const int r = tid >> 5, cc = tid & 31;
        LAt[r][cc] = a.LA[packed_tile_offset(J, J) + tid];
        LBt[r][cc] = a.b_ident ? (r == cc ? 1.0f : 0.0f) : a.LB[packed_tile_offset(I, I) + tid];
    }
    const int64_t xo = ws_tile_offset(I, J, a.nt) + p * TS + q;
    float h = a.X[xo];
    float g = a.Y[xo];
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
    a.Y[xo] = f_out;
    if (row < a.m && col < a.n) {
        const int64_t o = row * a.n + col;
        a.codes[o] = (int8_t)c_out;
        a.V[o] = (float)c_out * s;
        if (a.pre) a.pre[o] = x_out;
    }
    Et[p][q] = e_out;
    Ft[p][q] = f_out;
    __syncthreads();

    // Near pushes: wave w handles target k = w/2 + 1, column push (even w)
    // or row push (odd w), one 32x32x32 product on fp32 MFMA.
    const int kk = (w >> 1) + 1;
    const bool colpush = (w & 1) == 0;
    bool active = kk <= a.knear;
    int TI = I, TJ = J;
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
    if (!active) return;   // wave-uniform; no barrier follows
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
    // intra-wave handoff of the LDS tile (other lanes' writes)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    f32x16 acc = {0};
    const int lr = l & 31, lk = l >> 5;
#pragma unroll
    for (int k0 = 0; k0 < TS; k0 += 2) {
        float av, bv;
        if (colpush) {            // L^B[TI, I] (32x32) * E (32x32)
            av = Pw[w][lr][k0 + lk];
            bv = Et[k0 + lk][lr];
        } else {                  // F (32x32) * (L^A[TJ, J])^T
            av = Ft[lr][k0 + lk];
            bv = Pw[w][lr][k0 + lk];
        }
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc, 0, 0, 0);
    }
    float* out = colpush ? a.Y : a.X;
    const int64_t to = ws_tile_offset(TI, TJ, a.nt);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int rr = (r >> 2) * 8 + lk * 4 + (r & 3);
        out[to + rr * TS + lr] += acc[r];
    }
}

struct NodeArgs {
    int K, Mid, L;    // tile anti-diagonal range [K, L), split at Mid
    int knear;
    int mt, nt;
    int md_lo;        // first macro anti-diagonal of the grid
    float* X;
    float* Y;
    const float* LA;
    const float* LB;
    int b_ident;      // B = I: column pushes vanish
};

// Band push of one divide-and-conquer node on fp32 MFMA.
// Workgroup = 128x128 output macro tile (4x4 solver tiles), 4 waves of 64x64
// (2x2 blocks of v_mfma_f32_32x32x2f32).  blockIdx.z = 0: column push into Y;
// 1: row push into X.  The (source, target) validity masks are separable, so
// each K step stages zero tiles for invalid sources and the products of the
// remaining tiles are exact.
__global__ __launch_bounds__(256) void k_node(NodeArgs a) {
    __shared__ float As[MACRO * TS][TS + 1];
    __shared__ float Bs[TS][MACRO * TS + 1];
    const int mi = blockIdx.x;
    const int md = a.md_lo + (int)blockIdx.y;
    const int mj = md - mi;
    const int nmj = (a.nt + MACRO - 1) / MACRO;
    if (mj < 0 || mj >= nmj) return;
    const int I0 = mi * MACRO, J0 = mj * MACRO;
    if (I0 + J0 + 2 * (MACRO - 1) < a.Mid || I0 + J0 >= a.L) return;
    const bool colpush = blockIdx.z == 0;
    if (colpush && a.b_ident) return;
    int klo, khi;
    if (colpush) {
        klo = max(0, a.K - (J0 + MACRO - 1));
        khi = min(min(a.Mid - J0, I0 + MACRO - 1 - a.knear), a.mt);
    } else {
        klo = max(0, a.K - (I0 + MACRO - 1));
        khi = min(min(a.Mid - I0, J0 + MACRO - 1 - a.knear), a.nt);
    }
    if (klo >= khi) return;

    const int tid = threadIdx.x;
    const int wv = tid >> 6, l = tid & 63;
    const int wm = wv >> 1, wn = wv & 1;
    const int lr = l & 31, lk = l >> 5;
    f32x16 acc[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = f32x16{0};

    for (int kt = klo; kt < khi; ++kt) {
        // stage A (128 x 32) and B (32 x 128): tile t = 0..3 of each
#pragma unroll
        for (int t = 0; t < MACRO; ++t) {
            const int e0 = tid * 4;              // 256 threads x 4 = one tile
            const int r = e0 >> 5, cc = e0 & 31;
            // A operand
            const float* src = nullptr;
            if (colpush) {
                const int I = I0 + t;
                if (I < a.mt && kt <= I - a.knear - 1) src = a.LB + packed_tile_offset(I, kt);
            } else {
                const int I = I0 + t;
                if (I < a.mt && I + kt >= a.K && I + kt < a.Mid)
                    src = a.Y + ws_tile_offset(I, kt, a.nt);
            }
            f32x4 v = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            if (src) v = *reinterpret_cast<const f32x4*>(src + e0);
            As[t * TS + r][cc] = v[0];
            As[t * TS + r][cc + 1] = v[1];
            As[t * TS + r][cc + 2] = v[2];
            As[t * TS + r][cc + 3] = v[3];
            // B operand
            const float* bsrc = nullptr;
            if (colpush) {
                const int J = J0 + t;
                if (J < a.nt && kt + J >= a.K && kt + J < a.Mid)
                    bsrc = a.X + ws_tile_offset(kt, J, a.nt);
            } else {
                const int J = J0 + t;
                if (J < a.nt && kt <= J - a.knear - 1) bsrc = a.LA + packed_tile_offset(J, kt);
            }
            f32x4 u = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            if (bsrc) u = *reinterpret_cast<const f32x4*>(bsrc + e0);
            if (colpush) {       // E tile rows are the K index
                Bs[r][t * TS + cc] = u[0];
                Bs[r][t * TS + cc + 1] = u[1];
                Bs[r][t * TS + cc + 2] = u[2];
                Bs[r][t * TS + cc + 3] = u[3];
            } else {             // L^A tile (J, kt): element [jr][jc] -> Bs[jc][t*TS + jr]
                Bs[cc][t * TS + r] = u[0];
                Bs[cc + 1][t * TS + r] = u[1];
                Bs[cc + 2][t * TS + r] = u[2];
                Bs[cc + 3][t * TS + r] = u[3];
            }
        }
        __syncthreads();
#pragma unroll
        for (int k0 = 0; k0 < TS; k0 += 2) {
            float av[2], bv[2];
#pragma unroll
            for (int x = 0; x < 2; ++x) av[x] = As[wm * 64 + x * 32 + lr][k0 + lk];
#pragma unroll
            for (int y = 0; y < 2; ++y) bv[y] = Bs[k0 + lk][wn * 64 + y * 32 + lr];
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[x], bv[y], acc[x][y], 0, 0, 0);
        }
        __syncthreads();
    }

    float* out = colpush ? a.Y : a.X;
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const int I = I0 + wm * 2 + x, J = J0 + wn * 2 + y;
            if (I >= a.mt || J >= a.nt || I + J < a.Mid || I + J >= a.L) continue;
            const int64_t to = ws_tile_offset(I, J, a.nt);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rr = (r >> 2) * 8 + lk * 4 + (r & 3);
                out[to + rr * TS + lr] += acc[x][y][r];
            }
        }
}

// X <- W (tile-major, zero padding), Y <- 0.
__global__ void k_prep(const float* __restrict__ W, int64_t m, int64_t n, int mt, int nt,
                       float* __restrict__ X, float* __restrict__ Y) {
    const int64_t total = (int64_t)mt * nt * TILE_ELEMS;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t tile = e / TILE_ELEMS;
        const int w = (int)(e - tile * TILE_ELEMS);
        const int64_t I = tile / nt, J = tile - (tile / nt) * nt;
        const int64_t r = I * TS + w / TS, cc = J * TS + w % TS;
        X[e] = (r < m && cc < n) ? W[r * n + cc] : 0.0f;
        Y[e] = 0.0f;
    }
}

// ---------------------------------------------------------------------------
// host launchers

hipError_t launch_prep(hipStream_t s, const float* W, int64_t m, int64_t n, int mt, int nt,
                       float* X, float* Y) {
    int64_t total = (int64_t)mt * nt * TILE_ELEMS;
    int64_t g = (total + 255) / 256;
    if (g > 65535LL * 32) g = 65535LL * 32;
    hipLaunchKernelGGL(k_prep, dim3((unsigned)g), dim3(256), 0, s, W, m, n, mt, nt, X, Y);
    return hipGetLastError();
}

hipError_t launch_leaf(hipStream_t s, const LeafArgs& a, int ntiles) {
    hipLaunchKernelGGL(k_leaf, dim3((unsigned)ntiles), dim3(1024), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_node(hipStream_t s, const NodeArgs& a, int gx, int gy) {
    hipLaunchKernelGGL(k_node, dim3((unsigned)gx, (unsigned)gy, 2), dim3(256), 0, s, a);
    return hipGetLastError();
}

// Enqueue a whole solve.  evs (optional): 2 * (ops.size() + 1) events; a pair
// is recorded around the prep launch and around every schedule launch.
hipError_t run_schedule(hipStream_t s, const std::vector<SolveOp>& ops, const float* W, int64_t m,
                        int64_t n, int mt, int nt, float* X, float* Y, const float* LA,
                        const float* LB, int b_ident, const float* scale, float qmax,
                        int8_t* codes, float* V, float* pre, int knear, hipEvent_t* evs) {
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
    na.b_ident = b_ident;
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
            na.md_lo = op.md_lo;
            e = launch_node(s, na, op.gx, op.gy);
        }
        if (evs) hipEventRecord(evs[2 * i + 1], s);
        ++i;
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace bk
