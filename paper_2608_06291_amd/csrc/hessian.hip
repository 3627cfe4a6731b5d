// Kronecker-factor construction from calibration samples (Sec. 4 and App. A).
// Every factor the paper forms is a weighted Gram matrix of per-sample vectors,
// possibly multiplied entrywise by a fixed matrix:
//     C = s * (X^T diag(w) X) (.) M,    C_ij = s * M_ij * sum_k w_k X_ki X_kj,
// X the N x d matrix of samples (one row per sample):
//   K-FAC style (App. A):         A = E[a a^T], B = E[b b^T]                  (w = 1, M = 1)
//   single Shampoo step (App. A): A = E[|b|^2 a a^T], B = E[|a|^2 b b^T]      (w = squared norms)
//   MLP-local (App. A, b = D_g W_down^T): b b^T = (g g^T) (.) W_down^T W_down, so
//                                 B = E[g g^T] (.) D^T D with D^T D itself a Gram over the rows of
//                                 D = W_down, and tr(b^T b) = sum_i (D^T D)_ii g_i^2.
// k_sample_weights forms w_k = sum_i c_i X_ki^2 (c = 1: the squared norm).
// k_gram computes the upper-triangle 128 x 128 blocks of X^T diag(w) X on fp32
// MFMA, split over slices of the samples; k_gram_reduce adds the slices in a
// fixed order, applies s and M, writes the upper triangle and mirrors it.
#include <algorithm>
#include <cstdio>
#include <string>

#include "bakron.h"
#include "common.h"

namespace bk {

constexpr int GB = 128;        // Gram block edge
constexpr int GK = 32;         // samples per chunk
constexpr int GSTR = GK + 4;   // LDS row stride (floats) of a staged block

// ----------------------------------------------------------------------------
// w[k] = sum_i c[i] * X[k][i]^2 (c null: c = 1).  One wave per sample row.
template <bool VEC>
__global__ __launch_bounds__(256) void k_sample_weights(const float* __restrict__ X, int64_t N,
                                                        int64_t d, const float* __restrict__ c,
                                                        float* __restrict__ w) {
    const int64_t k = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int l = threadIdx.x & 63;
    if (k >= N) return;
    const float* row = X + k * d;
    float acc = 0.0f;
    if (VEC) {
        for (int64_t i = 4 * l; i < d; i += 256) {
            const f32x4 x = *reinterpret_cast<const f32x4*>(row + i);
            const f32x4 cc = c ? *reinterpret_cast<const f32x4*>(c + i) : f32x4{1.f, 1.f, 1.f, 1.f};
#pragma unroll
            for (int u = 0; u < 4; ++u) acc = fmaf(cc[u] * x[u], x[u], acc);
        }
    } else {
        for (int64_t i = l; i < d; i += 64) {
            const float x = row[i];
            acc = fmaf(c ? c[i] * x : x, x, acc);
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
    if (l == 0) w[k] = acc;
}

// dst[i] = src[i * (d + 1)]: the diagonal of a d x d matrix.
__global__ __launch_bounds__(256) void k_diag(const float* __restrict__ src, int64_t d,
                                              float* __restrict__ dst) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < d) dst[i] = src[i * (d + 1)];
}

// ----------------------------------------------------------------------------
// Upper-triangle block (bi, bj), bi <= bj, of X^T diag(w) X over the samples of
// one slice [k_lo, k_hi): part[slice][blk] (128 x 128, row-major).
// A chunk is 32 samples.  Thread t stages features 4 (t & 31) .. + 3 of both
// column ranges for samples 4 (t >> 5) .. + 3: four 16-byte row loads per
// operand, transposed in registers, written as four 16-byte LDS rows
// [feature][sample], so the MFMA operands below are contiguous along the
// sample index (lane half h takes sample 16h + s at step s of
// v_mfma_f32_32x32x2f32).  The first operand carries the weights.  4 waves,
// each 2 x 2 MFMA blocks of 32 x 32; LDS double-buffered, the next chunk in
// registers while the current one is multiplied.
struct GramArgs {
    const float* X;
    int64_t N, d;
    const float* w;
    int64_t slice_rows;   // samples per slice, a multiple of GK
    int nb, nblk;         // blocks per side, upper-triangle blocks
    int slices;
    float* part;          // [slices][nblk][GB * GB]
};

// Block t of a slice -> (bi, bj), bi <= bj.  The upper triangle is walked in
// 8 x 8 supertiles (row-major over supertiles, row-major inside each), so that
// consecutive blocks share few column ranges of X.
constexpr int GSUPER = 8;
__device__ inline void gram_block_of(int t, int nb, int& bi, int& bj) {
    const int nS = (nb + GSUPER - 1) / GSUPER;
    for (int SI = 0; SI < nS; ++SI) {
        const int r0 = SI * GSUPER, r1 = min(nb, r0 + GSUPER);
        for (int SJ = SI; SJ < nS; ++SJ) {
            const int c0 = SJ * GSUPER, c1 = min(nb, c0 + GSUPER);
            if (SI == SJ) {
                const int w = r1 - r0;
                if (t < w * (w + 1) / 2) {
                    int i = r0;
                    while (t >= r1 - i) {
                        t -= r1 - i;
                        ++i;
                    }
                    bi = i;
                    bj = i + t;
                    return;
                }
                t -= w * (w + 1) / 2;
            } else {
                const int cnt = (r1 - r0) * (c1 - c0);
                if (t < cnt) {
                    bi = r0 + t / (c1 - c0);
                    bj = c0 + t % (c1 - c0);
                    return;
                }
                t -= cnt;
            }
        }
    }
    bi = bj = 0;   // not reached for t < nb (nb + 1) / 2
}

// Work item of a k_gram workgroup.  Workgroups are dealt to the 8 XCDs in
// turn (workgroup v runs on XCD v mod 8), so XCD x is given the contiguous
// range x * per .. of the work list (slices in order, blocks of a slice in
// supertile order): the workgroups resident on one XCD then stream the same
// samples and few column ranges, which stay in that XCD's L2.
constexpr int GXCD = 8;
__device__ inline int gram_work_of(int v, int total) {
    const int per = (total + GXCD - 1) / GXCD;
    return (v % GXCD) * per + v / GXCD;
}

template <bool VEC>
__global__ __launch_bounds__(256, 2) void k_gram(GramArgs a) {
    __shared__ __attribute__((aligned(16))) float As[2][GB][GSTR];
    __shared__ __attribute__((aligned(16))) float Bs[2][GB][GSTR];
    const int wk = gram_work_of((int)blockIdx.x, a.nblk * a.slices);
    if (wk >= a.nblk * a.slices) return;   // padding of the last XCD's range
    const int slice = wk / a.nblk;
    const int blk = wk % a.nblk;
    int bi, bj;
    gram_block_of(blk, a.nb, bi, bj);
    const int64_t i0 = (int64_t)bi * GB, j0 = (int64_t)bj * GB;
    const int64_t k_lo = (int64_t)slice * a.slice_rows;
    const int64_t k_hi = min(a.N, k_lo + a.slice_rows);
    const int nch = k_hi > k_lo ? (int)((k_hi - k_lo + GK - 1) / GK) : 0;

    const int tid = threadIdx.x;
    const int wv = tid >> 6, l = tid & 63;
    const int wm = wv >> 1, wn = wv & 1;
    const int lr = l & 31, lk = l >> 5;
    const int f4 = 4 * (tid & 31), kq = 4 * (tid >> 5);
    const float* X = a.X;
    const int64_t d = a.d;
    // Loads are unconditional, from clamped (always valid) addresses, so that
    // they stay in flight across the MFMAs of the current chunk; the weights
    // and the masks of rows past the slice and columns past d are applied when
    // the registers are written to LDS.
    const bool a_in = i0 + f4 < d, b_in = j0 + f4 < d;
    const int64_t ia = a_in ? i0 + f4 : 0, ja = b_in ? j0 + f4 : 0;
    f32x4 ra[4], rb[4];
    float rw[4];
    int64_t kbase = 0;
    auto load = [&](int64_t k0) {
        kbase = k0;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t k = min(k0 + kq + r, k_hi - 1);
            const float* row = X + k * d;
            rw[r] = a.w ? a.w[k] : 1.0f;
            if (VEC) {
                ra[r] = *reinterpret_cast<const f32x4*>(row + ia);
                rb[r] = *reinterpret_cast<const f32x4*>(row + ja);
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    ra[r][u] = row[i0 + f4 + u < d ? i0 + f4 + u : 0];
                    rb[r][u] = row[j0 + f4 + u < d ? j0 + f4 + u : 0];
                }
            }
        }
    };
    auto store = [&](int sb) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const bool kin = kbase + kq + r < k_hi;
            const float wk = kin ? rw[r] : 0.0f;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool ca = VEC ? a_in : i0 + f4 + u < d;
                const bool cb = VEC ? b_in : j0 + f4 + u < d;
                ra[r][u] = ca ? ra[r][u] * wk : 0.0f;
                rb[r][u] = (cb && kin) ? rb[r][u] : 0.0f;
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            *reinterpret_cast<f32x4*>(&As[sb][f4 + u][kq]) = f32x4{ra[0][u], ra[1][u], ra[2][u], ra[3][u]};
            *reinterpret_cast<f32x4*>(&Bs[sb][f4 + u][kq]) = f32x4{rb[0][u], rb[1][u], rb[2][u], rb[3][u]};
        }
    };
    f32x16 acc[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = f32x16{0};
    if (nch > 0) {
        load(k_lo);
        store(0);
    }
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
        const int sb = c & 1;
        const bool more = c + 1 < nch;
        if (more) load(k_lo + (int64_t)(c + 1) * GK);
        f32x4 fa[2][4], fb[2][4];
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                fa[x][v] = *reinterpret_cast<const f32x4*>(&As[sb][(2 * wm + x) * TS + lr][lk * 16 + v * 4]);
                fb[x][v] = *reinterpret_cast<const f32x4*>(&Bs[sb][(2 * wn + x) * TS + lr][lk * 16 + v * 4]);
            }
#pragma unroll
        for (int st = 0; st < 16; ++st)
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[x][st >> 2][st & 3],
                                                                    fb[y][st >> 2][st & 3], acc[x][y],
                                                                    0, 0, 0);
        if (more) store(sb ^ 1);
        __syncthreads();
    }
    // acc[x][y][r] is entry (row (2wm + x) * 32 + (r >> 2) * 8 + lk * 4 + (r & 3),
    // column (2wn + y) * 32 + lr) of the block
    float* P = a.part + ((int64_t)slice * a.nblk + blk) * (GB * GB);
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = (2 * wm + x) * TS + (r >> 2) * 8 + lk * 4 + (r & 3);
                P[row * GB + (2 * wn + y) * TS + lr] = acc[x][y][r];
            }
}

// One 32 x 32 sub-tile of a block: sum the slices in order and scale; write
// the upper-triangle entries, C[i][j] = s * G_ij * M_ij (i <= j), and mirror
// them, C[j][i] = s * G_ij * M_ji (i < j), so that C is exactly symmetric when
// M is (the weighted products of a diagonal block are not bitwise symmetric).
// Sub-tiles below the diagonal of a diagonal block are skipped: their entries
// are the mirror of the sub-tile above.  Every entry of C is read (M) and
// written by one thread, so M may alias C.
__global__ __launch_bounds__(256) void k_gram_reduce(const float* __restrict__ part, int slices,
                                                     int nblk, int nb, int64_t d, float s,
                                                     const float* M, float* C) {
    __shared__ float T[TS][TS + 1];
    const int blk = (int)(blockIdx.x >> 4), sub = (int)(blockIdx.x & 15);
    int bi, bj;
    gram_block_of(blk, nb, bi, bj);
    const int sr = sub >> 2, sc = sub & 3;
    if (bi == bj && sr > sc) return;
    const bool diag = bi == bj && sr == sc;   // the sub-tile straddles the diagonal
    const int r = threadIdx.x >> 3, c4 = 4 * (threadIdx.x & 7);
    const int64_t bo = (int64_t)blk * (GB * GB) + (sr * TS + r) * GB + sc * TS + c4;
    f32x4 g = {0.f, 0.f, 0.f, 0.f};
    for (int sl = 0; sl < slices; ++sl)
        g += *reinterpret_cast<const f32x4*>(part + (int64_t)sl * nblk * (GB * GB) + bo);
    g *= s;
    const int64_t i = (int64_t)bi * GB + sr * TS + r;
    const int64_t jb = (int64_t)bj * GB + sc * TS + c4;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        if (i < d && jb + u < d && (!diag || r <= c4 + u)) {
            const int64_t o = i * d + jb + u;
            C[o] = M ? g[u] * M[o] : g[u];
        }
        T[r][c4 + u] = g[u];
    }
    __syncthreads();
    const int64_t il = (int64_t)bj * GB + sc * TS + r;   // mirrored row
    const int64_t jl = (int64_t)bi * GB + sr * TS + c4;  // mirrored columns
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        if (il < d && jl + u < d && (!diag || r > c4 + u)) {
            const int64_t o = il * d + jl + u;
            const float v = T[c4 + u][r];
            C[o] = M ? v * M[o] : v;
        }
    }
}

// ----------------------------------------------------------------------------
// Launch geometry of one Gram product.  The blocks of one slice are
// consecutive workgroups (they stream the same samples, which stay in L2);
// the slice count balances nblk * slices blocks over the 2 * ncu workgroup
// slots (two workgroups fit one CU), charging each slice its partial-sum
// traffic.
struct GramGeom {
    int nb, nblk, slices;
    int64_t slice_rows;
};

static GramGeom gram_geom(int64_t N, int64_t d, int ncu) {
    GramGeom g;
    g.nb = (int)((d + GB - 1) / GB);
    g.nblk = g.nb * (g.nb + 1) / 2;
    const int64_t nch = std::max<int64_t>(1, (N + GK - 1) / GK);
    const int64_t slots = 2 * (int64_t)std::max(ncu, 1);
    int best = 1;
    double best_t = 0.0;
    for (int S = 1; S <= 64 && S <= nch; ++S) {
        const int64_t per = (nch + S - 1) / S;
        const int64_t S_eff = (nch + per - 1) / per;
        // in chunk-times of one workgroup (2 * 128 * 128 * 32 flops at half a
        // CU's MFMA rate, about 3.4 us): the waves of blocks, plus writing and
        // reading back every 64 KiB partial at about 5 TB/s (0.0077 each)
        const double t = (double)((g.nblk * S_eff + slots - 1) / slots) * (double)per +
                         0.0077 * (double)(g.nblk * S_eff);
        if (S == 1 || t < best_t - 1e-9) {
            best_t = t;
            best = (int)S_eff;
        }
    }
    const int64_t per = (nch + best - 1) / best;
    g.slice_rows = per * GK;
    g.slices = (int)((nch + per - 1) / per);
    return g;
}

static size_t gram_part_bytes(const GramGeom& g) {
    return (size_t)g.slices * g.nblk * GB * GB * sizeof(float);
}

static hipError_t run_sample_weights(hipStream_t st, const float* X, int64_t N, int64_t d,
                                     const float* c, float* w) {
    if (N == 0) return hipSuccess;
    const bool vec = d % 4 == 0 && ((uintptr_t)X & 15) == 0 && (!c || ((uintptr_t)c & 15) == 0);
    const dim3 grid((unsigned)((N + 3) / 4));
    if (vec)
        hipLaunchKernelGGL(k_sample_weights<true>, grid, dim3(256), 0, st, X, N, d, c, w);
    else
        hipLaunchKernelGGL(k_sample_weights<false>, grid, dim3(256), 0, st, X, N, d, c, w);
    return hipGetLastError();
}

static hipError_t run_gram(hipStream_t st, const GramGeom& g, const float* X, int64_t N, int64_t d,
                           const float* w, float s, const float* M, float* C, float* part) {
    if (d == 0) return hipSuccess;
    GramArgs a{X, N, d, w, g.slice_rows, g.nb, g.nblk, g.slices, part};
    const bool vec = d % 4 == 0 && ((uintptr_t)X & 15) == 0;
    const int64_t total = (int64_t)g.nblk * g.slices;
    const dim3 grid((unsigned)(((total + GXCD - 1) / GXCD) * GXCD));
    if (vec)
        hipLaunchKernelGGL(k_gram<true>, grid, dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL(k_gram<false>, grid, dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_gram_reduce, dim3((unsigned)(g.nblk * 16)), dim3(256), 0, st, part,
                       g.slices, g.nblk, g.nb, d, s, M, C);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Per-sample quadratic forms w_k = x_k^T M x_k (M symmetric d x d): the
// weights tr(b^T B b) of the later Shampoo power steps (App. A).  Workgroup
// (row block R, column block J) computes the 128 x 128 tile of Y = X M
// (Y_kj = sum_t X_kt M_jt, M symmetric) on fp32 MFMA, then
// part[J][k] = sum_{j in J} Y_kj X_kj.  Both operands are rows with the
// inner index contiguous, staged as 16-byte copies (thread t: row t >> 1,
// inner quarter-chunk 16 (t & 1)).  k_quadform_reduce adds the column blocks
// in order.
struct QuadArgs {
    const float* X;
    int64_t N, d;
    const float* M;
    int nJ;
    float* part;   // [nJ][N]
};

template <bool VEC>
__global__ __launch_bounds__(256, 2) void k_quadform(QuadArgs a) {
    __shared__ __attribute__((aligned(16))) float As[2][GB][GSTR];
    __shared__ __attribute__((aligned(16))) float Bs[2][GB][GSTR];
    __shared__ float red[2][GB];
    const int J = (int)(blockIdx.x % (unsigned)a.nJ);
    const int64_t R = blockIdx.x / (unsigned)a.nJ;
    const int64_t k0 = R * GB, j0 = (int64_t)J * GB;
    const int64_t d = a.d;
    const int tid = threadIdx.x;
    const int wv = tid >> 6, l = tid & 63;
    const int wm = wv >> 1, wn = wv & 1;
    const int lr = l & 31, lk = l >> 5;
    const int srow = tid >> 1, sq = 16 * (tid & 1);
    const bool arow_in = k0 + srow < a.N, brow_in = j0 + srow < d;
    const float* xa = a.X + (arow_in ? k0 + srow : 0) * d;
    const float* mb = a.M + (brow_in ? j0 + srow : 0) * d;
    f32x4 ra[4], rb[4];
    int64_t tbase = 0;
    auto load = [&](int64_t t0) {
        tbase = t0;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int64_t t = t0 + sq + 4 * v;
            if (VEC) {
                const int64_t tc = t < d ? t : 0;   // d % 4 == 0: a whole chunk is in or out
                ra[v] = *reinterpret_cast<const f32x4*>(xa + tc);
                rb[v] = *reinterpret_cast<const f32x4*>(mb + tc);
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int64_t tc = t + u < d ? t + u : 0;
                    ra[v][u] = xa[tc];
                    rb[v][u] = mb[tc];
                }
            }
        }
    };
    auto store = [&](int sb) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool tin = tbase + sq + 4 * v + u < d;
                ra[v][u] = (tin && arow_in) ? ra[v][u] : 0.0f;
                rb[v][u] = (tin && brow_in) ? rb[v][u] : 0.0f;
            }
            *reinterpret_cast<f32x4*>(&As[sb][srow][sq + 4 * v]) = ra[v];
            *reinterpret_cast<f32x4*>(&Bs[sb][srow][sq + 4 * v]) = rb[v];
        }
    };
    f32x16 acc[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = f32x16{0};
    const int nch = (int)((d + GK - 1) / GK);
    load(0);
    store(0);
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
        const int sb = c & 1;
        const bool more = c + 1 < nch;
        if (more) load((int64_t)(c + 1) * GK);
        f32x4 fa[2][4], fb[2][4];
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                fa[x][v] = *reinterpret_cast<const f32x4*>(&As[sb][(2 * wm + x) * TS + lr][lk * 16 + v * 4]);
                fb[x][v] = *reinterpret_cast<const f32x4*>(&Bs[sb][(2 * wn + x) * TS + lr][lk * 16 + v * 4]);
            }
#pragma unroll
        for (int st = 0; st < 16; ++st)
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[x][st >> 2][st & 3],
                                                                    fb[y][st >> 2][st & 3], acc[x][y],
                                                                    0, 0, 0);
        if (more) store(sb ^ 1);
        __syncthreads();
    }
    // acc[x][y][r] = Y(row (2wm + x) * 32 + (r >> 2) * 8 + lk * 4 + (r & 3),
    //                  column (2wn + y) * 32 + lr); row sums of Y (.) X over the
    // wave's 64 columns, then over the lanes of a row, then over the two waves
    // that share the rows (wn = 0, 1)
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = (2 * wm + x) * TS + (r >> 2) * 8 + lk * 4 + (r & 3);
            const int64_t k = k0 + row;
            float v = 0.0f;
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int64_t j = j0 + (2 * wn + y) * TS + lr;
                const float xv = (k < a.N && j < d) ? a.X[k * d + j] : 0.0f;
                v = fmaf(acc[x][y][r], xv, v);
            }
#pragma unroll
            for (int off = 16; off >= 1; off >>= 1) v += __shfl_xor(v, off, 32);
            if (lr == 0) red[wn][row] = v;
        }
    __syncthreads();
    if (tid < GB && k0 + tid < a.N) a.part[(int64_t)J * a.N + k0 + tid] = red[0][tid] + red[1][tid];
}

__global__ __launch_bounds__(256) void k_quadform_reduce(const float* __restrict__ part, int nJ,
                                                         int64_t N, float* __restrict__ w) {
    const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (k >= N) return;
    float s = 0.0f;
    for (int J = 0; J < nJ; ++J) s += part[(int64_t)J * N + k];
    w[k] = s;
}

// C = A (.) B entrywise (n elements); C may alias A or B.
__global__ __launch_bounds__(256) void k_hadamard(const float* A, const float* B, int64_t n,
                                                  float* C) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e < n) C[e] = A[e] * B[e];
}

static size_t quadform_part_bytes(int64_t N, int64_t d) {
    return (size_t)((d + GB - 1) / GB) * (size_t)std::max<int64_t>(N, 1) * sizeof(float);
}

static hipError_t run_quadform(hipStream_t st, const float* X, int64_t N, int64_t d, const float* M,
                               float* w, float* part) {
    if (N == 0) return hipSuccess;
    const int nJ = (int)std::max<int64_t>(1, (d + GB - 1) / GB);
    QuadArgs a{X, N, d, M, nJ, part};
    const bool vec = d % 4 == 0 && ((uintptr_t)X & 15) == 0 && ((uintptr_t)M & 15) == 0;
    const dim3 grid((unsigned)(((N + GB - 1) / GB) * nJ));
    if (vec)
        hipLaunchKernelGGL(k_quadform<true>, grid, dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL(k_quadform<false>, grid, dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_quadform_reduce, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, st, part,
                       nJ, N, w);
    return hipGetLastError();
}

static int device_cus() {
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return ncu;
}

}  // namespace bk

// ============================================================================
// C ABI (declared in bakron.h)

using bk::GramGeom;

static bakron_status hess_fail(const char* msg) {
    bk::set_last_error(msg);
    return BAKRON_EINVAL;
}

static bakron_status hess_hip(hipError_t e, const char* what) {
    char buf[256];
    std::snprintf(buf, sizeof(buf), "%s: %s", what, hipGetErrorString(e));
    bk::set_last_error(buf);
    return e == hipErrorOutOfMemory ? BAKRON_ENOMEM : BAKRON_EHIP;
}

static inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// Dimension limits: blocks per side fit the launch grid comfortably.
static const int64_t HESS_DIM_MAX = (int64_t)1 << 17;
static const int64_t HESS_N_MAX = (int64_t)1 << 40;

// Workspace handshake shared by the factor-construction calls: with work ==
// NULL report the size; otherwise check it.
static bakron_status workspace_check(void* work, size_t* work_bytes, size_t need, bool* query) {
    *query = false;
    if (!work_bytes) return hess_fail("work_bytes is NULL");
    if (!work) {
        *work_bytes = need;
        *query = true;
        return BAKRON_OK;
    }
    if (*work_bytes < need) return hess_fail("workspace too small");
    if (((uintptr_t)work & 255) != 0) return hess_fail("workspace not 256-byte aligned");
    return BAKRON_OK;
}

extern "C" bakron_status bakron_sample_weights(const float* X, int64_t N, int64_t d, const float* c,
                                               float* w, hipStream_t stream) {
    bk::set_last_error("");
    if (N < 0 || d < 0 || N > HESS_N_MAX || d > HESS_DIM_MAX) return hess_fail("bad size");
    if (N > 0 && (!w || (d > 0 && !X))) return hess_fail("null pointer");
    hipError_t e = bk::run_sample_weights(stream, X, N, d, c, w);
    return e == hipSuccess ? BAKRON_OK : hess_hip(e, "bakron_sample_weights: launch");
}

extern "C" bakron_status bakron_gram(const float* X, int64_t N, int64_t d, const float* w, float s,
                                     const float* M, float* C, void* work, size_t* work_bytes,
                                     hipStream_t stream) {
    bk::set_last_error("");
    if (N < 0 || d < 0 || N > HESS_N_MAX || d > HESS_DIM_MAX) return hess_fail("bad size");
    const GramGeom g = bk::gram_geom(N, d, bk::device_cus());
    bool query;
    bakron_status st = workspace_check(work, work_bytes, bk::gram_part_bytes(g), &query);
    if (st != BAKRON_OK || query) return st;
    if (d > 0 && (!C || (N > 0 && !X))) return hess_fail("null pointer");
    hipError_t e = bk::run_gram(stream, g, X, N, d, w, s, M, C, static_cast<float*>(work));
    return e == hipSuccess ? BAKRON_OK : hess_hip(e, "bakron_gram: launch");
}

// Carves the workspace: [partials | weights x2 | extra], 256-byte aligned.
struct HessWork {
    float* part;
    float* w0;
    float* w1;
    float* extra;
};
static HessWork carve(void* work, size_t part, size_t wbytes) {
    char* p = static_cast<char*>(work);
    HessWork h;
    h.part = reinterpret_cast<float*>(p);
    h.w0 = reinterpret_cast<float*>(p + align256(part));
    h.w1 = reinterpret_cast<float*>(p + align256(part) + wbytes);
    h.extra = reinterpret_cast<float*>(p + align256(part) + 2 * wbytes);
    return h;
}

// Global (vector) case, App. A: K-FAC, or `iters` unnormalised power steps
// from (I, I).  Step 1 weighs by |b_k|^2 and |a_k|^2; step i > 1 by
// b_k^T B^(i-1) b_k and a_k^T A^(i-1) a_k, after which A and B are
// overwritten in place (the previous pair is no longer needed).
static bakron_status kron_factors_impl(const char* who, const float* a, const float* b, int64_t N,
                                       int64_t n, int64_t m, bool shampoo, int iters, float* A,
                                       float* B, void* work, size_t* work_bytes,
                                       hipStream_t stream) {
    if (N <= 0 || n <= 0 || m <= 0 || N > HESS_N_MAX || n > HESS_DIM_MAX || m > HESS_DIM_MAX ||
        iters < 1 || iters > 64)
        return hess_fail("bad size or iteration count");
    if (iters > 1 && ((N + bk::GB - 1) / bk::GB) * ((std::max(n, m) + bk::GB - 1) / bk::GB) >
                         ((int64_t)1 << 31) - 1)
        return hess_fail("too many samples for the power steps");
    const int ncu = bk::device_cus();
    const GramGeom ga = bk::gram_geom(N, n, ncu), gb = bk::gram_geom(N, m, ncu);
    size_t part = std::max(bk::gram_part_bytes(ga), bk::gram_part_bytes(gb));
    if (iters > 1)
        part = std::max({part, bk::quadform_part_bytes(N, n), bk::quadform_part_bytes(N, m)});
    const size_t wbytes = shampoo ? align256((size_t)N * sizeof(float)) : 0;
    bool query;
    bakron_status st = workspace_check(work, work_bytes, align256(part) + 2 * wbytes, &query);
    if (st != BAKRON_OK || query) return st;
    if (!a || !b || !A || !B) return hess_fail("null pointer");
    const HessWork h = carve(work, part, wbytes);
    const float inv = (float)(1.0 / (double)N);
    float* wa = shampoo ? h.w0 : nullptr;   // weights of B (from a)
    float* wb = shampoo ? h.w1 : nullptr;   // weights of A (from b)
    hipError_t e = hipSuccess;
    for (int it = 1; it <= (shampoo ? iters : 1); ++it) {
        if (shampoo && it == 1) {
            if ((e = bk::run_sample_weights(stream, a, N, n, nullptr, wa)) != hipSuccess ||
                (e = bk::run_sample_weights(stream, b, N, m, nullptr, wb)) != hipSuccess)
                return hess_hip(e, who);
        } else if (shampoo) {
            if ((e = bk::run_quadform(stream, a, N, n, A, wa, h.part)) != hipSuccess ||
                (e = bk::run_quadform(stream, b, N, m, B, wb, h.part)) != hipSuccess)
                return hess_hip(e, who);
        }
        if ((e = bk::run_gram(stream, ga, a, N, n, wb, inv, nullptr, A, h.part)) != hipSuccess ||
            (e = bk::run_gram(stream, gb, b, N, m, wa, inv, nullptr, B, h.part)) != hipSuccess)
            return hess_hip(e, who);
    }
    return BAKRON_OK;
}

// MLP-local case, App. A, b = D_g W_down^T: b b^T = (g g^T) (.) D^T D and
// tr(b^T X b) = g^T (X (.) D^T D) g.  Step 1 of Shampoo weighs A by
// g^T diag(D^T D) g and B by |x|^2; step i > 1 by g^T (B^(i-1) (.) D^T D) g
// and x^T A^(i-1) x.
static bakron_status mlp_local_impl(const char* who, const float* x, const float* g,
                                    const float* D, int64_t N, int64_t dm, int64_t dff,
                                    bool shampoo, int iters, float* A, float* B, void* work,
                                    size_t* work_bytes, hipStream_t stream) {
    if (N <= 0 || dm <= 0 || dff <= 0 || N > HESS_N_MAX || dm > HESS_DIM_MAX || dff > HESS_DIM_MAX ||
        iters < 1 || iters > 64)
        return hess_fail("bad size or iteration count");
    if (iters > 1 && ((N + bk::GB - 1) / bk::GB) * ((std::max(dm, dff) + bk::GB - 1) / bk::GB) >
                         ((int64_t)1 << 31) - 1)
        return hess_fail("too many samples for the power steps");
    const bool multi = shampoo && iters > 1;
    const int ncu = bk::device_cus();
    const GramGeom gx = bk::gram_geom(N, dm, ncu), gg = bk::gram_geom(N, dff, ncu),
                   gd = bk::gram_geom(dm, dff, ncu);
    size_t part = std::max({bk::gram_part_bytes(gx), bk::gram_part_bytes(gg),
                            bk::gram_part_bytes(gd)});
    if (multi)
        part = std::max({part, bk::quadform_part_bytes(N, dm), bk::quadform_part_bytes(N, dff)});
    const size_t wbytes = shampoo ? align256((size_t)N * sizeof(float)) : 0;
    // extra: the diagonal of D^T D (step 1), and D^T D itself kept apart from B
    // for the later steps
    const size_t cbytes = shampoo ? align256((size_t)dff * sizeof(float)) : 0;
    const size_t dbytes = multi ? (size_t)dff * (size_t)dff * sizeof(float) : 0;
    bool query;
    bakron_status st =
        workspace_check(work, work_bytes, align256(part) + 2 * wbytes + cbytes + dbytes, &query);
    if (st != BAKRON_OK || query) return st;
    if (!x || !g || !D || !A || !B) return hess_fail("null pointer");
    const HessWork h = carve(work, part, wbytes);
    const float inv = (float)(1.0 / (double)N);
    float* wx = shampoo ? h.w0 : nullptr;   // weights of B (from x)
    float* wg = shampoo ? h.w1 : nullptr;   // weights of A (from g)
    float* cdiag = h.extra;
    float* DtD = multi ? reinterpret_cast<float*>(reinterpret_cast<char*>(h.extra) + cbytes) : B;
    hipError_t e;
    // D^T D (rows of D = W_down as samples)
    if ((e = bk::run_gram(stream, gd, D, dm, dff, nullptr, 1.0f, nullptr, DtD, h.part)) != hipSuccess)
        return hess_hip(e, who);
    const int64_t nn = dff * dff;
    for (int it = 1; it <= (shampoo ? iters : 1); ++it) {
        if (shampoo && it == 1) {
            hipLaunchKernelGGL(bk::k_diag, dim3((unsigned)((dff + 255) / 256)), dim3(256), 0, stream,
                               DtD, dff, cdiag);
            if ((e = hipGetLastError()) != hipSuccess ||
                (e = bk::run_sample_weights(stream, g, N, dff, cdiag, wg)) != hipSuccess ||
                (e = bk::run_sample_weights(stream, x, N, dm, nullptr, wx)) != hipSuccess)
                return hess_hip(e, who);
        } else if (shampoo) {
            // B <- B^(i-1) (.) D^T D, the matrix of g's quadratic form
            hipLaunchKernelGGL(bk::k_hadamard, dim3((unsigned)((nn + 255) / 256)), dim3(256), 0, stream,
                               B, DtD, nn, B);
            if ((e = hipGetLastError()) != hipSuccess ||
                (e = bk::run_quadform(stream, g, N, dff, B, wg, h.part)) != hipSuccess ||
                (e = bk::run_quadform(stream, x, N, dm, A, wx, h.part)) != hipSuccess)
                return hess_hip(e, who);
        }
        // A = E[w_g x x^T]; B = E[w_x g g^T] (.) D^T D (in place over D^T D in
        // the one-step case)
        if ((e = bk::run_gram(stream, gx, x, N, dm, wg, inv, nullptr, A, h.part)) != hipSuccess ||
            (e = bk::run_gram(stream, gg, g, N, dff, wx, inv, DtD, B, h.part)) != hipSuccess)
            return hess_hip(e, who);
    }
    return BAKRON_OK;
}

extern "C" bakron_status bakron_kron_factors(const float* a, const float* b, int64_t N, int64_t n,
                                             int64_t m, int32_t style, float* A, float* B,
                                             void* work, size_t* work_bytes, hipStream_t stream) {
    bk::set_last_error("");
    if (style != BAKRON_KFAC && style != BAKRON_SHAMPOO) return hess_fail("bad style");
    return kron_factors_impl("bakron_kron_factors", a, b, N, n, m, style == BAKRON_SHAMPOO, 1, A, B,
                             work, work_bytes, stream);
}

extern "C" bakron_status bakron_kron_factors_iter(const float* a, const float* b, int64_t N,
                                                  int64_t n, int64_t m, int32_t iters, float* A,
                                                  float* B, void* work, size_t* work_bytes,
                                                  hipStream_t stream) {
    bk::set_last_error("");
    return kron_factors_impl("bakron_kron_factors_iter", a, b, N, n, m, true, iters, A, B, work,
                             work_bytes, stream);
}

extern "C" bakron_status bakron_mlp_local_factors(const float* x, const float* g, const float* D,
                                                  int64_t N, int64_t dm, int64_t dff, int32_t style,
                                                  float* A, float* B, void* work, size_t* work_bytes,
                                                  hipStream_t stream) {
    bk::set_last_error("");
    if (style != BAKRON_KFAC && style != BAKRON_SHAMPOO) return hess_fail("bad style");
    return mlp_local_impl("bakron_mlp_local_factors", x, g, D, N, dm, dff, style == BAKRON_SHAMPOO, 1,
                          A, B, work, work_bytes, stream);
}

extern "C" bakron_status bakron_mlp_local_factors_iter(const float* x, const float* g,
                                                       const float* D, int64_t N, int64_t dm,
                                                       int64_t dff, int32_t iters, float* A,
                                                       float* B, void* work, size_t* work_bytes,
                                                       hipStream_t stream) {
    bk::set_last_error("");
    return mlp_local_impl("bakron_mlp_local_factors_iter", x, g, D, N, dm, dff, true, iters, A, B,
                          work, work_bytes, stream);
}

extern "C" bakron_status bakron_quadform_weights(const float* X, int64_t N, int64_t d,
                                                 const float* M, float* w, void* work,
                                                 size_t* work_bytes, hipStream_t stream) {
    bk::set_last_error("");
    if (N < 0 || d < 0 || N > HESS_N_MAX || d > HESS_DIM_MAX ||
        ((N + bk::GB - 1) / bk::GB) * ((d + bk::GB - 1) / bk::GB) > ((int64_t)1 << 31) - 1)
        return hess_fail("bad size");
    bool query;
    bakron_status st = workspace_check(work, work_bytes, bk::quadform_part_bytes(N, d), &query);
    if (st != BAKRON_OK || query) return st;
    if (N > 0 && (!w || (d > 0 && (!X || !M)))) return hess_fail("null pointer");
    if (d == 0) {   // empty forms: w = 0 (the weight kernel with no features)
        hipError_t e = bk::run_sample_weights(stream, X, N, 0, nullptr, w);
        return e == hipSuccess ? BAKRON_OK : hess_hip(e, "bakron_quadform_weights");
    }
    hipError_t e = bk::run_quadform(stream, X, N, d, M, w, static_cast<float*>(work));
    return e == hipSuccess ? BAKRON_OK : hess_hip(e, "bakron_quadform_weights: launch");
}
