// Factor kernels: damping and the normalised error-feedback factor of one
// Kronecker factor X (n x n), computed in fp64 on the device.
//
//   X_d = X + damp * mean(diag X) * I                  (Sec. 4 opening; App. D)
//   R   = RevCholesky(X_d): lower, positive diagonal, R^T R = X_d   (Sec. 3.1)
//   L   = R^-1 diag(R): unit lower, equal to Cholesky(X_d^-1) with each column
//         divided by its diagonal entry (Alg. 1 / Alg. 2, first two lines).
//
// RevCholesky is obtained from an ordinary Cholesky of the index-reversed
// matrix: with P the reversal permutation, P X_d P = C C^T and R = P C^T P.
// Hence R^-1 = P C^-T P and L[i][j] = Cinv[n-1-j][n-1-i] * C[n-1-j][n-1-j].
//
// Blocked right-looking Cholesky (block NB) and a recursive triangular
// inverse, both driven by one fp64 GEMM on the matrix cores.  The result is rounded once to
// fp32 and stored as packed lower-triangular TS x TS tiles for the solver.
#include "common.h"

#include <functional>

namespace bk {

// One enqueue step of a factorisation: a few launches (or event records and
// waits) in stream order.
using FactorOp = std::function<hipError_t()>;

constexpr int NB = 64;  // factor block
constexpr int NB2 = 512;  // Cholesky panel (multiple of NB)

// ---------------------------------------------------------------------------
__global__ void k_diag_mean(const float* __restrict__ X, int64_t d, double* __restrict__ mean) {
    __shared__ double part[256];
    double s = 0.0;
    for (int64_t i = threadIdx.x; i < d; i += blockDim.x) s += (double)X[i * d + i];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *mean = part[0] / (double)d;
}

// Z[i][j] = X_d[d-1-i][d-1-j] (index-reversed, damped, fp64)
__global__ void k_flip_damp(const float* __restrict__ X, int64_t d, const double* __restrict__ mean,
                            double lam, double* __restrict__ Z) {
    const int64_t total = d * d;
    const double shift = lam * (*mean);
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = idx / d, j = idx - (idx / d) * d;
        double v = (double)X[(d - 1 - i) * d + (d - 1 - j)];
        if (i == j) v += shift;
        Z[idx] = v;
    }
}

// Unblocked Cholesky of the diagonal block Z[k0:k0+b, k0:k0+b] (lower part
// only), one wave: lane i holds row i of the block in registers; column j is
// finished by lane j's pivot (read by every lane through LDS), scaled in each
// lane, published to LDS and used by every later row for its trailing
// update.  The update runs over every column right of j in every lane, with
// the multiplier zeroed in lanes above the diagonal (i < j): entries right of
// a lane's diagonal then hold bounded values that are never read or stored,
// and no instruction is predicated per entry.  LDS operations of one wave
// complete in order, so no barrier is needed.  A non-positive or non-finite pivot sets *fail and records the
// pivot index in the reversed ordering.
__global__ __launch_bounds__(NB) void k_potrf_diag(double* __restrict__ Z, int64_t ld, int64_t k0,
                                                   int b, int* __restrict__ fail,
                                                   int64_t* __restrict__ fail_pivot) {
    if (*fail) return;
    __shared__ double col[NB];
    const int i = threadIdx.x;
    double row[NB];
#pragma unroll
    for (int c = 0; c < NB; ++c) row[c] = (i < b && c <= i && c < b) ? Z[(k0 + i) * ld + (k0 + c)] : 0.0;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        if (j >= b) continue;                                // uniform (last, partial block)
        if (i == j) col[j] = row[j];
        __builtin_amdgcn_wave_barrier();
        const double piv = col[j];
        if (!(piv > 0.0) || !isfinite(piv)) {                 // uniform: one value for all lanes
            if (i == 0) {
                *fail = 1;
                *fail_pivot = k0 + j;
            }
            return;
        }
        const double dj = sqrt(piv);
        if (i == j) row[j] = dj;
        else if (i > j) row[j] /= dj;
        __builtin_amdgcn_wave_barrier();
        col[i] = row[j];                                     // column j of the factor (rows > j)
        __builtin_amdgcn_wave_barrier();
        const double mj = (j <= i) ? row[j] : 0.0;
#pragma unroll
        for (int c = j + 1; c < NB; ++c) row[c] = fma(-mj, col[c], row[c]);
        __builtin_amdgcn_wave_barrier();
    }
    if (i < b) {
#pragma unroll
        for (int c = 0; c < NB; ++c)
            if (c <= i && c < b) Z[(k0 + i) * ld + (k0 + c)] = row[c];
    }
}

// Panel of the blocked Cholesky: every row r >= k0 + b of Z[:, k0:k0+b] is
// replaced by the solution x of x C_kk^T = Z[r, k0:k0+b] (C_kk the factored
// diagonal block, lower): x_j = (p_j - sum_{c<j} x_c C_jc) / C_jj, one thread
// per row, x in registers; each sum is split over four accumulators to
// shorten the dependent FMA chain.  C_kk is read through the scalar cache
// (its addresses are the same in every lane; Zd aliases Z, but the block's
// rows are never written here) and the reciprocals of its diagonal from LDS:
// 16% faster than broadcasting C_kk from LDS, with the same bits.
__global__ __launch_bounds__(256) void k_trsm_panel(double* __restrict__ Z,
                                                    const double* __restrict__ Zd, int64_t ld,
                                                    int64_t k0, int b, int64_t rows,
                                                    const int* __restrict__ fail) {
    if (*fail) return;
    __shared__ double rdiag[NB];
    if (threadIdx.x < NB)
        rdiag[threadIdx.x] = (int)threadIdx.x < b ? 1.0 / Zd[(k0 + threadIdx.x) * ld + (k0 + threadIdx.x)] : 0.0;
    __syncthreads();
    const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (r >= rows) return;
    const double* Ck = Zd + k0 * ld + k0;   // the factored diagonal block
    double* p = Z + (k0 + b + r) * ld + k0;
    double x[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        if (j < b) {   // uniform
            double a[4] = {p[j], 0.0, 0.0, 0.0};
#pragma unroll
            for (int c = 0; c < j; ++c) a[c & 3] = fma(-x[c], Ck[j * ld + c], a[c & 3]);
            x[j] = ((a[0] + a[1]) + (a[2] + a[3])) * rdiag[j];
        } else {
            x[j] = 0.0;
        }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j)
        if (j < b) p[j] = x[j];
}

// Inverse of lower-triangular diagonal blocks of C (size nbk <= NB each):
// block g covers rows/cols [k0 + g*NB, min(d, k0 + g*NB + NB)) of C and is
// written at rows/cols dst_off + g*NB of N (lower part only).  Thread j
// computes column j by forward substitution.
__global__ __launch_bounds__(NB) void k_inv_lower_blocks(const double* __restrict__ C, int64_t ldc,
                                                         double* __restrict__ N, int64_t ldn,
                                                         int64_t k0, int64_t d, int64_t dst_off,
                                                         const int* __restrict__ fail) {
    if (*fail) return;
    __shared__ double S[NB][NB + 1];
    __shared__ double Xs[NB][NB + 1];
    const int64_t base = k0 + (int64_t)blockIdx.x * NB;
    const int64_t dbase = dst_off + (int64_t)blockIdx.x * NB;
    const int b = (int)((d - base) < NB ? (d - base) : NB);
    const int t = threadIdx.x;
    for (int i = 0; i < b; ++i)
        if (t <= i) S[i][t] = C[(base + i) * ldc + (base + t)];
    __syncthreads();
    if (t < b) {
        const int j = t;
        for (int i = 0; i < b; ++i) {
            double v;
            if (i < j) v = 0.0;
            else if (i == j) v = 1.0 / S[i][i];
            else {
                double acc = 0.0;
                for (int k = j; k < i; ++k) acc += S[i][k] * Xs[k][j];
                v = -acc / S[i][i];
            }
            Xs[i][j] = v;
        }
        for (int i = j; i < b; ++i) N[(dbase + i) * ldn + (dbase + j)] = Xs[i][j];
    }
}

// C[M x N] = alpha * A[M x K] * op(B) + beta * C, row-major fp64, on fp64
// MFMA (v_mfma_f64_16x16x4f64: lane l supplies A[l % 16][l / 16] and
// B[l / 16][l % 16] of a k-step; register r of lane l holds
// D[l / 16 + 4 r][l % 16]).
// op(B) = B (K x N, ldb) or B^T (B is N x K, ldb).  lower_only skips the
// 64 x 64 blocks of C lying entirely above the diagonal (block column index >
// block row index): they are neither computed nor written.
// tri: bit 0 = A is lower triangular (A[i][k] = 0 for k > i), bit 1 = op(B)
// is lower triangular (op(B)[k][j] = 0 for k < j); the K loop of a block then
// skips the chunks that only meet those zeros.
// One workgroup per GT x GT block of C (GT = 64 or 128): GT / 16 waves, wave
// (wm, wn) computing rows 32 wm .. 32 wm + 31 and GT / 2 columns from
// wn * GT / 2 as 2 x (GT / 32) MFMA blocks.  K in chunks of 16 staged through
// double-buffered LDS as [k][row] / [k][col], the next chunk loaded into
// registers while the current one is multiplied.  The 128 x 128 block stages
// half as many bytes per flop.  Every entry of C sees the same MFMA sequence
// over the same K chunks in both block sizes, except that under `tri` a
// larger block may visit extra chunks whose products are exact zeros; those
// can only change the sign of an entry that is exactly zero, so zeros are
// stored as +0 and both block sizes give the same bits.
typedef double f64x4 __attribute__((ext_vector_type(4)));
constexpr int GK = 16;
template <int GT>
__global__ __launch_bounds__(4 * GT) void k_gemm(int64_t M, int64_t N, int64_t K, double alpha,
                                                 const double* __restrict__ A, int64_t lda,
                                                 const double* __restrict__ B, int64_t ldb,
                                                 int transB, double beta, double* __restrict__ C,
                                                 int64_t ldc, int lower_only, int tri,
                                                 const int* __restrict__ fail) {
    constexpr int PAD = GT + 2, YB = GT / 32;
    if (*fail) return;
    // block order: under tri the heaviest K ranges first, so that the longest
    // blocks do not start last (bit 0: the range grows with the block row, so
    // rows run bottom-up; bit 1: it shrinks with the block column, so blocks
    // run column by column from the left)
    const int64_t nbx = gridDim.x, nby = gridDim.y;
    const int64_t bid = (int64_t)blockIdx.y * nbx + blockIdx.x;
    int64_t bx = blockIdx.x, by = blockIdx.y;
    if (tri & 1) {
        by = nby - 1 - bid / nbx;
        bx = bid % nbx;
    } else if (tri & 2) {
        bx = bid / nby;
        by = bid % nby;
    }
    const int64_t r0 = by * GT, c0 = bx * GT;
    if (lower_only && c0 > r0 + GT - 1) return;
    // K range that can hold nonzero products for this block (GK-aligned start)
    const int64_t kbeg = (tri & 2) ? (c0 < K ? c0 / GK * GK : K) : 0;
    const int64_t kend = (tri & 1) ? (r0 + GT < K ? r0 + GT : K) : K;
    __shared__ double As[2][GK][PAD];
    __shared__ double Bs[2][GK][PAD];
    const int t = threadIdx.x;
    const int wv = t >> 6, l = t & 63;
    const int wm = wv >> 1, wn = wv & 1;
    const int li = l & 15, lk = l >> 4;
    // staging: A rows (and B^T rows) by t >> 2, k quarter 4 (t & 3); B rows
    // (k) by t / (GT / 4), column quarter 4 (t % (GT / 4))
    const int ar = t >> 2, aq = 4 * (t & 3);
    const int bk = t / (GT / 4), bq = 4 * (t % (GT / 4));
    double ra[4], rb[4];
    auto load = [&](int64_t k0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t gr = r0 + ar, gk = k0 + aq + u;
            ra[u] = (gr < M && gk < K) ? A[gr * lda + gk] : 0.0;
        }
        if (!transB) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t gk = k0 + bk, gc = c0 + bq + u;
                rb[u] = (gk < K && gc < N) ? B[gk * ldb + gc] : 0.0;
            }
        } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t gc = c0 + ar, gk = k0 + aq + u;
                rb[u] = (gk < K && gc < N) ? B[gc * ldb + gk] : 0.0;
            }
        }
    };
    auto store = [&](int sb) {
#pragma unroll
        for (int u = 0; u < 4; ++u) As[sb][aq + u][ar] = ra[u];
        if (!transB) {
#pragma unroll
            for (int u = 0; u < 4; ++u) Bs[sb][bk][bq + u] = rb[u];
        } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) Bs[sb][aq + u][ar] = rb[u];
        }
    };
    f64x4 acc[2][YB];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < YB; ++y) acc[x][y] = f64x4{0.0, 0.0, 0.0, 0.0};
    const int64_t nch = kend > kbeg ? (kend - kbeg + GK - 1) / GK : 0;
    if (nch > 0) {
        load(kbeg);
        store(0);
    }
    __syncthreads();
    for (int64_t c = 0; c < nch; ++c) {
        const int sb = (int)(c & 1);
        const bool more = c + 1 < nch;
        if (more) load(kbeg + (c + 1) * GK);
#pragma unroll
        for (int kk = 0; kk < GK / 4; ++kk) {
            const int kr = 4 * kk + lk;
            double a[2], b2[YB];
#pragma unroll
            for (int x = 0; x < 2; ++x) a[x] = As[sb][kr][wm * 32 + x * 16 + li];
#pragma unroll
            for (int y = 0; y < YB; ++y) b2[y] = Bs[sb][kr][wn * (GT / 2) + y * 16 + li];
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < YB; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[x], b2[y], acc[x][y], 0, 0, 0);
        }
        if (more) store(sb ^ 1);
        __syncthreads();
    }
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < YB; ++y) {
            const int64_t gc = c0 + wn * (GT / 2) + y * 16 + li;
            if (gc >= N) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t gr = r0 + wm * 32 + x * 16 + lk + 4 * r;
                if (gr >= M) continue;
                if (lower_only && (gc >> 6) > (gr >> 6)) continue;   // a 64 x 64 block above the diagonal
                double* cp = C + gr * ldc + gc;
                const double v = (beta == 0.0) ? alpha * acc[x][y][r] : alpha * acc[x][y][r] + beta * (*cp);
                *cp = v + 0.0;   // -0 -> +0: zeros do not depend on which chunks were visited
            }
        }
}

__global__ void k_copy2d(const double* __restrict__ src, int64_t lds, double* __restrict__ dst,
                         int64_t ldd, int64_t rows, int64_t cols, const int* __restrict__ fail) {
    if (*fail) return;
    const int64_t total = rows * cols;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = e / cols, c = e - (e / cols) * cols;
        dst[r * ldd + c] = src[r * lds + c];
    }
}

// L[i][j] = Cinv[d-1-j][d-1-i] * C[d-1-j][d-1-j] for j <= i < d, rounded to
// fp32 into packed TS x TS tiles; padding (index >= d) is the identity.
__global__ void k_pack_factor(const double* __restrict__ C, const double* __restrict__ Ninv,
                              int64_t d, int64_t ld, int64_t nt, float* __restrict__ out) {
    const int64_t ntiles = nt * (nt + 1) / 2;
    const int64_t total = ntiles * TILE_ELEMS;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t tile = e / TILE_ELEMS;
        const int w = (int)(e - tile * TILE_ELEMS);
        // invert tile = I(I+1)/2 + J
        int64_t I = (int64_t)((sqrt(8.0 * (double)tile + 1.0) - 1.0) * 0.5);
        while ((I + 1) * (I + 2) / 2 <= tile) ++I;
        while (I * (I + 1) / 2 > tile) --I;
        const int64_t J = tile - I * (I + 1) / 2;
        const int64_t i = I * TS + w / TS, j = J * TS + w % TS;
        float v;
        if (i >= d || j >= d) v = (i == j) ? 1.0f : 0.0f;
        else if (j > i) v = 0.0f;
        else {
            const int64_t a = d - 1 - j, c = d - 1 - i;
            v = (float)(Ninv[a * ld + c] * C[a * ld + a]);
        }
        out[e] = v;
    }
}

// Identity factor in packed storage (B = I: one-sided GPTQ, Sec. 1).
__global__ void k_pack_identity(int64_t nt, float* __restrict__ out) {
    const int64_t total = nt * (nt + 1) / 2 * TILE_ELEMS;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t tile = e / TILE_ELEMS;
        const int w = (int)(e - tile * TILE_ELEMS);
        int64_t I = (int64_t)((sqrt(8.0 * (double)tile + 1.0) - 1.0) * 0.5);
        while ((I + 1) * (I + 2) / 2 <= tile) ++I;
        while (I * (I + 1) / 2 > tile) --I;
        const int64_t J = tile - I * (I + 1) / 2;
        out[e] = (I == J && (w / TS) == (w % TS)) ? 1.0f : 0.0f;
    }
}

// Dense row-major export of a packed factor (testing aid).
__global__ void k_unpack_factor(const float* __restrict__ packed, int64_t d,
                                float* __restrict__ dst) {
    const int64_t total = d * d;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / d, j = e - (e / d) * d;
        float v = 0.0f;
        if (j <= i) v = packed[packed_tile_offset(i / TS, j / TS) + (i % TS) * TS + (j % TS)];
        dst[e] = v;
    }
}

// ---------------------------------------------------------------------------
// Host drivers

static inline unsigned grid1d(int64_t total, int threads = 256) {
    int64_t g = (total + threads - 1) / threads;
    if (g > 65535LL * 64) g = 65535LL * 64;
    if (g < 1) g = 1;
    return (unsigned)g;
}

// 128 x 128 blocks when there are enough of them to fill the chip twice
// over (counting only blocks on or below the diagonal for lower_only), else
// 64 x 64 blocks.
#ifndef GEMM128_MIN_BLOCKS
#define GEMM128_MIN_BLOCKS 512
#endif
static hipError_t gemm_f64(hipStream_t s, int64_t M, int64_t N, int64_t K, double alpha,
                         const double* A, int64_t lda, const double* B, int64_t ldb, int transB,
                         double beta, double* C, int64_t ldc, int lower, const int* fail,
                         int tri = 0) {
    if (M <= 0 || N <= 0) return hipSuccess;
    const int64_t bm = (M + 127) / 128, bn = (N + 127) / 128;
    int64_t active = bm * bn;
    if (lower) {   // blocks with block column <= block row
        active = 0;
        for (int64_t i = 0; i < bm; ++i) active += (i + 1 < bn ? i + 1 : bn);
    }
    if (active >= GEMM128_MIN_BLOCKS) {
        dim3 grid((unsigned)bn, (unsigned)bm);
        hipLaunchKernelGGL(k_gemm<128>, grid, dim3(512), 0, s, M, N, K, alpha, A, lda, B, ldb,
                           transB, beta, C, ldc, lower, tri, fail);
    } else {
        dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64));
        hipLaunchKernelGGL(k_gemm<64>, grid, dim3(256), 0, s, M, N, K, alpha, A, lda, B, ldb,
                           transB, beta, C, ldc, lower, tri, fail);
    }
    return hipGetLastError();
}

// Recursive lower-triangular inverse: Ninv[off:off+sz, off:off+sz] from C.
// Diagonal NB-blocks must already be inverted.  Appends its launches to ops.
static void trtri_ops(std::vector<FactorOp>& ops, hipStream_t s, const double* C, double* Ninv,
                      int64_t ld, int64_t off, int64_t sz, double* T, const int* fail) {
    if (sz <= NB) return;
    int64_t nblk = (sz + NB - 1) / NB;
    int64_t h = ((nblk + 1) / 2) * NB;
    if (h >= sz) h = sz - NB;
    trtri_ops(ops, s, C, Ninv, ld, off, h, T, fail);
    trtri_ops(ops, s, C, Ninv, ld, off + h, sz - h, T, fail);
    const int64_t n2 = sz - h;
    ops.push_back([=]() {
        // T (n2 x h) = C21 * N11 (N11 lower triangular)
        hipError_t e = gemm_f64(s, n2, h, h, 1.0, C + (off + h) * ld + off, ld, Ninv + off * ld + off,
                                ld, 0, 0.0, T, h, 0, fail, 2);
        if (e != hipSuccess) return e;
        // N21 = -N22 * T (N22 lower triangular)
        return gemm_f64(s, n2, h, n2, -1.0, Ninv + (off + h) * ld + (off + h), ld, T, h, 0, 0.0,
                        Ninv + (off + h) * ld + off, ld, 0, fail, 1);
    });
}

// The factorisation of one matrix as a list of enqueue steps (a few launches
// each, in stream order), so that the host can interleave the steps of two
// factorisations on their two streams: enqueued one after the other, the
// second stream would sit idle while the host issues the first one's
// hundreds of launches.  Z, Ninv: d*d doubles; T: d*d/4 + d*NB doubles;
// flag: 1 int + 1 int64 (fail, pivot) zeroed by the caller.  With s2 (and
// its two events) the Cholesky looks one panel ahead; s2's work is ordered
// before everything enqueued on s after the last step.
void factor_ops(std::vector<FactorOp>& ops, hipStream_t s, hipStream_t s2, hipEvent_t ev_panel,
                hipEvent_t ev_rest, const float* X, int64_t d, double lam, double* Z, double* Ninv,
                double* T, double* mean, int* fail, int64_t* fail_pivot, float* packed, int64_t nt) {
    ops.push_back([=]() {
        hipLaunchKernelGGL(k_diag_mean, dim3(1), dim3(256), 0, s, X, d, mean);
        hipLaunchKernelGGL(k_flip_damp, dim3(grid1d(d * d)), dim3(256), 0, s, X, d, mean, lam, Z);
        return hipGetLastError();
    });
    // Two-level right-looking Cholesky: panels of NB2 columns, each factored
    // in NB-column steps (diagonal block, substitution for every row below,
    // update of the panel's remaining columns), then one rank-NB2 update of
    // the trailing matrix, which reads and writes it NB2 / NB times less
    // often than rank-NB updates would.  With s2 the trailing update of a
    // panel is split: the columns of the next panel on s, the rest on s2,
    // where it overlaps the next panel's factorisation (a chain of small,
    // latency-bound launches).  The rest update of panel p writes only
    // columns that panel p + 1 does not touch, and the next-panel update of
    // panel p + 1 waits for it, so every entry receives the same updates in
    // the same order either way.
    for (int64_t p0 = 0; p0 < d; p0 += NB2) {
        const int64_t pend = (d - p0) < NB2 ? d : p0 + NB2;
        for (int64_t k0 = p0; k0 < pend; k0 += NB) {
            const int b = (int)((pend - k0) < NB ? (pend - k0) : NB);
            ops.push_back([=]() {
                hipLaunchKernelGGL(k_potrf_diag, dim3(1), dim3(NB), 0, s, Z, d, k0, b, fail, fail_pivot);
                const int64_t rest = d - k0 - b;
                if (rest <= 0) return hipGetLastError();
                // panel solve: P <- P C_kk^-T by substitution
                hipLaunchKernelGGL(k_trsm_panel, dim3((unsigned)((rest + 255) / 256)), dim3(256), 0,
                                   s, Z, Z, d, k0, b, rest, fail);
                // the panel's remaining columns: Z[k0+b:, k0+b:pend] -= P P[k0+b:pend]^T
                return gemm_f64(s, rest, pend - k0 - b, b, -1.0, Z + (k0 + b) * d + k0, d,
                                Z + (k0 + b) * d + k0, d, 1, 1.0, Z + (k0 + b) * d + (k0 + b), d, 1,
                                fail);
            });
        }
        const int64_t rest = d - pend;
        if (rest <= 0) continue;
        const double* P = Z + pend * d + p0;   // the factored panel's rows below it
        const int64_t kp = pend - p0;
        // split point: the end of the next panel (no split without s2)
        const int64_t nend = (s2 && d - pend > NB2) ? pend + NB2 : d;
        const bool wait_prev = s2 && p0 > 0;
        ops.push_back([=]() {
            hipError_t e;
            if (nend < d) {   // Z[nend:, nend:] -= P P^T on s2, after this panel
                if ((e = hipEventRecord(ev_panel, s)) != hipSuccess) return e;
                if ((e = hipStreamWaitEvent(s2, ev_panel, 0)) != hipSuccess) return e;
                e = gemm_f64(s2, d - nend, d - nend, kp, -1.0, P + (nend - pend) * d, d,
                             P + (nend - pend) * d, d, 1, 1.0, Z + nend * d + nend, d, 1, fail);
                if (e != hipSuccess) return e;
            }
            // the previous panel's rest update also wrote these columns
            if (wait_prev && (e = hipStreamWaitEvent(s, ev_rest, 0)) != hipSuccess) return e;
            // Z[pend:, pend:nend] -= P P[pend:nend]^T on s
            e = gemm_f64(s, rest, nend - pend, kp, -1.0, P, d, P, d, 1, 1.0, Z + pend * d + pend, d, 1,
                         fail);
            if (e != hipSuccess) return e;
            if (nend < d) e = hipEventRecord(ev_rest, s2);
            return e;
        });
    }
    ops.push_back([=]() {
        // Ninv = C^-1 (lower); upper part must be zero for the recursive GEMMs
        hipError_t e = hipMemsetAsync(Ninv, 0, sizeof(double) * d * d, s);
        if (e != hipSuccess) return e;
        const int64_t nblk = (d + NB - 1) / NB;
        hipLaunchKernelGGL(k_inv_lower_blocks, dim3((unsigned)nblk), dim3(NB), 0, s, Z, d, Ninv, d,
                           (int64_t)0, d, (int64_t)0, fail);
        return hipGetLastError();
    });
    trtri_ops(ops, s, Z, Ninv, d, 0, d, T, fail);
    ops.push_back([=]() {
        hipLaunchKernelGGL(k_pack_factor, dim3(grid1d(nt * (nt + 1) / 2 * TILE_ELEMS)), dim3(256), 0,
                           s, Z, Ninv, d, d, nt, packed);
        return hipGetLastError();
    });
}

hipError_t pack_identity(hipStream_t s, int64_t nt, float* packed) {
    hipLaunchKernelGGL(k_pack_identity, dim3(grid1d(nt * (nt + 1) / 2 * TILE_ELEMS)), dim3(256), 0,
                       s, nt, packed);
    return hipGetLastError();
}

hipError_t unpack_factor(hipStream_t s, const float* packed, int64_t d, float* dst) {
    hipLaunchKernelGGL(k_unpack_factor, dim3(grid1d(d * d)), dim3(256), 0, s, packed, d, dst);
    return hipGetLastError();
}

}  // namespace bk
