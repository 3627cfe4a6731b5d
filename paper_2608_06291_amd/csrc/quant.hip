// Quantiser set-up around the solve (Sec. 3.1, App. D): the MSE scale search
// and the block-diagonal output factor of an attention projection.
//
// MSE scales (App. D: max-abs per row over the largest code, optionally
// shrunk by up to 2x by an MSE search).  For every row i (or row segment of
// `group` columns) and candidate k = 0..grid:
//   base = fl32(max_j |W_ij| / hi),  p_k = fl32(1 - maxshrink * k / grid),
//   s_k = fl32(base * p_k),
//   err_k = sum_j (W_ij - fl32(s_k * c_ij))^2,  c_ij = clamp(rint(fl32(W_ij / s_k)), lo, hi)
// (c = 0 when s_k = 0), summed in fp64; the scale is s_k of the first
// minimum.  The integer decisions are taken with IEEE fp32 division, rint
// and products, so they are reproducible; only the fp64 summation order is
// the kernel's own.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <string>

#include "bakron.h"
#include "common.h"

namespace bk {

constexpr int MSE_THREADS = 256;   // one candidate per thread: grid <= 255

// One workgroup per (row, column segment).  The segment's max-abs first
// (a block reduction), then every thread evaluates its candidate over the
// segment's columns; thread 0 picks the first minimum.
__global__ __launch_bounds__(MSE_THREADS) void k_mse_scales(const float* __restrict__ W, int64_t n,
                                                            int seg, int nseg, int grid,
                                                            double maxshrink, float lo, float hi,
                                                            float* __restrict__ scale) {
    __shared__ float red[MSE_THREADS];
    __shared__ float sv[MSE_THREADS];
    __shared__ double err[MSE_THREADS];
    const int i = (int)(blockIdx.x / (unsigned)nseg), g = (int)(blockIdx.x % (unsigned)nseg);
    const int64_t c0 = (int64_t)g * seg, c1 = std::min<int64_t>(n, c0 + seg);
    const float* row = W + (int64_t)i * n;
    const int t = threadIdx.x;
    float mx = 0.0f;
    for (int64_t j = c0 + t; j < c1; j += MSE_THREADS) mx = fmaxf(mx, fabsf(row[j]));
    red[t] = mx;
    __syncthreads();
    for (int h = MSE_THREADS / 2; h > 0; h >>= 1) {
        if (t < h) red[t] = fmaxf(red[t], red[t + h]);
        __syncthreads();
    }
    const float base = red[0] / hi;
    if (t <= grid) {
        const float p = (float)(1.0 - maxshrink * (double)t / (double)grid);
        const float s = grid > 0 ? base * p : base;
        double e = 0.0;
        for (int64_t j = c0; j < c1; ++j) {
            const float w = row[j];
            float v = 0.0f;
            if (s > 0.0f) {
                const float c = fminf(fmaxf(rintf(w / s), lo), hi);
                v = s * c;
            }
            const double d = (double)w - (double)v;
            e = fma(d, d, e);
        }
        err[t] = e;
        sv[t] = s;
    }
    __syncthreads();
    if (t == 0) {
        int best = 0;
        for (int k = 1; k <= grid; ++k)
            if (err[k] < err[best]) best = k;
        scale[(int64_t)i * nseg + g] = sv[best];
    }
}

// Dst (m x m, m = nblocks * hb) = blockdiag(blocks): every entry written
// (zeros off the blocks).
__global__ __launch_bounds__(256) void k_blockdiag(const float* __restrict__ blocks, int64_t hb,
                                                   int64_t m, float* __restrict__ dst) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= m * m) return;
    const int64_t r = e / m, c = e % m;
    const int64_t h = r / hb;
    dst[e] = (c / hb == h) ? blocks[h * hb * hb + (r - h * hb) * hb + (c - h * hb)] : 0.0f;
}

}  // namespace bk

extern "C" bakron_status bakron_mse_scales(const float* W, int64_t m, int64_t n, int32_t bits,
                                           int32_t alphabet, int32_t group_size, int32_t grid,
                                           double maxshrink, float* scale, hipStream_t stream) {
    bk::set_last_error("");
    if (!W || !scale || m <= 0 || n <= 0 || m > ((int64_t)1 << 31) - 1 || n > ((int64_t)1 << 40)) {
        bk::set_last_error("bakron_mse_scales: null pointer or bad size");
        return BAKRON_EINVAL;
    }
    if (bits < 2 || bits > 8 ||
        (alphabet != BAKRON_ALPHABET_SYMMETRIC && alphabet != BAKRON_ALPHABET_ASYMMETRIC)) {
        bk::set_last_error("bakron_mse_scales: bad bits or alphabet");
        return BAKRON_EINVAL;
    }
    if (group_size < 0 || grid < 0 || grid >= bk::MSE_THREADS || !(maxshrink >= 0.0) ||
        !(maxshrink < 1.0)) {
        bk::set_last_error("bakron_mse_scales: need group_size >= 0, 0 <= grid <= 255, "
                           "0 <= maxshrink < 1");
        return BAKRON_EINVAL;
    }
    const int64_t seg = group_size > 0 ? group_size : n;
    const int64_t nseg = (n + seg - 1) / seg;
    if (m * nseg > ((int64_t)1 << 31) - 1) {
        bk::set_last_error("bakron_mse_scales: too many row segments");
        return BAKRON_EINVAL;
    }
    const int h = 1 << (bits - 1);
    const float lo = alphabet == BAKRON_ALPHABET_ASYMMETRIC ? (float)-h : (float)-(h - 1);
    const float hi = (float)(h - 1);
    hipLaunchKernelGGL(bk::k_mse_scales, dim3((unsigned)(m * nseg)), dim3(bk::MSE_THREADS), 0, stream,
                       W, n, (int)seg, (int)nseg, grid, maxshrink, lo, hi, scale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        char buf[200];
        std::snprintf(buf, sizeof(buf), "bakron_mse_scales: launch: %s", hipGetErrorString(e));
        bk::set_last_error(buf);
        return BAKRON_EHIP;
    }
    return BAKRON_OK;
}

extern "C" bakron_status bakron_factor_blockdiag(const float* A, int64_t n, const float* B_blocks,
                                                 int64_t nblocks, int64_t hb, float damp,
                                                 hipStream_t stream, bakron_factors** out) {
    bk::set_last_error("");
    if (!B_blocks || nblocks <= 0 || hb <= 0 || nblocks * hb > ((int64_t)1 << 20)) {
        bk::set_last_error("bakron_factor_blockdiag: invalid block arguments");
        return BAKRON_EINVAL;
    }
    const int64_t m = nblocks * hb;
    float* Bfull = nullptr;
    hipError_t e = hipMalloc(&Bfull, sizeof(float) * (size_t)m * (size_t)m);
    if (e != hipSuccess) {
        bk::set_last_error("bakron_factor_blockdiag: hipMalloc");
        return e == hipErrorOutOfMemory ? BAKRON_ENOMEM : BAKRON_EHIP;
    }
    hipLaunchKernelGGL(bk::k_blockdiag, dim3((unsigned)((m * m + 255) / 256)), dim3(256), 0, stream,
                       B_blocks, hb, m, Bfull);
    e = hipGetLastError();
    bakron_status st;
    if (e != hipSuccess) {
        bk::set_last_error("bakron_factor_blockdiag: launch");
        st = BAKRON_EHIP;
    } else {
        // bakron_factor synchronises `stream` before returning, so the
        // assembled matrix is no longer in use when it is freed below
        st = bakron_factor(A, n, Bfull, m, damp, stream, out);
    }
    hipFree(Bfull);   // waits for the work that still uses it
    return st;
}
