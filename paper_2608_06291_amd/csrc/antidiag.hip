// BaKron-antidiagonal (Alg. 3): the anti-diagonal-parallel form of the
// vectorised-weight rounding without the divide-and-conquer.  It is the
// reference point of the paper's runtime comparison (Table 3: BaKron against
// BaKron-antidiagonal, which the paper notes is essentially the iterative
// form of YAQA) and reaches the same output as the BaKron solver (Thm 3.2).
//
// For every element anti-diagonal k = 0 .. m+n-2 in order:
//   round:  for the entries (i, k-i): x = W~/s_ij, c = clamp(rint x, lo, hi),
//           V = s_ij c, E = V - W~ (the error Delta of Alg. 3);
//   update: W~ += L^B * antidiag_k(E) * L^A^T, i.e. for every (p, q)
//           W~_pq += sum_i L^B[p][i] E[i][k-i] L^A[q][k-i]  (a rank-r product,
//           r = number of entries on the diagonal).
// Total work is quartic, O(m^2 n^2) (Table 1); each step is one dense product
// whose K dimension runs over the diagonal's entries.
#include "common.h"

namespace bk {

// Round the entries (i, k - i), i in [i0, i1], of the working copy Wt
// (row-major m x n); the error of row i goes to delta[i].
__global__ __launch_bounds__(256) void k_ad_round(const float* __restrict__ Wt, int64_t m, int64_t n,
                                                  int k, int i0, int i1, QuantArgs q,
                                                  int8_t* __restrict__ codes,
                                                  float* __restrict__ V, float* __restrict__ pre,
                                                  float* __restrict__ delta) {
    const int i = i0 + (int)(blockIdx.x * 256 + threadIdx.x);
    if (i > i1) return;
    const int64_t o = (int64_t)i * n + (k - i);
    const float w = Wt[o];
    const float s = entry_scale(q, i, k - i, m, n);
    const float inv_s = s > 0.0f ? 1.0f / s : 0.0f;   // zero scale: alphabet {0}
    const float x = w * inv_s;
    const float c = __builtin_amdgcn_fmed3f(rintf(x), q.qlo, q.qhi);
    codes[o] = (int8_t)(int)c;
    V[o] = c * s;
    if (pre) pre[o] = s > 0.0f ? x : __builtin_nanf("");
    delta[i] = fmaf(c, s, -w);
}

// Rank-r update of one 64 x 64 block of Wt after diagonal k (i in [i0, i1]):
//   C[p][q] += sum_i (L^B[p][i] delta[i]) * L^A[q][k - i].
// Only i with i <= p and k - i <= q contribute (triangular factors), so the
// block walks i over [max(i0, k - q_max), min(i1, p_max)] in chunks aligned to
// the factor's 32-column tiles: the L^B operand of a chunk is one tile row per
// block row (two 16-byte loads per thread), the L^A operand 32 consecutive
// columns read backwards.  v_mfma_f32_32x32x2f32, 4 waves with one 32 x 32
// quarter each (lane half h takes k = 16h + s at step s); chunks are
// prefetched two ahead in two register sets.  Blocks that hold no entry past
// diagonal k return at once.
constexpr int AD_B = 64;
constexpr int AD_STRIDE = TS + 4;
__global__ __launch_bounds__(256) void k_ad_update(float* __restrict__ Wt, int64_t m, int64_t n,
                                                   int k, int i0, int i1,
                                                   const float* __restrict__ LA,
                                                   const float* __restrict__ LB,
                                                   const float* __restrict__ delta, int nbq) {
    __shared__ __attribute__((aligned(16))) float As[2][AD_B][AD_STRIDE];
    __shared__ __attribute__((aligned(16))) float Bs[2][AD_B][AD_STRIDE];
    const int P0 = (int)(blockIdx.x / nbq) * AD_B, Q0 = (int)(blockIdx.x % nbq) * AD_B;
    const int pmax = min((int)m - 1, P0 + AD_B - 1), qmax = min((int)n - 1, Q0 + AD_B - 1);
    if (pmax + qmax <= k) return;   // every entry of the block is on diagonal <= k
    const int lo = max(i0, k - qmax), hi = min(i1, pmax);
    if (lo > hi) return;
    const int c_lo = lo >> 5, c_hi = hi >> 5;   // factor tile columns of the chunks

    const int tid = threadIdx.x;
    const int wv = tid >> 6, l = tid & 63;
    const int wm = wv >> 1, wn = wv & 1;
    const int lr = l & 31, lk = l >> 5;
    // staging: thread tid fills row tid >> 2, chunk columns t = 8 (tid & 3) .. + 7
    const int srow = tid >> 2, st0 = 8 * (tid & 3);
    const int p = P0 + srow, q = Q0 + srow;
    f32x4 ra[2][2];
    float rb[2][8];
    auto load = [&](int c, int r) {
        const int ib = 32 * c + st0;   // first i of this thread's 8 columns
        if (p < m && c <= (p >> 5)) {
            const f32x4* src = reinterpret_cast<const f32x4*>(LB + packed_tile_offset(p >> 5, c) +
                                                              (p & 31) * TS + st0);
            const f32x4 d0 = *reinterpret_cast<const f32x4*>(delta + ib);
            const f32x4 d1 = *reinterpret_cast<const f32x4*>(delta + ib + 4);
            f32x4 a0 = src[0], a1 = src[1];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                a0[u] = (ib + u >= lo && ib + u <= hi) ? a0[u] * d0[u] : 0.0f;
                a1[u] = (ib + 4 + u >= lo && ib + 4 + u <= hi) ? a1[u] * d1[u] : 0.0f;
            }
            ra[r][0] = a0;
            ra[r][1] = a1;
        } else {
            ra[r][0] = f32x4{0.f, 0.f, 0.f, 0.f};
            ra[r][1] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int j = k - (ib + u);
            rb[r][u] = (q < n && j >= 0 && j <= q && ib + u >= lo && ib + u <= hi)
                           ? LA[packed_tile_offset(q >> 5, j >> 5) + (q & 31) * TS + (j & 31)]
                           : 0.0f;
        }
    };
    auto store = [&](int sb, int r) {
        *reinterpret_cast<f32x4*>(&As[sb][srow][st0]) = ra[r][0];
        *reinterpret_cast<f32x4*>(&As[sb][srow][st0 + 4]) = ra[r][1];
#pragma unroll
        for (int u = 0; u < 8; ++u) Bs[sb][srow][st0 + u] = rb[r][u];
    };
    f32x16 acc = {0};
    // chunk c is multiplied from buffer (c - c_lo) & 1; while it is, chunk c + 2
    // loads into register set (c - c_lo) & 1 and chunk c + 1 (other set) is
    // written to the other buffer
    auto chunk = [&](int c, int sb) {
        if (c + 2 <= c_hi) load(c + 2, sb);
        f32x4 fa[4], fb[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            fa[v] = *reinterpret_cast<const f32x4*>(&As[sb][wm * 32 + lr][lk * 16 + v * 4]);
            fb[v] = *reinterpret_cast<const f32x4*>(&Bs[sb][wn * 32 + lr][lk * 16 + v * 4]);
        }
#pragma unroll
        for (int st = 0; st < 16; ++st)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[st >> 2][st & 3], fb[st >> 2][st & 3], acc,
                                                       0, 0, 0);
        if (c + 1 <= c_hi) store(sb ^ 1, sb ^ 1);
        __syncthreads();
    };
    load(c_lo, 0);
    if (c_lo + 1 <= c_hi) load(c_lo + 1, 1);
    store(0, 0);
    __syncthreads();
    for (int c = c_lo; c <= c_hi; c += 2) {
        chunk(c, 0);
        if (c + 1 <= c_hi) chunk(c + 1, 1);
    }
    // C[row][col] of this wave's quarter: row (r >> 2) * 8 + lk * 4 + (r & 3), column lr
    const int qo = Q0 + wn * 32 + lr;
    if (qo >= n) return;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int po = P0 + wm * 32 + (r >> 2) * 8 + lk * 4 + (r & 3);
        if (po < m) Wt[(int64_t)po * n + qo] += acc[r];
    }
}

// Enqueues the whole of Alg. 3 on one stream: copy W into the working array,
// then round and update one anti-diagonal after the other.  delta holds
// 32 * ceil(m / 32) floats (one per row, read in whole tile-aligned chunks).
hipError_t run_antidiag(hipStream_t st, const float* W, int64_t m, int64_t n, float* Wt,
                        float* delta, const float* LA, const float* LB, const QuantArgs& q,
                        int8_t* codes, float* V, float* pre) {
    hipError_t e = hipMemcpyAsync(Wt, W, sizeof(float) * (size_t)(m * n), hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
    const int nbp = (int)((m + AD_B - 1) / AD_B), nbq = (int)((n + AD_B - 1) / AD_B);
    for (int k = 0; k <= (int)(m + n - 2); ++k) {
        const int i0 = k - (int)(n - 1) > 0 ? k - (int)(n - 1) : 0;
        const int i1 = k < (int)(m - 1) ? k : (int)(m - 1);
        const int cnt = i1 - i0 + 1;
        hipLaunchKernelGGL(k_ad_round, dim3((unsigned)((cnt + 255) / 256)), dim3(256), 0, st, Wt, m,
                           n, k, i0, i1, q, codes, V, pre, delta);
        if (k < (int)(m + n - 2))
            hipLaunchKernelGGL(k_ad_update, dim3((unsigned)(nbp * nbq)), dim3(256), 0, st, Wt, m, n, k,
                               i0, i1, LA, LB, delta, nbq);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace bk
