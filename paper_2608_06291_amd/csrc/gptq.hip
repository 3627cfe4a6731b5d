// One-sided rounding for B = I (GPTQ, Alg. 1 applied to every row of W with
// the Hessian A; Sec. 1 and Table 1: n sequential steps, O(mn^2) work).
//
// With B = I the feedback of Eq. (1) never crosses rows:
//     W~_pq = W0_pq + sum_{j<q} E_pj L^A_qj ,   E = V - W~ ,
// so the rows are independent and each row is a sequential pass over its n
// columns.  Two levels of blocking (GPTQ's lazy batch updates):
//   * ranges of GR column tiles (1024 columns).  Once a range is rounded, its
//     errors are pushed into every later column of a working copy W' of W
//     in one full-chip product on fp32 MFMA (k_gptq_push), so the bulk of
//     the O(mn^2) work does not depend on how many rows there are;
//   * inside a range, blocks of 32 columns (one factor tile), k_gptq:
//     1. lazy feedback: W~[rows, blk] = W'[rows, blk] + E[rows, range start
//        .. blk] L^A[blk, ...]^T, a dense product on fp32 MFMA over the
//        earlier blocks of the range;
//     2. the 32 columns of the block in order: quantise column j of every
//        row, then add E[:, j] L^A[q, j] to the later columns q of the block.
// The sums are the same elementary updates of Eq. (1), in another order.
//
// A k_gptq workgroup owns 16 rows and walks the blocks of one range.  In
// step 1 each of its 4 waves multiplies a quarter of the source tiles with
// v_mfma_f32_16x16x4f32 (A = the 16 error rows, B = the factor tile rows, so
// D[i][j] = sum_k E[i][k] L^A[j][k]), with the operands of its next two
// tiles in flight; the four partial sums meet in LDS.  In step 2 each wave
// owns 4 rows, 16 lanes per row with the block columns c and c + 16 in
// registers; the error of column j is broadcast along its 16 lanes with a
// lane shuffle, so no barrier is needed inside the block.
#include "common.h"

namespace bk {

struct GptqArgs {
    int64_t m, n;
    int nt;           // column tiles
    int64_t ldE;      // row stride of the error workspace (nt * 32)
    const float* Wb;  // base values of the range: W (the first range) or W'
    int64_t ldWb;     // their row stride
    const float* LA;  // packed unit-lower factor tiles
    float* E;         // errors, ceil(m/16)*16 x nt*32 row-major (workspace)
    int b_begin, b_end;   // the column tiles of this launch
    QuantArgs q;
    int8_t* codes;
    float* V;
    float* pre;       // may be null
};

constexpr int GR = 32;   // column tiles per range (1024 columns; the default of run_gptq)

__device__ inline f32x4 ld4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }

__device__ inline void mfma16_8(f32x4 a0, f32x4 a1, f32x4 b0, f32x4 b1, f32x4& acc) {
#pragma unroll
    for (int t = 0; t < 4; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[t], b0[t], acc, 0, 0, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[t], b1[t], acc, 0, 0, 0);
}

constexpr int GW = 4;   // waves per workgroup

__global__ __launch_bounds__(64 * GW) void k_gptq(GptqArgs a) {
    __shared__ float part[GW][16][33];   // per wave: partial 16 x 32 lazy products
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), l = tid & 63;
    const int64_t row0 = (int64_t)blockIdx.x * 16;
    // step 1 lane roles: A row i16, k chunk [8 s, 8 s + 8) of every source tile
    const int i16 = l & 15, s = l >> 4;
    // step 2 lane roles: row rr of the 16, block columns c16 and c16 + 16
    const int rr = 4 * w + (l >> 4), c16 = l & 15;
    const int64_t row = row0 + rr;
    const float qlo = a.q.qlo, qhi = a.q.qhi;
    const float nan = __builtin_nanf("");

    for (int b = a.b_begin; b < a.b_end; ++b) {
        // 1. lazy feedback from the range's source tiles kt < b (a quarter per wave),
        // two tiles in flight: set 0 holds tiles w, w + 2 GW, ..., set 1
        // tiles w + GW, w + 3 GW, ...
        f32x4 acc0 = {0.0f, 0.0f, 0.0f, 0.0f}, acc1 = {0.0f, 0.0f, 0.0f, 0.0f};
        {
            const float* erow = a.E + (row0 + i16) * a.ldE + 8 * s;
            const float* lt = a.LA + packed_tile_offset(b, 0) + i16 * TS + 8 * s;
            f32x4 e0[2], e1[2], l0[2], l1[2], m0[2], m1[2];
            auto ld = [&](int kt, int q) {
                e0[q] = ld4(erow + kt * TS);
                e1[q] = ld4(erow + kt * TS + 4);
                l0[q] = ld4(lt + kt * TILE_ELEMS);
                l1[q] = ld4(lt + kt * TILE_ELEMS + 4);
                m0[q] = ld4(lt + kt * TILE_ELEMS + 16 * TS);
                m1[q] = ld4(lt + kt * TILE_ELEMS + 16 * TS + 4);
            };
            auto mul = [&](int q) {
                mfma16_8(e0[q], e1[q], l0[q], l1[q], acc0);   // output columns 0..15 of the block
                mfma16_8(e0[q], e1[q], m0[q], m1[q], acc1);   // output columns 16..31
            };
            int kt = a.b_begin + w;
            if (kt < b) ld(kt, 0);
            if (kt + GW < b) ld(kt + GW, 1);
            for (; kt + GW < b; kt += 2 * GW) {
                {
                    const f32x4 x0 = e0[0], x1 = e1[0], y0 = l0[0], y1 = l1[0], z0 = m0[0], z1 = m1[0];
                    if (kt + 2 * GW < b) ld(kt + 2 * GW, 0);
                    mfma16_8(x0, x1, y0, y1, acc0);
                    mfma16_8(x0, x1, z0, z1, acc1);
                }
                {
                    const f32x4 x0 = e0[1], x1 = e1[1], y0 = l0[1], y1 = l1[1], z0 = m0[1], z1 = m1[1];
                    if (kt + 3 * GW < b) ld(kt + 3 * GW, 1);
                    mfma16_8(x0, x1, y0, y1, acc0);
                    mfma16_8(x0, x1, z0, z1, acc1);
                }
            }
            if (kt < b) mul(0);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            part[w][4 * s + r][i16] = acc0[r];
            part[w][4 * s + r][16 + i16] = acc1[r];
        }
        __syncthreads();

        // 2. the block's 32 columns in order, 16 lanes per row
        const int64_t col0 = (int64_t)b * TS + c16, col1 = col0 + 16;
        float h0 = part[0][rr][c16], h1 = part[0][rr][16 + c16];
#pragma unroll
        for (int v = 1; v < GW; ++v) {
            h0 += part[v][rr][c16];
            h1 += part[v][rr][16 + c16];
        }
        if (row < a.m && col0 < a.n) h0 += a.Wb[row * a.ldWb + col0];
        if (row < a.m && col1 < a.n) h1 += a.Wb[row * a.ldWb + col1];
        const float s0 = entry_scale(a.q, row, col0, a.m, a.n);
        const float s1 = entry_scale(a.q, row, col1, a.m, a.n);
        const float is0 = s0 > 0.0f ? 1.0f / s0 : 0.0f;   // zero scale: alphabet {0}
        const float is1 = s1 > 0.0f ? 1.0f / s1 : 0.0f;
        // L^A[col][blk] of the lane's two columns, strictly below the diagonal
        float c0[TS], c1[TS];
        {
            const float* d = a.LA + packed_tile_offset(b, b);
#pragma unroll
            for (int j = 0; j < TS; j += 4) {
                const f32x4 u = ld4(d + c16 * TS + j), v = ld4(d + (16 + c16) * TS + j);
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    c0[j + t] = (j + t < c16) ? u[t] : 0.0f;
                    c1[j + t] = (j + t < 16 + c16) ? v[t] : 0.0f;
                }
            }
        }
        float e0 = 0.0f, e1 = 0.0f, x0 = 0.0f, x1 = 0.0f;
#pragma unroll
        for (int j = 0; j < TS; ++j) {
            const bool hi = j >= 16;                       // column j sits in slot 1
            const float hv = hi ? h1 : h0, iv = hi ? is1 : is0, sv = hi ? s1 : s0;
            const float xv = hv * iv;
            const float cq = __builtin_amdgcn_fmed3f(rintf(xv), qlo, qhi);
            const float ev = fmaf(cq, sv, -hv);
            // the owner of column j is lane (j & 15) of the row's 16 lanes
            const float ej = __shfl(ev, (l & 48) | (j & 15), 64);
            if (c16 == (j & 15)) {
                if (hi) { e1 = ev; x1 = xv; } else { e0 = ev; x0 = xv; }
            }
            h0 = fmaf(ej, c0[j], h0);
            h1 = fmaf(ej, c1[j], h1);
        }
        // errors for the later blocks (every workspace row and column is
        // written, padding included: its errors are 0); outputs
        a.E[row * a.ldE + col0] = e0;
        a.E[row * a.ldE + col1] = e1;
        if (row < a.m) {
            if (col0 < a.n) {
                const int64_t o = row * a.n + col0;
                const float r = __builtin_amdgcn_fmed3f(rintf(x0), qlo, qhi);
                a.codes[o] = (int8_t)(int)r;
                a.V[o] = r * s0;
                if (a.pre) a.pre[o] = s0 > 0.0f ? x0 : nan;
            }
            if (col1 < a.n) {
                const int64_t o = row * a.n + col1;
                const float r = __builtin_amdgcn_fmed3f(rintf(x1), qlo, qhi);
                a.codes[o] = (int8_t)(int)r;
                a.V[o] = r * s1;
                if (a.pre) a.pre[o] = s1 > 0.0f ? x1 : nan;
            }
        }
        __syncthreads();   // the block's errors and the partial sums are reused
    }
}

// The push of a finished range: Wout[p][q] = Win[p][q] + sum_k E[p][k] L^A[q][k]
// over the range's columns k, for every later column q >= qb.  One workgroup
// per MT x MT block of 32 x 32 tiles of W', 4 waves in a 2 x 2 arrangement,
// each MT/2 x MT/2 blocks of v_mfma_f32_32x32x2f32; the range's K in chunks
// of one tile (32), staged through double-buffered LDS with 16-byte rows,
// the chunks two ahead prefetched into registers while the current one is
// multiplied (within a chunk lane half h supplies k = 16 h + s at step s).
// The same pipeline as the two-sided node push, on row-major E and W'.
struct PushArgs {
    int64_t m, m16, n;
    int nt;
    int64_t ldE;
    const float* E;
    const float* LA;
    const float* Win;
    int64_t ldIn;
    float* Wout;
    int64_t ldOut;
    int kb, ke;       // the range's column tiles
    int64_t qb;       // first column of the later ranges (a multiple of 32)
};

constexpr int PSTR = TS + 4;   // LDS row stride (floats): 16-byte rows

template <int MT>
__global__ __launch_bounds__(256, (MT == 4 ? 2 : 4)) void k_gptq_push(PushArgs a) {
    constexpr int WB = MT / 2;
    __shared__ __attribute__((aligned(16))) float As[2][MT * TS][PSTR];
    __shared__ __attribute__((aligned(16))) float Bs[2][MT * TS][PSTR];
    const int tid = threadIdx.x;
    const int wv = tid >> 6, l = tid & 63;
    const int wm = wv >> 1, wn = wv & 1;
    const int lr = l & 31, lk = l >> 5;
    const int srow = tid >> 3, sk = (tid & 7) * 4;   // staging: one float4 of each tile
    const int64_t p0 = (int64_t)blockIdx.y * (MT * TS), q0 = a.qb + (int64_t)blockIdx.x * (MT * TS);
    const int Q0 = (int)(q0 / TS);

    f32x4 ra[2][MT], rb[2][MT];
    auto load = [&](int kt, int r) {
#pragma unroll
        for (int t = 0; t < MT; ++t) {
            const int64_t p = p0 + t * TS + srow;
            const bool kin = kt < a.ke;
            ra[r][t] = (kin && p < a.m16) ? *reinterpret_cast<const f32x4*>(a.E + p * a.ldE + (int64_t)kt * TS + sk)
                                          : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            rb[r][t] = (kin && Q0 + t < a.nt)
                           ? *reinterpret_cast<const f32x4*>(a.LA + packed_tile_offset(Q0 + t, kt) + tid * 4)
                           : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
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
    auto chunk = [&](int kt, int s, int r) {
        load(kt + 2, r);   // past the range: zeros, nothing read
        f32x4 fa[WB][4], fb[WB][4];
#pragma unroll
        for (int x = 0; x < WB; ++x)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                fa[x][v] = *reinterpret_cast<const f32x4*>(&As[s][(wm * WB + x) * TS + lr][lk * 16 + v * 4]);
#pragma unroll
        for (int y = 0; y < WB; ++y)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                fb[y][v] = *reinterpret_cast<const f32x4*>(&Bs[s][(wn * WB + y) * TS + lr][lk * 16 + v * 4]);
#pragma unroll
        for (int st = 0; st < 16; ++st) {
#pragma unroll
            for (int x = 0; x < WB; ++x)
#pragma unroll
                for (int y = 0; y < WB; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[x][st >> 2][st & 3],
                                                                    fb[y][st >> 2][st & 3], acc[x][y], 0, 0, 0);
        }
        if (kt + 1 < a.ke) store(s ^ 1, r ^ 1);
        __syncthreads();
    };
    load(a.kb, 0);
    load(a.kb + 1, 1);
    store(0, 0);
    __syncthreads();
    for (int kt = a.kb; kt < a.ke; kt += 2) {
        chunk(kt, 0, 0);
        if (kt + 1 < a.ke) chunk(kt + 1, 1, 1);
    }
#pragma unroll
    for (int x = 0; x < WB; ++x)
#pragma unroll
        for (int y = 0; y < WB; ++y) {
            const int64_t q = q0 + (wn * WB + y) * TS + lr;
            if (q >= a.n) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t p = p0 + (wm * WB + x) * TS + (r >> 2) * 8 + lk * 4 + (r & 3);
                if (p < a.m) a.Wout[p * a.ldOut + q] = a.Win[p * a.ldIn + q] + acc[x][y][r];
            }
        }
}

// errors (ceil(m/16)*16 x nt*32) and the working copy W' (the same shape)
size_t gptq_workspace_floats(int64_t m, int64_t n) {
    return 2 * (size_t)((m + 15) / 16 * 16) * (size_t)((n + TS - 1) / TS * TS);
}

// range_tiles: column tiles per range (0: GR).  Per range one k_gptq launch
// and, unless it is the last, one push: 1024-column ranges measured fastest
// on the paper's Table 3 shapes (128 to 2048 columns tried).
hipError_t run_gptq(hipStream_t st, const float* W, int64_t m, int64_t n, const float* LA, float* E,
                    const QuantArgs& q, int8_t* codes, float* V, float* pre, int range_tiles) {
    const int R = range_tiles > 0 ? range_tiles : GR;
    const int nt = (int)((n + TS - 1) / TS);
    const int64_t ldE = (int64_t)nt * TS, m16 = (m + 15) / 16 * 16;
    float* Wt = E + m16 * ldE;
    GptqArgs a;
    a.m = m;
    a.n = n;
    a.nt = nt;
    a.ldE = ldE;
    a.LA = LA;
    a.E = E;
    a.q = q;
    a.codes = codes;
    a.V = V;
    a.pre = pre;
    for (int b0 = 0; b0 < nt; b0 += R) {
        const int b1 = b0 + R < nt ? b0 + R : nt;
        a.b_begin = b0;
        a.b_end = b1;
        a.Wb = b0 == 0 ? W : Wt;
        a.ldWb = b0 == 0 ? n : ldE;
        hipLaunchKernelGGL(k_gptq, dim3((unsigned)(m16 / 16)), dim3(64 * GW), 0, st, a);
        if (b1 < nt) {
            PushArgs pa;
            pa.m = m;
            pa.m16 = m16;
            pa.n = n;
            pa.ldE = ldE;
            pa.E = E;
            pa.LA = LA;
            pa.Win = b0 == 0 ? W : Wt;
            pa.ldIn = b0 == 0 ? n : ldE;
            pa.Wout = Wt;
            pa.ldOut = ldE;
            pa.kb = b0;
            pa.ke = b1;
            pa.qb = (int64_t)b1 * TS;
            pa.nt = nt;
            // 128 x 128 blocks when they fill the chip twice over, else 64 x 64
            const int64_t big = ((n - pa.qb + 127) / 128) * ((m + 127) / 128);
            if (big >= 512) {
                const dim3 grid((unsigned)((n - pa.qb + 127) / 128), (unsigned)((m + 127) / 128));
                hipLaunchKernelGGL(k_gptq_push<4>, grid, dim3(256), 0, st, pa);
            } else {
                const dim3 grid((unsigned)((n - pa.qb + 63) / 64), (unsigned)((m + 63) / 64));
                hipLaunchKernelGGL(k_gptq_push<2>, grid, dim3(256), 0, st, pa);
            }
        }
    }
    return hipGetLastError();
}

}  // namespace bk
