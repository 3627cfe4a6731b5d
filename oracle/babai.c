/*
 * oracle/babai.c -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * Plain, slow fp64 reference for the sequential rounding that BaKron computes.
 * Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
 * load this file's library.  It shares no code with the HIP solver.
 *
 * What it computes (paper: Sec. 3.2, Alg. 2 "BaKron-naive"; Thm 3.2 states that
 * BaKron-antidiagonal, BaKron-recursive and BaKron return the same output):
 *   GPTQ / Babai nearest-plane on vec(W) with the Kronecker Hessian A (x) B,
 *   written in the unvectorised weight domain.  Entries are visited row by
 *   row; after an entry is quantised, its error Delta is fed back to every
 *   entry below and to the right through the rank-one update
 *       W <- W + L^B_i * Delta * (L^A_j)^T ,
 *   where L^A, L^B are the column-normalised (unit-diagonal) lower factors
 *   Cholesky(A^{-1}), Cholesky(B^{-1}).  The factors are inputs here; the
 *   Python side of the oracle forms them.
 *
 * "round" is replaced by "quantise to the nearest alphabet element"
 * (Sec. 3.1): an alphabet of consecutive integers {lo..hi} (symmetric
 * {-l..l} as in App. D, or the (b+1)-bit {-2^b..2^b-1} of Sec. 3.1) and a
 * scale per entry s_ij (per row and/or column, Sec. 3.1; the caller expands
 * row, group and column scales), i.e.
 *   c = clamp(rint(x), lo, hi),   x = W~_ij / s_ij,   v = s_ij * c.
 * Ties are broken half-to-even (App. B asks only for a fixed tie rule).
 * The paper's timed runs are float32 (Sec. 6), so the integer decision is
 * taken on x rounded to float32; x itself is reported in fp64.
 * A zero scale means the entry's alphabet is {0}.
 *
 * Optional tie forcing (the parity protocol): where the oracle's own x lies
 * within tie_window grid steps of a rounding boundary k+1/2 (k in
 * [lo, hi-1]), the code given in `forced` is adopted instead and the entry is
 * counted as excused; both choices are valid outputs of the sequential rule
 * up to the tie convention.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static int quantise_code(double x, int qlo, int qhi)
{
    float xf = (float)x;
    float r = rintf(xf);             /* half-to-even under the default FE mode */
    if (r > (float)qhi) r = (float)qhi;
    if (r < (float)qlo) r = (float)qlo;
    return (int)r;
}

static int near_boundary(double x, int qlo, int qhi, double window)
{
    if (!(window > 0.0)) return 0;
    /* boundaries are k + 1/2 for k = qlo .. qhi-1 */
    double k = floor(x);
    double d = fabs(x - (k + 0.5));
    if (d >= window) return 0;
    return (k >= qlo && k <= qhi - 1) ? 1 : 0;
}

/*
 * Alg. 2 (BaKron-naive) with quantise in place of round.
 *   W0  : m x n row-major input weights
 *   LA  : n x n row-major, unit lower triangular (normalised Cholesky(A^-1))
 *   LB  : m x m row-major, unit lower triangular (normalised Cholesky(B^-1))
 *   S   : m x n row-major per-entry scales (>= 0)
 *   qlo, qhi: the alphabet {qlo..qhi}
 *   forced: NULL, or m x n codes to adopt at near-boundary entries
 * Outputs: codes (m x n), V = s_ij * code (m x n), pre = x = W~/s (m x n; NaN
 * for zero scales), counters.  Returns 0, or -1 on allocation failure.
 * max_entries > 0 stops after that many entries in visiting order (a bounded
 * timing sample; later outputs are left untouched); <= 0 processes all.
 */
int oracle_babai_naive(int64_t m, int64_t n, const double *W0, const double *LA,
                       const double *LB, const double *S, int qlo, int qhi,
                       const int8_t *forced, double tie_window, int8_t *codes,
                       double *V, double *pre, int64_t *n_excused, int64_t *n_flip,
                       int64_t max_entries)
{
    double *W = (double *)malloc(sizeof(double) * (size_t)(m * n));
    double *LAT = (double *)malloc(sizeof(double) * (size_t)(n * n));
    if (!W || !LAT) { free(W); free(LAT); return -1; }
    memcpy(W, W0, sizeof(double) * (size_t)(m * n));
    /* LAT[j*n + q] = LA[q*n + j]: column j of L^A stored contiguously */
    for (int64_t q = 0; q < n; ++q)
        for (int64_t j = 0; j < n; ++j) LAT[j * n + q] = LA[q * n + j];
    int64_t exc = 0, flip = 0, done = 0;

    for (int64_t i = 0; i < m; ++i) {
        for (int64_t j = 0; j < n; ++j) {
            if (max_entries > 0 && done >= max_entries) goto out;
            ++done;
            const double s = S[i * n + j];
            const double w = W[i * n + j];
            int c;
            double x;
            if (s == 0.0) {
                c = 0;
                x = NAN;
            } else {
                x = w / s;
                c = quantise_code(x, qlo, qhi);
                if (forced && near_boundary(x, qlo, qhi, tie_window)) {
                    ++exc;
                    if ((int)forced[i * n + j] != c) ++flip;
                    c = (int)forced[i * n + j];
                }
            }
            const double v = s * (double)c;
            const double delta = v - w;
            codes[i * n + j] = (int8_t)c;
            V[i * n + j] = v;
            pre[i * n + j] = x;
            /* W <- W + L^B_i * delta * (L^A_j)^T ; nonzero only for p>=i, q>=j */
            const double *la = LAT + j * n;
            for (int64_t p = i; p < m; ++p) {
                const double t = LB[p * m + i] * delta;
                if (t == 0.0) continue;
                double *row = W + p * n;
                for (int64_t q = j; q < n; ++q) row[q] += t * la[q];
            }
        }
    }
out:
    free(W);
    free(LAT);
    if (n_excused) *n_excused = exc;
    if (n_flip) *n_flip = flip;
    return 0;
}

/*
 * Closed-form special case: A and B both AR(1) Toeplitz matrices
 * [rho^|i-j|] (no damping).  Then the normalised factor Cholesky(X^{-1}) is
 * I - rho * (sub-diagonal) (a consequence of the definitions in Sec. 3.1,
 * pinned in the tests), and the feedback of Eq. (1) reaches only the three
 * neighbours up, left and up-left:
 *   W~_pq = W0_pq - rhoB*E_{p-1,q} - rhoA*E_{p,q-1} + rhoA*rhoB*E_{p-1,q-1},
 *   E = V - W~.
 * O(mn) at any size; used as an exact reference for full-size structured runs.
 * Tie forcing as for oracle_babai_naive.
 */
int oracle_ar1_diffusion(int64_t m, int64_t n, const double *W0, double rhoA,
                         double rhoB, const double *S, int qlo, int qhi, const int8_t *forced,
                         double tie_window, int8_t *codes, double *V, double *pre,
                         int64_t *n_excused, int64_t *n_flip)
{
    double *E = (double *)malloc(sizeof(double) * (size_t)(m * n));
    if (!E) return -1;
    int64_t exc = 0, flip = 0;
    for (int64_t p = 0; p < m; ++p) {
        for (int64_t q = 0; q < n; ++q) {
            const double s = S[p * n + q];
            double wt = W0[p * n + q];
            if (p > 0) wt -= rhoB * E[(p - 1) * n + q];
            if (q > 0) wt -= rhoA * E[p * n + q - 1];
            if (p > 0 && q > 0) wt += rhoA * rhoB * E[(p - 1) * n + q - 1];
            int c;
            double x;
            if (s == 0.0) { c = 0; x = NAN; }
            else {
                x = wt / s;
                c = quantise_code(x, qlo, qhi);
                if (forced && near_boundary(x, qlo, qhi, tie_window)) {
                    ++exc;
                    if ((int)forced[p * n + q] != c) ++flip;
                    c = (int)forced[p * n + q];
                }
            }
            const double v = s * (double)c;
            codes[p * n + q] = (int8_t)c;
            V[p * n + q] = v;
            pre[p * n + q] = x;
            E[p * n + q] = v - wt;
        }
    }
    free(E);
    if (n_excused) *n_excused = exc;
    if (n_flip) *n_flip = flip;
    return 0;
}

/*
 * BaKron-recursive (Alg. 5, Sec. 3.4): the same row-major sequential rounding
 * as oracle_babai_naive, with the feedback batched by divide and conquer.
 * A block of rows [r0, r1) x columns [c0, c1) is solved by splitting its
 * larger dimension in half (at floor(./2): columns when it has fewer rows than
 * columns, else rows), solving the first half, adding the first half's errors
 * to the second half in one product, and solving the second half:
 *   columns:  W~[:, 2nd] += L^B[blk, blk] * E[:, 1st] * (L^A[2nd, 1st])^T
 *   rows:     W~[2nd, :] += L^B[2nd, 1st] * E[1st, :] * (L^A[blk, blk])^T
 * where E = V - W~ of the processed entries (the workspace keeps every
 * processed entry's pre-rounding value in place).  Blocks no larger than
 * base x base are solved by Alg. 2 restricted to the block.  By Thm 3.2 the
 * result is the same as Alg. 2's: every entry receives the same elementary
 * updates before it is quantised, only summed in another order.
 *
 * The products go to a BLAS dgemm passed in by the caller (Fortran interface,
 * column-major) when their size M*N*K reaches blas_min, and to a plain triple
 * loop otherwise (gemm may be NULL: loops only).
 *
 * Arguments and outputs as oracle_babai_naive (no early stop).  Returns 0, or
 * -1 on allocation failure.
 */
typedef void (*oracle_dgemm_t)(const char *ta, const char *tb, const int *m, const int *n,
                               const int *k, const double *alpha, const double *a,
                               const int *lda, const double *b, const int *ldb,
                               const double *beta, double *c, const int *ldc);

typedef struct {
    int64_t m, n;
    double *Wt;            /* workspace: W0 + feedback received; pre-rounding value once processed */
    double *E;             /* E = V - W~ of processed entries */
    double *T;             /* product scratch */
    const double *LA, *LB, *S;
    int qlo, qhi;
    const int8_t *forced;
    double tie_window;
    int8_t *codes;
    double *V, *pre;
    int64_t exc, flip, base, blas_min;
    oracle_dgemm_t gemm;
} rec_ctx;

/* row-major C (M x N, ldc) = beta * C + A (M x K, lda) * B (K x N, ldb) */
static void mm_nn(const rec_ctx *c, int64_t M, int64_t N, int64_t K, const double *A, int64_t lda,
                  const double *B, int64_t ldb, double *C, int64_t ldc, double beta)
{
    if (M <= 0 || N <= 0) return;
    if (c->gemm && M * N * K >= c->blas_min && K > 0) {
        const int m_ = (int)N, n_ = (int)M, k_ = (int)K, la = (int)ldb, lb = (int)lda, lc = (int)ldc;
        const double one = 1.0;
        c->gemm("N", "N", &m_, &n_, &k_, &one, B, &la, A, &lb, &beta, C, &lc);
        return;
    }
    for (int64_t i = 0; i < M; ++i) {
        double *ci = C + i * ldc;
        if (beta == 0.0) for (int64_t j = 0; j < N; ++j) ci[j] = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double a = A[i * lda + k];
            const double *bk = B + k * ldb;
            for (int64_t j = 0; j < N; ++j) ci[j] += a * bk[j];
        }
    }
}

/* row-major C (M x N, ldc) = beta * C + A (M x K, lda) * B^T, B (N x K, ldb) */
static void mm_nt(const rec_ctx *c, int64_t M, int64_t N, int64_t K, const double *A, int64_t lda,
                  const double *B, int64_t ldb, double *C, int64_t ldc, double beta)
{
    if (M <= 0 || N <= 0) return;
    if (c->gemm && M * N * K >= c->blas_min && K > 0) {
        const int m_ = (int)N, n_ = (int)M, k_ = (int)K, la = (int)ldb, lb = (int)lda, lc = (int)ldc;
        const double one = 1.0;
        c->gemm("T", "N", &m_, &n_, &k_, &one, B, &la, A, &lb, &beta, C, &lc);
        return;
    }
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j) {
            double acc = 0.0;
            for (int64_t k = 0; k < K; ++k) acc += A[i * lda + k] * B[j * ldb + k];
            C[i * ldc + j] = (beta == 0.0 ? 0.0 : beta * C[i * ldc + j]) + acc;   /* beta = 0: C is not read */
        }
}

/* Alg. 2 on the block [r0, r1) x [c0, c1) with the block's own factor parts */
static void rec_leaf(rec_ctx *c, int64_t r0, int64_t r1, int64_t c0, int64_t c1)
{
    const int64_t m = c->m, n = c->n;
    for (int64_t i = r0; i < r1; ++i) {
        for (int64_t j = c0; j < c1; ++j) {
            const double s = c->S[i * n + j];
            const double w = c->Wt[i * n + j];
            int code;
            double x;
            if (s == 0.0) {
                code = 0;
                x = NAN;
            } else {
                x = w / s;
                code = quantise_code(x, c->qlo, c->qhi);
                if (c->forced && near_boundary(x, c->qlo, c->qhi, c->tie_window)) {
                    ++c->exc;
                    if ((int)c->forced[i * n + j] != code) ++c->flip;
                    code = (int)c->forced[i * n + j];
                }
            }
            const double v = s * (double)code;
            const double delta = v - w;
            c->codes[i * n + j] = (int8_t)code;
            c->V[i * n + j] = v;
            c->pre[i * n + j] = x;
            c->E[i * n + j] = delta;
            /* rank-one update of the rest of the block (the entry itself keeps W~) */
            for (int64_t p = i; p < r1; ++p) {
                const double t = c->LB[p * m + i] * delta;
                double *row = c->Wt + p * n;
                for (int64_t q = (p == i ? j + 1 : j); q < c1; ++q) row[q] += t * c->LA[q * n + j];
            }
        }
    }
}

static void rec_solve(rec_ctx *c, int64_t r0, int64_t r1, int64_t c0, int64_t c1)
{
    const int64_t h = r1 - r0, w = c1 - c0, m = c->m, n = c->n;
    if (h <= 0 || w <= 0) return;
    if (h <= c->base && w <= c->base) {
        rec_leaf(c, r0, r1, c0, c1);
        return;
    }
    if (h < w) {
        const int64_t cm = c0 + w / 2, w1 = cm - c0, w2 = c1 - cm;
        rec_solve(c, r0, r1, c0, cm);
        /* T = L^B[blk, blk] E[blk, 1st];  W~[blk, 2nd] += T L^A[2nd, 1st]^T */
        mm_nn(c, h, w1, h, c->LB + r0 * m + r0, m, c->E + r0 * n + c0, n, c->T, w1, 0.0);
        mm_nt(c, h, w2, w1, c->T, w1, c->LA + cm * n + c0, n, c->Wt + r0 * n + cm, n, 1.0);
        rec_solve(c, r0, r1, cm, c1);
    } else {
        const int64_t rm = r0 + h / 2, h1 = rm - r0, h2 = r1 - rm;
        rec_solve(c, r0, rm, c0, c1);
        /* T = E[1st, blk] L^A[blk, blk]^T;  W~[2nd, blk] += L^B[2nd, 1st] T */
        mm_nt(c, h1, w, w, c->E + r0 * n + c0, n, c->LA + c0 * n + c0, n, c->T, w, 0.0);
        mm_nn(c, h2, w, h1, c->LB + rm * m + r0, m, c->T, w, c->Wt + rm * n + c0, n, 1.0);
        rec_solve(c, rm, r1, c0, c1);
    }
}

int oracle_babai_recursive(int64_t m, int64_t n, const double *W0, const double *LA,
                           const double *LB, const double *S, int qlo, int qhi,
                           const int8_t *forced, double tie_window, int8_t *codes, double *V,
                           double *pre, int64_t *n_excused, int64_t *n_flip, int64_t base,
                           int64_t blas_min, oracle_dgemm_t gemm)
{
    rec_ctx c;
    memset(&c, 0, sizeof(c));
    const size_t mn = (size_t)(m * n);
    c.Wt = (double *)malloc(sizeof(double) * mn);
    c.E = (double *)malloc(sizeof(double) * mn);
    c.T = (double *)malloc(sizeof(double) * (mn / 2 + 1));
    if (!c.Wt || !c.E || !c.T) { free(c.Wt); free(c.E); free(c.T); return -1; }
    memcpy(c.Wt, W0, sizeof(double) * mn);
    c.m = m; c.n = n; c.LA = LA; c.LB = LB; c.S = S; c.qlo = qlo; c.qhi = qhi;
    c.forced = forced; c.tie_window = tie_window; c.codes = codes; c.V = V; c.pre = pre;
    c.base = base < 1 ? 1 : base;
    c.blas_min = blas_min;
    c.gemm = gemm;
    rec_solve(&c, 0, m, 0, n);
    free(c.Wt); free(c.E); free(c.T);
    if (n_excused) *n_excused = c.exc;
    if (n_flip) *n_flip = c.flip;
    return 0;
}
