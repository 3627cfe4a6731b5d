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
