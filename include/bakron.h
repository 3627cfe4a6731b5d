/*
 * bakron.h -- C ABI of libbakron.so, an MI355X (gfx950) solver for BaKron
 * (arXiv 2608.06291): sequential Babai / GPTQ rounding of an m x n weight
 * matrix W under a Kronecker-factored Hessian A (x) B (A: n x n acting on the
 * input/column side, B: m x m acting on the output/row side).
 *
 * Problem statement (Sec. 3.2, Alg. 2; Alg. 6 is the solver; Thm 3.2 states
 * that all variants return the same output): given W, A, B, return the
 * quantised V obtained by visiting the entries in any order compatible with
 * "(i,j) before (p,q) whenever i<=p and j<=q", quantising each entry at its
 * current value, and feeding the error back to the later entries through
 * the unit-lower factors L^A = normalised Cholesky(A^-1) and
 * L^B = normalised Cholesky(B^-1).  "round" is replaced by quantisation to
 * an integer alphabet with scales per row, column or column group
 * (Sec. 3.1; App. D; see bakron_quantizer), ties to even.
 *
 * Conventions for every entry point:
 *   - All matrices are row-major, contiguous, fp32 unless stated otherwise.
 *   - Pointers marked "device" must be HIP device (or managed) memory on the
 *     device current at the call; the library never frees caller memory.
 *   - Errors found on the host (null pointers, bad sizes, bad bits, shape
 *     mismatch with the factor handle) return BAKRON_EINVAL before any work
 *     is enqueued.  HIP runtime failures return BAKRON_EHIP.  Allocation
 *     failures return BAKRON_ENOMEM.
 *   - Not thread-safe per handle: one solve at a time per bakron_factors
 *     (the handle owns the solve workspace).
 */
#ifndef BAKRON_H
#define BAKRON_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BAKRON_OK = 0,
    BAKRON_EINVAL = 1,   /* invalid argument (host-side validation)            */
    BAKRON_ENOTSPD = 2,  /* a damped factor matrix is not positive definite    */
    BAKRON_ENOMEM = 3,   /* device or host allocation failed                   */
    BAKRON_EHIP = 4      /* a HIP runtime call failed                          */
} bakron_status;

/* Opaque, library-owned, device-resident: the two normalised factors in
 * fp32 plus the cached solve workspace for the last (m, n) solved. */
typedef struct bakron_factors bakron_factors;

/* Quantisation alphabets (Sec. 3.1).  bits in [2, 8]; h = 2^(bits-1):
 *   SYMMETRIC   {-(h-1) .. h-1}  (App. D's {-l..l}, l = h - 1)
 *   ASYMMETRIC  {-h .. h-1}      (the (b+1)-bit alphabet {-2^b .. 2^b-1}) */
typedef enum {
    BAKRON_ALPHABET_SYMMETRIC = 0,
    BAKRON_ALPHABET_ASYMMETRIC = 1
} bakron_alphabet;

/* Quantiser (Sec. 3.1: scaling factors per row and/or column; App. D).
 * Entry (i, j) is quantised as c = clamp(rint(W~_ij / s_ij), lo, hi) and
 * V_ij = s_ij * c, with the scale
 *   s_ij = base_ij * (col_scale ? col_scale[j] : 1)     (one fp32 product)
 *   base_ij = group_size > 0 ? scale[i * ceil(n / group_size) + j / group_size]
 *                            : scale[i]
 * All scales must be finite and >= 0.  bakron_solve_debug checks this and
 * returns BAKRON_EINVAL otherwise; bakron_solve does not look (a device
 * reduction plus a synchronisation would break its asynchrony): there a
 * negative scale acts as 0 and a NaN scale gives NaN in V.  s_ij = 0 makes the
 * entry's alphabet {0}.  The caller
 * chooses the scales (App. D: max_j |W_ij| / l per row, optionally shrunk by
 * an MSE search: bakron_mse_scales).
 *   bits        alphabet size, in [2, 8]
 *   scale       DEVICE pointer: m per-row scales (group_size = 0), or an
 *               m x ceil(n / group_size) row-major matrix of per-(row, column
 *               group) scales
 *   alphabet    bakron_alphabet
 *   group_size  0, or the number of consecutive columns sharing a scale
 *   col_scale   DEVICE pointer to n per-column factors, or NULL
 * Zero-initialise the struct and set bits and scale for the per-row symmetric
 * quantiser of App. D. */
typedef struct {
    int32_t bits;
    const float *scale;
    int32_t alphabet;
    int32_t group_size;
    const float *col_scale;
} bakron_quantizer;

/*
 * bakron_factor -- damp and factor the Kronecker factors once (App. B: the
 * factorisations are done only at the top level).
 *
 *   A     device, n x n, symmetric positive semi-definite (undamped Gram)
 *   n     > 0
 *   B     device, m x m, symmetric PSD, or NULL for B = I_m (one-sided
 *         GPTQ, Sec. 1); then m may be any value and is not checked
 *   m     > 0 when B != NULL
 *   damp  >= 0, finite: X <- X + damp * mean(diag X) * I, each matrix with
 *         its own mean diagonal (Sec. 4 opening; App. D)
 *   stream  HIP stream the work is ordered on (0 = default stream).  The
 *         call also creates non-blocking streams of its own, forked from
 *         and joined back into `stream`, and destroys them before it
 *         returns: one for B (A and B are factored concurrently) and, for a
 *         factor of 8192 or more, one that runs its trailing updates one
 *         panel ahead
 *   out   receives the handle on BAKRON_OK; untouched otherwise
 *
 * Computes, in fp64 on the device, L^X = R_X^-1 diag(R_X) where
 * R_X = RevCholesky(X_d) (Sec. 3.1 definition); this equals the normalised
 * Cholesky(X_d^-1) of Alg. 2.  The fp32 result is kept in the handle.
 * Synchronises `stream` once to report BAKRON_ENOTSPD (a non-positive or
 * non-finite pivot); bakron_factors_error() then names the matrix and pivot.
 */
bakron_status bakron_factor(const float *A, int64_t n, const float *B, int64_t m,
                            float damp, hipStream_t stream, bakron_factors **out);

/*
 * bakron_solve -- the BaKron rounding (Alg. 6), asynchronous on `stream`.
 *
 *   W      device, m x n, not modified
 *   m, n   must equal the handle's sizes (n always; m when B was given)
 *   f      handle from bakron_factor
 *   q      quantiser (alphabet and scales, see bakron_quantizer)
 *   codes  device, m x n int8 output in the alphabet
 *   V      device, m x n fp32 output, V_ij = s_ij * codes_ij (one fp32 product)
 *
 * The first call for a given (m, n) allocates the workspace (about 8*m*n
 * bytes plus one int per 32 x 32 tile) and builds the launch plans (and may
 * synchronise the host, see below); later calls with the same (m, n)
 * allocate nothing and never synchronise the host.
 * The work is ordered after everything enqueued on `stream` before the call,
 * and everything enqueued on `stream` after it is ordered after the solve.
 * On a stream other than the legacy default stream (0 / hipStreamLegacy) the
 * solve may fork onto two streams of the handle, restricted to disjoint CU
 * sets (the divide-and-conquer pushes into later segments overlap with the
 * segment launches), and joins back into `stream` with events.  It does so
 * for the shapes where a cost model of both schedules, built when the shape
 * is first planned, favours the overlap (near-square layers up to about
 * 4096 x 4096), always with the environment variable BAKRON_DEFER=1, and
 * never with BAKRON_DEFER=0.  When the cost model picks the two-stream plan
 * (BAKRON_DEFER unset), the first solve of that shape on the handle runs
 * both plans twice each, times them with events on `stream` (one host
 * synchronisation), keeps the faster for the handle and returns the outputs
 * of its last run (not while per-launch profiling is enabled, which keeps
 * the model's choice).  On the legacy default stream, which
 * synchronises implicitly with such streams, and while `stream` is being
 * captured into a graph, everything runs on `stream`.  Unless
 * BAKRON_DEFER=0, the first solve planned on a device creates the two
 * CU-restricted streams, whichever plan its shape uses; the library keeps
 * them, with the launch plans, until the process exits.  The results are
 * bitwise the same either way.  Kernel faults surface as
 * BAKRON_EHIP on a later call or at the caller's synchronisation.
 *
 * With B = NULL at bakron_factor (B = I) the rows are independent and the
 * solve is Alg. 1 on every row (GPTQ with Hessian A, Sec. 1), all on
 * `stream`: the columns are taken in ranges of 1024; per range one launch
 * rounds it (one workgroup per 16 rows, blocks of 32 columns, the feedback
 * of the range's earlier blocks applied lazily) and one launch pushes its
 * errors into every later column of a working copy of W.  Its workspace is
 * 8 * ceil(m/16)*16 * ceil(n/32)*32 + 256 bytes, allocated on the first call
 * for a shape.  The environment variable BAKRON_GPTQ=0 at handle creation sends
 * such solves through the two-sided solver instead (same codes up to fp32
 * summation order).  Debug switches read at handle creation:
 * BAKRON_KNEAR=k (0..8) sets how many tile anti-diagonals a tile pulls from
 * itself instead of receiving them from node pushes; BAKRON_MACRO=4 or 2
 * forces 128 x 128 or 64 x 64 macro tiles in every node push;
 * BAKRON_GPTQ_RANGE=t (1..64) sets the one-sided range to t column tiles of
 * 32 (the tests use it to run several ranges on small shapes).
 */
bakron_status bakron_solve(const float *W, int64_t m, int64_t n, const bakron_factors *f,
                           bakron_quantizer q, int8_t *codes, float *V, hipStream_t stream);

/*
 * bakron_solve_debug -- bakron_solve that also writes, for every entry, the
 * pre-rounding value in grid units x_ij = W~_ij / s_ij (device, m x n fp32;
 * NaN where s_ij = 0), the value at which the entry was quantised.
 * Used to measure the numerical margin against the fp64 oracle.
 * Before enqueuing the solve it validates the quantiser's scales on the device
 * (every scale, and every col_scale factor, finite and >= 0) and synchronises
 * `stream` once to read the result: BAKRON_EINVAL (nothing else enqueued) if
 * one is negative, NaN or infinite.  Not capturable into a graph.
 */
bakron_status bakron_solve_debug(const float *W, int64_t m, int64_t n, const bakron_factors *f,
                                 bakron_quantizer q, int8_t *codes, float *V, float *pre,
                                 hipStream_t stream);

/*
 * bakron_solve_antidiag -- the same rounding by BaKron-antidiagonal (Alg. 3):
 * element anti-diagonal after element anti-diagonal, each rounded in
 * parallel and followed by the full update W~ += L^B * antidiag_k(E) * L^A^T.
 * Thm 3.2: the output equals bakron_solve's (up to fp32 summation order, i.e.
 * possibly different codes at entries within rounding noise of a boundary).
 * Its total work is O(m^2 n^2) against BaKron's O(mn(m+n)) (Table 1); it is
 * the reference point of the paper's runtime comparison (Table 3) and is
 * provided for that comparison, not as a production path.
 *
 * Arguments, layouts, ownership and errors as bakron_solve; pre may be NULL
 * (else as bakron_solve_debug).  Adds m + n - 1 pairs of launches on
 * `stream`.  Workspace: 4 * (m * n + 32 * ceil(m / 32)) bytes, allocated on the first
 * call for a shape and kept on the handle (separate from bakron_solve's).
 * Dimensions above 2^30 -> BAKRON_EINVAL.
 */
bakron_status bakron_solve_antidiag(const float *W, int64_t m, int64_t n, const bakron_factors *f,
                                    bakron_quantizer q, int8_t *codes, float *V, float *pre,
                                    hipStream_t stream);

/*
 * bakron_factor_blockdiag -- bakron_factor with an output factor that is
 * block-diagonal, B = blockdiag(B_0, .., B_{nblocks-1}): the per-head output
 * Grams of an attention projection assembled into one matrix spanning the
 * whole projection (App. D; BaKron puts no block structure on B, and
 * errors then never propagate between heads).
 *   B_blocks  device, nblocks x hb x hb (block h row-major at h * hb * hb),
 *             each symmetric PSD; m = nblocks * hb, at most 2^20
 *   damp      relative to the mean diagonal of the assembled B (all blocks),
 *             as in bakron_factor
 * Other arguments, results and errors as bakron_factor.  Assembles B in a
 * temporary m x m fp32 device buffer (freed before returning).
 */
bakron_status bakron_factor_blockdiag(const float *A, int64_t n, const float *B_blocks,
                                      int64_t nblocks, int64_t hb, float damp, hipStream_t stream,
                                      bakron_factors **out);

/*
 * bakron_mse_scales -- App. D's scale choice: for each row (group_size = 0)
 * or each (row, group of group_size columns) of W, the scale
 *   s_k = fl32(base * p_k),  base = fl32(max |W_ij| / hi),
 *   p_k = fl32(1 - maxshrink * k / grid),  k = 0 .. grid
 * (hi the alphabet's largest code) that minimises the squared error of
 * round-to-nearest quantisation, sum_j (W_ij - fl32(s_k c_ij))^2 with
 * c_ij = clamp(rint(fl32(W_ij / s_k)), lo, hi), summed in fp64; the first
 * minimum (least shrink) wins.  grid = 0 gives the max-abs scale.
 *   W          device, m x n fp32
 *   bits, alphabet  as bakron_quantizer
 *   group_size 0 or the column-group width
 *   grid       in [0, 255] (App. D's "shrink by up to 2x": maxshrink 0.5)
 *   maxshrink  in [0, 1)
 *   scale      device output: m floats, or m x ceil(n / group_size), usable
 *              as bakron_quantizer.scale
 * One launch on `stream`.  Errors: BAKRON_EINVAL for bad arguments.
 */
bakron_status bakron_mse_scales(const float *W, int64_t m, int64_t n, int32_t bits,
                                int32_t alphabet, int32_t group_size, int32_t grid,
                                double maxshrink, float *scale, hipStream_t stream);

/* Debug aid: with the environment variable BAKRON_POISON=1 when a handle is
 * created, every solve on it first fills the whole solve workspace (except the
 * sticky status word of bakron_solve_check) with NaN / -1 bytes (an extra
 * launch); the results are unchanged, which shows that no workspace word is
 * read before the solve writes it.  BAKRON_SPIN_LIMIT=k (1 <= k <= 2^22),
 * read at every solve, lowers the number of polls after which a tile-ordering
 * wait gives up, to exercise that path (bakron_solve_check) from the host. */

/* Frees the handle, its factors and its workspace (synchronises the device
 * work that used them).  NULL is a no-op. */
void bakron_factors_free(bakron_factors *f);

/* Static, never NULL. */
const char *bakron_status_string(bakron_status s);

/* Last error message recorded on the handle ("" if none); valid until the
 * next call on the handle. */
const char *bakron_factors_error(const bakron_factors *f);

/* Message of the last failed bakron_factor call in this thread ("" if none). */
const char *bakron_last_error(void);

/*
 * bakron_factor_export -- copy a normalised factor out of the handle as a
 * dense row-major fp32 matrix (which = 0: L^A, n x n; which = 1: L^B, m x m).
 * dst is a device pointer.  Asynchronous on `stream`.  For testing.
 */
bakron_status bakron_factor_export(const bakron_factors *f, int which, float *dst,
                                   hipStream_t stream);

/*
 * Measurement hook (not needed for solving).  While enabled, every
 * bakron_solve on the handle records a HIP event pair around each kernel
 * launch on its stream (which adds a few microseconds per launch).  After the
 * caller has synchronised that stream, bakron_profile_read fills stats[k] for
 * the last profiled solve, per kernel class k:
 *   0 workspace initialisation
 *   1 segment: rounding of the tiles of a range of tile anti-diagonals
 *     (Alg. 6 leaves and the lowest recursion levels), near field included
 *   2 node push: divide-and-conquer band update (Alg. 6 internal nodes)
 * with
 *   ms          summed launch durations
 *   launches    number of launches
 *   flops       algorithmic work: 2*32^3 flops per (source, target) tile pair
 *               fed back (Eq. (1)), plus the in-tile pairs of solved tiles;
 *               for class 0, bytes moved instead
 *   mfma_flops  flops executed on the matrix cores, zero-masked tiles included
 * Classes beyond nstats are dropped.  Returns BAKRON_EINVAL if no profiled
 * solve has been enqueued since enabling.
 */
typedef struct {
    double ms;
    int64_t launches;
    double flops;
    double mfma_flops;
} bakron_kernel_stat;

bakron_status bakron_profile_enable(bakron_factors *f, int on);
bakron_status bakron_profile_read(const bakron_factors *f, bakron_kernel_stat *stats, int nstats);

/*
 * bakron_solve_check -- diagnostic (not needed for solving; synchronises
 * `stream`).  The solve orders the tiles inside one launch with bounded
 * waits on per-tile ready flags.  *failed receives 1 if a wait gave up in any
 * solve on this handle since the last check (or since the workspace for the
 * current shape was created), else 0; the record is then cleared.  The record
 * is sticky on the device: once a wait has given up, every wait of every later
 * solve returns at once, so all outputs since the failure are invalid.  A
 * correct run never gives up: every awaited tile is held by a running
 * workgroup.
 */
bakron_status bakron_solve_check(const bakron_factors *f, hipStream_t stream, int32_t *failed);

/*
 * bakron_solve_noalloc -- bakron_solve for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results (bitwise), ordering on
 * `stream` and errors as bakron_solve, except:
 *   - the solve workspace (two fp32 tile arrays of 4 * 1024 * ceil(m/32) *
 *     ceil(n/32) bytes each, one int per tile and per segment launch) and the
 *     node work list live in a static device array of 136 MiB that the
 *     library holds on every GPU it runs on until the process exits; a layer
 *     whose workspace and work list do not fit (more than about 17000 32 x 32
 *     tiles, e.g. beyond 4096 x 4096) gives BAKRON_EINVAL before any work is
 *     enqueued;
 *   - it never calls hipMalloc / hipFree or any allocating routine; the first
 *     call for a shape builds its launch plan in host memory (cached), and
 *     every call copies the plan's work list (host -> device, a few MB at
 *     most) into the array on `stream`;
 *   - everything runs on `stream` (the one-stream plan; no fork);
 *   - the current device must be the handle's device (else BAKRON_EINVAL).
 * Every call on a GPU uses that GPU's one array, which keeps the last call's
 * contents: calls that overlap in time on one GPU (on different streams, or
 * from different threads or handles) race and give wrong results; serialise
 * them.  bakron_solve_check on a handle that ran this call also reports (and
 * clears) a give-up recorded in the array's status word, which is shared by
 * every handle on the GPU.
 */
bakron_status bakron_solve_noalloc(const float *W, int64_t m, int64_t n, const bakron_factors *f,
                                   bakron_quantizer q, int8_t *codes, float *V,
                                   hipStream_t stream);

/* ------------------------------------------------------------------------
 * Kronecker-factor construction from calibration samples (Sec. 4, App. A).
 *
 * The Hessian of a linear unit W (m x n) is an expectation of Kronecker
 * products, H = E[a a^T (x) b b^T], a the unit's input, b the gradient of the
 * loss with respect to its output (global case, both vectors) or the
 * MLP-local matrix b = D_g W_down^T.  Two Kronecker approximations H ~ A (x) B
 * are formed (App. A):
 *   K-FAC style     A = E[a a^T],               B = E[b b^T];
 *   Shampoo style   one power-iteration step of the best Kronecker
 *                   approximation (rearrangement of H) from A0 = I, B0 = I:
 *                   A = E[tr(b^T b) a a^T],     B = E[tr(a^T a) b b^T].
 * E is the sample mean (1/N) sum_k.  All of them reduce to one primitive,
 * the weighted masked Gram matrix C = s * (X^T diag(w) X) (.) M.
 *
 * Conventions of this group (in addition to those above):
 *   - sample matrices are N x d row-major fp32, one sample per row;
 *   - computed in fp32 on the matrix cores (fp32 products, fp32 sums); the
 *     summation order is fixed for a given device and shape, so repeated calls
 *     give bitwise the same result;
 *   - workspace protocol: with work == NULL the call stores the number of
 *     workspace bytes it needs in *work_bytes and does nothing else (no GPU
 *     work, pointers not checked); otherwise work is a device buffer of
 *     *work_bytes >= that size, 256-byte aligned, owned by the caller, which
 *     must not use it until the enqueued work completes.  The size depends on
 *     the sizes and on the CU count of the current device;
 *   - asynchronous on `stream`; error messages via bakron_last_error().
 * ------------------------------------------------------------------------ */

typedef enum {
    BAKRON_KFAC = 0,     /* A = E[a a^T],           B = E[b b^T]           */
    BAKRON_SHAMPOO = 1   /* A = E[tr(b^T b) a a^T], B = E[tr(a^T a) b b^T] */
} bakron_kron_style;

/*
 * bakron_gram -- C = s * (X^T diag(w) X) (.) M, i.e.
 *   C_ij = s * M_ij * sum_k w_k X_ki X_kj      (i, j < d)
 * the Gram accumulation of the Hessian factors (Sec. 4; App. A).
 *
 *   X   device, N x d;  N >= 0 (N = 0 gives C = 0), 0 <= d <= 2^17
 *   w   device, N per-sample weights, or NULL for w = 1
 *   s   scale (1/N for a sample mean)
 *   M   device, d x d entrywise factor, or NULL for M = 1; may be the same
 *       buffer as C (then it is overwritten with the result)
 *   C   device, d x d output, both triangles written
 * Two launches.  Errors: BAKRON_EINVAL for bad sizes, NULL X (N, d > 0) or C
 * (d > 0), or a bad workspace.
 */
bakron_status bakron_gram(const float *X, int64_t N, int64_t d, const float *w, float s,
                          const float *M, float *C, void *work, size_t *work_bytes,
                          hipStream_t stream);

/*
 * bakron_sample_weights -- w_k = sum_i c_i X_ki^2 for k < N: the per-sample
 * Shampoo weights of App. A (c = NULL: tr(a^T a) = |a_k|^2 of vector
 * samples; c = diag(W_down^T W_down): the MLP-local tr(b^T b) =
 * g^T diag(W_down^T W_down) g).
 *   X  device, N x d;  c  device, d floats, or NULL for c = 1;  w  device, N.
 * One launch, no workspace.
 */
bakron_status bakron_sample_weights(const float *X, int64_t N, int64_t d, const float *c, float *w,
                                    hipStream_t stream);

/*
 * bakron_kron_factors -- Kronecker factors of a global (backpropagated)
 * Hessian from N paired vector samples (Sec. 4; App. A):
 *   a  device, N x n (inputs of the unit)
 *   b  device, N x m (gradients at the unit's output)
 *   style  bakron_kron_style
 *   A  device, n x n output;  B  device, m x m output
 * N >= 1, n, m in [1, 2^17].  Workspace as above.
 */
bakron_status bakron_kron_factors(const float *a, const float *b, int64_t N, int64_t n, int64_t m,
                                  int32_t style, float *A, float *B, void *work, size_t *work_bytes,
                                  hipStream_t stream);

/*
 * bakron_mlp_local_factors -- Kronecker factors of the MLP-local Hessians of
 * a gated MLP, MLP(x) = W_down (W_up x (.) sigma(W_gate x)) (App. A):
 *   H_up   = E[x x^T (x) (g g^T (.) W_down^T W_down)],  g = sigma(W_gate x)
 *   H_gate = E[x x^T (x) (f f^T (.) W_down^T W_down)],  f = sigma'(W_gate x) (.) W_up x
 * i.e. b = D_g W_down^T, b b^T = g g^T (.) D^T D and tr(b^T b) =
 * g^T diag(D^T D) g, with D = W_down:
 *   K-FAC:    A = E[x x^T],                  B = E[g g^T] (.) D^T D
 *   Shampoo:  A = E[(g^T diag(D^T D) g) x x^T], B = E[|x|^2 g g^T] (.) D^T D
 *
 *   x  device, N x dm (inputs of the MLP)
 *   g  device, N x dff: the features g (for W_up) or f (for W_gate)
 *   D  device, dm x dff: W_down
 *   A  device, dm x dm output;  B  device, dff x dff output
 * N >= 1, dm, dff in [1, 2^17].  Workspace as above.
 */
bakron_status bakron_mlp_local_factors(const float *x, const float *g, const float *D, int64_t N,
                                       int64_t dm, int64_t dff, int32_t style, float *A, float *B,
                                       void *work, size_t *work_bytes, hipStream_t stream);

/*
 * bakron_quadform_weights -- w_k = x_k^T M x_k for every sample (row) x_k of
 * X: the per-sample weights tr(b^T B^(i) b) of the later Shampoo power steps
 * (App. A: A^(i+1) = E[tr(b^T B^(i) b) a a^T]).
 *   X  device, N x d;  M  device, d x d, SYMMETRIC (M_tj is read as M_jt);
 *   w  device, N outputs.  0 <= d <= 2^17.
 * Two launches (X M on fp32 MFMA with the row sums fused, then the sum over
 * column blocks in a fixed order).  Workspace as above: ceil(d / 128) * N
 * floats.
 */
bakron_status bakron_quadform_weights(const float *X, int64_t N, int64_t d, const float *M,
                                      float *w, void *work, size_t *work_bytes, hipStream_t stream);

/*
 * bakron_kron_factors_iter, bakron_mlp_local_factors_iter -- the Shampoo-style
 * factors after `iters` unnormalised power steps on the rearranged Hessian
 * from A^(0) = I, B^(0) = I (App. A; iters = 1 is BAKRON_SHAMPOO):
 *   A^(i+1) = E[tr(b^T B^(i) b) a a^T],   B^(i+1) = E[tr(a^T A^(i) a) b b^T]
 * with, in the MLP-local case (b = D_g W_down^T, D = W_down),
 *   tr(b^T X b) = g^T (X (.) D^T D) g,   b b^T = (g g^T) (.) D^T D.
 * Each step is one more pass over the calibration samples.  The iterates are
 * not normalised (the rounding is invariant to scaling A or B); their size
 * grows geometrically with iters, so keep iters small (<= 64 accepted).
 * Arguments otherwise as bakron_kron_factors / bakron_mlp_local_factors; the
 * MLP-local workspace holds one more dff x dff matrix when iters > 1.
 */
bakron_status bakron_kron_factors_iter(const float *a, const float *b, int64_t N, int64_t n,
                                       int64_t m, int32_t iters, float *A, float *B, void *work,
                                       size_t *work_bytes, hipStream_t stream);
bakron_status bakron_mlp_local_factors_iter(const float *x, const float *g, const float *D,
                                            int64_t N, int64_t dm, int64_t dff, int32_t iters,
                                            float *A, float *B, void *work, size_t *work_bytes,
                                            hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* BAKRON_H */
