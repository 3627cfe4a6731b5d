"""fp64 CPU oracle for the BaKron solver -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline leg
may import this module.  It shares no code with the HIP solver in
``paper_2608_06291_amd/``; neither imports the other.

Contents, each following a passage of arXiv 2608.06291:

* :func:`damp` -- regularisation: add a multiple of the mean diagonal to the
  diagonal (Sec. 4 opening; App. D uses 0.5, the workloads here use 0.01).
* :func:`normalized_factor` -- ``Cholesky(X^-1)`` with every column divided by
  its diagonal entry (Alg. 1 / Alg. 2, first two lines).  Literal route:
  explicit inverse, then Cholesky (LAPACK via numpy, fp64).
* :func:`babai` -- the sequential rounding itself: Alg. 2 (BaKron-naive) in C
  (``babai.c``), optionally tie-forced.
* :func:`babai_recursive` -- the same rounding sequence by Alg. 5
  (BaKron-recursive, Sec. 3.4): split the larger dimension in half, solve
  the first half, feed its errors to the second half in one product (fp64
  BLAS-3), solve the second half; Alg. 2 on small blocks.  O(mn(m+n)) work,
  so it reaches the full-size layers.
* :func:`normalized_factor_rev` -- the same factor by the RevCholesky route
  (Sec. 3.1 definition): L = R^-1 diag(R), for sizes where the explicit
  inverse of the literal route is too slow; the two routes are pinned equal.
* :func:`ar1_diffusion` -- exact O(mn) special case for AR(1) Toeplitz A, B.
* :func:`rev_cholesky` / :func:`certificate` -- closed-form check of any
  candidate output: by Eq. (1) the final workspace is
  ``V = W0 + L^B E (L^A)^T``, so ``E = R^_B (V - W0) R^_A^T`` with
  ``R^_X = (L^X)^-1`` = RevCholesky(X) with rows divided by their diagonal
  (Sec. 3.1 definition of RevCholesky), and the pre-rounding values are
  ``W~ = V - E``.  V is a valid sequential-rounding output iff
  ``V = quantise(W~)`` entrywise up to ties.
* :func:`alphabet_bounds`, :func:`entry_scales` -- the quantiser of Sec. 3.1:
  an alphabet {lo..hi} (symmetric, or the (b+1)-bit {-2^b..2^b-1}) and
  scales per row and/or column (row or column-group scales times column
  factors).
* :func:`mse_scales` -- App. D's scale choice: max-abs per row over the
  largest positive code, shrunk by up to 2x where that lowers the row's
  squared round-to-nearest error.
* :func:`objective` -- ``tr((W - V)^T B (W - V) A)``, which equals
  ``vec(W - V)^T (A (x) B) vec(W - V)`` by Prop. 3.1.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "babai.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile babai.c into liboracle.so with gcc (plain C, -O2, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fno-fast-math",
             "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        dp = ctypes.POINTER(ctypes.c_double)
        i8p = ctypes.POINTER(ctypes.c_int8)
        i64p = ctypes.POINTER(ctypes.c_int64)
        lib.oracle_babai_naive.restype = ctypes.c_int
        lib.oracle_babai_naive.argtypes = [
            ctypes.c_int64, ctypes.c_int64, dp, dp, dp, dp, ctypes.c_int, ctypes.c_int,
            i8p, ctypes.c_double, i8p, dp, dp, i64p, i64p, ctypes.c_int64]
        lib.oracle_babai_recursive.restype = ctypes.c_int
        lib.oracle_babai_recursive.argtypes = [
            ctypes.c_int64, ctypes.c_int64, dp, dp, dp, dp, ctypes.c_int, ctypes.c_int,
            i8p, ctypes.c_double, i8p, dp, dp, i64p, i64p, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_void_p]
        lib.oracle_ar1_diffusion.restype = ctypes.c_int
        lib.oracle_ar1_diffusion.argtypes = [
            ctypes.c_int64, ctypes.c_int64, dp, ctypes.c_double, ctypes.c_double,
            dp, ctypes.c_int, ctypes.c_int, i8p, ctypes.c_double, i8p, dp, dp, i64p, i64p]
        _lib = lib
    return _lib


def _dptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _i8ptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int8))


def qmax_of_bits(bits: int) -> int:
    """Symmetric alphabet {-l..l} with l = 2^(bits-1) - 1 (App. D uses l = 3)."""
    return (1 << (int(bits) - 1)) - 1


def alphabet_bounds(bits: int, alphabet: str = "sym"):
    """(lo, hi) of the quantisation alphabet {lo..hi} (Sec. 3.1): "sym" is
    {-l..l}, l = 2^(bits-1) - 1 (App. D); "asym" is the (b+1)-bit alphabet
    {-2^b .. 2^b - 1} with b = bits - 1."""
    if alphabet == "sym":
        l = qmax_of_bits(bits)
        return -l, l
    if alphabet == "asym":
        h = 1 << (int(bits) - 1)
        return -h, h - 1
    raise ValueError(alphabet)


def entry_scales(scale, m: int, n: int, group_size: int = 0, col_scale=None) -> np.ndarray:
    """Per-entry scales s_ij (Sec. 3.1: factors per row and/or column).

    scale: m per-row scales, or with group_size g > 0 an m x ceil(n/g) matrix
    of per-(row, column group) scales (group of column j: j // g); an m x n
    array is taken as given.  col_scale: None or n per-column factors, which
    multiply the row/group scale in fp32 (the stored scales are fp32).
    Returned as fp64 holding the fp32 values."""
    S = np.asarray(scale, dtype=np.float32)
    if S.shape == (m, n) and group_size == 0 and col_scale is None:
        return S.astype(np.float64)
    if group_size > 0:
        G = -(-n // group_size)
        base = S.reshape(m, G)[:, np.arange(n) // group_size]
    else:
        base = np.broadcast_to(S.reshape(m, 1), (m, n))
    if col_scale is not None:
        base = (base * np.asarray(col_scale, dtype=np.float32).reshape(1, n)).astype(np.float32)
    return np.ascontiguousarray(base, dtype=np.float64)


def damp(X, lam: float) -> np.ndarray:
    """X + lam * mean(diag X) * I in fp64 (Sec. 4 opening, App. D)."""
    X = np.asarray(X, dtype=np.float64)
    d = X.shape[0]
    out = X.copy()
    out[np.diag_indices(d)] += float(lam) * float(np.mean(np.diag(X)))
    return out


def normalized_factor(X, lam: float) -> np.ndarray:
    """Unit-lower L = Cholesky(X_d^-1) with column j divided by L_jj (Alg. 2)."""
    Xd = damp(X, lam)
    Linv = np.linalg.cholesky(np.linalg.inv(Xd))
    return Linv / np.diag(Linv)[None, :]


def rev_cholesky(Xd, fortran: bool = False) -> np.ndarray:
    """Lower R with positive diagonal and R^T R = Xd (Sec. 3.1 definition).

    With P the reversal permutation, P Xd P = C C^T gives R = P C^T P.
    C is LAPACK's fp64 Cholesky (dpotrf) of the column-major copy of P Xd P.
    The result is row-major, or column-major with fortran=True."""
    from scipy.linalg import lapack
    Xd = np.asarray(Xd, dtype=np.float64)
    C, info = lapack.dpotrf(np.asfortranarray(Xd[::-1, ::-1]), lower=1, clean=1, overwrite_a=1)
    if info != 0:
        raise np.linalg.LinAlgError(f"dpotrf info {info}: not positive definite")
    R = C[::-1, ::-1].T
    return np.asfortranarray(R) if fortran else np.ascontiguousarray(R)


def babai(W, LA, LB, scale, bits: int, forced=None, tie_window: float = 0.0,
          max_entries: int = 0, alphabet: str = "sym"):
    """Sequential rounding of Alg. 2 (row-major), in C.  Returns a dict with
    codes (int8), V (fp64), pre (x = W~/s, fp64), n_excused, n_flip.
    scale: per-row (m) or per-entry (m x n, see :func:`entry_scales`).
    max_entries > 0 stops after that many entries (timing samples only)."""
    lib = _load()
    W = np.ascontiguousarray(W, dtype=np.float64)
    m, n = W.shape
    LA = np.ascontiguousarray(LA, dtype=np.float64)
    LB = np.ascontiguousarray(LB, dtype=np.float64)
    s = entry_scales(scale, m, n)
    qlo, qhi = alphabet_bounds(bits, alphabet)
    assert LA.shape == (n, n) and LB.shape == (m, m)
    codes = np.zeros((m, n), np.int8)
    V = np.zeros((m, n), np.float64)
    pre = np.zeros((m, n), np.float64)
    exc = ctypes.c_int64(0)
    flip = ctypes.c_int64(0)
    fp = None
    if forced is not None:
        forced = np.ascontiguousarray(forced, dtype=np.int8)
        assert forced.shape == (m, n)
        fp = _i8ptr(forced)
    rc = lib.oracle_babai_naive(m, n, _dptr(W), _dptr(LA), _dptr(LB), _dptr(s),
                                qlo, qhi, fp, float(tie_window),
                                _i8ptr(codes), _dptr(V), _dptr(pre),
                                ctypes.byref(exc), ctypes.byref(flip), int(max_entries))
    if rc != 0:
        raise MemoryError("oracle_babai_naive: allocation failed")
    return dict(codes=codes, V=V, pre=pre, n_excused=int(exc.value),
                n_flip=int(flip.value))


def blas_dgemm_pointer():
    """Address of the fp64 BLAS dgemm (Fortran interface) that scipy exports
    for compiled extensions; used by babai_recursive for its products."""
    import scipy.linalg.cython_blas as cb
    cap = cb.__pyx_capi__["dgemm"]
    get_name = ctypes.pythonapi.PyCapsule_GetName
    get_name.restype = ctypes.c_char_p
    get_name.argtypes = [ctypes.py_object]
    get_ptr = ctypes.pythonapi.PyCapsule_GetPointer
    get_ptr.restype = ctypes.c_void_p
    get_ptr.argtypes = [ctypes.py_object, ctypes.c_char_p]
    return get_ptr(cap, get_name(cap))


def blas_threads() -> int:
    """Threads of the BLAS behind blas_dgemm_pointer (scipy's OpenBLAS)."""
    try:
        import threadpoolctl
        for info in threadpoolctl.threadpool_info():
            if info.get("user_api") == "blas" and "scipy.libs" in info.get("filepath", ""):
                return int(info["num_threads"])
        for info in threadpoolctl.threadpool_info():
            if info.get("user_api") == "blas":
                return int(info["num_threads"])
    except Exception:
        pass
    return 1


def babai_recursive(W, LA, LB, scale, bits: int, forced=None, tie_window: float = 0.0,
                    alphabet: str = "sym", base: int = 8, blas_min: int = 32768,
                    use_blas: bool = True):
    """The rounding of :func:`babai` (same codes) by Alg. 5 in C: feedback
    batched by divide and conquer, products through fp64 BLAS dgemm when
    M*N*K >= blas_min (plain loops below, or everywhere if not use_blas),
    Alg. 2 on blocks of at most base x base.  Returns the same dict."""
    lib = _load()
    W = np.ascontiguousarray(W, dtype=np.float64)
    m, n = W.shape
    LA = np.ascontiguousarray(LA, dtype=np.float64)
    LB = np.ascontiguousarray(LB, dtype=np.float64)
    s = entry_scales(scale, m, n)
    qlo, qhi = alphabet_bounds(bits, alphabet)
    assert LA.shape == (n, n) and LB.shape == (m, m)
    codes = np.zeros((m, n), np.int8)
    V = np.zeros((m, n), np.float64)
    pre = np.zeros((m, n), np.float64)
    exc = ctypes.c_int64(0)
    flip = ctypes.c_int64(0)
    fp = None
    if forced is not None:
        forced = np.ascontiguousarray(forced, dtype=np.int8)
        assert forced.shape == (m, n)
        fp = _i8ptr(forced)
    gemm = blas_dgemm_pointer() if use_blas else None
    rc = lib.oracle_babai_recursive(m, n, _dptr(W), _dptr(LA), _dptr(LB), _dptr(s), qlo, qhi, fp,
                                    float(tie_window), _i8ptr(codes), _dptr(V), _dptr(pre),
                                    ctypes.byref(exc), ctypes.byref(flip), int(base),
                                    int(blas_min), gemm)
    if rc != 0:
        raise MemoryError("oracle_babai_recursive: allocation failed")
    return dict(codes=codes, V=V, pre=pre, n_excused=int(exc.value), n_flip=int(flip.value))


def normalized_factor_rev(X, lam: float) -> np.ndarray:
    """The factor of :func:`normalized_factor` by the RevCholesky route:
    R = RevCholesky(X_d) (lower, R^T R = X_d, Sec. 3.1), L = R^-1 diag(R).
    Equal in exact arithmetic to normalised Cholesky(X_d^-1): X_d^-1 =
    R^-1 R^-T with R^-1 lower, so R^-1 D^-1 (D = diag(R^-1) = diag(R)^-1) is
    the Cholesky factor, and normalising its columns gives R^-1 diag(R)."""
    from scipy.linalg import lapack
    R = rev_cholesky(damp(X, lam), fortran=True)
    d = np.diag(R).copy()
    Rinv, info = lapack.dtrtri(R, lower=1, overwrite_c=1)
    if info != 0:
        raise np.linalg.LinAlgError(f"dtrtri info {info}")
    del R
    L = np.tril(Rinv)
    L *= d[None, :]
    return np.ascontiguousarray(L)


def solve(W, A, B, damp_lambda: float, scale, bits: int, forced=None,
          tie_window: float = 0.0, alphabet: str = "sym", method: str = "naive"):
    """Factors by the literal route, then :func:`babai` (method "naive",
    Alg. 2) or :func:`babai_recursive` (method "recursive", Alg. 5; the
    same codes).  B=None means I_m."""
    W = np.asarray(W, dtype=np.float64)
    m, n = W.shape
    LA = normalized_factor(A, damp_lambda)
    LB = np.eye(m) if B is None else normalized_factor(B, damp_lambda)
    run = {"naive": babai, "recursive": babai_recursive}[method]
    return run(W, LA, LB, scale, bits, forced=forced, tie_window=tie_window, alphabet=alphabet)


def naive_macs(m: int, n: int, entries: int | None = None) -> float:
    """Multiply-adds of Alg. 2's rank-one updates: entry (i, j) updates the
    (m - i) x (n - j) block below-right of it; over the first `entries`
    entries in row-major order (all if None)."""
    if entries is None or entries >= m * n:
        return m * (m + 1) / 2.0 * n * (n + 1) / 2.0
    full_rows, rest = divmod(int(entries), n)
    row_sum = n * (n + 1) / 2.0
    total = sum((m - i) * row_sum for i in range(full_rows))
    total += (m - full_rows) * sum(n - j for j in range(rest))
    return float(total)


def ar1_diffusion(W, rhoA: float, rhoB: float, scale, bits: int, forced=None,
                  tie_window: float = 0.0, alphabet: str = "sym"):
    """Exact output for A = [rhoA^|i-j|], B = [rhoB^|i-j|] without damping."""
    lib = _load()
    W = np.ascontiguousarray(W, dtype=np.float64)
    m, n = W.shape
    s = entry_scales(scale, m, n)
    qlo, qhi = alphabet_bounds(bits, alphabet)
    codes = np.zeros((m, n), np.int8)
    V = np.zeros((m, n), np.float64)
    pre = np.zeros((m, n), np.float64)
    exc = ctypes.c_int64(0)
    flip = ctypes.c_int64(0)
    fp = None
    if forced is not None:
        forced = np.ascontiguousarray(forced, dtype=np.int8)
        assert forced.shape == (m, n)
        fp = _i8ptr(forced)
    rc = lib.oracle_ar1_diffusion(m, n, _dptr(W), float(rhoA), float(rhoB), _dptr(s),
                                  qlo, qhi, fp, float(tie_window), _i8ptr(codes),
                                  _dptr(V), _dptr(pre), ctypes.byref(exc), ctypes.byref(flip))
    if rc != 0:
        raise MemoryError("oracle_ar1_diffusion: allocation failed")
    return dict(codes=codes, V=V, pre=pre, n_excused=int(exc.value), n_flip=int(flip.value))


def near_boundary(x, bits: int, window: float, alphabet: str = "sym") -> np.ndarray:
    """Entries whose grid value x lies within `window` of a boundary k+1/2,
    k in [lo, hi-1]; NaN (zero scale) is never near a boundary."""
    lo, hi = alphabet_bounds(bits, alphabet)
    x = np.asarray(x, dtype=np.float64)
    k = np.floor(x)
    with np.errstate(invalid="ignore"):
        near = (np.abs(x - (k + 0.5)) < window) & (k >= lo) & (k <= hi - 1)
    return near & np.isfinite(x)


def quantise_codes(x, bits: int, alphabet: str = "sym") -> np.ndarray:
    """clamp(rint(float32(x)), lo, hi); NaN (zero scale) maps to 0."""
    lo, hi = alphabet_bounds(bits, alphabet)
    xf = np.asarray(x, dtype=np.float64).astype(np.float32)
    with np.errstate(invalid="ignore"):
        c = np.clip(np.rint(xf), lo, hi)
    c = np.where(np.isfinite(xf), c, 0)
    return c.astype(np.int8)


def certificate(W, A, B, damp_lambda: float, scale, codes, bits: int,
                rows=None, RA=None, RB=None):
    """Pre-rounding values implied by a candidate output (closed form).

    Returns x = W~/s for the requested rows (all rows if None), computed as
    W~ = V - R^_B (V - W0) R^_A^T with V = s_i * codes in fp64.  RA/RB may
    pass precomputed RevCholesky factors of the damped matrices.
    """
    W = np.asarray(W, dtype=np.float64)
    m, n = W.shape
    S = entry_scales(scale, m, n)
    V = S * np.asarray(codes, dtype=np.float64)
    if RA is None:
        RA = rev_cholesky(damp(A, damp_lambda))
    if B is None:
        RB = np.eye(m)
    elif RB is None:
        RB = rev_cholesky(damp(B, damp_lambda))
    RhA = RA / np.diag(RA)[:, None]
    RhB = RB / np.diag(RB)[:, None]
    D = V - W
    if rows is None:
        E = RhB @ D @ RhA.T
        Vr = V
    else:
        rows = np.asarray(rows)
        E = (RhB[rows, :] @ D) @ RhA.T
        Vr = V[rows]
    Wt = Vr - E
    Sr = S if rows is None else S[rows]
    with np.errstate(divide="ignore", invalid="ignore"):
        x = Wt / Sr
    x[Sr == 0.0] = np.nan
    return x


def certify(W, A, B, damp_lambda: float, scale, codes, bits: int, window: float = 1e-4,
            alphabet: str = "sym", row_block: int = 4096):
    """Certificate, verdict and objective of a candidate output in one pass,
    for every entry of a full-size layer (fp64, BLAS-3 triangular products).

    With R_X = RevCholesky(X_d) (lower, R_X^T R_X = X_d), D = V - W0 and
    T = R_B D R_A^T:
      * pre-rounding values (closed form of Eq. (1), as :func:`certificate`):
        W~ = V - diag(R_B)^-1 T diag(R_A)^-1, x = W~ / s;
      * objective (Prop. 3.1): tr(D^T B_d D A_d) = |R_B D R_A^T|_F^2 = |T|_F^2.
    Returns dict(verdict of :func:`verdict`, objective, x (m x n fp64)).
    B = None means B = I.  Rows of T are formed in blocks of row_block."""
    from scipy.linalg import blas
    W = np.asarray(W, dtype=np.float64)
    m, n = W.shape
    S = entry_scales(scale, m, n)
    V = S * np.asarray(codes, dtype=np.float64)
    RA = rev_cholesky(damp(A, damp_lambda))
    dA = np.diag(RA).copy()
    D = V - W
    # U = D R_A^T (right triangular product), column-major for BLAS
    U = blas.dtrmm(1.0, np.asfortranarray(RA), np.asfortranarray(D), side=1, lower=1, trans_a=1)
    del D
    if B is None:
        T = np.ascontiguousarray(U)
        dB = np.ones(m)
    else:
        RB = rev_cholesky(damp(B, damp_lambda))
        dB = np.diag(RB).copy()
        T = np.empty((m, n), np.float64)
        # T[rows] = R_B[rows, :r1] U[:r1]: R_B lower, so row block [r0, r1)
        # needs only the first r1 rows of U
        for r0 in range(0, m, row_block):
            r1 = min(m, r0 + row_block)
            T[r0:r1] = RB[r0:r1, :r1] @ U[:r1]
        del RB
    del U
    obj = float(np.sum(T * T))
    Wt = V - T / dB[:, None] / dA[None, :]
    del T
    with np.errstate(divide="ignore", invalid="ignore"):
        x = Wt / S
    x[S == 0.0] = np.nan
    return dict(verdict=verdict(codes, x, bits, window, alphabet), objective=obj, x=x)


def verdict(codes, x, bits: int, window: float = 1e-4, alphabet: str = "sym"):
    """Compare candidate codes with quantise(x) along the candidate's own
    trajectory.  violations: differ and not near a boundary (must be 0);
    flips: differ at near-boundary entries (excused, rate-limited)."""
    codes = np.asarray(codes)
    own = quantise_codes(x, bits, alphabet)
    near = near_boundary(x, bits, window, alphabet)
    diff = own != codes
    return dict(violations=int(np.count_nonzero(diff & ~near)),
                flips=int(np.count_nonzero(diff & near)),
                near=int(np.count_nonzero(near)),
                total=int(codes.size))


def objective(W, V, A, B, damp_lambda: float) -> float:
    """tr((W - V)^T B_d (W - V) A_d) in fp64 with the damped factors."""
    D = np.asarray(W, dtype=np.float64) - np.asarray(V, dtype=np.float64)
    Ad = damp(A, damp_lambda)
    BD = D if B is None else damp(B, damp_lambda) @ D
    return float(np.sum(BD * (D @ Ad)))


def mse_scale_candidates(W, bits: int, alphabet: str = "sym", grid: int = 100,
                         maxshrink: float = 0.5) -> np.ndarray:
    """Candidate scales of every row, m x (grid + 1), fp32 values (App. D):
    s_k = fl32(fl32(max_j |W_ij| / hi) * p_k), p_k = fl32(1 - maxshrink k / grid),
    hi the largest positive code of the alphabet (grid = 0: s = the base)."""
    W32 = np.asarray(W, dtype=np.float32)
    _, hi = alphabet_bounds(bits, alphabet)
    base = (np.max(np.abs(W32), axis=1) / np.float32(hi)).astype(np.float32)
    if grid == 0:
        return base[:, None].copy()
    p = np.array([1.0 - maxshrink * k / grid for k in range(grid + 1)]).astype(np.float32)
    return (base[:, None] * p[None, :]).astype(np.float32)


def mse_scales(W, bits: int, alphabet: str = "sym", grid: int = 100,
               maxshrink: float = 0.5, group_size: int = 0):
    """App. D: per row, the candidate scale (max-abs over the largest code,
    shrunk by p_k in [1 - maxshrink, 1]) whose round-to-nearest quantisation
    has the least squared error sum_j (W_ij - fl32(s c_ij))^2, with
    c_ij = clamp(rint(fl32(W_ij / s)), lo, hi); the first (least shrunk)
    candidate wins ties.  With group_size g > 0 the same per (row, group of g
    columns), giving m x ceil(n/g) scales.  Returns (scales fp32, errors fp64
    (rows x segments x (grid + 1)) or (m, grid + 1) without groups)."""
    W32 = np.asarray(W, dtype=np.float32)
    m, n = W32.shape
    if group_size > 0:
        outs = [mse_scales(W32[:, g0:g0 + group_size], bits, alphabet, grid, maxshrink)
                for g0 in range(0, n, group_size)]
        return (np.stack([o[0] for o in outs], axis=1),
                np.stack([o[1] for o in outs], axis=1))
    lo, hi = alphabet_bounds(bits, alphabet)
    cand = mse_scale_candidates(W32, bits, alphabet, grid, maxshrink)
    err = np.zeros((m, cand.shape[1]), np.float64)
    for k in range(cand.shape[1]):
        s = cand[:, k:k + 1]
        with np.errstate(divide="ignore", invalid="ignore"):
            x = (W32 / s).astype(np.float32)
        c = np.where(s > 0, np.clip(np.rint(x), lo, hi), 0).astype(np.float32)
        v = (s * c).astype(np.float32)
        err[:, k] = np.sum((W32.astype(np.float64) - v.astype(np.float64)) ** 2, axis=1)
    best = np.argmin(err, axis=1)       # first minimum
    return cand[np.arange(m), best].astype(np.float32), err
