"""fp64 CPU oracle for the Kronecker-factor construction -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline leg
may import this module.  It shares no code with the HIP path in
``paper_2608_06291_amd/``.

Everything follows App. A of arXiv 2608.06291 in its own notation, written from
the definitions (plain numpy in fp64, one sample at a time where the paper's
expression is per sample):

* :func:`expect_outer` -- ``E[w a a^T]`` over the calibration samples, E the
  sample mean.  Samples may be vectors (rows of an N x d array) or matrices
  (N x d x p), for which ``a a^T`` is the d x d matrix product.
* :func:`full_hessian` -- ``H = E[a a^T (x) b b^T]`` (App. A: the form shared by
  the global and the local Hessians), tiny sizes only.
* :func:`expect_outer_entries` -- single entries of the same mean (sampled
  checks at full size).
* :func:`trace_quad` -- ``tr(a^T X a)`` per sample (the Shampoo weights).
* :func:`kfac_factors` -- ``A = E[a a^T]``, ``B = E[b b^T]`` (K-FAC style,
  App. A: independence assumption).
* :func:`shampoo_factors` -- the unnormalised power iteration of App. A,
  ``A^(i+1) = E[tr(b^T B^(i) b) a a^T]``, ``B^(i+1) = E[tr(a^T A^(i) a) b b^T]``
  from ``A^(0) = I``, ``B^(0) = I``; one step is the "single iteration"
  Shampoo-style factor pair.
* :func:`rearrange` -- the Van Loan--Pitsianis rearrangement R with
  ``R(A (x) B) = vec(A) vec(B)^T`` (App. A), used by the pins.
* :func:`mlp_local_b` -- App. A's MLP-local ``b = D_g W_down^T`` (or ``D_f``),
  built explicitly per sample (no Hadamard identity).
* :func:`glu_features` -- ``g = sigma(W_gate x)`` and
  ``f = sigma'(W_gate x) (.) W_up x`` for SiLU, the gated MLP of App. A.

vec stacks columns (Prop. 3.1): ``vec(W)`` of an m x n matrix lists column 0
first; ``H = A (x) B`` with A acting on the input side (n x n) and B on the
output side (m x m), so a sample gradient ``b a^T`` has ``vec = a (x) b``.
"""
from __future__ import annotations

import numpy as np


def _as_samples(a) -> np.ndarray:
    """N x d x p view of vector (N x d) or matrix (N x d x p) samples, fp64."""
    a = np.asarray(a, np.float64)
    if a.ndim == 2:
        return a[:, :, None]
    if a.ndim != 3:
        raise ValueError("samples must be N x d or N x d x p")
    return a


def expect_outer(a, w=None) -> np.ndarray:
    """E[w_k a_k a_k^T] = (1/N) sum_k w_k a_k a_k^T (App. A's sample mean)."""
    s = _as_samples(a)
    N, d, _ = s.shape
    out = np.zeros((d, d), np.float64)
    for k in range(N):
        wk = 1.0 if w is None else float(w[k])
        out += wk * (s[k] @ s[k].T)
    return out / N


def expect_outer_entries(X, pairs, w=None) -> np.ndarray:
    """Entries (i, j) of E[w_k x_k x_k^T] for vector samples, one at a time:
    (1/N) sum_k w_k X_ki X_kj (for sampled checks at sizes where the whole
    matrix is out of reach)."""
    X = np.asarray(X)
    N = X.shape[0]
    wk = None if w is None else np.asarray(w, np.float64)
    out = np.empty(len(pairs), np.float64)
    for t, (i, j) in enumerate(pairs):
        p = X[:, i].astype(np.float64) * X[:, j].astype(np.float64)
        out[t] = (p if wk is None else wk * p).sum() / N
    return out


def trace_quad(a, X=None) -> np.ndarray:
    """tr(a_k^T X a_k) for every sample k (X = None: the identity)."""
    s = _as_samples(a)
    out = np.empty(s.shape[0], np.float64)
    for k in range(s.shape[0]):
        ak = s[k]
        out[k] = np.trace(ak.T @ ak) if X is None else np.trace(ak.T @ X @ ak)
    return out


def kfac_factors(a, b):
    """K-FAC style pair (App. A): A = E[a a^T], B = E[b b^T]."""
    return expect_outer(a), expect_outer(b)


def shampoo_factors(a, b, iters: int = 1, normalise: bool = False):
    """Shampoo-style pair (App. A): `iters` steps of the power iteration on
    R(H) from A^(0) = I_n, B^(0) = I_m, both factors updated from the previous
    pair.  The paper's iteration is unnormalised; with ``normalise`` every
    iterate is divided by its Frobenius norm (same directions, no overflow)."""
    sa, sb = _as_samples(a), _as_samples(b)
    A = np.eye(sa.shape[1])
    B = np.eye(sb.shape[1])
    for _ in range(iters):
        A_next = expect_outer(sa, trace_quad(sb, B))
        B_next = expect_outer(sb, trace_quad(sa, A))
        A, B = A_next, B_next
        if normalise:
            A = A / np.linalg.norm(A)
            B = B / np.linalg.norm(B)
    return A, B


def full_hessian(a, b) -> np.ndarray:
    """H = E[a a^T (x) b b^T] as an explicit (n m) x (n m) matrix (tiny sizes)."""
    sa, sb = _as_samples(a), _as_samples(b)
    N = sa.shape[0]
    n, m = sa.shape[1], sb.shape[1]
    H = np.zeros((n * m, n * m), np.float64)
    for k in range(N):
        H += np.kron(sa[k] @ sa[k].T, sb[k] @ sb[k].T)
    return H / N


def rearrange(H, n: int, m: int) -> np.ndarray:
    """Van Loan--Pitsianis rearrangement of an (n m) x (n m) matrix viewed as an
    n x n grid of m x m blocks: row i + n j of R(H) is vec of block (i, j), so
    that R(A (x) B) = vec(A) vec(B)^T (block (i, j) of A (x) B is A_ij B)."""
    H = np.asarray(H, np.float64)
    R = np.empty((n * n, m * m), np.float64)
    for j in range(n):
        for i in range(n):
            blk = H[i * m:(i + 1) * m, j * m:(j + 1) * m]
            R[i + n * j] = blk.reshape(-1, order="F")
    return R


def mlp_local_b(gate_feat, W_down) -> np.ndarray:
    """b_k = D_{g_k} W_down^T (dff x dm) for every sample (App. A, MLP-local)."""
    g = np.asarray(gate_feat, np.float64)
    D = np.asarray(W_down, np.float64)
    return np.stack([np.diag(g[k]) @ D.T for k in range(g.shape[0])])


def mlp_local_factors(x, gate_feat, W_down, style: str = "kfac", iters: int = 1):
    """Kronecker factors of the MLP-local Hessian E[x x^T (x) b b^T] with
    b = D_g W_down^T (pass f instead of g for W_gate), App. A."""
    b = mlp_local_b(gate_feat, W_down)
    if style == "kfac":
        return kfac_factors(x, b)
    if style == "shampoo":
        return shampoo_factors(x, b, iters=iters)
    raise ValueError(style)


def silu(z):
    return z / (1.0 + np.exp(-z))


def silu_prime(z):
    sg = 1.0 / (1.0 + np.exp(-z))
    return sg * (1.0 + z * (1.0 - sg))


def glu_features(x, W_gate, W_up):
    """g = sigma(W_gate x) and f = sigma'(W_gate x) (.) W_up x per sample
    (App. A, gated MLP; sigma = SiLU).  x: N x dm, W_*: dff x dm."""
    x = np.asarray(x, np.float64)
    z = x @ np.asarray(W_gate, np.float64).T
    u = x @ np.asarray(W_up, np.float64).T
    return silu(z), silu_prime(z) * u
