"""Pins for the Kronecker-factor oracle (App. A), CPU only.

Each test ties the oracle to something other than itself: the gradients and
Jacobians of the actual loss and gated MLP taken by torch autograd (fp64), the
exact factorisation of H for independent samples, the defining property of the
Van Loan--Pitsianis rearrangement, the power iteration checked against a
library SVD, and a closed-form AR(1) expectation.  A transposed Kronecker
order, a wrong vec convention, a dropped 1/N, a wrong trace weight or a wrong
SiLU derivative each fail one of them.
"""
import numpy as np
import pytest
import torch

import workloads


def _rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([7001, *key])))


def _vec(M):
    """Column-stacking vec (Prop. 3.1) of a torch or numpy matrix."""
    return M.T.reshape(-1)


# ---------------------------------------------------------------- global case
def test_full_hessian_is_gradient_outer_product(oracle_mod):
    """H = E[a a^T (x) b b^T] is E[vec(G) vec(G)^T] for the per-sample weight
    gradient G of a loss whose output gradient is b (App. A, global case):
    autograd of l_k(W) = b_k^T W a_k gives G = b a^T."""
    h = oracle_mod.hessian
    r = _rng(1)
    N, n, m = 6, 3, 4
    a, b = r.standard_normal((N, n)), r.standard_normal((N, m))
    H = np.zeros((n * m, n * m))
    for k in range(N):
        W = torch.zeros((m, n), dtype=torch.float64, requires_grad=True)
        loss = torch.from_numpy(b[k]) @ W @ torch.from_numpy(a[k])
        (G,) = torch.autograd.grad(loss, W)
        v = _vec(G).numpy()
        H += np.outer(v, v)
    H /= N
    np.testing.assert_allclose(h.full_hessian(a, b), H, rtol=1e-13, atol=1e-13)
    # GPTQ's special case: b runs over the rows of I_m with every a, so
    # H = E[a a^T] (x) I_m / m
    A = h.expect_outer(a)
    Hg = h.full_hessian(np.repeat(a, m, 0), np.tile(np.eye(m), (N, 1)))
    np.testing.assert_allclose(m * Hg, np.kron(A, np.eye(m)), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("matrix_b", [False, True])
def test_kfac_exact_for_independent_samples(oracle_mod, matrix_b):
    """If the samples are every pairing of an a-set with a b-set, a and b are
    independent and E[a a^T (x) b b^T] = E[a a^T] (x) E[b b^T] exactly."""
    h = oracle_mod.hessian
    r = _rng(2, int(matrix_b))
    Na, Nb, n, m = 4, 3, 3, 5
    aset = r.standard_normal((Na, n))
    bset = r.standard_normal((Nb, m, 2)) if matrix_b else r.standard_normal((Nb, m))
    a = np.repeat(aset, Nb, axis=0)
    b = np.tile(bset, (Na, 1, 1)) if matrix_b else np.tile(bset, (Na, 1))
    A, B = h.kfac_factors(a, b)
    H = h.full_hessian(a, b)
    np.testing.assert_allclose(np.kron(A, B), H, rtol=1e-12, atol=1e-13)
    # the other Kronecker order is not H (n != m): the order is pinned
    assert not np.allclose(np.kron(B, A), H)


def test_rearrangement_defining_property(oracle_mod):
    """R(A (x) B) = vec(A) vec(B)^T and R preserves the Frobenius norm."""
    h = oracle_mod.hessian
    r = _rng(3)
    n, m = 3, 4
    A, B = r.standard_normal((n, n)), r.standard_normal((m, m))
    R = h.rearrange(np.kron(A, B), n, m)
    np.testing.assert_allclose(R, np.outer(_vec(A), _vec(B)), rtol=1e-14, atol=1e-14)
    H = r.standard_normal((n * m, n * m))
    assert np.isclose(np.linalg.norm(h.rearrange(H, n, m)), np.linalg.norm(H), rtol=1e-14)


@pytest.mark.parametrize("matrix_b", [False, True])
def test_shampoo_single_step_is_power_step(oracle_mod, matrix_b):
    """One Shampoo step from (I, I) is u = R(H) vec(I_m), v = R(H)^T vec(I_n)."""
    h = oracle_mod.hessian
    r = _rng(4, int(matrix_b))
    N, n, m = 7, 3, 4
    a = r.standard_normal((N, n)) * r.lognormal(0, 0.5, (N, 1))
    b = r.standard_normal((N, m, 3)) if matrix_b else r.standard_normal((N, m))
    A1, B1 = h.shampoo_factors(a, b, iters=1)
    R = h.rearrange(h.full_hessian(a, b), n, m)
    np.testing.assert_allclose(_vec(A1), R @ _vec(np.eye(m)), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(_vec(B1), R.T @ _vec(np.eye(n)), rtol=1e-12, atol=1e-13)


def test_shampoo_iteration_converges_to_best_kronecker(oracle_mod):
    """Many power steps give the top singular pair of R(H) (library SVD), i.e.
    the best Kronecker approximation in Frobenius norm (App. A, Van Loan)."""
    h = oracle_mod.hessian
    r = _rng(5)
    N, n, m = 9, 3, 4
    a = r.standard_normal((N, n)) * r.lognormal(0, 1.0, (N, 1))
    b = r.standard_normal((N, m)) * r.lognormal(0, 1.0, (N, 1))
    H = h.full_hessian(a, b)
    R = h.rearrange(H, n, m)
    U, S, Vt = np.linalg.svd(R)
    A, B = h.shampoo_factors(a, b, iters=400, normalise=True)
    u, v = _vec(A), _vec(B)
    assert abs(abs(u @ U[:, 0]) - 1.0) < 1e-9
    assert abs(abs(v @ Vt[0]) - 1.0) < 1e-9
    # the converged pair, scaled by its best multiple (the top singular value),
    # attains the SVD bound ||H - A (x) B||^2 = sum of the other sigma^2
    K1 = np.kron(A, B)
    best = np.linalg.norm(H - (np.sum(K1 * H) / np.sum(K1 * K1)) * K1)
    np.testing.assert_allclose(best ** 2, np.sum(S[1:] ** 2), rtol=1e-8)
    # K-FAC is never better than the best Kronecker approximation
    Ak, Bk = h.kfac_factors(a, b)
    K = np.kron(Ak, Bk)
    c = np.sum(K * H) / np.sum(K * K)
    assert np.linalg.norm(H - c * K) >= best - 1e-12


# ---------------------------------------------------------------- MLP-local
def _mlp_case(seed, N=5, dm=3, dff=4):
    r = _rng(6, seed)
    x = r.standard_normal((N, dm))
    Wg = r.standard_normal((dff, dm)) / np.sqrt(dm)
    Wu = r.standard_normal((dff, dm)) / np.sqrt(dm)
    Wd = r.standard_normal((dm, dff)) / np.sqrt(dff)
    return x, Wg, Wu, Wd


def _mlp_torch(x, Wg, Wu, Wd):
    z = Wg @ x
    return Wd @ ((Wu @ x) * (z * torch.sigmoid(z)))


@pytest.mark.parametrize("which", ["up", "gate"])
def test_mlp_local_hessian_is_gauss_newton_of_the_mlp(oracle_mod, which):
    """E[x x^T (x) b b^T] with b = D_g W_down^T (up) or D_f W_down^T (gate)
    equals E[J^T J] for the Jacobian J of the gated MLP's output with respect
    to vec(W_up) or vec(W_gate), taken by autograd (App. A, l2 output loss)."""
    h = oracle_mod.hessian
    x, Wg, Wu, Wd = _mlp_case(1)
    N, dm = x.shape
    dff = Wg.shape[0]
    T = lambda v: torch.from_numpy(v)  # noqa: E731
    JtJ = np.zeros((dm * dff, dm * dff))
    for k in range(N):
        def f(vecW):
            W = vecW.reshape(dm, dff).T   # inverse of column-stacking vec
            if which == "up":
                return _mlp_torch(T(x[k]), T(Wg), W, T(Wd))
            return _mlp_torch(T(x[k]), W, T(Wu), T(Wd))
        W0 = Wu if which == "up" else Wg
        J = torch.autograd.functional.jacobian(f, _vec(T(W0)).clone()).numpy()
        JtJ += J.T @ J
    JtJ /= N
    g, fgate = h.glu_features(x, Wg, Wu)
    feat = g if which == "up" else fgate
    H = h.full_hessian(x, h.mlp_local_b(feat, Wd))
    np.testing.assert_allclose(H, JtJ, rtol=1e-11, atol=1e-13)


def test_mlp_local_hadamard_and_trace_identities(oracle_mod):
    """App. A: b b^T = (g g^T) (.) W_down^T W_down and
    tr(b^T b) = g^T diag(W_down^T W_down) g, checked on the explicit b."""
    h = oracle_mod.hessian
    x, Wg, Wu, Wd = _mlp_case(2, N=6, dm=4, dff=5)
    g, _ = h.glu_features(x, Wg, Wu)
    b = h.mlp_local_b(g, Wd)
    DtD = Wd.T @ Wd
    A, B = h.kfac_factors(x, b)
    np.testing.assert_allclose(B, h.expect_outer(g) * DtD, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(h.trace_quad(b), np.einsum("ki,i,ki->k", g, np.diag(DtD), g),
                               rtol=1e-12)


def test_silu_derivative(oracle_mod):
    h = oracle_mod.hessian
    z = np.linspace(-8, 8, 101)
    zt = torch.from_numpy(z).requires_grad_(True)
    (d,) = torch.autograd.grad(torch.nn.functional.silu(zt).sum(), zt)
    np.testing.assert_allclose(h.silu_prime(z), d.numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(h.silu(z), torch.nn.functional.silu(torch.from_numpy(z)).numpy(),
                               rtol=1e-13, atol=1e-15)


# ---------------------------------------------------------------- closed form
def test_ar1_samples_expectation(oracle_mod):
    """E[a a^T] of the AR(1) sample recipe tends to the Toeplitz rho^|i-j|;
    with N samples every entry is within 6 standard errors (sd <= sqrt(2/N))."""
    N, d, rho = 20000, 6, 0.6
    a = workloads.ar1_samples(N, d, rho, _rng(8)).astype(np.float64)
    A = oracle_mod.hessian.expect_outer(a)
    assert np.max(np.abs(A - workloads.ar1_toeplitz(d, rho))) < 6 * np.sqrt(2.0 / N)


def test_expect_outer_entries_match_the_matrix(oracle_mod):
    h = oracle_mod.hessian
    r = _rng(9)
    X = r.standard_normal((50, 7))
    w = r.lognormal(0, 1, 50)
    pairs = [(0, 0), (2, 5), (6, 1), (3, 3)]
    E = h.expect_outer(X, w)
    np.testing.assert_allclose(h.expect_outer_entries(X, pairs, w), [E[i, j] for i, j in pairs],
                               rtol=1e-13)
