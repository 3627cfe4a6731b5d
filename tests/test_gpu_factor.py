"""GPU factor kernels (damping, RevCholesky, triangular inverse, normalise)
against the fp64 oracle's literal route Cholesky(X_d^-1), the AR(1) closed
form, and the non-SPD error path.

Tolerance: the device computes in fp64 and rounds once to fp32, so each
entry of L is within half an fp32 ulp of the exact value plus the fp64
error of the two routes (about cond(X_d) * 1e-16 relative).  For the
well-conditioned damped Grams here |L_ij| <= ~4, giving the bound
|L_gpu - L_ref| <= 1e-6 * max(1, |L_ref|).
"""
import numpy as np
import pytest

import workloads
from gpu_util import knear, log

pytestmark = pytest.mark.gpu


def _factor(A, B, damp):
    import torch
    import paper_2608_06291_amd as pk
    dev = torch.device("cuda:0")
    At = torch.from_numpy(np.ascontiguousarray(A, np.float32)).to(dev)
    Bt = None if B is None else torch.from_numpy(np.ascontiguousarray(B, np.float32)).to(dev)
    return pk.factor(At, Bt, damp)


@pytest.mark.parametrize("d", [1, 2, 5, 31, 32, 33, 63, 64, 65, 100, 129, 200, 257])
def test_factor_matches_oracle(oracle_mod, d):
    p = workloads.make_random(d, d, seed=d, rhoA=0.6, rhoB=0.3)
    f = _factor(p["A"], p["B"], 0.01)
    LA = f.export("A").cpu().numpy().astype(np.float64)
    LB = f.export("B").cpu().numpy().astype(np.float64)
    f.close()
    for L, X in ((LA, p["A"]), (LB, p["B"])):
        ref = oracle_mod.normalized_factor(X, 0.01)
        err = np.abs(L - ref) / np.maximum(1.0, np.abs(ref))
        log(f"[factor] d={d} max scaled err {err.max():.3e}")
        assert err.max() <= 1e-6
        assert np.all(np.diag(L) == 1.0)
        assert np.all(np.triu(L, 1) == 0.0)


def test_factor_large_block_paths(oracle_mod):
    """Several 64-blocks of the blocked Cholesky and the recursive inverse."""
    d = 700
    p = workloads.make_random(d, 48, seed=1)        # B is the 700 x 700 one
    f = _factor(p["A"], p["B"], 0.01)
    LB = f.export("B").cpu().numpy().astype(np.float64)
    f.close()
    ref = oracle_mod.normalized_factor(p["B"], 0.01)
    err = np.abs(LB - ref) / np.maximum(1.0, np.abs(ref))
    log(f"[factor] d={d} max scaled err {err.max():.3e}")
    assert err.max() <= 1e-6


def test_factor_ar1_closed_form():
    """X = [rho^|i-j|] (exact in fp32 for rho = 1/2), no damping:
    L = I - rho * subdiag."""
    d = 1000
    f = _factor(workloads.ar1_toeplitz(d, 0.5), None, 0.0)
    L = f.export("A").cpu().numpy().astype(np.float64)
    f.close()
    ref = np.eye(d) - 0.5 * np.eye(d, k=-1)
    assert np.abs(L - ref).max() <= 1e-6


def test_factor_ar1_closed_form_large():
    """The same closed form at sizes that take the 128 x 128 fp64 GEMM blocks,
    the heavy-first triangular products and the one-panel look-ahead of the
    trailing updates (factors of 8192 and more), with partial 512-column
    panels and partial blocks: A 9000 x 9000, B 8300 x 8300.  The Cholesky
    factor of the AR(1) matrix is dense, so every trailing update carries
    nonzero data, and the inverse must cancel to the bidiagonal L."""
    import torch
    dev = torch.device("cuda:0")

    def ar1(d):
        i = torch.arange(d, device=dev, dtype=torch.float32)
        return 0.5 ** (i[:, None] - i[None, :]).abs()

    import paper_2608_06291_amd as pk
    log("case factor AR(1) closed form, A 9000, B 8300")
    f = pk.factor(ar1(9000), ar1(8300), 0.0)
    for which, d in (("A", 9000), ("B", 8300)):
        L = f.export(which)
        ref = torch.eye(d, device=dev, dtype=torch.float32)
        idx = torch.arange(1, d, device=dev)
        ref[idx, idx - 1] = -0.5
        err = float((L - ref).abs().max())
        log(f"[factor] AR(1) {which} d={d} max err {err:.3e}")
        assert err <= 1e-6
        del L, ref
    f.close()


def test_factor_identity_B_and_export_errors():
    import paper_2608_06291_amd as pk
    f = _factor(workloads.ar1_toeplitz(40, 0.5), None, 0.01)
    with pytest.raises(pk.BakronError):
        f.export("B")
    f.close()


def test_not_spd_reports_enotspd():
    """Undamped rank-deficient Gram (rank 8 < 40) is not positive definite."""
    import paper_2608_06291_amd as pk
    rng = np.random.default_rng(0)
    X = rng.standard_normal((40, 8))
    G = (X @ X.T / 8).astype(np.float32)
    with pytest.raises(pk.BakronError) as ei:
        _factor(G, None, 0.0)
    assert ei.value.status == pk.BAKRON_ENOTSPD
    assert "not positive definite" in str(ei.value)
    # with damping the same matrix factors fine
    f = _factor(G, None, 0.01)
    f.close()
    # negative diagonal, also caught
    with pytest.raises(pk.BakronError):
        _factor(-np.eye(10, dtype=np.float32), None, 0.0)


def test_invalid_arguments():
    import torch
    import paper_2608_06291_amd as pk
    dev = torch.device("cuda:0")
    A = torch.eye(8, device=dev)
    f = pk.factor(A, None, 0.01)
    W = torch.zeros((4, 8), device=dev)
    s = torch.ones(4, device=dev)
    for bits in (1, 9):
        with pytest.raises(pk.BakronError) as ei:
            pk.solve(W, f, bits, s)
        assert ei.value.status == pk.BAKRON_EINVAL
    with pytest.raises(pk.BakronError):
        pk.solve(torch.zeros((4, 7), device=dev), f, 4, s)   # n mismatch
    f.close()
    with knear(None):
        pass
