"""Pins for the oracle's Alg. 5 (BaKron-recursive, Sec. 3.4) against its Alg. 2
(BaKron-naive): by Thm 3.2 both visit every entry with the same elementary
updates applied, so the codes must be identical and the pre-rounding values
equal up to fp64 summation order.  Also pins the RevCholesky factor route
against the literal inverse-then-Cholesky route, and Alg. 5 against the
exact AR(1) three-neighbour recursion at a size Alg. 2 does not reach
quickly.  A planted slip in the recursion (a dropped or misplaced product, a
wrong split, a missing leaf update) changes the codes on these shapes."""
import numpy as np
import pytest

import workloads

SHAPES = [(1, 1), (1, 37), (37, 1), (2, 3), (5, 6), (13, 9), (33, 31), (65, 97), (97, 200),
          (130, 67)]


def _factors(o, p):
    LA = o.normalized_factor(p["A"], p["damp"])
    LB = np.eye(p["W"].shape[0]) if p["B"] is None else o.normalized_factor(p["B"], p["damp"])
    return LA, LB


def _same(r1, r2):
    assert np.array_equal(r1["codes"], r2["codes"])
    assert np.array_equal(np.isnan(r1["pre"]), np.isnan(r2["pre"]))
    d = np.nanmax(np.abs(r1["pre"] - r2["pre"])) if r1["pre"].size else 0.0
    assert d < 1e-9, d
    assert np.allclose(r1["V"], r2["V"], rtol=0, atol=1e-15)


@pytest.mark.parametrize("m,n", SHAPES)
@pytest.mark.parametrize("base", [1, 3, 8])
def test_recursive_equals_naive(oracle_mod, m, n, base):
    o = oracle_mod
    p = workloads.make_random(m, n, seed=m * 7 + n)
    LA, LB = _factors(o, p)
    r1 = o.babai(p["W"], LA, LB, p["scale"], p["bits"])
    # products through BLAS everywhere, and through plain loops everywhere
    for blas_min in (1, 1 << 62):
        r2 = o.babai_recursive(p["W"], LA, LB, p["scale"], p["bits"], base=base,
                               blas_min=blas_min)
        _same(r1, r2)


def test_recursive_config1(oracle_mod):
    o = oracle_mod
    p = workloads.make(1, seed=0)
    LA, LB = _factors(o, p)
    _same(o.babai(p["W"], LA, LB, p["scale"], p["bits"]),
          o.babai_recursive(p["W"], LA, LB, p["scale"], p["bits"]))


@pytest.mark.parametrize("variant", ["B=I", "bits2", "asym+groups", "zero-rows"])
def test_recursive_variants(oracle_mod, variant):
    o = oracle_mod
    p = workloads.make_random(70, 90, seed=5, identity_B=(variant == "B=I"),
                              bits=2 if variant == "bits2" else 4)
    LA, LB = _factors(o, p)
    scale, alphabet = p["scale"], "sym"
    if variant == "asym+groups":
        alphabet = "asym"
        g = np.random.default_rng(1).uniform(0.5, 1.5, (70, 3)).astype(np.float32)
        scale = o.entry_scales(g * p["scale"][:, None], 70, 90, group_size=32)
    if variant == "zero-rows":
        scale = p["scale"].copy()
        scale[[0, 17, 69]] = 0.0
    r1 = o.babai(p["W"], LA, LB, scale, p["bits"], alphabet=alphabet)
    r2 = o.babai_recursive(p["W"], LA, LB, scale, p["bits"], alphabet=alphabet)
    _same(r1, r2)


def test_recursive_tie_forcing(oracle_mod):
    """Forced replay: adopting another candidate's codes inside the tie window
    works the same way in both (same excused entries, same flips)."""
    o = oracle_mod
    p = workloads.make_random(60, 70, seed=9)
    LA, LB = _factors(o, p)
    r = o.babai(p["W"], LA, LB, p["scale"], p["bits"])
    # a candidate that differs from the oracle at its near-ties: flip every
    # entry within 0.3 of a boundary towards the other side
    x = r["pre"]
    near = o.near_boundary(x, p["bits"], 0.3)
    cand = r["codes"].copy()
    cand[near] = np.where(x[near] > np.floor(x[near]) + 0.5, np.floor(x[near]),
                          np.floor(x[near]) + 1).astype(np.int8)
    f1 = o.babai(p["W"], LA, LB, p["scale"], p["bits"], forced=cand, tie_window=0.3)
    f2 = o.babai_recursive(p["W"], LA, LB, p["scale"], p["bits"], forced=cand, tie_window=0.3)
    _same(f1, f2)
    assert f1["n_excused"] == f2["n_excused"] > 0
    assert f1["n_flip"] == f2["n_flip"] > 0


def test_rev_factor_route_equals_literal(oracle_mod):
    o = oracle_mod
    for d, seed in ((1, 0), (7, 1), (64, 2), (300, 3)):
        X = workloads.make_random(d, d, seed=seed)["A"]
        np.testing.assert_allclose(o.normalized_factor_rev(X, 0.01), o.normalized_factor(X, 0.01),
                                   rtol=0, atol=1e-10)


def test_recursive_ar1_closed_form(oracle_mod):
    """A, B AR(1) Toeplitz without damping: the normalised factors are
    I - rho * subdiag, and the exact O(mn) three-neighbour recursion gives the
    codes at a size where Alg. 2 is slow."""
    o = oracle_mod
    rng = np.random.default_rng(23)
    m, n = 700, 650
    W = (rng.standard_normal((m, n)) * 0.02).astype(np.float32)
    s = workloads.row_scales(W, 3)
    LA = o.normalized_factor_rev(workloads.ar1_toeplitz(n, 0.5), 0.0)
    LB = o.normalized_factor_rev(workloads.ar1_toeplitz(m, 0.25), 0.0)
    r1 = o.ar1_diffusion(W, 0.5, 0.25, s, 3)
    r2 = o.babai_recursive(W, LA, LB, s, 3)
    assert np.array_equal(r1["codes"], r2["codes"])
    assert np.nanmax(np.abs(r1["pre"] - r2["pre"])) < 1e-7
