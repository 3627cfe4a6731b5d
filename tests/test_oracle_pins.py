"""Pins for the fp64 oracle, checked against what the paper and the mathematics
fix (CPU only).  Each test would catch a plausible slip in the oracle: a
dropped feedback term, a transposed factor, a wrong traversal order, a wrong
vec convention, a wrong tie rule, a missing clamp error.
"""
import json
import os

import numpy as np
import pytest

import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_problem(m, n, seed, bits=4, identity_B=False, rhoA=0.5, rhoB=0.3):
    return workloads.make_random(m, n, seed, bits=bits, rhoA=rhoA, rhoB=rhoB,
                                 identity_B=identity_B)


# ---------------------------------------------------------------- quantiser
def test_quantiser_ties_clamp_zero_scale(oracle_mod):
    o = oracle_mod
    # half-to-even ties, clamp to +-l (App. D alphabet; App. B fixed tie rule)
    x = np.array([0.5, 1.5, 2.5, -0.5, -1.5, 7.49, 7.5, 100.0, -100.0, np.nan])
    assert o.quantise_codes(x, 4).tolist() == [0, 2, 2, 0, -2, 7, 7, 7, -7, 0]
    # zero-scale row: alphabet {0}, V = 0, error = -W~ fed back
    W = np.array([[0.3, -0.2, 0.1], [0.4, 0.5, 0.6]])
    A = workloads.ar1_toeplitz(3, 0.5)
    r = o.solve(W, A, None, 0.0, np.array([0.0, 0.1]), 4)
    assert r["codes"][0].tolist() == [0, 0, 0]
    assert np.all(r["V"][0] == 0.0)
    assert np.all(np.isnan(r["pre"][0]))


# ---------------------------------------------------------------- golden
@pytest.mark.parametrize("name", ["hand_2x2_ar1.json", "hand_1x3_clamp.json",
                                  "hand_2x2_damp.json"])
def test_hand_worked_examples(oracle_mod, name):
    o = oracle_mod
    g = json.load(open(os.path.join(GOLDEN, name)))
    W = np.array(g["W"], np.float64)
    r = o.solve(W, np.array(g["A"]), np.array(g["B"]), g["damp"], np.array(g["scale"]), g["bits"])
    assert r["codes"].tolist() == g["codes"]
    np.testing.assert_allclose(r["pre"], np.array(g["pre"]), atol=1e-12)
    if "L" in g:
        np.testing.assert_allclose(o.normalized_factor(np.array(g["A"]), 0.0),
                                   np.array(g["L"]), atol=1e-14)
    # damping with each factor's own mean diagonal, and the factors it leads to
    for X, key, lkey in (("A", "Ad", "LA"), ("B", "Bd", "LB")):
        if key in g:
            np.testing.assert_allclose(o.damp(np.array(g[X]), g["damp"]), np.array(g[key]),
                                       rtol=0, atol=1e-15)
            np.testing.assert_allclose(o.normalized_factor(np.array(g[X]), g["damp"]),
                                       np.array(g[lkey]), rtol=0, atol=1e-15)


# ---------------------------------------------------------------- brute force
def _gptq_vector(w, H, scale_vec, bits):
    """Alg. 1 (GPTQ on one vector) with per-coordinate scale, plain numpy."""
    from oracle.oracle import quantise_codes
    L = np.linalg.cholesky(np.linalg.inv(H))
    L = L / np.diag(L)[None, :]
    w = np.array(w, np.float64).copy()
    codes = np.zeros(w.shape[0], np.int8)
    for i in range(w.shape[0]):
        s = scale_vec[i]
        c = 0 if s == 0 else int(quantise_codes(np.array([w[i] / s]), bits)[0])
        codes[i] = c
        delta = s * c - w[i]
        w = w + delta * L[:, i]
    return codes


@pytest.mark.parametrize("m,n", [(1, 5), (5, 1), (3, 4), (4, 3), (5, 6), (6, 6), (7, 9)])
def test_explicit_kronecker_hessian(oracle_mod, m, n):
    """GPTQ on vec(W) (column-major, Sec. 3.1) with H = A_d (x) B_d, explicit
    mn x mn Hessian and its own Cholesky(H^-1), equals the 2-D oracle (Alg. 2)."""
    o = oracle_mod
    p = _rand_problem(m, n, seed=m * 10 + n)
    W = p["W"].astype(np.float64)
    Ad, Bd = o.damp(p["A"], p["damp"]), o.damp(p["B"], p["damp"])
    H = np.kron(Ad, Bd)
    w = W.reshape(-1, order="F")
    svec = np.tile(p["scale"].astype(np.float64), n)          # vec index i + m*j
    codes_vec = _gptq_vector(w, H, svec, p["bits"])
    ref = codes_vec.reshape((m, n), order="F")
    got = o.solve(W, p["A"], p["B"], p["damp"], p["scale"], p["bits"])["codes"]
    assert np.array_equal(got, ref)


def test_explicit_kronecker_hessian_config1(oracle_mod):
    """The 64 x 64 configuration itself: Alg. 1 on vec(W) with the explicit
    4096 x 4096 Hessian A_d (x) B_d and its own Cholesky(H^-1) gives the codes
    of the 2-D oracle (Alg. 2) on every entry, and the same pre-rounding
    values up to fp64 rounding."""
    import workloads
    o = oracle_mod
    c = workloads.make(1, seed=0)
    W = c["W"].astype(np.float64)
    m, n = W.shape
    Ad, Bd = o.damp(c["A"], c["damp"]), o.damp(c["B"], c["damp"])
    H = np.kron(Ad, Bd)
    L = np.linalg.cholesky(np.linalg.inv(H))
    L = L / np.diag(L)[None, :]
    w = W.reshape(-1, order="F").copy()
    svec = np.tile(c["scale"].astype(np.float64), n)
    from oracle.oracle import quantise_codes
    codes = np.zeros(m * n, np.int8)
    x = np.zeros(m * n)
    for i in range(m * n):
        x[i] = w[i] / svec[i]
        codes[i] = int(quantise_codes(np.array([x[i]]), c["bits"])[0])
        w[i + 1:] += (svec[i] * codes[i] - w[i]) * L[i + 1:, i]
    got = o.solve(W, c["A"], c["B"], c["damp"], c["scale"], c["bits"])
    assert np.array_equal(got["codes"], codes.reshape((m, n), order="F"))
    assert np.max(np.abs(got["pre"] - x.reshape((m, n), order="F"))) < 1e-8


@pytest.mark.parametrize("m,n", [(2, 3), (3, 3), (4, 5)])
def test_obs_constrained_reminimisation(oracle_mod, m, n):
    """Sec. 3.2 OBS view: after fixing the processed set S, the free entries F
    minimise the quadratic, v_F = w_F - H_FF^-1 H_FS (q_S - w_S); the next entry
    in row-major order is quantised at that value."""
    o = oracle_mod
    p = _rand_problem(m, n, seed=77 + m + n)
    W = p["W"].astype(np.float64)
    H = np.kron(o.damp(p["A"], p["damp"]), o.damp(p["B"], p["damp"]))
    w = W.reshape(-1, order="F")
    s = p["scale"].astype(np.float64)
    order = [i + m * j for i in range(m) for j in range(n)]   # row-major in vec index
    q = np.zeros(m * n)
    codes = np.zeros((m, n), np.int8)
    done = []
    for k in order:
        free = [t for t in range(m * n) if t not in done]
        v = w.copy()
        if done:
            S = np.array(done)
            F = np.array(free)
            v[F] = w[F] - np.linalg.solve(H[np.ix_(F, F)], H[np.ix_(F, S)] @ (q[S] - w[S]))
        i, j = k % m, k // m
        c = int(o.quantise_codes(np.array([v[k] / s[i]]), p["bits"])[0])
        codes[i, j] = c
        q[k] = s[i] * c
        done.append(k)
    got = o.solve(W, p["A"], p["B"], p["damp"], p["scale"], p["bits"])["codes"]
    assert np.array_equal(got, codes)


# ---------------------------------------------------------------- special cases
@pytest.mark.parametrize("m,n", [(4, 17), (9, 33), (16, 64)])
def test_B_identity_is_gptq_per_row(oracle_mod, m, n):
    """Sec. 1: B = I is GPTQ with H = A, row by row (Alg. 1)."""
    o = oracle_mod
    p = _rand_problem(m, n, seed=5 + m, identity_B=True)
    Ad = o.damp(p["A"], p["damp"])
    got = o.solve(p["W"], p["A"], None, p["damp"], p["scale"], p["bits"])["codes"]
    for i in range(m):
        ref = _gptq_vector(p["W"][i].astype(np.float64), Ad,
                           np.full(n, float(p["scale"][i])), p["bits"])
        assert np.array_equal(got[i], ref), i


@pytest.mark.parametrize("m,n", [(17, 4), (33, 9)])
def test_A_identity_is_gptq_per_column(oracle_mod, m, n):
    o = oracle_mod
    p = _rand_problem(m, n, seed=9 + n)
    Bd = o.damp(p["B"], p["damp"])
    got = o.solve(p["W"], np.eye(n, dtype=np.float32), p["B"], p["damp"], p["scale"],
                  p["bits"])["codes"]
    for j in range(n):
        ref = _gptq_vector(p["W"][:, j].astype(np.float64), Bd,
                           p["scale"].astype(np.float64), p["bits"])
        assert np.array_equal(got[:, j], ref), j


def test_diagonal_hessians_give_round_to_nearest(oracle_mod):
    rng = np.random.default_rng(3)
    m, n = 11, 13
    W = rng.standard_normal((m, n)) * 0.02
    A = np.diag(rng.uniform(0.5, 2.0, n))
    B = np.diag(rng.uniform(0.5, 2.0, m))
    s = np.max(np.abs(W), axis=1) / 7
    got = oracle_mod.solve(W, A, B, 0.01, s, 4)["codes"]
    assert np.array_equal(got, oracle_mod.quantise_codes(W / s[:, None], 4))


def test_fine_grid_returns_W(oracle_mod):
    """North-star check 3 (Eq. (1) with Cor. 3.4's no-clamping premise): with one
    scale s for every row and a grid fine enough that nothing clamps, every
    error obeys |E| <= s/2, so V - W0 = L^B E L^A^T gives
    |V - W|_max <= (s/2) max_p |L^B_p,:|_1 max_q |L^A_q,:|_1 -> 0 with s."""
    o = oracle_mod
    m, n = 24, 20
    p = _rand_problem(m, n, seed=11, bits=8)
    W = p["W"].astype(np.float64)
    LA = o.normalized_factor(p["A"], p["damp"])
    LB = o.normalized_factor(p["B"], p["damp"])
    growth = np.max(np.abs(LB).sum(1)) * np.max(np.abs(LA).sum(1))
    s0 = np.max(np.abs(W)) / 100.0         # finest grid: |W|/s <= 100 inside the INT8 range
    errs = []
    for s in (64 * s0, 16 * s0, 4 * s0, s0):
        r = o.babai(W, LA, LB, np.full(m, s), 8)
        # the premise: no entry clamps (|x| < l + 1/2 = 127.5), so |E| <= s/2
        assert np.max(np.abs(r["pre"])) < 127.5
        assert np.max(np.abs(r["V"] - r["pre"] * s)) <= 0.5 * s * (1 + 1e-12)
        err = np.max(np.abs(r["V"] - W))
        assert err <= 0.5 * s * growth * (1 + 1e-9)
        errs.append(err)
    # V -> W: the error falls with the grid step
    assert errs[0] > errs[1] > errs[2] > errs[3]


def test_error_bound_cor34(oracle_mod):
    """Cor. 3.4 in the integer domain (uniform scale, no clamping):
    |R_B (V-W) R_A^T|_F^2 <= 1/4 sum_ij R_B,ii^2 R_A,jj^2 <= 1/4 tr(A) tr(B)."""
    o = oracle_mod
    p = _rand_problem(20, 24, seed=21, bits=8)
    s = 0.002
    W = p["W"].astype(np.float64) / s
    Ad, Bd = o.damp(p["A"], p["damp"]), o.damp(p["B"], p["damp"])
    r = o.solve(W, p["A"], p["B"], p["damp"], np.ones(20), 8)
    assert np.all(np.abs(r["pre"]) < 127.5)
    RA, RB = o.rev_cholesky(Ad), o.rev_cholesky(Bd)
    lhs = np.linalg.norm(RB @ (r["V"] - W) @ RA.T) ** 2
    mid = 0.25 * np.sum(np.outer(np.diag(RB) ** 2, np.diag(RA) ** 2))
    rhs = 0.25 * np.trace(Ad) * np.trace(Bd)
    assert lhs <= mid * (1 + 1e-9) <= rhs * (1 + 1e-9)


def test_transpose_symmetry(oracle_mod):
    """Swapping the roles of rows and columns (W^T with A, B exchanged) gives the
    transposed codes when the scale is one scalar (the order-free Eq. (2))."""
    o = oracle_mod
    p = _rand_problem(13, 9, seed=31)
    s = np.float64(np.max(np.abs(p["W"])) / 7)
    r1 = o.solve(p["W"], p["A"], p["B"], p["damp"], np.full(13, s), 4)
    r2 = o.solve(p["W"].T, p["B"], p["A"], p["damp"], np.full(9, s), 4)
    assert np.array_equal(r1["codes"], r2["codes"].T)


def test_hessian_scale_invariance(oracle_mod):
    """Scaling A or B by a constant changes nothing (App. A, Shampoo remark);
    powers of two keep every rounding step bit-identical."""
    o = oracle_mod
    p = _rand_problem(10, 12, seed=41)
    r1 = o.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], 4)
    r2 = o.solve(p["W"], 4.0 * p["A"], 0.25 * p["B"], p["damp"], p["scale"], 4)
    assert np.array_equal(r1["codes"], r2["codes"])
    np.testing.assert_array_equal(r1["pre"], r2["pre"])
    r3 = o.solve(p["W"], 3.0 * p["A"].astype(np.float64), 0.7 * p["B"].astype(np.float64),
                 p["damp"], p["scale"], 4)
    assert np.array_equal(r1["codes"], r3["codes"])
    np.testing.assert_allclose(r1["pre"], r3["pre"], atol=1e-10)


# ---------------------------------------------------------------- factors
def test_ar1_factor_closed_form(oracle_mod):
    """For X = [rho^|i-j|], normalised Cholesky(X^-1) = I - rho*subdiag."""
    for rho in (0.5, 0.25, 0.8):
        d = 40
        idx = np.arange(d)
        X = rho ** np.abs(idx[:, None] - idx[None, :]).astype(np.float64)   # fp64 Toeplitz
        L = oracle_mod.normalized_factor(X, 0.0)
        ref = np.eye(d) - rho * np.eye(d, k=-1)
        np.testing.assert_allclose(L, ref, atol=1e-12)


def test_factor_routes_agree(oracle_mod):
    """Cholesky(X^-1) normalised == inverse of RevCholesky(X) row-normalised."""
    o = oracle_mod
    p = _rand_problem(30, 45, seed=51)
    for X in (p["A"], p["B"]):
        L = o.normalized_factor(X, p["damp"])
        R = o.rev_cholesky(o.damp(X, p["damp"]))
        Rh = R / np.diag(R)[:, None]
        np.testing.assert_allclose(np.linalg.inv(Rh), L, atol=1e-10)
        assert np.allclose(np.diag(L), 1.0) and np.allclose(np.triu(L, 1), 0.0)


def test_ar1_diffusion_matches_naive(oracle_mod):
    o = oracle_mod
    rng = np.random.default_rng(61)
    m, n = 40, 50
    W = rng.standard_normal((m, n)) * 0.02
    s = np.max(np.abs(W), axis=1) / 3
    A = workloads.ar1_toeplitz(n, 0.5).astype(np.float64)
    B = workloads.ar1_toeplitz(m, 0.25).astype(np.float64)
    r1 = o.solve(W, A, B, 0.0, s, 3)
    r2 = o.ar1_diffusion(W, 0.5, 0.25, s, 3)
    assert np.array_equal(r1["codes"], r2["codes"])
    np.testing.assert_allclose(r1["pre"], r2["pre"], atol=1e-10)


# ---------------------------------------------------------------- certificate
def test_certificate_reproduces_trajectory(oracle_mod):
    o = oracle_mod
    p = _rand_problem(37, 29, seed=71, bits=3)
    r = o.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], p["bits"])
    x = o.certificate(p["W"], p["A"], p["B"], p["damp"], p["scale"], r["codes"], p["bits"])
    np.testing.assert_allclose(x, r["pre"], atol=1e-9)
    v = o.verdict(r["codes"], x, p["bits"])
    assert v["violations"] == 0 and v["flips"] == 0
    xr = o.certificate(p["W"], p["A"], p["B"], p["damp"], p["scale"], r["codes"], p["bits"],
                       rows=np.array([0, 5, 36]))
    np.testing.assert_allclose(xr, r["pre"][[0, 5, 36]], atol=1e-9)


def test_certificate_detects_planted_error(oracle_mod):
    """A wrong code anywhere is caught (planted in the oracle's output, on CPU)."""
    o = oracle_mod
    p = _rand_problem(20, 20, seed=81)
    r = o.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], p["bits"])
    bad = r["codes"].copy()
    i, j = 7, 11
    bad[i, j] = bad[i, j] + 1 if bad[i, j] < 7 else bad[i, j] - 1
    x = o.certificate(p["W"], p["A"], p["B"], p["damp"], p["scale"], bad, p["bits"])
    v = o.verdict(bad, x, p["bits"])
    assert v["violations"] >= 1


def test_tie_forcing_adopts_forced_codes(oracle_mod):
    """With a huge window every interior entry is excused and the forced codes
    are adopted; the replay stays a valid trajectory (certificate)."""
    o = oracle_mod
    p = _rand_problem(12, 12, seed=91)
    r = o.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], p["bits"])
    forced = np.clip(r["codes"].astype(np.int16) + 1, -7, 7).astype(np.int8)
    rf = o.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], p["bits"], forced=forced,
                 tie_window=0.6)
    inner = np.abs(rf["pre"]) < 7.0
    assert np.array_equal(rf["codes"][inner], forced[inner])
    assert rf["n_excused"] >= int(np.count_nonzero(inner))
    x = o.certificate(p["W"], p["A"], p["B"], p["damp"], p["scale"], rf["codes"], p["bits"])
    np.testing.assert_allclose(x, rf["pre"], atol=1e-9)


def test_objective_is_kronecker_quadratic(oracle_mod):
    """Prop. 3.1: tr(D^T B D A) = vec(D)^T (A (x) B) vec(D), vec column-major."""
    o = oracle_mod
    p = _rand_problem(6, 7, seed=101)
    r = o.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], p["bits"])
    D = p["W"].astype(np.float64) - r["V"]
    d = D.reshape(-1, order="F")
    H = np.kron(o.damp(p["A"], p["damp"]), o.damp(p["B"], p["damp"]))
    ref = float(d @ H @ d)
    assert abs(o.objective(p["W"], r["V"], p["A"], p["B"], p["damp"]) - ref) <= 1e-12 * abs(ref)


def test_babai_beats_round_to_nearest(oracle_mod):
    """Sanity on the objective: sequential feedback lowers tr(D^T B D A) versus
    plain rounding on a correlated workload (config 1)."""
    o = oracle_mod
    c = workloads.make(1, seed=0)
    r = o.solve(c["W"], c["A"], c["B"], c["damp"], c["scale"], c["bits"])
    rtn = o.quantise_codes(c["W"].astype(np.float64) / c["scale"][:, None], c["bits"])
    Vr = c["scale"][:, None].astype(np.float64) * rtn
    assert o.objective(c["W"], r["V"], c["A"], c["B"], c["damp"]) < \
        o.objective(c["W"], Vr, c["A"], c["B"], c["damp"])


@pytest.mark.parametrize("m,n,identity_B", [(40, 30, False), (30, 45, False), (25, 33, True)])
def test_certify_matches_certificate_and_objective(oracle_mod, m, n, identity_B):
    """The one-pass full-size certify() (triangular products, objective as
    |R_B D R_A^T|_F^2) agrees with certificate() + verdict() and with the
    explicit objective tr(D^T B_d D A_d); a planted wrong code is caught."""
    o = oracle_mod
    p = _rand_problem(m, n, seed=m + n, identity_B=identity_B)
    r = o.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], p["bits"])
    c = o.certify(p["W"], p["A"], p["B"], p["damp"], p["scale"], r["codes"], p["bits"],
                  row_block=7)
    x = o.certificate(p["W"], p["A"], p["B"], p["damp"], p["scale"], r["codes"], p["bits"])
    np.testing.assert_allclose(c["x"], x, rtol=0, atol=1e-10)
    np.testing.assert_allclose(c["x"], r["pre"], rtol=0, atol=1e-9)
    assert c["verdict"]["violations"] == 0 and c["verdict"]["flips"] == 0
    obj = o.objective(p["W"], r["V"], p["A"], p["B"], p["damp"])
    assert abs(c["objective"] - obj) <= 1e-12 * obj
    bad = r["codes"].copy()
    bad[m // 2, n // 3] += 1 if bad[m // 2, n // 3] < 7 else -1
    cb = o.certify(p["W"], p["A"], p["B"], p["damp"], p["scale"], bad, p["bits"])
    assert cb["verdict"]["violations"] >= 1
