"""Pins for the oracle's quantiser variants (Sec. 3.1, App. D), CPU only:
the (b+1)-bit alphabet {-2^b..2^b-1}, scales per row and/or column (row or
column-group scales times column factors), the MSE scale search, and a
block-diagonal output factor B assembled from per-head Grams."""
import itertools

import numpy as np
import pytest

import workloads


def _q(x, lo, hi):
    """Nearest alphabet element in fp32, half to even (the fixed tie rule)."""
    return int(min(max(np.rint(np.float32(x)), lo), hi))


def _gptq_vector(w, H, svec, lo, hi):
    """Alg. 1 on one vector with a per-coordinate scale and alphabet {lo..hi},
    written independently of the oracle: Cholesky(H^-1), unit columns."""
    L = np.linalg.cholesky(np.linalg.inv(H))
    L = L / np.diag(L)[None, :]
    w = np.array(w, np.float64).copy()
    codes = np.zeros(w.shape[0], np.int64)
    for i in range(w.shape[0]):
        s = svec[i]
        c = 0 if s == 0 else _q(w[i] / s, lo, hi)
        codes[i] = c
        w = w + (s * c - w[i]) * L[:, i]
    return codes


def _rng(*k):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([7100, *k])))


def test_alphabets(oracle_mod):
    o = oracle_mod
    assert o.alphabet_bounds(4, "sym") == (-7, 7)
    assert o.alphabet_bounds(2, "asym") == (-2, 1)
    assert o.alphabet_bounds(8, "asym") == (-128, 127)
    x = np.array([-2.6, -2.5, -1.5, -0.5, 0.5, 1.4, 1.5, 3.0, np.nan])
    assert o.quantise_codes(x, 2, "asym").tolist() == [-2, -2, -2, 0, 0, 1, 1, 1, 0]
    assert o.quantise_codes(x, 2, "sym").tolist() == [-1, -1, -1, 0, 0, 1, 1, 1, 0]
    # boundaries of {-2..1}: -1.5, -0.5, 0.5 only
    near = o.near_boundary(np.array([-2.5, -1.5, -0.5, 0.5, 1.5]), 2, 1e-3, "asym")
    assert near.tolist() == [False, True, True, True, False]


def test_entry_scales_definition(oracle_mod):
    r = _rng(1)
    m, n, g = 3, 10, 4
    G = r.uniform(0.5, 2, (m, 3)).astype(np.float32)
    c = r.uniform(0.5, 2, n).astype(np.float32)
    S = oracle_mod.entry_scales(G, m, n, group_size=g, col_scale=c)
    for i, j in itertools.product(range(m), range(n)):
        assert S[i, j] == float(np.float32(G[i, j // g] * c[j]))
    rs = r.uniform(0.5, 2, m).astype(np.float32)
    S2 = oracle_mod.entry_scales(rs, m, n)
    assert np.all(S2 == rs.astype(np.float64)[:, None])


@pytest.mark.parametrize("alphabet,group,cols", [("asym", 0, False), ("sym", 3, True),
                                                  ("asym", 2, True), ("sym", 0, True)])
@pytest.mark.parametrize("m,n", [(3, 4), (5, 6), (4, 7)])
def test_explicit_kronecker_hessian_general_quantiser(oracle_mod, alphabet, group, cols, m, n):
    """GPTQ on vec(W) (column-major) with H = A_d (x) B_d and the per-entry
    scales and alphabet of the variant equals the 2-D oracle."""
    o = oracle_mod
    p = workloads.make_random(m, n, seed=40 + m * 7 + n + group, bits=3)
    r = _rng(2, m, n, group)
    W = p["W"].astype(np.float64)
    G = -(-n // group) if group else 1
    rowscale = (r.uniform(0.3, 1.0, (m, G)) * np.abs(W).max() / 3).astype(np.float32)
    scale = rowscale if group else rowscale[:, 0]
    col = r.uniform(0.5, 1.5, n).astype(np.float32) if cols else None
    S = o.entry_scales(scale, m, n, group_size=group, col_scale=col)
    lo, hi = o.alphabet_bounds(3, alphabet)
    H = np.kron(o.damp(p["A"], p["damp"]), o.damp(p["B"], p["damp"]))
    ref = _gptq_vector(W.reshape(-1, order="F"), H, S.reshape(-1, order="F"), lo, hi)
    got = o.solve(W, p["A"], p["B"], p["damp"], S, 3, alphabet=alphabet)["codes"]
    assert np.array_equal(got, ref.reshape((m, n), order="F"))


def test_B_identity_with_column_scales_is_gptq_per_row(oracle_mod):
    o = oracle_mod
    m, n = 6, 20
    p = workloads.make_random(m, n, seed=3, identity_B=True)
    col = _rng(3).uniform(0.5, 1.5, n).astype(np.float32)
    S = o.entry_scales(p["scale"], m, n, col_scale=col)
    Ad = o.damp(p["A"], p["damp"])
    got = o.solve(p["W"], p["A"], None, p["damp"], S, 4, alphabet="asym")["codes"]
    for i in range(m):
        ref = _gptq_vector(p["W"][i].astype(np.float64), Ad, S[i], -8, 7)
        assert np.array_equal(got[i], ref), i


def test_diagonal_hessians_round_to_nearest_grouped_asym(oracle_mod):
    o = oracle_mod
    r = _rng(4)
    m, n, g = 7, 12, 5
    W = r.standard_normal((m, n)) * 0.02
    G = (r.uniform(0.5, 1.0, (m, 3)) * 0.02 / 2).astype(np.float32)
    A = np.diag(r.uniform(0.5, 2.0, n))
    B = np.diag(r.uniform(0.5, 2.0, m))
    S = o.entry_scales(G, m, n, group_size=g)
    got = o.solve(W, A, B, 0.01, S, 3, alphabet="asym")["codes"]
    assert np.array_equal(got, o.quantise_codes(W / S, 3, "asym"))


# ---------------------------------------------------------------- MSE scales
def test_mse_scales_brute_force(oracle_mod):
    """Every candidate of every row evaluated with scalar fp32 arithmetic; the
    chosen scale is the first minimiser (App. D: shrink by up to 2x)."""
    o = oracle_mod
    r = _rng(5)
    W = (r.standard_t(3, (6, 9)) * 0.01).astype(np.float32)
    W[2] = 0.0                                       # all candidates tie: no shrink
    for alphabet in ("sym", "asym"):
        lo, hi = o.alphabet_bounds(3, alphabet)
        got, _ = o.mse_scales(W, 3, alphabet, grid=20, maxshrink=0.5)
        for i in range(W.shape[0]):
            base = np.float32(np.max(np.abs(W[i])) / np.float32(hi))
            best, best_e = None, None
            for k in range(21):
                s = np.float32(base * np.float32(1.0 - 0.5 * k / 20))
                e = 0.0
                for wv in W[i]:
                    c = 0 if s == 0 else _q(np.float32(wv / s), lo, hi)
                    e += (float(wv) - float(np.float32(s * np.float32(c)))) ** 2
                if best_e is None or e < best_e:
                    best, best_e = s, e
            assert got[i] == best, (alphabet, i)
    assert got[2] == 0.0


def test_mse_scales_exact_grid_and_outlier(oracle_mod):
    o = oracle_mod
    # a row already on the grid of its max-abs scale: no shrink (zero error)
    s0 = np.float32(0.01)
    W = (np.array([[-7, -3, 0, 2, 5, 7]], np.float32) * s0).astype(np.float32)
    got, err = o.mse_scales(W, 4, "sym")
    assert got[0] == np.float32(np.max(np.abs(W)) / 7) and err[0, 0] == 0.0
    # one entry 1.0 among many 0.5 with l = 3: the max-abs scale 1/3 puts 0.5
    # at 1.5 grid steps (error 1/6 each, 1.75 in all); the candidate 1/4 puts it
    # on the grid and only clips the 1.0 to 0.75 (error 0.0625), so the search
    # shrinks to a scale at least as good as 1/4
    W = np.full((1, 64), 0.5, np.float32)
    W[0, 0] = 1.0
    got, err = o.mse_scales(W, 3, "sym")
    assert got[0] < np.float32(1.0 / 3) and abs(err[0, 0] - 1.75) < 1e-5
    assert err[0].min() <= 0.0625 + 1e-12


# ---------------------------------------------------------------- block-diagonal B
def test_block_diagonal_B_decouples_heads(oracle_mod):
    """With B = blockdiag(B_1..B_H) (the per-head output Grams of an attention
    projection assembled into one matrix, App. D), no feedback crosses heads:
    the solve equals the per-head solves stacked (damping applied beforehand)."""
    o = oracle_mod
    H, hb, n = 3, 5, 8
    p = workloads.make_random(H * hb, n, seed=8)
    r = _rng(8)
    blocks = []
    for h in range(H):
        Z = r.standard_normal((hb, 3 * hb))
        blocks.append(Z @ Z.T / (3 * hb) + 0.1 * np.eye(hb))
    B = np.zeros((H * hb, H * hb))
    for h in range(H):
        B[h * hb:(h + 1) * hb, h * hb:(h + 1) * hb] = blocks[h]
    Ad = o.damp(p["A"], p["damp"])
    full = o.solve(p["W"], Ad, B, 0.0, p["scale"], 4)["codes"]
    for h in range(H):
        rows = slice(h * hb, (h + 1) * hb)
        part = o.solve(p["W"][rows], Ad, blocks[h], 0.0, p["scale"][rows], 4)["codes"]
        assert np.array_equal(full[rows], part), h
    # and the normalised factor of the block-diagonal matrix is block-diagonal
    LB = o.normalized_factor(B, 0.0)
    for h in range(H):
        rows = slice(h * hb, (h + 1) * hb)
        np.testing.assert_allclose(LB[rows, rows], o.normalized_factor(blocks[h], 0.0),
                                   atol=1e-12)
        LB[rows, rows] = 0
    assert np.max(np.abs(LB)) < 1e-12
