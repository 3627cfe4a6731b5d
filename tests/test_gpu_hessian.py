"""GPU parity of the Kronecker-factor construction (App. A) with the fp64
oracle, through the C ABI (bakron_gram, bakron_sample_weights,
bakron_kron_factors, bakron_mlp_local_factors).

Tolerance (fp32 arithmetic, derived from the summation): every entry of a
factor is a sum of N products w_k x_ki x_kj accumulated in fp32 (one rounding
per product, per weight multiply, per addition, per scale and mask
multiply), and each Shampoo weight a sum of d squares; the recursive-summation
bound gives
    |C_gpu - C| <= (N + d + 8) u * s |M_ij| sum_k |w_k x_ki x_kj|,  u = 2^-24,
checked entry by entry, plus a typical-error check: the relative Frobenius
error stays below 20 sqrt(N + d) u.
"""
import numpy as np
import pytest

import workloads
from gpu_util import log

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


def _dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to("cuda:0")


def _check(got, expect, abssum, N, d, label):
    got = np.asarray(got, np.float64)
    err = np.abs(got - expect)
    bound = (N + d + 8) * U32 * abssum + 1e-30
    worst = float(np.max(err / bound)) if err.size else 0.0
    fro = float(np.linalg.norm(got - expect) / max(np.linalg.norm(expect), 1e-300))
    log(f"[{label}] max err/bound {worst:.3e}  rel fro {fro:.3e}")
    assert worst <= 1.0, label
    assert fro <= 20 * np.sqrt(N + d) * U32, label


def _abssum(X, w=None, s=1.0, M=None):
    """s |M| (.) sum_k |w_k| |x_k| |x_k|^T in fp64 (the error-bound scale)."""
    Xa = np.abs(np.asarray(X, np.float64))
    wa = np.ones(Xa.shape[0]) if w is None else np.abs(np.asarray(w, np.float64))
    S = (Xa * wa[:, None]).T @ Xa * abs(s)
    return S if M is None else S * np.abs(np.asarray(M, np.float64))


@pytest.mark.parametrize("N,d", [(1, 1), (7, 5), (33, 130), (1000, 200), (4097, 260), (3000, 258),
                                 (64, 640)])
@pytest.mark.parametrize("weighted,masked", [(False, False), (True, True)])
def test_gram_parity(oracle_mod, N, d, weighted, masked):
    import torch
    import paper_2608_06291_amd as pk
    h = oracle_mod.hessian
    log(f"case gram N={N} d={d} w={weighted} M={masked}")
    r = np.random.Generator(np.random.PCG64(np.random.SeedSequence([4000, N, d])))
    X = workloads.ar1_samples(N, d, 0.5, r, norm_sigma=0.5)
    w = r.standard_normal(N).astype(np.float32) if weighted else None   # signed weights too
    M = None
    if masked:
        Z = r.standard_normal((d, 3))
        M = (Z @ Z.T).astype(np.float32)
    s = np.float32(0.37)
    C = pk.gram(_dev(X), None if w is None else _dev(w), float(s), None if M is None else _dev(M))
    torch.cuda.synchronize()
    C = C.cpu().numpy()
    expect = float(s) * N * h.expect_outer(X, w)
    if M is not None:
        expect = expect * M.astype(np.float64)
    _check(C, expect, _abssum(X, w, float(s), M), N, d, f"gram{N}x{d}")
    if M is None:
        assert np.array_equal(C, C.T), "C must be exactly symmetric"


def test_gram_in_place_mask_empty_and_deterministic(oracle_mod):
    import torch
    import paper_2608_06291_amd as pk
    h = oracle_mod.hessian
    r = np.random.Generator(np.random.PCG64(np.random.SeedSequence([4001])))
    N, d = 2500, 300
    X = workloads.ar1_samples(N, d, 0.3, r)
    Z = r.standard_normal((d, 5))
    M = (Z @ Z.T).astype(np.float32)
    Xd = _dev(X)
    log("case gram in-place M")
    C = _dev(M)
    pk.gram(Xd, None, 1.0 / N, C, C)
    ref = pk.gram(Xd, None, 1.0 / N, _dev(M))
    torch.cuda.synchronize()
    assert torch.equal(C, ref), "in-place mask must equal the out-of-place result"
    expect = h.expect_outer(X) * M.astype(np.float64)
    _check(C.cpu().numpy(), expect, _abssum(X, None, 1.0 / N, M), N, d, "gram-inplace")
    log("case gram repeat bitwise")
    for _ in range(2):
        again = pk.gram(Xd, None, 1.0 / N, _dev(M))
        torch.cuda.synchronize()
        assert torch.equal(again, ref)
    log("case gram N=0")
    C0 = torch.full((7, 7), 3.0, device="cuda:0")
    pk.gram(torch.empty((0, 7), device="cuda:0"), None, 1.0, None, C0)
    torch.cuda.synchronize()
    assert torch.count_nonzero(C0).item() == 0


@pytest.mark.parametrize("N,d,withc", [(1, 3, False), (513, 200, True), (300, 258, True),
                                       (100, 4096, False)])
def test_sample_weights_parity(oracle_mod, N, d, withc):
    import torch
    import paper_2608_06291_amd as pk
    log(f"case sample weights N={N} d={d} c={withc}")
    r = np.random.Generator(np.random.PCG64(np.random.SeedSequence([4002, N, d])))
    X = workloads.ar1_samples(N, d, 0.5, r, norm_sigma=1.0)
    c = r.lognormal(0, 1, d).astype(np.float32) if withc else None
    w = pk.sample_weights(_dev(X), None if c is None else _dev(c))
    torch.cuda.synchronize()
    w = w.cpu().numpy().astype(np.float64)
    # tr(a^T C a) with C = diag(c): the oracle's per-sample trace
    expect = oracle_mod.hessian.trace_quad(X, None if c is None else np.diag(c.astype(np.float64)))
    # positive terms: relative bound (d + 2) u
    assert np.all(np.abs(w - expect) <= (d + 2) * U32 * np.abs(expect) + 1e-30)


@pytest.mark.parametrize("style", ["kfac", "shampoo"])
@pytest.mark.parametrize("N,n,m", [(1, 4, 3), (3000, 200, 130), (777, 257, 64)])
def test_kron_factors_parity(oracle_mod, style, N, n, m):
    import torch
    import paper_2608_06291_amd as pk
    h = oracle_mod.hessian
    log(f"case kron factors {style} N={N} n={n} m={m}")
    p = workloads.kron_samples(N, n, m, seed=1)
    A, B = pk.kron_factors(_dev(p["a"]), _dev(p["b"]), style)
    torch.cuda.synchronize()
    if style == "kfac":
        eA, eB = h.kfac_factors(p["a"], p["b"])
        wA = wB = None
    else:
        eA, eB = h.shampoo_factors(p["a"], p["b"], iters=1)
        wA, wB = h.trace_quad(p["b"]), h.trace_quad(p["a"])
    _check(A.cpu().numpy(), eA, _abssum(p["a"], wA, 1.0 / N), N, max(n, m), f"kron-A-{style}")
    _check(B.cpu().numpy(), eB, _abssum(p["b"], wB, 1.0 / N), N, max(n, m), f"kron-B-{style}")


@pytest.mark.parametrize("style", ["kfac", "shampoo"])
@pytest.mark.parametrize("which", ["g", "f"])
@pytest.mark.parametrize("N,dm,dff", [(2, 3, 5), (600, 96, 160), (300, 130, 258)])
def test_mlp_local_factors_parity(oracle_mod, style, which, N, dm, dff):
    """The oracle forms b = D_g W_down^T explicitly per sample; the GPU uses
    b b^T = (g g^T) (.) W_down^T W_down and tr(b^T b) = g^T diag(D^T D) g."""
    import torch
    import paper_2608_06291_amd as pk
    h = oracle_mod.hessian
    log(f"case mlp-local {style} feat={which} N={N} dm={dm} dff={dff}")
    p = workloads.mlp_samples(N, dm, dff, seed=2)
    x, g, D = p["x"], p[which], p["Wd"]
    A, B = pk.mlp_local_factors(_dev(x), _dev(g), _dev(D), style)
    torch.cuda.synchronize()
    eA, eB = h.mlp_local_factors(x, g, D, style)
    DtD_abs = np.abs(D.astype(np.float64)).T @ np.abs(D.astype(np.float64))
    if style == "kfac":
        wA = wB = None
    else:
        wA = h.trace_quad(h.mlp_local_b(g, D))
        wB = h.trace_quad(x)
    # D^T D is itself an fp32 Gram over dm rows: its error adds dm to the chain
    _check(A.cpu().numpy(), eA, _abssum(x, wA, 1.0 / N), N + dff, dm, f"mlp-A-{style}-{which}")
    _check(B.cpu().numpy(), eB, _abssum(g, wB, 1.0 / N, DtD_abs), N + dm, max(dm, dff),
           f"mlp-B-{style}-{which}")


@pytest.mark.parametrize("N,d", [(1, 1), (300, 130), (1000, 258), (513, 256)])
def test_quadform_weights_parity(oracle_mod, N, d):
    """w_k = x_k^T M x_k against the oracle's per-sample trace tr(x^T M x):
    a sum of d inner sums of d products each, so the fp32 bound is
    (2d + 8) u |x|^T |M| |x| per sample."""
    import torch
    import paper_2608_06291_amd as pk
    log(f"case quadform N={N} d={d}")
    r = np.random.Generator(np.random.PCG64(np.random.SeedSequence([4100, N, d])))
    X = workloads.ar1_samples(N, d, 0.4, r, norm_sigma=0.5)
    Z = r.standard_normal((d, d + 3))
    M = (Z @ Z.T / d).astype(np.float32)
    w = pk.quadform_weights(_dev(X), _dev(M))
    torch.cuda.synchronize()
    w = w.cpu().numpy().astype(np.float64)
    expect = oracle_mod.hessian.trace_quad(X, M.astype(np.float64))
    Xa = np.abs(X.astype(np.float64))
    bound = (2 * d + 8) * U32 * np.einsum("kj,jt,kt->k", Xa, np.abs(M.astype(np.float64)), Xa)
    assert np.all(np.abs(w - expect) <= bound + 1e-30)


def _iter_tol(N, d, iters):
    """Relative Frobenius tolerance of `iters` power steps: each step adds a
    Gram's and a quadratic form's fp32 error on top of the previous pair's."""
    return iters * 40 * np.sqrt(N + 2 * d) * U32


@pytest.mark.parametrize("iters", [2, 3])
@pytest.mark.parametrize("N,n,m", [(2000, 200, 130), (257, 33, 70)])
def test_kron_factors_power_steps(oracle_mod, iters, N, n, m):
    import torch
    import paper_2608_06291_amd as pk
    h = oracle_mod.hessian
    log(f"case shampoo iters={iters} N={N} n={n} m={m}")
    p = workloads.kron_samples(N, n, m, seed=3)
    A, B = pk.kron_factors(_dev(p["a"]), _dev(p["b"]), "shampoo", iters=iters)
    torch.cuda.synchronize()
    eA, eB = h.shampoo_factors(p["a"], p["b"], iters=iters)
    for got, exp, d, lab in ((A, eA, n, "A"), (B, eB, m, "B")):
        got = got.cpu().numpy().astype(np.float64)
        rel = np.linalg.norm(got - exp) / np.linalg.norm(exp)
        log(f"[shampoo{iters}] {lab} rel fro {rel:.2e}")
        assert rel <= _iter_tol(N, d, iters), (lab, rel)
        assert np.array_equal(got, got.T)


@pytest.mark.parametrize("iters", [2, 3])
def test_mlp_local_power_steps(oracle_mod, iters):
    """The oracle forms b = D_g W_down^T and tr(b^T B b) explicitly; the GPU
    uses g^T (B (.) D^T D) g."""
    import torch
    import paper_2608_06291_amd as pk
    h = oracle_mod.hessian
    N, dm, dff = 300, 64, 96
    log(f"case mlp-local shampoo iters={iters}")
    p = workloads.mlp_samples(N, dm, dff, seed=4)
    A, B = pk.mlp_local_factors(_dev(p["x"]), _dev(p["g"]), _dev(p["Wd"]), "shampoo", iters=iters)
    torch.cuda.synchronize()
    eA, eB = h.mlp_local_factors(p["x"], p["g"], p["Wd"], "shampoo", iters=iters)
    for got, exp, lab in ((A, eA, "A"), (B, eB, "B")):
        got = got.cpu().numpy().astype(np.float64)
        rel = np.linalg.norm(got - exp) / np.linalg.norm(exp)
        log(f"[mlp shampoo{iters}] {lab} rel fro {rel:.2e}")
        assert rel <= _iter_tol(N + dm, dff, iters), (lab, rel)


def test_power_step_one_is_single_shampoo():
    """iters = 1 through the iterating entry point is the one-step pair, bit
    for bit."""
    import torch
    import paper_2608_06291_amd as pk
    p = workloads.kron_samples(700, 100, 60, seed=5)
    a, b = _dev(p["a"]), _dev(p["b"])
    A1, B1 = pk.kron_factors(a, b, "shampoo")
    lib = pk.load()
    import ctypes
    A2 = torch.empty_like(A1)
    B2 = torch.empty_like(B1)
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    pk._lib._with_workspace(lambda wk, nb: lib.bakron_kron_factors_iter(
        pk._lib._ptr(a), pk._lib._ptr(b), 700, 100, 60, 1, pk._lib._ptr(A2), pk._lib._ptr(B2), wk,
        nb, st), a.device)
    torch.cuda.synchronize()
    assert torch.equal(A1, A2) and torch.equal(B1, B2)


def _sampled_pairs(rng, d, k=40):
    pr = [(int(i), int(j)) for i, j in rng.integers(0, d, (k, 2))]
    return pr + [(i, i) for i in rng.integers(0, d, 8).tolist()]


@pytest.mark.parametrize("workload", ["global-kfac", "global-shampoo", "mlp-local-kfac"])
def test_factors_full_size_sampled(oracle_mod, workload):
    """bench.py --factors' launch configuration at the paper's calibration size
    (256 x 2048 samples): 48 entries of each factor against the oracle's
    per-entry means, within the summation bound of each entry."""
    import torch
    import paper_2608_06291_amd as pk
    h = oracle_mod.hessian
    N = 256 * 2048
    dev = torch.device("cuda:0")
    log(f"case full-size factors {workload} N={N}")
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([4200, len(workload)])))
    if workload.startswith("global"):
        p = workloads.kron_samples_torch(N, 4096, 4096, 0, dev)
        a, b, D = p["a"], p["b"], None
        style = workload.split("-")[1]
        A, B = pk.kron_factors(a, b, style)
    else:
        p = workloads.mlp_samples_torch(N, 4096, 14336, 0, dev, "g")
        a, b, D = p["x"], p["feat"], p["Wd"]
        style = "kfac"
        A, B = pk.mlp_local_factors(a, b, D, style)
    torch.cuda.synchronize()
    for X, F, wsrc, mask, lab in ((a, A, b, None, "A"), (b, B, a, D, "B")):
        d = X.shape[1]
        pr = _sampled_pairs(rng, d)
        idx = sorted({i for q in pr for i in q})
        cols = X[:, idx].double().cpu().numpy()
        pos = {c: t for t, c in enumerate(idx)}
        q = [(pos[i], pos[j]) for i, j in pr]
        w = None
        if style == "shampoo":   # |other sample|^2 as the weight, fp64 on the CPU
            w = np.empty(N)
            for k0 in range(0, N, 65536):
                blk = wsrc[k0:k0 + 65536].double()
                w[k0:k0 + 65536] = (blk * blk).sum(1).cpu().numpy()
        expect = h.expect_outer_entries(cols, q, w)
        absum = h.expect_outer_entries(np.abs(cols), q, None if w is None else np.abs(w))
        if mask is not None:
            dcols = mask[:, idx].double().cpu().numpy()
            m_e = mask.shape[0] * h.expect_outer_entries(dcols, q)
            m_a = mask.shape[0] * h.expect_outer_entries(np.abs(dcols), q)
            expect, absum = expect * m_e, absum * np.abs(m_a)
        got = np.array([F[i, j].item() for i, j in pr])
        bound = (N + 2 * d + 8) * U32 * absum
        worst = float(np.max(np.abs(got - expect) / (bound + 1e-30)))
        log(f"[full {workload}] {lab} max err/bound {worst:.3e}")
        assert worst <= 1.0, (workload, lab)
    del a, b, D, A, B, p
    torch.cuda.empty_cache()
