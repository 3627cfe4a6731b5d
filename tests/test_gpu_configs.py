"""Full-size configurations, in the launch configuration bench.py times (a
stream of its own, where node pushes into later segments overlap with the
segment launches on a CU-restricted side stream).

At these sizes the sequential oracle cannot replay every entry, so parity is
checked two ways:
  * certificate (property that holds at any size): with the GPU's codes, the
    closed form W~ = V - R^_B (V - W0) R^_A^T gives the value at which each
    entry must have been quantised along the GPU's own trajectory; every code
    must equal quantise(W~/s) except within 1e-4 grid steps of a boundary
    (computed in fp64 on the host for sampled rows; all rows for 4096^2);
  * structured exact oracle: A, B AR(1) Toeplitz without damping, whose
    factors are bidiagonal, so the O(mn) three-neighbour recursion is the
    exact sequential rounding at the full shape.
"""
import numpy as np
import pytest

import workloads
from gpu_util import TIE_WINDOW, MAX_FLIP_RATE, gpu_run, log, v_is_scale_times_code

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _run(p, debug):
    """gpu_run on a non-default stream, as bench.py runs the solver."""
    import torch
    with torch.cuda.stream(torch.cuda.Stream()):
        return gpu_run(p, debug=debug)


def _rows(m, full):
    if full:
        return None
    rng = np.random.default_rng(m)
    base = [0, 1, 31, 32, 33, 63, 64, m // 2, m - 33, m - 32, m - 1]
    return np.unique(np.concatenate([base, rng.choice(m, 37, replace=False)]))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cid", [2, 3, 4, 5])
def test_config_certificate(oracle_mod, cid):
    o = oracle_mod
    log(f"case config {cid}: generating")
    c = workloads.make(cid, seed=0, device="cuda")
    m, n = c["W"].shape
    log(f"case config {cid}: solving {m}x{n}")
    codes, V, pre = _run(c, True)
    assert v_is_scale_times_code(V, codes, c["scale"])
    l = (1 << (c["bits"] - 1)) - 1
    assert np.all(np.abs(codes.astype(np.int32)) <= l)
    rows = _rows(m, full=(cid == 2))
    log(f"case config {cid}: certificate on {'all' if rows is None else len(rows)} rows")
    x = o.certificate(c["W"], c["A"], c["B"], c["damp"], c["scale"], codes, c["bits"], rows=rows)
    cr = codes if rows is None else codes[rows]
    pr = pre if rows is None else pre[rows]
    v = o.verdict(cr, x, c["bits"], window=TIE_WINDOW)
    fin = np.isfinite(x)
    margin = float(np.max(np.abs(pr[fin].astype(np.float64) - x[fin])))
    log(f"[config{cid}] {v} margin={margin:.3e}")
    assert v["violations"] == 0
    assert v["flips"] <= MAX_FLIP_RATE * v["total"]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("cid", [2, 4, 5])
def test_config_shape_ar1_exact(oracle_mod, cid):
    cfg = workloads.CONFIGS[cid]
    W = workloads.make_weights(cfg, seed=1)
    s = workloads.row_scales(W, cfg.bits)
    p = dict(W=W, A=workloads.ar1_toeplitz(cfg.n, 0.5), B=workloads.ar1_toeplitz(cfg.m, 0.25),
             scale=s, bits=cfg.bits, damp=0.0)
    log(f"case AR(1) at config {cid} shape {cfg.m}x{cfg.n}")
    codes, V, pre = _run(p, False)
    r = oracle_mod.ar1_diffusion(W, 0.5, 0.25, s, cfg.bits, forced=codes, tie_window=TIE_WINDOW)
    viol = int(np.count_nonzero(r["codes"] != codes))
    log(f"[ar1 config{cid}] violations={viol} flips={r['n_flip']} excused={r['n_excused']}")
    assert viol == 0
    assert r["n_flip"] <= MAX_FLIP_RATE * W.size
    assert v_is_scale_times_code(V, codes, s)


@pytest.mark.timeout(600)
def test_config2_two_stream_plan_bitwise():
    """The 4096x4096 layer on a stream of its own (node pushes overlapped on the
    side stream) and on the legacy default stream (everything on one stream):
    bitwise identical codes, V and pre-rounding values."""
    c = workloads.make(2, seed=0, device="cuda")
    log("case config 2 two-stream vs one-stream plan")
    c1, v1, x1 = _run(c, True)
    c0, v0, x0 = gpu_run(c, debug=True)
    assert np.array_equal(c0, c1)
    assert np.array_equal(v0.view(np.uint32), v1.view(np.uint32))
    assert np.array_equal(x0.view(np.uint32), x1.view(np.uint32))


@pytest.mark.timeout(900)
def test_config2_general_quantiser_certificate(oracle_mod):
    """The 4096 x 4096 layer with the general quantiser (asymmetric INT4
    alphabet, MSE-searched 128-column group scales, per-column factors), at
    full size on a stream of its own: the closed-form certificate on sampled
    rows with per-entry scales."""
    import torch
    import paper_2608_06291_amd as pk
    o = oracle_mod
    log("case config 2 general quantiser: generating")
    c = workloads.make(2, seed=0, device="cuda")
    m, n = c["W"].shape
    # the scales: the GPU search is itself checked against the oracle's
    # elsewhere; here the oracle's own search provides them
    scale, _ = o.mse_scales(c["W"], 4, "asym", group_size=128)
    col = np.random.Generator(np.random.PCG64(77)).uniform(0.8, 1.25, n).astype(np.float32)
    p = dict(c, scale=scale, alphabet="asym", group_size=128, col_scale=col)
    log("case config 2 general quantiser: solving")
    codes, V, pre = _run(p, True)
    S = o.entry_scales(scale, m, n, group_size=128, col_scale=col)
    assert v_is_scale_times_code(V, codes, S)
    assert np.all((codes >= -8) & (codes <= 7))
    rows = _rows(m, full=False)
    x = o.certificate(c["W"], c["A"], c["B"], c["damp"], S, codes, 4, rows=rows)
    v = o.verdict(codes[rows], x, 4, window=TIE_WINDOW, alphabet="asym")
    fin = np.isfinite(x)
    margin = float(np.max(np.abs(pre[rows][fin].astype(np.float64) - x[fin])))
    log(f"[config2-general] {v} margin={margin:.3e}")
    assert v["violations"] == 0
    assert v["flips"] <= MAX_FLIP_RATE * v["total"]
    del torch, pk
