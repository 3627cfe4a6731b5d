"""B = NULL (B = I): the one-sided GPTQ kernel (Alg. 1 on every row with the
Hessian A, blocked lazy updates on fp32 MFMA) against the fp64 oracle run
with B = I, element by element under the tie-forced protocol; ragged shapes
that span several 16-row groups and 32-column blocks, every quantiser
variant, the two-sided solver forced with BAKRON_GPTQ=0 on the same inputs,
determinism and a poisoned workspace."""
import os

import numpy as np
import pytest

import workloads
from gpu_util import check_against_oracle, gpu_run, log

pytestmark = pytest.mark.gpu


def _problem(m, n, seed, bits=4):
    return workloads.make_random(m, n, seed, bits=bits, identity_B=True)


class _env:
    def __init__(self, **kv):
        self.kv = kv

    def __enter__(self):
        self.old = {k: os.environ.get(k) for k in self.kv}
        os.environ.update({k: str(v) for k, v in self.kv.items()})

    def __exit__(self, *a):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


@pytest.mark.parametrize("m,n", [(1, 1), (1, 37), (37, 1), (5, 37), (16, 32), (17, 33), (33, 65),
                                 (130, 257), (257, 97), (64, 64)])
def test_gptq_shapes(oracle_mod, m, n):
    p = _problem(m, n, seed=500 + m + 7 * n)
    log(f"case one-sided m={m} n={n}")
    codes, V, pre = gpu_run(p)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"gptq{m}x{n}")


@pytest.mark.parametrize("rng_tiles,m,n", [(1, 65, 97), (3, 130, 257), (2, 257, 97), (5, 200, 300),
                                             (1, 16, 70)])
def test_gptq_multi_range(oracle_mod, rng_tiles, m, n):
    """Column ranges of a few tiles (BAKRON_GPTQ_RANGE), so that small ragged
    shapes run several ranges and the pushes between them (partial last
    range, partial row and column blocks of the push)."""
    p = _problem(m, n, seed=900 + rng_tiles + m + 3 * n)
    log(f"case one-sided m={m} n={n} range={rng_tiles} tiles")
    with _env(BAKRON_GPTQ_RANGE=rng_tiles):
        codes, V, pre = gpu_run(p)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"gptq{m}x{n}r{rng_tiles}")


@pytest.mark.parametrize("rng_tiles", [None, 2])
@pytest.mark.parametrize("variant", ["bits2", "bits8", "asym+groups+cols", "zero-rows"])
def test_gptq_quantisers(oracle_mod, variant, rng_tiles):
    m, n = 90, 150
    p = _problem(m, n, seed=61, bits={"bits2": 2, "bits8": 8}.get(variant, 4))
    if variant == "asym+groups+cols":
        g = 32
        rng = np.random.default_rng(5)
        p["scale"] = (p["scale"][:, None] * rng.uniform(0.6, 1.4, (m, -(-n // g)))).astype(np.float32)
        p["group_size"] = g
        p["alphabet"] = "asym"
        p["col_scale"] = rng.uniform(0.8, 1.25, n).astype(np.float32)
    if variant == "zero-rows":
        p["scale"] = p["scale"].copy()
        p["scale"][[0, 45, 89]] = 0.0
    log(f"case one-sided quantiser {variant}, range {rng_tiles}")
    env = {} if rng_tiles is None else {"BAKRON_GPTQ_RANGE": rng_tiles}
    with _env(**env):
        codes, V, pre = gpu_run(p)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"gptq-{variant}-r{rng_tiles}")


def test_gptq_against_two_sided_solver(oracle_mod):
    """The same B = I problem through the two-sided solver (BAKRON_GPTQ=0):
    both agree with the oracle."""
    p = _problem(200, 300, seed=62)
    log("case one-sided vs two-sided solver")
    with _env(BAKRON_GPTQ=0):
        c2, v2, x2 = gpu_run(p, k=1)
    check_against_oracle(p, c2, v2, x2, oracle_mod, label="two-sided-B=I")
    c1, v1, x1 = gpu_run(p)
    check_against_oracle(p, c1, v1, x1, oracle_mod, label="one-sided")
    assert np.max(np.abs(x1.astype(np.float64) - x2)) < 1e-3


def test_gptq_large_with_recursive_oracle(oracle_mod):
    """1000 x 2080: many row groups and column blocks; the oracle replays the
    sequence with Alg. 5 (same codes as Alg. 2)."""
    p = _problem(1000, 2080, seed=63)
    log("case one-sided 1000x2080")
    codes, V, pre = gpu_run(p)
    check_against_oracle(p, codes, V, pre, oracle_mod, label="gptq-1000x2080", method="recursive")


@pytest.mark.parametrize("rng_tiles", [None, 2])
def test_gptq_deterministic_and_poison_free(rng_tiles):
    """Repeated solves are bitwise equal, and so is a solve whose workspace
    (errors and the working copy of W) was filled with NaN first: nothing is
    read before it is written, also across ranges (2-tile ranges)."""
    p = _problem(150, 230, seed=64)
    log(f"case one-sided determinism and poisoned workspace, range {rng_tiles}")
    env = {} if rng_tiles is None else {"BAKRON_GPTQ_RANGE": rng_tiles}
    with _env(**env):
        (c1, v1, x1), (c2, v2, x2) = gpu_run(p, repeat=2)
    with _env(BAKRON_POISON=1, **env):
        c3, v3, x3 = gpu_run(p)
    for c, v, x in ((c2, v2, x2), (c3, v3, x3)):
        assert np.array_equal(c1, c)
        assert np.array_equal(v1.view(np.uint32), v.view(np.uint32))
        assert np.array_equal(np.nan_to_num(x1).view(np.uint32), np.nan_to_num(x).view(np.uint32))


@pytest.mark.timeout(600)
def test_gptq_certificate_wide_table3_shape(oracle_mod):
    """A Table 3 shape with the longest sequential chain per row, 2048 x 8192
    (A the AR(1) Toeplitz matrix rho^|i-j| with rho = 0.5, W ~ N(0, 0.02^2),
    INT4 per-row scales, 1% damping, B = I): the certificate (closed form of
    Eq. (1)) along the kernel's own trajectory, on every entry, and the
    objective."""
    import json
    o = oracle_mod
    m, n = 2048, 8192
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([3000, m, n])))
    W = (rng.standard_normal((m, n)) * 0.02).astype(np.float32)
    p = dict(W=W, A=workloads.ar1_toeplitz(n, 0.5), B=None, scale=workloads.row_scales(W, 4), bits=4,
             damp=0.01)
    log("case one-sided 2048x8192 certificate")
    codes, V, pre = gpu_run(p)
    cert = o.certify(p["W"], p["A"], None, p["damp"], p["scale"], codes, p["bits"], window=1e-4)
    v, x = cert["verdict"], cert["x"]
    fin = np.isfinite(x)
    margin = float(np.max(np.abs(pre[fin].astype(np.float64) - x[fin])))
    log("[gptq-2048x8192] " + json.dumps(dict(**v, margin_grid_steps=margin, objective=cert["objective"])))
    assert v["violations"] == 0
    assert v["flips"] <= 1e-4 * m * n
    assert margin < 1e-4


def test_gptq_handle_alternating_row_counts():
    """With B = NULL the row count is free per call: one handle solving
    300, 130 and again 300 rows (the workspace is reallocated at each change
    of shape) gives bitwise the results of a fresh handle per shape."""
    import torch
    import paper_2608_06291_amd as pk
    dev = torch.device("cuda:0")
    n = 230
    p300 = _problem(300, n, seed=71)
    p130 = _problem(130, n, seed=72)
    p130["A"] = p300["A"]                 # one factor A for both row counts
    refs = {}
    for key, p in (("300", p300), ("130", p130)):
        refs[key] = gpu_run(p)
    log("case one-sided handle with alternating row counts")
    f = pk.factor(torch.from_numpy(p300["A"]).to(dev), None, p300["damp"])
    for key, p in (("300", p300), ("130", p130), ("300", p300)):
        W = torch.from_numpy(p["W"]).to(dev)
        s = torch.from_numpy(p["scale"]).to(dev)
        c, v, x = pk.solve(W, f, p["bits"], s, debug=True)
        torch.cuda.synchronize()
        assert f.check()
        c0, v0, x0 = refs[key]
        assert np.array_equal(c.cpu().numpy(), c0)
        assert np.array_equal(v.cpu().numpy().view(np.uint32), v0.view(np.uint32))
        assert np.array_equal(np.nan_to_num(x.cpu().numpy()).view(np.uint32),
                              np.nan_to_num(x0).view(np.uint32))
    f.close()
