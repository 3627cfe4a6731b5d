"""GPU parity: the HIP solver (through the C ABI) against the fp64 oracle,
element by element, on seeded inputs that span several 32x32 tiles with
ragged tails, plus the degenerate shapes."""
import numpy as np
import pytest

import workloads
from gpu_util import check_against_oracle, gpu_run, gpu_run_antidiag, log

pytestmark = pytest.mark.gpu


def _problem(m, n, seed, bits=4, identity_B=False):
    return workloads.make_random(m, n, seed, bits=bits, identity_B=identity_B)


SHAPES = [(1, 1), (1, 37), (37, 1), (2, 3), (31, 33), (32, 32), (33, 31), (64, 64),
          (65, 97), (130, 67), (97, 200), (257, 129)]


@pytest.mark.parametrize("m,n", SHAPES)
def test_parity_shapes(oracle_mod, m, n):
    p = _problem(m, n, seed=m * 1000 + n)
    log(f"case shape m={m} n={n}")
    codes, V, pre = gpu_run(p)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"shape{m}x{n}")


def _sweep_cases(count=24):
    """Seeded random cases: shape (ragged in both directions, up to 200 x 200),
    alphabet size, near-field distance and B = I."""
    rng = np.random.Generator(np.random.PCG64(20261202))
    cases = []
    for _ in range(count):
        m, n = (int(x) for x in rng.integers(1, 201, size=2))
        bits = int(rng.choice([2, 3, 4, 8]))
        k = [None, 0, 2, 5, 8][int(rng.integers(0, 5))]
        ident = bool(rng.random() < 0.2)
        cases.append((m, n, bits, k, ident, int(rng.integers(0, 1 << 30))))
    return cases


@pytest.mark.parametrize("m,n,bits,k,ident,seed", _sweep_cases())
def test_parity_random_sweep(oracle_mod, m, n, bits, k, ident, seed):
    """Element-wise tie-forced parity on a seeded random sweep of shapes,
    alphabets, near-field distances and one-sided (B = I) problems."""
    p = workloads.make_random(m, n, seed, bits=bits, identity_B=ident)
    log(f"case sweep m={m} n={n} bits={bits} knear={k} identity_B={ident} seed={seed}")
    codes, V, pre = gpu_run(p, k=k)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"sweep{m}x{n}b{bits}k{k}i{int(ident)}")


@pytest.mark.parametrize("k", [0, 1, 3, 8])
@pytest.mark.parametrize("m,n", [(200, 300), (300, 200), (161, 161)])
def test_parity_node_paths(oracle_mod, m, n, k):
    """Small KNEAR sends most tile pairs through the divide-and-conquer nodes
    (KNEAR 0: every segment is one tile anti-diagonal and nothing is pulled);
    KNEAR 8 is the largest near field the segment kernel supports."""
    p = _problem(m, n, seed=7 + m + n)
    log(f"case node-path m={m} n={n} knear={k}")
    codes, V, pre = gpu_run(p, k=k)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"knear{k}-{m}x{n}")


@pytest.mark.parametrize("bits", [2, 3, 8])
def test_parity_bits(oracle_mod, bits):
    p = _problem(96, 130, seed=bits, bits=bits)
    log(f"case bits={bits}")
    codes, V, pre = gpu_run(p, k=2)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"bits{bits}")


@pytest.mark.parametrize("m,n,k", [(65, 97, None), (200, 300, 1)])
def test_parity_B_identity(oracle_mod, m, n, k):
    """B = NULL: one-sided GPTQ with H = A (Sec. 1)."""
    p = _problem(m, n, seed=3, identity_B=True)
    log(f"case B=I m={m} n={n}")
    codes, V, pre = gpu_run(p, k=k)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"BI-{m}x{n}")


def test_zero_scale_rows(oracle_mod):
    p = _problem(70, 90, seed=11)
    p["scale"] = p["scale"].copy()
    p["scale"][[0, 33, 69]] = 0.0
    codes, V, pre = gpu_run(p, k=1)
    assert np.all(codes[[0, 33, 69]] == 0) and np.all(V[[0, 33, 69]] == 0)
    assert np.all(np.isnan(pre[[0, 33, 69]]))
    check_against_oracle(p, codes, V, pre, oracle_mod, label="zero-scale")


def test_config1_tiny_layer(oracle_mod):
    """Configuration 1 (64x64, INT4) in full."""
    p = workloads.make(1, seed=0)
    codes, V, pre = gpu_run(p)
    res = check_against_oracle(p, codes, V, pre, oracle_mod, label="config1")
    assert res["margin"] < 1e-3


def test_determinism(oracle_mod):
    """Two solves give bitwise-identical codes, V and pre (no float atomics)."""
    p = _problem(150, 170, seed=5)
    (c1, v1, x1), (c2, v2, x2) = gpu_run(p, k=2, repeat=2)
    assert np.array_equal(c1, c2)
    assert np.array_equal(v1.view(np.uint32), v2.view(np.uint32))
    assert np.array_equal(np.nan_to_num(x1).view(np.uint32), np.nan_to_num(x2).view(np.uint32))


def test_ar1_structured_exact(oracle_mod):
    """A, B AR(1) Toeplitz, no damping: exact O(mn) oracle (3-tap diffusion)."""
    rng = np.random.default_rng(17)
    m, n = 333, 290
    W = (rng.standard_normal((m, n)) * 0.02).astype(np.float32)
    p = dict(W=W, A=workloads.ar1_toeplitz(n, 0.5), B=workloads.ar1_toeplitz(m, 0.25),
             scale=workloads.row_scales(W, 3), bits=3, damp=0.0)
    codes, V, pre = gpu_run(p, k=2)
    r = oracle_mod.ar1_diffusion(W, 0.5, 0.25, p["scale"], 3, forced=codes, tie_window=1e-4)
    assert np.count_nonzero(r["codes"] != codes) == 0
    assert r["n_flip"] <= 1e-4 * m * n


@pytest.mark.parametrize("m,n,k", [(600, 500, 8), (300, 420, 1), (1100, 300, 8), (300, 1100, 8)])
def test_side_stream_bitwise(m, n, k):
    """On a non-default stream with BAKRON_DEFER=1 (read when a handle first
    plans a shape), node pushes into later segments run on a CU-restricted
    side stream, also on the tall and wide shapes where the cost model would
    keep one stream; on the legacy default stream and with BAKRON_DEFER=0
    everything runs on the caller's stream.  Every target tile receives the
    same additions in the same order either way, so the results must be
    bitwise identical."""
    import os
    import torch
    p = _problem(m, n, seed=m + 3 * n)
    log(f"case side stream m={m} n={n} knear={k}")
    old = os.environ.get("BAKRON_DEFER")
    try:
        os.environ["BAKRON_DEFER"] = "0"
        c0, v0, x0 = gpu_run(p, k=k)
        os.environ["BAKRON_DEFER"] = "1"
        with torch.cuda.stream(torch.cuda.Stream()):
            c1, v1, x1 = gpu_run(p, k=k, repeat=2)[1]
        c2, v2, x2 = gpu_run(p, k=k)
    finally:
        if old is None:
            os.environ.pop("BAKRON_DEFER", None)
        else:
            os.environ["BAKRON_DEFER"] = old
    for c, v, x in ((c1, v1, x1), (c2, v2, x2)):
        assert np.array_equal(c0, c)
        assert np.array_equal(v0.view(np.uint32), v.view(np.uint32))
        assert np.array_equal(x0.view(np.uint32), x.view(np.uint32))


@pytest.mark.parametrize("m,n,k,identity_B", [(257, 129, None, False), (100, 97, 0, False),
                                               (130, 70, 3, True)])
def test_poisoned_workspace_bitwise(m, n, k, identity_B):
    """With BAKRON_POISON=1 the handle fills its whole workspace with NaN / -1
    bytes before every solve; the results must equal an unpoisoned solve bit
    for bit (no word of the workspace is read before the solve writes it)."""
    import os
    p = workloads.make_random(m, n, seed=404, identity_B=identity_B)
    log(f"case poisoned workspace m={m} n={n} k={k} B=I={identity_B}")
    ref = gpu_run(p, k=k)
    old = os.environ.get("BAKRON_POISON")
    os.environ["BAKRON_POISON"] = "1"
    try:
        got = gpu_run(p, k=k, repeat=2)
        ad = gpu_run_antidiag(p)
    finally:
        if old is None:
            del os.environ["BAKRON_POISON"]
        else:
            os.environ["BAKRON_POISON"] = old
    for c, v, x in got:
        assert np.array_equal(c, ref[0])
        assert np.array_equal(v.view(np.uint32), ref[1].view(np.uint32))
        assert np.array_equal(np.isnan(x), np.isnan(ref[2]))
    ref_ad = gpu_run_antidiag(p)
    assert np.array_equal(ad[0], ref_ad[0]) and np.array_equal(ad[1].view(np.uint32),
                                                               ref_ad[1].view(np.uint32))


@pytest.mark.parametrize("macro,k", [(4, 8), (4, 0), (2, 8)])
def test_parity_forced_macro_tile(oracle_mod, macro, k):
    """BAKRON_MACRO=4 makes every node push use the 128 x 128 macro tiles
    (otherwise chosen only for nodes with >= 512 items, i.e. at full size),
    =2 the 64 x 64 ones, on a shape whose tile counts (32 x 34) are not
    multiples of 4, so the partial macro tiles and their masks run; every
    entry against the oracle's tie-forced replay (Alg. 5, the same sequence
    as Alg. 2)."""
    import os
    m, n = 1000, 1060
    p = _problem(m, n, seed=4000 + macro + k)
    log(f"case forced macro tile {macro} knear={k} m={m} n={n}")
    old = os.environ.get("BAKRON_MACRO")
    os.environ["BAKRON_MACRO"] = str(macro)
    try:
        codes, V, pre = gpu_run(p, k=k)
    finally:
        if old is None:
            del os.environ["BAKRON_MACRO"]
        else:
            os.environ["BAKRON_MACRO"] = old
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"macro{macro}-k{k}",
                         method="recursive")
