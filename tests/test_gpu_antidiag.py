"""GPU parity of BaKron-antidiagonal (Alg. 3, bakron_solve_antidiag) with the
fp64 oracle, and its agreement with the BaKron solver (Thm 3.2: both reach
the same rounding)."""
import numpy as np
import pytest

import workloads
from gpu_util import check_against_oracle, gpu_run, gpu_run_antidiag, log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("m,n", [(1, 1), (2, 3), (37, 29), (64, 64), (65, 130), (130, 67)])
def test_antidiag_parity(oracle_mod, m, n):
    p = workloads.make_random(m, n, seed=500 + m * 7 + n)
    log(f"case antidiag m={m} n={n}")
    codes, V, pre = gpu_run_antidiag(p)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"antidiag{m}x{n}")


@pytest.mark.parametrize("bits,identity_B", [(2, False), (4, True)])
def test_antidiag_variants(oracle_mod, bits, identity_B):
    p = workloads.make_random(70, 90, seed=31, bits=bits, identity_B=identity_B)
    log(f"case antidiag bits={bits} B=I={identity_B}")
    codes, V, pre = gpu_run_antidiag(p)
    check_against_oracle(p, codes, V, pre, oracle_mod, label=f"antidiag-b{bits}-I{identity_B}")


def test_antidiag_matches_bakron():
    """Same codes as the divide-and-conquer solver except at entries whose
    pre-rounding value lies within rounding noise of a boundary."""
    p = workloads.make_random(300, 260, seed=77)
    log("case antidiag vs bakron 300x260")
    ca, _, pa = gpu_run_antidiag(p)
    cb, _, pb = gpu_run(p)
    diff = ca != cb
    log(f"[antidiag] differing codes {int(diff.sum())} of {diff.size}")
    if diff.any():
        # the first differing entry in row-major order has no differing entry
        # above-left of it, so both solvers rounded the same value up to fp32
        # noise: it must lie next to a rounding boundary
        i, j = np.unravel_index(np.flatnonzero(diff)[0], diff.shape)
        frac = abs(float(pa[i, j]) - np.floor(float(pa[i, j])) - 0.5)
        assert frac < 1e-3, (i, j, float(pa[i, j]), float(pb[i, j]))
    else:
        fin = np.isfinite(pa) & np.isfinite(pb)
        assert float(np.max(np.abs(pa[fin] - pb[fin]))) < 1e-3
