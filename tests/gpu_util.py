"""Helpers for GPU parity tests: run the HIP solver through the C ABI (via the
ctypes binding) and compare with the fp64 oracle under the tie-forced
protocol.

Protocol (the parity tolerance): the oracle replays the sequential rounding
and, wherever its own pre-rounding value lies within TIE_WINDOW = 1e-4 grid
steps of a rounding boundary, adopts the GPU's code (both are valid outputs up
to the tie rule).  Then
  * violations = entries where the GPU differs from that replay: must be 0;
  * flips      = excused entries where the GPU's code differs from the
                 oracle's own rounding: at most 1e-4 of all entries;
  * objective  = tr((W-V)^T B_d (W-V) A_d) within 1e-5 relative, beyond the
                 difference that the fp32 representation of V alone explains.
"""
import contextlib
import os
import sys

import numpy as np

TIE_WINDOW = 1e-4
MAX_FLIP_RATE = 1e-4
OBJ_RTOL = 1e-5


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@contextlib.contextmanager
def knear(k):
    """Factor handles read BAKRON_KNEAR at creation; small values route most
    (source, target) pairs through the divide-and-conquer node products."""
    old = os.environ.get("BAKRON_KNEAR")
    if k is None:
        yield
        return
    os.environ["BAKRON_KNEAR"] = str(k)
    try:
        yield
    finally:
        if old is None:
            del os.environ["BAKRON_KNEAR"]
        else:
            os.environ["BAKRON_KNEAR"] = old


def gpu_run(p, debug=True, k=None, repeat=1):
    """Factor + solve on cuda:0; returns numpy codes, V, pre (pre None if not debug)."""
    import torch
    import paper_2608_06291_amd as pk
    dev = torch.device("cuda:0")
    A = torch.from_numpy(np.ascontiguousarray(p["A"], np.float32)).to(dev)
    B = None if p["B"] is None else torch.from_numpy(np.ascontiguousarray(p["B"], np.float32)).to(dev)
    W = torch.from_numpy(np.ascontiguousarray(p["W"], np.float32)).to(dev)
    s = torch.from_numpy(np.ascontiguousarray(p["scale"], np.float32)).to(dev)
    with knear(k):
        f = pk.factor(A, B, p["damp"])
    outs = []
    for _ in range(repeat):
        # poison outputs so unwritten entries cannot pass
        codes = torch.full(W.shape, 100, dtype=torch.int8, device=dev)
        V = torch.full(W.shape, float("nan"), dtype=torch.float32, device=dev)
        pre = torch.full(W.shape, float("nan"), dtype=torch.float32, device=dev) if debug else None
        r = pk.solve(W, f, p["bits"], s, codes=codes, V=V, pre=pre, debug=debug)
        torch.cuda.synchronize()
        assert f.check(), "a tile-ordering wait of the solve gave up"
        outs.append(tuple(None if t is None else t.cpu().numpy() for t in
                          (r[0], r[1], r[2] if debug else None)))
    f.close()
    return outs[0] if repeat == 1 else outs


def v_is_scale_times_code(V, codes, scale):
    """V_ij must be the single fp32 product s_i * c_ij."""
    ref = (scale.astype(np.float32)[:, None] * codes.astype(np.float32)).astype(np.float32)
    return np.array_equal(V.view(np.uint32), ref.view(np.uint32)) or np.array_equal(V, ref)


def check_against_oracle(p, codes, V, pre, oracle, label=""):
    """Full element-by-element comparison with the tie-forced oracle replay."""
    m, n = p["W"].shape
    assert codes.dtype == np.int8 and codes.shape == (m, n)
    l = (1 << (p["bits"] - 1)) - 1
    assert np.all(np.abs(codes.astype(np.int32)) <= l), f"{label}: code outside alphabet"
    assert v_is_scale_times_code(V, codes, p["scale"]), f"{label}: V != s*c"
    forced = oracle.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], p["bits"],
                          forced=codes, tie_window=TIE_WINDOW)
    viol = int(np.count_nonzero(forced["codes"] != codes))
    flips = forced["n_flip"]
    res = dict(violations=viol, flips=flips, excused=forced["n_excused"], total=m * n)
    if pre is not None:
        fin = np.isfinite(forced["pre"])
        res["margin"] = float(np.max(np.abs(pre[fin].astype(np.float64) - forced["pre"][fin]))) \
            if fin.any() else 0.0
    og = oracle.objective(p["W"], V.astype(np.float64), p["A"], p["B"], p["damp"])
    oo = oracle.objective(p["W"], forced["V"], p["A"], p["B"], p["damp"])
    # The GPU returns V in fp32 (|dV| <= 2^-24 |V| per entry), so the two
    # objectives can differ by up to 2 eps sqrt(obj(D) obj(V)) + eps^2 obj(V)
    # with obj(V) = tr(V^T B V A); this floor matters only when V ~ W.
    ov = oracle.objective(np.zeros_like(forced["V"]), forced["V"], p["A"], p["B"], p["damp"])
    eps = 2.0 ** -24
    floor = 2 * eps * np.sqrt(abs(oo) * abs(ov)) + eps * eps * abs(ov)
    res["obj_rel"] = max(abs(og - oo) - floor, 0.0) / max(abs(oo), 1e-300)
    log(f"[parity] {label} m={m} n={n} {res}")
    assert viol == 0, f"{label}: {viol} non-excused code mismatches"
    assert flips <= MAX_FLIP_RATE * m * n, f"{label}: flip rate {flips}/{m*n}"
    assert res["obj_rel"] <= OBJ_RTOL, f"{label}: objective rel diff {res['obj_rel']}"
    if flips == 0:
        # forcing changed nothing, so the free-running oracle must agree exactly
        free = oracle.solve(p["W"], p["A"], p["B"], p["damp"], p["scale"], p["bits"])
        assert np.array_equal(free["codes"], codes), f"{label}: free-running mismatch"
    return res


def gpu_run_antidiag(p):
    """Factor + BaKron-antidiagonal solve on cuda:0; returns numpy codes, V, pre."""
    import torch
    import paper_2608_06291_amd as pk
    dev = torch.device("cuda:0")
    A = torch.from_numpy(np.ascontiguousarray(p["A"], np.float32)).to(dev)
    B = None if p["B"] is None else torch.from_numpy(np.ascontiguousarray(p["B"], np.float32)).to(dev)
    W = torch.from_numpy(np.ascontiguousarray(p["W"], np.float32)).to(dev)
    s = torch.from_numpy(np.ascontiguousarray(p["scale"], np.float32)).to(dev)
    f = pk.factor(A, B, p["damp"])
    codes = torch.full(W.shape, 100, dtype=torch.int8, device=dev)
    V = torch.full(W.shape, float("nan"), dtype=torch.float32, device=dev)
    pre = torch.full(W.shape, float("nan"), dtype=torch.float32, device=dev)
    pk.solve_antidiag(W, f, p["bits"], s, codes=codes, V=V, pre=pre)
    torch.cuda.synchronize()
    out = (codes.cpu().numpy(), V.cpu().numpy(), pre.cpu().numpy())
    f.close()
    return out
