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


def quant_kwargs(p):
    """Quantiser of a problem dict for the binding: alphabet, group size and
    per-column factors (absent: the per-row symmetric quantiser)."""
    import torch
    kw = dict(alphabet=p.get("alphabet", "sym"), group_size=p.get("group_size", 0))
    if p.get("col_scale") is not None:
        kw["col_scale"] = torch.from_numpy(np.ascontiguousarray(p["col_scale"], np.float32)).to("cuda:0")
    return kw


def oracle_scales(p, oracle):
    """Per-entry scales of the problem's quantiser (m x n, fp32 values)."""
    m, n = p["W"].shape
    return oracle.entry_scales(p["scale"], m, n, group_size=p.get("group_size", 0),
                               col_scale=p.get("col_scale"))


def gpu_run(p, debug=True, k=None, repeat=1):
    """Factor + solve on cuda:0; returns numpy codes, V, pre (pre None if not debug)."""
    import torch
    import paper_2608_06291_amd as pk
    dev = torch.device("cuda:0")
    A = torch.from_numpy(np.ascontiguousarray(p["A"], np.float32)).to(dev)
    B = None if p["B"] is None else torch.from_numpy(np.ascontiguousarray(p["B"], np.float32)).to(dev)
    W = torch.from_numpy(np.ascontiguousarray(p["W"], np.float32)).to(dev)
    s = torch.from_numpy(np.ascontiguousarray(p["scale"], np.float32)).to(dev)
    qk = quant_kwargs(p)
    with knear(k):
        if p.get("B_blocks") is not None:
            Bb = torch.from_numpy(np.ascontiguousarray(p["B_blocks"], np.float32)).to(dev)
            f = pk.factor_blockdiag(A, Bb, p["damp"])
        else:
            f = pk.factor(A, B, p["damp"])
    outs = []
    for _ in range(repeat):
        # poison outputs so unwritten entries cannot pass
        codes = torch.full(W.shape, 100, dtype=torch.int8, device=dev)
        V = torch.full(W.shape, float("nan"), dtype=torch.float32, device=dev)
        pre = torch.full(W.shape, float("nan"), dtype=torch.float32, device=dev) if debug else None
        r = pk.solve(W, f, p["bits"], s, codes=codes, V=V, pre=pre, debug=debug, **qk)
        torch.cuda.synchronize()
        assert f.check(), "a tile-ordering wait of the solve gave up"
        outs.append(tuple(None if t is None else t.cpu().numpy() for t in
                          (r[0], r[1], r[2] if debug else None)))
    f.close()
    return outs[0] if repeat == 1 else outs


def v_is_scale_times_code(V, codes, scale):
    """V_ij must be the single fp32 product s_ij * c_ij (scale: per row or
    per entry)."""
    S = np.asarray(scale, np.float32)
    S = S[:, None] if S.ndim == 1 else S
    ref = (S * codes.astype(np.float32)).astype(np.float32)
    return np.array_equal(V.view(np.uint32), ref.view(np.uint32)) or np.array_equal(V, ref)


def check_against_oracle(p, codes, V, pre, oracle, label="", method="naive"):
    """Full element-by-element comparison with the tie-forced oracle replay
    (method "naive": Alg. 2; "recursive": Alg. 5, the same sequence, for
    shapes where the quartic Alg. 2 is slow)."""
    m, n = p["W"].shape
    assert codes.dtype == np.int8 and codes.shape == (m, n)
    alphabet = p.get("alphabet", "sym")
    lo, hi = oracle.alphabet_bounds(p["bits"], alphabet)
    assert np.all((codes.astype(np.int32) >= lo) & (codes.astype(np.int32) <= hi)), \
        f"{label}: code outside alphabet"
    S = oracle_scales(p, oracle)
    assert v_is_scale_times_code(V, codes, S), f"{label}: V != s*c"
    B = p["B"]
    if p.get("B_blocks") is not None:
        B = block_diag(p["B_blocks"])
    forced = oracle.solve(p["W"], p["A"], B, p["damp"], S, p["bits"],
                          forced=codes, tie_window=TIE_WINDOW, alphabet=alphabet, method=method)
    viol = int(np.count_nonzero(forced["codes"] != codes))
    flips = forced["n_flip"]
    res = dict(violations=viol, flips=flips, excused=forced["n_excused"], total=m * n)
    if pre is not None:
        fin = np.isfinite(forced["pre"])
        res["margin"] = float(np.max(np.abs(pre[fin].astype(np.float64) - forced["pre"][fin]))) \
            if fin.any() else 0.0
    og = oracle.objective(p["W"], V.astype(np.float64), p["A"], B, p["damp"])
    oo = oracle.objective(p["W"], forced["V"], p["A"], B, p["damp"])
    # The GPU returns V in fp32 (|dV| <= 2^-24 |V| per entry), so the two
    # objectives can differ by up to 2 eps sqrt(obj(D) obj(V)) + eps^2 obj(V)
    # with obj(V) = tr(V^T B V A); this floor matters only when V ~ W.
    ov = oracle.objective(np.zeros_like(forced["V"]), forced["V"], p["A"], B, p["damp"])
    eps = 2.0 ** -24
    floor = 2 * eps * np.sqrt(abs(oo) * abs(ov)) + eps * eps * abs(ov)
    res["obj_rel"] = max(abs(og - oo) - floor, 0.0) / max(abs(oo), 1e-300)
    log(f"[parity] {label} m={m} n={n} {res}")
    assert viol == 0, f"{label}: {viol} non-excused code mismatches"
    assert flips <= MAX_FLIP_RATE * m * n, f"{label}: flip rate {flips}/{m*n}"
    assert res["obj_rel"] <= OBJ_RTOL, f"{label}: objective rel diff {res['obj_rel']}"
    if flips == 0:
        # forcing changed nothing, so the free-running oracle must agree exactly
        free = oracle.solve(p["W"], p["A"], B, p["damp"], S, p["bits"], alphabet=alphabet,
                            method=method)
        assert np.array_equal(free["codes"], codes), f"{label}: free-running mismatch"
    return res


def block_diag(blocks):
    """The m x m block-diagonal matrix of nblocks x hb x hb blocks (fp32)."""
    blocks = np.asarray(blocks, np.float32)
    nb, hb, _ = blocks.shape
    out = np.zeros((nb * hb, nb * hb), np.float32)
    for h in range(nb):
        out[h * hb:(h + 1) * hb, h * hb:(h + 1) * hb] = blocks[h]
    return out


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
    pk.solve_antidiag(W, f, p["bits"], s, codes=codes, V=V, pre=pre, **quant_kwargs(p))
    torch.cuda.synchronize()
    out = (codes.cpu().numpy(), V.cpu().numpy(), pre.cpu().numpy())
    f.close()
    return out
