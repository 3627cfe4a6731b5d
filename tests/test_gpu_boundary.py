"""Boundary behaviour of the solve entry points on the GPU: the debug-mode
scale validation (BAKRON_EINVAL for a negative, NaN or infinite scale) and the
sticky give-up record of the tile-ordering waits (bakron_solve_check).

The give-up path is forced from the host: BAKRON_SPIN_LIMIT=1 makes every
wait that finds its flag unset give up after one poll, so the kernels still
run to completion and only the output is marked invalid."""
import os

import numpy as np
import pytest

import workloads
from gpu_util import check_against_oracle, log

pytestmark = pytest.mark.gpu


def _setup(m, n, seed):
    import torch
    import paper_2608_06291_amd as pk
    dev = torch.device("cuda:0")
    p = workloads.make_random(m, n, seed=seed)
    A = torch.from_numpy(p["A"]).to(dev)
    B = torch.from_numpy(p["B"]).to(dev)
    W = torch.from_numpy(p["W"]).to(dev)
    s = torch.from_numpy(p["scale"]).to(dev)
    f = pk.factor(A, B, p["damp"])
    return p, f, W, s


@pytest.mark.parametrize("bad", [float("nan"), -1e-3, float("inf")])
def test_debug_solve_rejects_bad_scales(bad):
    import torch
    import paper_2608_06291_amd as pk
    log(f"case debug scale validation bad={bad}")
    m, n = 70, 90
    p, f, W, s = _setup(m, n, seed=12)
    codes = torch.full((m, n), 100, dtype=torch.int8, device=W.device)
    V = torch.full((m, n), 5.0, device=W.device)
    pre = torch.full((m, n), 5.0, device=W.device)
    # per-row scale
    s_bad = s.clone()
    s_bad[37] = bad
    with pytest.raises(pk.BakronError) as ei:
        pk.solve(W, f, 4, s_bad, codes=codes, V=V, pre=pre, debug=True)
    assert ei.value.status == pk.BAKRON_EINVAL
    assert "scale" in f.error()
    # per-(row, group) scale
    g = 32
    sg = s[:, None].repeat(1, -(-n // g)).contiguous()
    sg[m - 1, 2] = bad
    with pytest.raises(pk.BakronError) as ei:
        pk.solve(W, f, 4, sg, codes=codes, V=V, pre=pre, debug=True, group_size=g)
    assert ei.value.status == pk.BAKRON_EINVAL
    # per-column factor
    col = torch.ones(n, device=W.device)
    col[n - 1] = bad
    with pytest.raises(pk.BakronError) as ei:
        pk.solve(W, f, 4, s, codes=codes, V=V, pre=pre, debug=True, col_scale=col)
    assert ei.value.status == pk.BAKRON_EINVAL
    torch.cuda.synchronize()
    # nothing was enqueued: the outputs keep their poison
    assert bool((codes == 100).all()) and bool((V == 5.0).all()) and bool((pre == 5.0).all())
    # a zero scale is valid (alphabet {0}); the same handle then solves normally
    s0 = s.clone()
    s0[3] = 0.0
    c, v, x = pk.solve(W, f, 4, s0, codes=codes, V=V, pre=pre, debug=True)
    torch.cuda.synchronize()
    assert f.check()
    assert bool((c[3] == 0).all()) and bool(torch.isnan(x[3]).all())
    f.close()


def test_give_up_record_is_sticky_until_checked(oracle_mod):
    import torch
    import paper_2608_06291_amd as pk
    log("case sticky give-up record (BAKRON_SPIN_LIMIT=1)")
    m, n = 600, 600
    p, f, W, s = _setup(m, n, seed=33)
    old = os.environ.get("BAKRON_SPIN_LIMIT")
    try:
        os.environ["BAKRON_SPIN_LIMIT"] = "1"
        pk.solve(W, f, p["bits"], s)
        torch.cuda.synchronize()
    finally:
        if old is None:
            os.environ.pop("BAKRON_SPIN_LIMIT", None)
        else:
            os.environ["BAKRON_SPIN_LIMIT"] = old
    # a solve with the normal limit after the failure is still reported: the
    # record survives until it is read
    pk.solve(W, f, p["bits"], s)
    torch.cuda.synchronize()
    assert not f.check()
    # reading cleared it; the next solve is complete and correct
    assert f.check()
    codes, V, pre = pk.solve(W, f, p["bits"], s, debug=True)
    torch.cuda.synchronize()
    assert f.check()
    check_against_oracle(p, codes.cpu().numpy(), V.cpu().numpy(), pre.cpu().numpy(), oracle_mod,
                         label="after-check")
    f.close()


def test_two_handles_on_two_streams_bitwise():
    """Two handles (two shapes) solved on two user streams, their solves
    enqueued back to back with no synchronisation in between: both share the
    device's CU-restricted streams and the process-wide plan cache, and each
    result is bitwise the same as the handle's solve alone."""
    import torch
    import paper_2608_06291_amd as pk
    from gpu_util import gpu_run
    dev = torch.device("cuda:0")
    cases = [(1024, 1024, 11), (700, 900, 12)]
    probs = [workloads.make_random(m, n, seed=s) for m, n, s in cases]
    log("case two handles on two streams: references")
    refs = [gpu_run(p) for p in probs]
    hs, outs, ins = [], [], []
    streams = [torch.cuda.Stream(dev) for _ in cases]
    for p, st in zip(probs, streams):
        with torch.cuda.stream(st):
            A = torch.from_numpy(p["A"]).to(dev)
            B = torch.from_numpy(p["B"]).to(dev)
            W = torch.from_numpy(p["W"]).to(dev)
            s = torch.from_numpy(p["scale"]).to(dev)
            f = pk.factor(A, B, p["damp"])
            m, n = W.shape
            o = (torch.full((m, n), 100, dtype=torch.int8, device=dev),
                 torch.full((m, n), float("nan"), dtype=torch.float32, device=dev),
                 torch.full((m, n), float("nan"), dtype=torch.float32, device=dev))
            pk.solve(W, f, p["bits"], s, codes=o[0], V=o[1], pre=o[2], debug=True)   # first solve of the shape
        hs.append(f)
        outs.append(o)
        ins.append((W, s, p["bits"]))
    torch.cuda.synchronize()
    log("case two handles on two streams: interleaved solves")
    for _ in range(3):
        for f, o, (W, s, bits), st in zip(hs, outs, ins, streams):
            with torch.cuda.stream(st):
                pk.solve(W, f, bits, s, codes=o[0], V=o[1], pre=o[2], debug=True)
    torch.cuda.synchronize()
    for f, o, (c0, v0, x0) in zip(hs, outs, refs):
        assert f.check()
        c, v, x = (t.cpu().numpy() for t in o)
        assert np.array_equal(c, c0)
        assert np.array_equal(v.view(np.uint32), v0.view(np.uint32))
        assert np.array_equal(np.nan_to_num(x).view(np.uint32), np.nan_to_num(x0).view(np.uint32))
        f.close()
