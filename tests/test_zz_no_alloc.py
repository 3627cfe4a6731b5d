"""bakron_solve_noalloc (workspace in the library's static per-device scratch,
no device allocation) against bakron_solve, through the C ABI: codes and V
bitwise equal on two calls in a row, the second with a smaller layer, then
the first shape again (the scratch keeps the previous call's contents, so
each call must set up what it reads); a layer too large for the scratch is
refused before any work is enqueued."""
import numpy as np
import pytest

import workloads
from gpu_util import log

pytestmark = pytest.mark.gpu


def _inputs(m, n, seed, identity_B=False):
    import torch
    dev = torch.device("cuda:0")
    p = workloads.make_random(m, n, seed=seed, identity_B=identity_B)
    t = {k: (None if p[k] is None else torch.from_numpy(p[k]).to(dev)) for k in ("A", "B", "W", "scale")}
    return p, t


def _both(pk, t, f, bits, **qk):
    import torch
    dev = t["W"].device
    m, n = t["W"].shape
    c0 = torch.full((m, n), 100, dtype=torch.int8, device=dev)
    v0 = torch.full((m, n), float("nan"), device=dev)
    c1 = torch.full((m, n), 100, dtype=torch.int8, device=dev)
    v1 = torch.full((m, n), float("nan"), device=dev)
    pk.solve(t["W"], f, bits, t["scale"], codes=c0, V=v0, **qk)
    pk.solve_noalloc(t["W"], f, bits, t["scale"], codes=c1, V=v1, **qk)
    torch.cuda.synchronize()
    assert f.check()
    assert torch.equal(c0, c1)
    assert torch.equal(v0.view(torch.int32), v1.view(torch.int32))
    return c1


@pytest.mark.parametrize("shapes,identity_B", [([(700, 650), (300, 260), (700, 650)], False),
                                               ([(520, 400), (97, 130)], True)])
def test_noalloc_matches_solve(shapes, identity_B):
    import torch
    import paper_2608_06291_amd as pk
    for i, (m, n) in enumerate(shapes):
        log(f"case noalloc call {i} m={m} n={n} B=I={identity_B}")
        p, t = _inputs(m, n, seed=8800 + i, identity_B=identity_B)
        f = pk.factor(t["A"], t["B"], p["damp"])
        c = _both(pk, t, f, p["bits"])
        assert int(c.abs().max()) <= (1 << (p["bits"] - 1)) - 1
        f.close()
        del t
        torch.cuda.synchronize()


def test_noalloc_group_scales_and_knear0():
    import os
    import torch
    import paper_2608_06291_amd as pk
    m, n = 333, 290
    log(f"case noalloc group scales knear=0 m={m} n={n}")
    p, t = _inputs(m, n, seed=8900)
    old = os.environ.get("BAKRON_KNEAR")
    os.environ["BAKRON_KNEAR"] = "0"
    try:
        f = pk.factor(t["A"], t["B"], p["damp"])
    finally:
        if old is None:
            del os.environ["BAKRON_KNEAR"]
        else:
            os.environ["BAKRON_KNEAR"] = old
    g = 64
    sg = t["scale"][:, None].repeat(1, -(-n // g)).contiguous()
    sg *= torch.linspace(0.8, 1.2, sg.shape[1], device=sg.device)[None, :]
    _both(pk, dict(t, scale=sg), f, 3, alphabet="asym", group_size=g)
    f.close()


def test_noalloc_refuses_layers_beyond_the_scratch():
    import torch
    import paper_2608_06291_amd as pk
    log("case noalloc too large")
    dev = torch.device("cuda:0")
    n = 64
    A = torch.eye(n, device=dev)
    f = pk.factor(A, None, 0.0)
    m = 300000            # ceil(m/32) * 2 tiles * 8 KiB > 136 MiB
    W = torch.zeros((m, n), device=dev)
    s = torch.ones(m, device=dev)
    codes = torch.full((m, n), 100, dtype=torch.int8, device=dev)
    with pytest.raises(pk.BakronError) as ei:
        pk.solve_noalloc(W, f, 4, s, codes=codes)
    assert ei.value.status == pk.BAKRON_EINVAL
    assert "scratch" in f.error()
    torch.cuda.synchronize()
    assert bool((codes == 100).all())
    f.close()
