"""GPU run of the Sec. 5 recursive flow on a toy layer stack: every layer's
factors, scales and BaKron rounding through the C ABI, checked against an
fp64 reference written here independently of the flow module (forward and
backward in numpy, the oracle's factors, scale search and sequential
rounding under the tie-forced protocol)."""
import math

import numpy as np
import pytest

import workloads
from gpu_util import check_against_oracle, log

pytestmark = pytest.mark.gpu


def _reference_pairs(h, W, x0, g_out):
    """(a_l, b_l) for every layer in fp64: forward, then one full backward."""
    xs, ys = [np.asarray(x0, np.float64)], []
    for Wl in W:
        y = xs[-1] @ np.asarray(Wl, np.float64).T
        ys.append(y)
        xs.append(h.silu(y))
    g = np.asarray(g_out, np.float64)
    bs = [None] * len(W)
    for l in range(len(W) - 1, -1, -1):
        bs[l] = h.silu_prime(ys[l]) * g
        g = bs[l] @ np.asarray(W[l], np.float64)
    return [(xs[l], bs[l]) for l in range(len(W))]


@pytest.mark.parametrize("style,iters", [("kfac", 1), ("shampoo", 2)])
def test_recursive_flow_on_gpu(oracle_mod, style, iters):
    import torch
    from paper_2608_06291_amd import flow
    h = oracle_mod.hessian
    L, d, N, bits, damp = 5, 96, 1024, 3, 0.01
    m = workloads.toy_mlp(L, d, N, seed=1)
    log(f"case flow {style} iters={iters} L={L} d={d} N={N}")
    dev = torch.device("cuda:0")
    stack = flow.LayerStack([torch.from_numpy(W).to(dev) for W in m["W"]])
    step, res = flow.bakron_layer_step(stack, bits, damp, style=style, iters=iters)
    st = flow.recursive_flow(stack, torch.from_numpy(m["x0"]).to(dev),
                             torch.from_numpy(m["g_out"]).to(dev), step)
    torch.cuda.synchronize()
    assert st.order == list(range(L))
    assert st.peak_live_pairs == math.ceil(math.log2(L)) + 1
    pairs = _reference_pairs(h, m["W"], m["x0"], m["g_out"])
    for l in range(L):
        a, b = pairs[l]
        A, B = (h.kfac_factors(a, b) if style == "kfac" else h.shampoo_factors(a, b, iters=iters))
        gA = res[l]["A"].cpu().numpy().astype(np.float64)
        rel = np.linalg.norm(gA - A) / np.linalg.norm(A)
        assert rel < 1e-4, (l, rel)   # fp32 forward/backward and factor sums
        scale, _ = oracle_mod.mse_scales(m["W"][l], bits)
        gs = res[l]["scale"].cpu().numpy()
        assert np.array_equal(gs, scale), l
        p = dict(W=m["W"][l], A=A, B=B, damp=damp, scale=scale, bits=bits)
        check_against_oracle(p, res[l]["codes"].cpu().numpy(), res[l]["V"].cpu().numpy(), None,
                             oracle_mod, label=f"flow-{style}-layer{l}")
