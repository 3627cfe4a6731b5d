"""CPU checks of the Sec. 5 flow orchestration (paper_2608_06291_amd/flow.py)
with torch fp64 on the CPU: the recursion hands every layer the same input and
output gradient as the naive flow (a full backward pass per layer), those
gradients are autograd's, and the layer-evaluation and memory counts follow
O(l log l) and O(log l)."""
import math

import pytest
import torch

from paper_2608_06291_amd import flow


def _stack(L, d, seed):
    g = torch.Generator().manual_seed(seed)
    W = [torch.randn((d, d), generator=g, dtype=torch.float64) / math.sqrt(d) for _ in range(L)]
    x0 = torch.randn((16, d), generator=g, dtype=torch.float64)
    gout = torch.randn((16, d), generator=g, dtype=torch.float64)
    return flow.LayerStack(W), x0, gout


def _collect(fn, stack, x0, gout):
    got = {}
    st = fn(stack, x0, gout, lambda l, a, b: got.__setitem__(l, (a.clone(), b.clone())))
    return got, st


@pytest.mark.parametrize("L", [1, 2, 3, 5, 8, 13])
def test_recursive_flow_matches_naive_flow(L):
    stack, x0, gout = _stack(L, 6, L)
    rec, st_r = _collect(flow.recursive_flow, stack, x0, gout)
    nai, st_n = _collect(flow.naive_flow, stack, x0, gout)
    assert sorted(rec) == list(range(L)) and st_r.order == list(range(L))
    for l in range(L):
        assert torch.equal(rec[l][0], nai[l][0]) and torch.equal(rec[l][1], nai[l][1]), l
    # naive: l + (L - l) forwards and L - l backwards for layer l
    assert st_n.layer_forwards == L * L
    assert st_n.layer_backwards == L * (L + 1) // 2


def test_flow_gradients_are_autograd():
    """b_l = dL/dy_l for L = sum(g_out * f(x0)): hooks on the autograd graph."""
    L = 5
    stack, x0, gout = _stack(L, 7, 99)
    rec, _ = _collect(flow.recursive_flow, stack, x0, gout)
    ys = []
    x = x0.clone().requires_grad_(True)
    for l in range(L):
        y = x @ stack.W[l].t()
        y.retain_grad()
        ys.append(y)
        x = torch.nn.functional.silu(y)
    (x * gout).sum().backward()
    xs = [x0]
    for l in range(L - 1):
        xs.append(torch.nn.functional.silu(ys[l]).detach())
    for l in range(L):
        torch.testing.assert_close(rec[l][1], ys[l].grad, rtol=1e-12, atol=1e-14)
        torch.testing.assert_close(rec[l][0], xs[l], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("L", [2, 4, 7, 16, 32, 33])
def test_recursive_flow_costs(L):
    """O(l log l) layer evaluations and O(log l) live (activation, gradient)
    pairs: each level forwards its whole range and backpropagates its second
    half, each leaf one forward and one backward."""
    stack, x0, gout = _stack(L, 3, 7)
    _, st = _collect(flow.recursive_flow, stack, x0, gout)

    def cost(n):          # (forwards, backwards) of a range of n layers
        if n == 1:
            return 1, 1
        h = n // 2
        f1, b1 = cost(h)
        f2, b2 = cost(n - h)
        return n + f1 + f2, (n - h) + b1 + b2
    assert (st.layer_forwards, st.layer_backwards) == cost(L)
    depth = math.ceil(math.log2(L)) + 1
    assert st.peak_live_pairs == depth
    assert st.layer_forwards + st.layer_backwards <= 3 * L * math.ceil(math.log2(L)) + 2 * L
