"""Quantisation flows over a stack of layers (Sec. 5).

The global (backpropagated) Hessian of layer l needs, for every calibration
sample, the layer's input a = x_l and the gradient b of the loss with respect
to the layer's output y_l = W_l x_l.  Sec. 5 gets them for all layers with a
recursion over the layer range [lo, hi), given the input x_lo of its first
layer and the gradient g_hi of the loss with respect to the output of its
last layer:

  * one layer: hand (x_lo, b = dL/dy_lo) to the per-layer step (Kronecker
    factors, factorisation, BaKron);
  * otherwise, with mid = (lo + hi) // 2: forward x_lo through [lo, mid) to
    x_mid, forward x_mid through [mid, hi) and backpropagate g_hi to g_mid,
    then recurse on [lo, mid) with (x_lo, g_mid) and on [mid, hi) with
    (x_mid, g_hi).

Every level of the recursion evaluates each layer at most twice (forward, and
backward for the second half), so the flow costs O(l log l) layer
evaluations and keeps O(log l) pairs of mid-layer activations alive, against
O(l^2) evaluations for a full backward pass per layer, or O(l) stored Hessians
for one pass that accumulates all layers (Sec. 5, Table 2).

The activations and gradients at the split points are computed once, from the
weights as they are when the range is split (the weights of both halves are
still unquantised at that point).

The model is a stack of square linear layers with SiLU after each,
  y_l = W_l x_l,  x_{l+1} = SiLU(y_l),
evaluated with torch on the device (it stands in for the network being
quantised; its forward and backward are the network's own computation).  The
per-layer step runs in libbakron's kernels through the C ABI.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass
class FlowStats:
    """Counters of one flow run."""
    layer_forwards: int = 0       # single-layer forward evaluations
    layer_backwards: int = 0      # single-layer backward evaluations
    peak_live_pairs: int = 0      # largest number of (activation, gradient) pairs held at once
    order: list = field(default_factory=list)   # layers in the order they were quantised


def _silu(torch, y):
    return y * torch.sigmoid(y)


def _silu_prime(torch, y):
    s = torch.sigmoid(y)
    return s * (1.0 + y * (1.0 - s))


class LayerStack:
    """y_l = W_l x_l, x_{l+1} = SiLU(y_l) for a list of square weights (torch
    tensors on one device, samples as rows: X is N x d, y = X W_l^T)."""

    def __init__(self, weights):
        self.W = list(weights)

    def __len__(self):
        return len(self.W)

    def forward_layer(self, l, x, stats):
        import torch
        stats.layer_forwards += 1
        y = x @ self.W[l].t()
        return y, _silu(torch, y)

    def backward_layer(self, l, y, g_out, stats):
        """dL/dy_l and dL/dx_l from dL/dx_{l+1} (y_l kept from the forward)."""
        import torch
        stats.layer_backwards += 1
        b = _silu_prime(torch, y) * g_out
        return b, b @ self.W[l]


def recursive_flow(stack: LayerStack, x0, g_out, layer_step, stats: FlowStats | None = None):
    """Sec. 5's recursion over all layers of `stack`.  layer_step(l, a, b) is
    called once per layer, in layer order, with its input a (N x d) and output
    gradient b (N x d).  Returns the stats."""
    stats = stats or FlowStats()
    live = [0]

    def rec(lo, hi, x_lo, g_hi):
        live[0] += 1
        stats.peak_live_pairs = max(stats.peak_live_pairs, live[0])
        if hi - lo == 1:
            y, _ = stack.forward_layer(lo, x_lo, stats)
            b, _ = stack.backward_layer(lo, y, g_hi, stats)
            del y
            stats.order.append(lo)
            layer_step(lo, x_lo, b)
        else:
            mid = (lo + hi) // 2
            x = x_lo
            for l in range(lo, mid):
                _, x = stack.forward_layer(l, x, stats)
            x_mid = x
            ys = []
            for l in range(mid, hi):
                y, x = stack.forward_layer(l, x, stats)
                ys.append(y)
            del x
            g = g_hi
            for l in range(hi - 1, mid - 1, -1):
                _, g = stack.backward_layer(l, ys.pop(), g, stats)
            g_mid = g
            rec(lo, mid, x_lo, g_mid)
            del g_mid
            rec(mid, hi, x_mid, g_hi)
        live[0] -= 1

    rec(0, len(stack), x0, g_out)
    return stats


def naive_flow(stack: LayerStack, x0, g_out, layer_step, stats: FlowStats | None = None):
    """The O(l^2) baseline of Sec. 5: for every layer, a forward pass to it
    and a full backward pass from the output."""
    stats = stats or FlowStats()
    for l in range(len(stack)):
        x = x0
        for k in range(l):
            _, x = stack.forward_layer(k, x, stats)
        a = x
        ys = []
        for k in range(l, len(stack)):
            y, x = stack.forward_layer(k, x, stats)
            ys.append(y)
        g = g_out
        for k in range(len(stack) - 1, l - 1, -1):
            b, g = stack.backward_layer(k, ys.pop(), g, stats)
        stats.order.append(l)
        layer_step(l, a, b)
    return stats


def bakron_layer_step(stack: LayerStack, bits: int, damp: float, style: str = "kfac",
                      iters: int = 1, alphabet: str = "sym", mse: bool = True, results=None):
    """The per-layer step of the global-Hessian flow: Kronecker factors of the
    layer's Hessian from its (a, b) samples (App. A), factorisation, scales
    (App. D: max-abs with the MSE shrink) and the BaKron rounding of W_l, all
    in libbakron.  Stores (codes, V, scale, A, B) per layer in `results`."""
    from . import _lib as lib
    results = {} if results is None else results

    def step(l, a, b):
        A, B = lib.kron_factors(a.contiguous(), b.contiguous(), style, iters=iters)
        f = lib.factor(A, B, damp)
        W = stack.W[l].contiguous()
        s = lib.mse_scales(W, bits, alphabet, grid=100 if mse else 0)
        codes, V = lib.solve(W, f, bits, s, alphabet=alphabet)
        f.close()
        results[l] = dict(codes=codes, V=V, scale=s, A=A, B=B)

    return step, results
