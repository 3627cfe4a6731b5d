"""Seeded synthetic workloads for the BaKron solver (shared by tests, bench, smoke).

This module only *generates inputs*; it holds none of the solver's arithmetic
(no damping, no factors, no rounding).  Everything is fp64 internally and
rounded once to fp32, so the solver and the oracle receive bit-identical
arrays.

The paper measures solver speed on matrices it does not describe (Table 3) and
quality on real LLM layers with Pile calibration data (App. D).  Neither is
available here, so these LLM-shaped synthetic layers stand in for them:

* W: Gaussian N(0, sigma^2) (optionally heavy-tailed Student-t nu=5 scaled to
  std sigma; optionally a few outlier columns scaled x10).
* A = X X^T / N with X (n x N): each sample column is an AR(1) sequence along
  the feature index, x_0 = e_0, x_t = rho x_{t-1} + sqrt(1-rho^2) e_t, plus an
  optional rank-r spike U Z (U orthonormal n x r, Z ~ N(0, 10)).
* B = G G^T / N likewise with G (m x N).
* Per-row scale s_i = max_j |W_ij| / l in fp32, l = 2^(bits-1) - 1.
* damp = 0.01 (relative to each matrix's own mean diagonal); applied by the
  solver and by the oracle, never here.

RNG: numpy PCG64 seeded by SeedSequence([config_id, seed, stream]) with
streams W=0, X(for A)=1, G(for B)=2, spike=3, outliers=4.

Calibration samples for the Kronecker-factor construction (App. A) come from
kron_samples (global case: inputs a and output gradients b) and mlp_samples
(gated MLP: inputs x, weights, features g and f), with *_torch versions of the
same recipes for full-size workloads drawn on the GPU.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

STREAM_W, STREAM_X, STREAM_G, STREAM_SPIKE, STREAM_OUT = 0, 1, 2, 3, 4


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    m: int
    n: int
    sigma: float
    NA: int
    rhoA: float
    NB: int
    rhoB: float
    bits: int
    spikeA: int = 0
    outlier_frac: float = 0.0
    heavy_tail: bool = False
    damp: float = 0.01
    notes: str = field(default="", compare=False)


CONFIGS = {
    1: Config(1, "tiny-64x64", 64, 64, 0.02, 256, 0.5, 256, 0.3, 4),
    2: Config(2, "attn-proj-4096x4096", 4096, 4096, 0.02, 8192, 0.6, 8192, 0.2, 4,
              spikeA=32, outlier_frac=0.001),
    3: Config(3, "mlp-up-11008x4096", 11008, 4096, 0.015, 8192, 0.5, 8192, 0.2, 3),
    4: Config(4, "mlp-down-4096x11008", 4096, 11008, 0.01, 16384, 0.5, 16384, 0.3, 2,
              heavy_tail=True),
    5: Config(5, "llama70b-mlp-28672x8192", 28672, 8192, 0.01, 32768, 0.5, 32768, 0.2, 4,
              spikeA=64),
}


def _rng(cid: int, seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([cid, seed, stream])))


def qmax_of_bits(bits: int) -> int:
    return (1 << (int(bits) - 1)) - 1


def gram_ar1(d: int, N: int, rho: float, rng: np.random.Generator, spike_rank: int = 0,
             spike_rng: np.random.Generator | None = None, chunk: int = 4096,
             device: str = "cpu") -> np.ndarray:
    """X X^T / N for X (d x N) of AR(1) sample columns (+ optional spike), fp64.

    Samples are drawn in chunks of `chunk` columns (bounded memory); the Gram
    is accumulated in fp64, on `device` ("cpu" uses numpy; "cuda" uses torch
    fp64 matmul) -- input generation only.
    """
    U = None
    if spike_rank > 0:
        q, _ = np.linalg.qr(spike_rng.standard_normal((d, spike_rank)))
        U = q
    c = np.sqrt(1.0 - rho * rho)
    use_torch = device != "cpu"
    if use_torch:
        import torch
        G = torch.zeros((d, d), dtype=torch.float64, device=device)
    else:
        G = np.zeros((d, d), np.float64)
    done = 0
    while done < N:
        k = min(chunk, N - done)
        eps = rng.standard_normal((d, k))
        X = np.empty((d, k), np.float64)
        X[0] = eps[0]
        for t in range(1, d):
            X[t] = rho * X[t - 1] + c * eps[t]
        if U is not None:
            Z = spike_rng.standard_normal((spike_rank, k)) * np.sqrt(10.0)
            X += U @ Z
        if use_torch:
            Xt = torch.from_numpy(X).to(device)
            G.addmm_(Xt, Xt.T)
            del Xt
        else:
            G += X @ X.T
        done += k
    if use_torch:
        G = G.cpu().numpy()
    G /= float(N)
    return 0.5 * (G + G.T)


def ar1_samples(N: int, d: int, rho: float, rng: np.random.Generator, spike_rank: int = 0,
                spike_rng: np.random.Generator | None = None,
                norm_sigma: float = 0.0) -> np.ndarray:
    """N calibration samples as the rows of an N x d fp32 matrix: each an
    AR(1) sequence along the feature index (the recipe of gram_ar1), plus an
    optional rank-r spike, times an optional per-sample log-normal magnitude
    exp(norm_sigma * z_k) (tokens and gradients of very different norms)."""
    c = np.sqrt(1.0 - rho * rho)
    eps = rng.standard_normal((N, d))
    X = np.empty((N, d), np.float64)
    X[:, 0] = eps[:, 0]
    for t in range(1, d):
        X[:, t] = rho * X[:, t - 1] + c * eps[:, t]
    if spike_rank > 0:
        q, _ = np.linalg.qr(spike_rng.standard_normal((d, spike_rank)))
        X += (spike_rng.standard_normal((N, spike_rank)) * np.sqrt(10.0)) @ q.T
    if norm_sigma > 0:
        X *= np.exp(norm_sigma * rng.standard_normal((N, 1)))
    return X.astype(np.float32)


def kron_samples(N: int, n: int, m: int, seed: int) -> dict:
    """Paired samples of a global Hessian: inputs a (N x n: AR(1), rho 0.5,
    rank-4 spike, log-normal token norms sigma 0.5) and output gradients b
    (N x m: AR(1), rho 0.2, log-normal norms sigma 1.0), fp32."""
    r = [np.random.Generator(np.random.PCG64(np.random.SeedSequence([2000, N, n, m, seed, k])))
         for k in range(3)]
    a = ar1_samples(N, n, 0.5, r[0], spike_rank=min(4, n), spike_rng=r[2], norm_sigma=0.5)
    b = ar1_samples(N, m, 0.2, r[1], norm_sigma=1.0)
    return dict(a=a, b=b)


def mlp_samples(N: int, dm: int, dff: int, seed: int) -> dict:
    """A gated MLP, MLP(x) = W_down (W_up x (.) SiLU(W_gate x)), with Gaussian
    weights (W_gate, W_up ~ N(0, 1/dm), W_down ~ N(0, 1/dff)) and inputs x as
    in kron_samples; the features g = SiLU(W_gate x) and
    f = SiLU'(W_gate x) (.) W_up x are this forward pass, in fp64, rounded
    once to fp32 (the module's own computation, not the Hessian's)."""
    r = [np.random.Generator(np.random.PCG64(np.random.SeedSequence([3000, N, dm, dff, seed, k])))
         for k in range(3)]
    x = ar1_samples(N, dm, 0.5, r[0], spike_rank=min(4, dm), spike_rng=r[2], norm_sigma=0.5)
    Wg = r[1].standard_normal((dff, dm)) / np.sqrt(dm)
    Wu = r[1].standard_normal((dff, dm)) / np.sqrt(dm)
    Wd = r[1].standard_normal((dm, dff)) / np.sqrt(dff)
    z = x.astype(np.float64) @ Wg.T
    u = x.astype(np.float64) @ Wu.T
    sg = 1.0 / (1.0 + np.exp(-z))
    g = z * sg
    f = sg * (1.0 + z * (1.0 - sg)) * u
    return dict(x=x, Wg=Wg.astype(np.float32), Wu=Wu.astype(np.float32),
                Wd=Wd.astype(np.float32), g=g.astype(np.float32), f=f.astype(np.float32))


def ar1_samples_torch(N: int, d: int, rho: float, gen, device, spike_rank: int = 0,
                      norm_sigma: float = 0.0):
    """The recipe of ar1_samples drawn with torch's generator `gen` on `device`
    in fp32 (for full-size workloads; different random numbers from the numpy
    version).  Returns an N x d contiguous fp32 tensor."""
    import torch
    # the recursion x_0 = e_0, x_t = rho x_{t-1} + c e_t unrolled: x = L e with
    # L[t][s] = rho^(t-s) * (1 if s == 0 else c), one product for all samples
    c = float(np.sqrt(1.0 - rho * rho))
    t = torch.arange(d, device=device, dtype=torch.float64)
    L = torch.where(t[:, None] >= t[None, :], rho ** (t[:, None] - t[None, :]).clamp(min=0),
                    torch.zeros((), dtype=torch.float64, device=device))
    L[:, 1:] *= c
    eps = torch.randn((N, d), generator=gen, device=device)
    X = eps @ L.t().to(torch.float32)
    del eps
    if spike_rank > 0:
        q, _ = torch.linalg.qr(torch.randn((d, spike_rank), generator=gen, device=device))
        X.addmm_(torch.randn((N, spike_rank), generator=gen, device=device) * np.sqrt(10.0), q.t())
    if norm_sigma > 0:
        X.mul_(torch.exp(norm_sigma * torch.randn((N, 1), generator=gen, device=device)))
    return X.contiguous()


def kron_samples_torch(N: int, n: int, m: int, seed: int, device) -> dict:
    """kron_samples' recipe on the device (torch generator seeded by seed)."""
    import torch
    gen = torch.Generator(device=device).manual_seed(2000 + seed)
    a = ar1_samples_torch(N, n, 0.5, gen, device, spike_rank=min(4, n), norm_sigma=0.5)
    b = ar1_samples_torch(N, m, 0.2, gen, device, norm_sigma=1.0)
    return dict(a=a, b=b)


def mlp_samples_torch(N: int, dm: int, dff: int, seed: int, device, feature: str = "g") -> dict:
    """mlp_samples' recipe on the device in fp32, with only the requested
    feature ("g" for W_up, "f" for W_gate)."""
    import torch
    gen = torch.Generator(device=device).manual_seed(3000 + seed)
    x = ar1_samples_torch(N, dm, 0.5, gen, device, spike_rank=min(4, dm), norm_sigma=0.5)
    Wg = torch.randn((dff, dm), generator=gen, device=device) / np.sqrt(dm)
    Wu = torch.randn((dff, dm), generator=gen, device=device) / np.sqrt(dm)
    Wd = (torch.randn((dm, dff), generator=gen, device=device) / np.sqrt(dff)).contiguous()
    z = x @ Wg.t()
    if feature == "g":
        feat = torch.nn.functional.silu(z, inplace=True)
    else:
        sg = torch.sigmoid(z)
        z.mul_(1.0 - sg).add_(1.0).mul_(sg)        # SiLU'(z) = sg (1 + z (1 - sg))
        del sg
        feat = z.mul_(x @ Wu.t())
    return dict(x=x, Wg=Wg, Wu=Wu, Wd=Wd, feat=feat.contiguous())


def toy_mlp(L: int, d: int, N: int, seed: int) -> dict:
    """A stack of L square layers (y = W x, then SiLU) for the flow of Sec. 5:
    W_l ~ N(0, 2/d), inputs x0 as in kron_samples (AR(1) rows with a spike and
    log-normal norms), and output gradients g_out ~ N(0, 1) standing in for
    the gradients of sampled-label losses (App. D), all fp32."""
    r = [np.random.Generator(np.random.PCG64(np.random.SeedSequence([4000, L, d, N, seed, k])))
         for k in range(3)]
    W = [(r[0].standard_normal((d, d)) * np.sqrt(2.0 / d)).astype(np.float32) for _ in range(L)]
    x0 = ar1_samples(N, d, 0.5, r[1], spike_rank=min(4, d), spike_rng=r[2], norm_sigma=0.5)
    g_out = r[2].standard_normal((N, d)).astype(np.float32)
    return dict(W=W, x0=x0, g_out=g_out)


def make_weights(cfg: Config, seed: int) -> np.ndarray:
    rng = _rng(cfg.cid, seed, STREAM_W)
    if cfg.heavy_tail:
        W = rng.standard_t(5.0, size=(cfg.m, cfg.n)) * (cfg.sigma / np.sqrt(5.0 / 3.0))
    else:
        W = rng.standard_normal((cfg.m, cfg.n)) * cfg.sigma
    if cfg.outlier_frac > 0:
        k = int(round(cfg.outlier_frac * cfg.n))
        cols = _rng(cfg.cid, seed, STREAM_OUT).choice(cfg.n, size=k, replace=False)
        W[:, cols] *= 10.0
    return W.astype(np.float32)


def row_scales(W: np.ndarray, bits: int) -> np.ndarray:
    """s_i = max_j |W_ij| / l in fp32 (App. D: max-abs per row over l)."""
    l = np.float32(qmax_of_bits(bits))
    return (np.max(np.abs(W.astype(np.float32)), axis=1) / l).astype(np.float32)


def make(cid: int, seed: int = 0, device: str = "cpu") -> dict:
    """Canonical fp32 inputs for configuration `cid`.

    Returns dict(W, A, B, scale, bits, damp, cfg, sha256) with W (m x n),
    A (n x n) and B (m x m) undamped symmetric Grams, all fp32 row-major.
    """
    cfg = CONFIGS[cid]
    W = make_weights(cfg, seed)
    A = gram_ar1(cfg.n, cfg.NA, cfg.rhoA, _rng(cid, seed, STREAM_X), cfg.spikeA,
                 _rng(cid, seed, STREAM_SPIKE), device=device).astype(np.float32)
    B = gram_ar1(cfg.m, cfg.NB, cfg.rhoB, _rng(cid, seed, STREAM_G),
                 device=device).astype(np.float32)
    s = row_scales(W, cfg.bits)
    out = dict(W=W, A=A, B=B, scale=s, bits=cfg.bits, damp=cfg.damp, cfg=cfg)
    out["sha256"] = {k: hashlib.sha256(np.ascontiguousarray(out[k]).tobytes()).hexdigest()
                     for k in ("W", "A", "B", "scale")}
    return out


def make_random(m: int, n: int, seed: int, bits: int = 4, rhoA: float = 0.5,
                rhoB: float = 0.3, NA: int | None = None, NB: int | None = None,
                sigma: float = 0.02, identity_B: bool = False) -> dict:
    """Small random problem of any shape (parity cases): same recipe as the
    configs with N = 4*max(dim, 16) samples unless given."""
    rng_w = np.random.Generator(np.random.PCG64(np.random.SeedSequence([1000, m, n, seed, 0])))
    W = (rng_w.standard_normal((m, n)) * sigma).astype(np.float32)
    NA = NA or 4 * max(n, 16)
    NB = NB or 4 * max(m, 16)
    rx = np.random.Generator(np.random.PCG64(np.random.SeedSequence([1000, m, n, seed, 1])))
    rg = np.random.Generator(np.random.PCG64(np.random.SeedSequence([1000, m, n, seed, 2])))
    A = gram_ar1(n, NA, rhoA, rx).astype(np.float32)
    B = None if identity_B else gram_ar1(m, NB, rhoB, rg).astype(np.float32)
    return dict(W=W, A=A, B=B, scale=row_scales(W, bits), bits=bits, damp=0.01)


def ar1_toeplitz(d: int, rho: float) -> np.ndarray:
    """Population AR(1) covariance [rho^|i-j|] in fp32 (exact closed-form case)."""
    idx = np.arange(d)
    return (rho ** np.abs(idx[:, None] - idx[None, :])).astype(np.float32)
