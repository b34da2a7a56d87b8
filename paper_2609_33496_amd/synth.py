"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers: it holds none of the method's arithmetic (no
quantizer, no statistic, no routing), and it is the one piece of code that both the HIP
path's tests/benchmark and the CPU oracle's tests use.  Everything is numpy ``default_rng``
(PCG64) so an array is reproducible from its seed alone.

The paper's real tensors (SDXL / SDXL-Turbo / PixArt-alpha checkpoints and their
activations on COCO-2014 captions) are not available; these recipes stand in for them:

* ``single_layer``: X [256, 640] Student-t (nu = 4) with 1% of the columns scaled x20 as
  outliers; W [640, 640] N(0, 0.02^2) with each output channel scaled by exp(N(0, 0.5^2)).
* ``hetero_weights``: output channels drawn from a mix of families (Gaussian 50 %, Laplace
  10 %, uniform 15 %, Student-t3 10 %, Gaussian with 0.5 % x10 outliers 10 %, Gaussian with a
  log-normal(0, 1) scale per 32-block 5 %), each at unit variance, times 0.02 and a per-row
  factor exp(N(0, 0.5^2)).  Per-row Gaussians alone make a single format win everywhere;
  real trained weights are not Gaussian per row.
* ``diffusion_acts``: activations at timestep t of a scaled-linear schedule,
  sqrt(abar_t) * GMM + sqrt(1 - abar_t) * lam * t3, with a 4-component Gaussian mixture
  (means +-0.5, +-1.5, sigma 0.1, equal weights) and a per-layer factor lam ~ U(0.5, 2)
  on the Student-t (nu = 3) term, so kurtosis falls as t -> 0 and layers cross the routing
  gates at different timesteps.  abar_t is the workload's own schedule tensor, computed the
  way diffusion pipelines store it (binary32 linspace of sqrt(beta), binary32 cumprod).
"""
from __future__ import annotations

import numpy as np


def rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(list(key))


def single_layer(seed: int = 0, M: int = 256, K: int = 640, N: int = 640):
    """Single linear layer: X [M, K] t4 with round(1% of K) outlier columns x20; W [N, K]."""
    g = rng(seed, 1)
    X = g.standard_t(4.0, size=(M, K)).astype(np.float32)
    n_out = int(round(0.01 * K))
    cols = g.choice(K, size=n_out, replace=False)
    X[:, cols] *= np.float32(20.0)
    W = (g.normal(0.0, 0.02, size=(N, K)) * np.exp(g.normal(0.0, 0.5, size=(N, 1)))).astype(np.float32)
    return X, W


FAMILIES = ("gauss", "laplace", "uniform", "t3", "outlier", "blockvar")
FAMILY_P = (0.50, 0.10, 0.15, 0.10, 0.10, 0.05)


def hetero_weights(seed: int, N: int, K: int, families=None):
    """W [N, K] float32 with heterogeneous per-channel distributions (see module doc).
    Returns (W, family_index[N])."""
    g = rng(seed, 2)
    fam = g.choice(len(FAMILIES), size=N, p=FAMILY_P) if families is None else np.asarray(families)
    W = np.empty((N, K), np.float64)
    for f, name in enumerate(FAMILIES):
        rows = np.nonzero(fam == f)[0]
        if rows.size == 0:
            continue
        shape = (rows.size, K)
        if name == "gauss":
            v = g.normal(size=shape)
        elif name == "laplace":
            v = g.laplace(scale=1.0 / np.sqrt(2.0), size=shape)
        elif name == "uniform":
            v = g.uniform(-np.sqrt(3.0), np.sqrt(3.0), size=shape)
        elif name == "t3":
            v = g.standard_t(3.0, size=shape) / np.sqrt(3.0)
        elif name == "outlier":
            v = g.normal(size=shape)
            v[g.random(size=shape) < 0.005] *= 10.0
        else:  # blockvar
            v = g.normal(size=shape)
            nb = K // 32
            sc = np.exp(g.normal(0.0, 1.0, size=(rows.size, nb)))
            v[:, :nb * 32] *= np.repeat(sc, 32, axis=1)
        W[rows] = v
    W *= 0.02 * np.exp(g.normal(0.0, 0.5, size=(N, 1)))
    return W.astype(np.float32), fam


def alphas_cumprod(T: int = 1000, beta0: float = 0.00085, beta1: float = 0.012, scaled: bool = True):
    """The workload's noise-schedule tensor, as diffusion pipelines store it (binary32)."""
    if scaled:
        betas = np.linspace(np.float32(beta0) ** 0.5, np.float32(beta1) ** 0.5, T, dtype=np.float32) ** 2
    else:
        betas = np.linspace(beta0, beta1, T, dtype=np.float32)
    return np.cumprod(np.float32(1.0) - betas, dtype=np.float32)


def layer_lambda(seed: int, layer: int) -> float:
    return float(rng(seed, 3, layer).uniform(0.5, 2.0))


def diffusion_acts(seed: int, layer: int, t: int, M: int, K: int, abar=None, step: int = 0):
    """Activation X [M, K] of `layer` at timestep t (see module doc)."""
    if abar is None:
        abar = alphas_cumprod()
    a = float(abar[t])
    g = rng(seed, 4, layer, t, step)
    means = np.array([-1.5, -0.5, 0.5, 1.5])
    comp = g.integers(0, 4, size=(M, K))
    gmm = means[comp] + 0.1 * g.normal(size=(M, K))
    noise = layer_lambda(seed, layer) * g.standard_t(3.0, size=(M, K))
    return (np.sqrt(a) * gmm + np.sqrt(1.0 - a) * noise).astype(np.float32)


# --------------------------------------------------------------------------------------------
# layer sets of the workloads (K -> N per linear; M tokens)
# --------------------------------------------------------------------------------------------
def sdxl_block_layers(d: int = 1280):
    """SDXL-like transformer-block linear set at width d: QKV d->3d, out-proj d->d,
    GEGLU d->8d, FF-out 4d->d.  Returns [(name, K, N)]."""
    return [("qkv", d, 3 * d), ("out", d, d), ("geglu", d, 8 * d), ("ff_out", 4 * d, d)]


def pixart_block_layers(d: int = 1152):
    """PixArt-alpha-like DiT block: QKV, proj, MLP fc1/fc2 and cross-attention KV from the
    4096-wide text encoder.  Returns [(name, K, N, M_tokens)]."""
    return [("qkv", d, 3 * d, 8192), ("proj", d, d, 8192), ("fc1", d, 4 * d, 8192),
            ("fc2", 4 * d, d, 8192), ("cross_kv", 4096, d, 240)]


# --------------------------------------------------------------------------------------------
# the same recipes drawn on the GPU (torch, seeded per array), for the benchmark's full-size
# stacks (1.64 G weights, 1.5 G activations) where drawing on the host would take minutes.
# Only normal and uniform draws: Laplace by inverting its CDF, Student-t with integral nu as
# a normal over the root of a chi-square built from nu squared normals.
# --------------------------------------------------------------------------------------------
def _gen(device, *key: int):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(rng(*key).integers(0, 2 ** 62)))
    return g


def _student_t_dev(nu: int, shape, g, device):
    import torch
    z = torch.randn(shape, generator=g, device=device)
    chi = torch.zeros(shape, device=device)
    for _ in range(nu):
        chi += torch.randn(shape, generator=g, device=device) ** 2
    return z / torch.sqrt(chi / nu)


def hetero_weights_dev(seed: int, N: int, K: int, device="cuda"):
    """hetero_weights' families and proportions, drawn on `device` (float32 [N, K])."""
    import torch
    g = _gen(device, seed, 12)
    fam = torch.multinomial(torch.tensor(FAMILY_P, device=device), N, replacement=True, generator=g)
    W = torch.empty((N, K), dtype=torch.float32, device=device)
    for f, name in enumerate(FAMILIES):
        rows = torch.nonzero(fam == f).flatten()
        if rows.numel() == 0:
            continue
        shape = (rows.numel(), K)
        if name == "gauss":
            v = torch.randn(shape, generator=g, device=device)
        elif name == "laplace":
            u = torch.rand(shape, generator=g, device=device) - 0.5
            v = -torch.sign(u) * torch.log1p(-2.0 * u.abs()) / np.sqrt(2.0)
        elif name == "uniform":
            v = (torch.rand(shape, generator=g, device=device) * 2.0 - 1.0) * np.sqrt(3.0)
        elif name == "t3":
            v = _student_t_dev(3, shape, g, device) / np.sqrt(3.0)
        elif name == "outlier":
            v = torch.randn(shape, generator=g, device=device)
            v = torch.where(torch.rand(shape, generator=g, device=device) < 0.005, v * 10.0, v)
        else:  # blockvar
            v = torch.randn(shape, generator=g, device=device)
            nb = K // 32
            sc = torch.exp(torch.randn((rows.numel(), nb), generator=g, device=device))
            v[:, :nb * 32] *= torch.repeat_interleave(sc, 32, dim=1)
        W[rows] = v
    W *= 0.02 * torch.exp(0.5 * torch.randn((N, 1), generator=g, device=device))
    return W


def diffusion_acts_dev(seed: int, layer: int, t: int, M: int, K: int, device="cuda", step: int = 0):
    """diffusion_acts' mixture at timestep t, drawn on `device` (float32 [M, K])."""
    import torch
    a = float(alphas_cumprod()[t])
    g = _gen(device, seed, 14, layer, t, step)
    means = torch.tensor([-1.5, -0.5, 0.5, 1.5], device=device)
    comp = torch.randint(0, 4, (M, K), generator=g, device=device)
    gmm = means[comp] + 0.1 * torch.randn((M, K), generator=g, device=device)
    noise = layer_lambda(seed, layer) * _student_t_dev(3, (M, K), g, device)
    return (np.sqrt(a) * gmm + np.sqrt(1.0 - a) * noise).to(torch.float32)


def sdxl_stack_layers():
    """The 70-block SDXL-like linear stack: 10 blocks at width 640 then 60 at width 1280, each
    with the block linear set.  Returns [(name, K, N, width)] in order (280 linears)."""
    out = []
    for d, nblk in ((640, 10), (1280, 60)):
        for b in range(nblk):
            for name, K, N in sdxl_block_layers(d):
                out.append((f"d{d}.{name}", K, N, d))
    return out
