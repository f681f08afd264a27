"""Seeded synthetic inputs for the CosmoFlow conv stack.

This module holds NO arithmetic of the method (no convolution, activation or
pooling); it only draws random inputs, weights and upstream gradients, and
lists the layer shapes of each workload.  Both the GPU path and the oracle are
fed from here, so the two never compute an input for each other.

The paper's training data (N-body simulations binned into 128^3 particle-count
histograms, Section IV-C) is not available; these cubes stand in for it with
the same shape (128^3 single-channel fp32 volumes) and the same mean of 8
particles per voxel (512^3 particles in 256^3 voxels).

Recipes
  iid     lambda = exp(N(0,1)) per voxel, count ~ Poisson(lambda),
          x = log1p(count).
  grf     Gaussian random field with power spectrum P(k) ~ k^-2.5 (white
          noise filtered in Fourier space, P(0) = 0), standardised, turned
          into a lognormal density rho of mean 1 and variance 2
          (rho = exp(sigma*g - sigma^2/2), sigma^2 = ln 3), Poisson-sampled at
          mean 8*rho, then x = log1p(count).
  weights He-normal: N(0, 2/fan_in), fan_in = k^3 * C_in (untruncated).
  dy      upstream gradient N(0, 1).
"""
from __future__ import annotations

import hashlib

import numpy as np

# ---------------------------------------------------------------------------
# Workloads.  Each layer: conv kernel k (cubic), stride, output channels,
# whether a 2^3 stride-2 average pool follows.  Padding is TensorFlow SAME.
# ---------------------------------------------------------------------------

def stack_layers(c0: int = 1, c5: int = 128):
    """The six-layer CosmoFlow-shaped stack (first three layers pooled)."""
    return [
        dict(k=3, stride=1, cin=c0, cout=16, pool=True),
        dict(k=4, stride=1, cin=16, cout=32, pool=True),
        dict(k=4, stride=2, cin=32, cout=64, pool=True),
        dict(k=3, stride=1, cin=64, cout=64, pool=False),
        dict(k=2, stride=1, cin=64, cout=c5, pool=False),
        dict(k=2, stride=1, cin=c5, cout=c5, pool=False),
    ]


def paper_layers():
    """The first three conv layers of the paper's own network, the ones whose
    geometry the per-layer FLOP products of Table I pin (Section V-B): VALID
    padding, stride 1, each followed by the 2^3 stride-2 pool;
    128^3 -> 126^3 -> 63^3 -> 60^3 -> 30^3 -> 27^3 -> 13^3."""
    return [
        dict(k=3, stride=1, cin=1, cout=16, pool=True, pad="valid"),
        dict(k=4, stride=1, cin=16, cout=32, pool=True, pad="valid"),
        dict(k=4, stride=1, cin=32, cout=64, pool=True, pad="valid"),
    ]


WORKLOADS = {
    # single layer, forward only
    "layer1_32c": dict(size=32, batch=1, dtype="f32", c0=1, recipe="iid",
                       layers=stack_layers()[:1], backward=False, cfg=0),
    "stack_64c_b1_f32": dict(size=64, batch=1, dtype="f32", c0=1, recipe="iid",
                             layers=stack_layers(), backward=True, cfg=1),
    "stack_128c_b1_f32": dict(size=128, batch=1, dtype="f32", c0=1, recipe="grf",
                              layers=stack_layers(), backward=True, cfg=2),
    "stack_128c_b8_bf16": dict(size=128, batch=8, dtype="bf16", c0=1, recipe="grf",
                               layers=stack_layers(), backward=True, cfg=3),
    "stack_256c4_b2_bf16": dict(size=256, batch=2, dtype="bf16", c0=4, recipe="grf",
                                layers=stack_layers(c0=4, c5=256), backward=True, cfg=4),
    # the paper's own geometry (VALID) for its first three conv layers
    "paper_c1c3_64_b1_f32": dict(size=64, batch=1, dtype="f32", c0=1, recipe="iid",
                                 layers=paper_layers(), backward=True, cfg=5),
    "paper_c1c3_128_b1_f32": dict(size=128, batch=1, dtype="f32", c0=1, recipe="grf",
                                  layers=paper_layers(), backward=True, cfg=6),
    "paper_c1c3_128_b8_bf16": dict(size=128, batch=8, dtype="bf16", c0=1, recipe="grf",
                                   layers=paper_layers(), backward=True, cfg=7),
}

ALPHA = 0.01


def iid_lognormal_poisson(shape, seed: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    lam = np.exp(rng.standard_normal(shape))
    counts = rng.poisson(lam)
    return np.log1p(counts).astype(np.float32)


def grf_lognormal_poisson(size: int, seed: int, mean_count: float = 8.0,
                          slope: float = -2.5) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    noise = rng.standard_normal((size, size, size))
    f = np.fft.rfftn(noise)
    k1 = np.fft.fftfreq(size) * size
    k3 = np.fft.rfftfreq(size) * size
    kk = np.sqrt(k1[:, None, None] ** 2 + k1[None, :, None] ** 2 + k3[None, None, :] ** 2)
    amp = np.zeros_like(kk)
    nz = kk > 0
    amp[nz] = kk[nz] ** (slope / 2.0)
    g = np.fft.irfftn(f * amp, s=(size, size, size))
    g = (g - g.mean()) / g.std()
    sigma2 = np.log(3.0)
    rho = np.exp(np.sqrt(sigma2) * g - sigma2 / 2.0)
    counts = rng.poisson(mean_count * rho)
    return np.log1p(counts).astype(np.float32)


def make_input(name: str, sample_seed_base: int | None = None) -> np.ndarray:
    """NDHWC float32 input batch of a workload."""
    wl = WORKLOADS[name]
    S, B, C = wl["size"], wl["batch"], wl["c0"]
    base = 10000 * wl["cfg"] if sample_seed_base is None else sample_seed_base
    x = np.empty((B, S, S, S, C), np.float32)
    for b in range(B):
        for c in range(C):
            seed = base + 100 * c + b
            if wl["recipe"] == "iid":
                x[b, ..., c] = iid_lognormal_poisson((S, S, S), seed)
            else:
                x[b, ..., c] = grf_lognormal_poisson(S, seed)
    return x


def he_normal(k: int, cin: int, cout: int, seed: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    std = np.sqrt(2.0 / (k * k * k * cin))
    return (rng.standard_normal((k, k, k, cin, cout)) * std).astype(np.float32)


def make_weights(name: str):
    wl = WORKLOADS[name]
    ws, bs = [], []
    for i, L in enumerate(wl["layers"]):
        ws.append(he_normal(L["k"], L["cin"], L["cout"], 20000 + 100 * wl["cfg"] + i))
        bs.append(np.zeros(L["cout"], np.float32))
    return ws, bs


#: widths of the fully-connected head (Section III-A: three FC layers, three
#: outputs; the first two widths are in the paper's missing Fig. 2 -- a reading)
HEAD_WIDTHS = (128, 64, 3)

#: parameter ranges of the simulations (Section IV-C): Omega_M, sigma_8, n_s
PARAM_RANGES = ((0.25, 0.35), (0.78, 0.95), (0.9, 1.0))


def make_head(name: str, features: int, widths=HEAD_WIDTHS):
    """He-normal FC weights [in][out] (seed 40000 + 100 cfg + layer), zero
    biases, and per-sample targets drawn uniformly from the simulations'
    parameter ranges (seed 50000 + cfg)."""
    wl = WORKLOADS[name]
    dims = [features, *widths]
    ws, bs = [], []
    for i in range(len(widths)):
        rng = np.random.Generator(np.random.PCG64(40000 + 100 * wl["cfg"] + i))
        ws.append((rng.standard_normal((dims[i], dims[i + 1])) * np.sqrt(2.0 / dims[i])).astype(np.float32))
        bs.append(np.zeros(dims[i + 1], np.float32))
    rng = np.random.Generator(np.random.PCG64(50000 + wl["cfg"]))
    tgt = np.stack([rng.uniform(lo, hi, wl["batch"]) for lo, hi in PARAM_RANGES], 1).astype(np.float32)
    return ws, bs, tgt


def normal(shape, seed: int, scale: float = 1.0) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    return (rng.standard_normal(shape) * scale).astype(np.float32)


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()
