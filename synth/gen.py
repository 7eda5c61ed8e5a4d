"""Synthetic workloads standing in for the paper's evaluation data.

The paper evaluates on TabPFN-3 train-to-train attention (tabular rows, Results:
TabPFN-3) and on Wan 2.1-14B video self-attention (Results: Wan 2.1-14B T2V).
Neither the weights nor the datasets are available, so every input here is a
seeded draw with the shapes and structure of those workloads:

* Gaussian-mixture rows (queries and keys share the component centres and draw
  their labels independently, so they are co-located), for the tabular shapes;
* a smooth spatio-temporal Gaussian random field plus noise on a (T, H, W)
  latent grid, tokens shuffled, for the video shapes.

All arrays are float32 of shape [B*H, N, d]. For bf16 workloads the values are
rounded to bf16 (round to nearest even) here, so that the float32 arrays hold
exactly the values the GPU receives. Random generator: NumPy PCG64 seeded with
``[config, head]``; draw order per head: mixture parameters, Q, K, V, token
permutation.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); return float32.
    Finite inputs only (the largest finite pattern plus the rounding increment
    still fits in 32 bits)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    b = (b + (np.uint32(0x7FFF) + lsb)) & np.uint32(0xFFFF0000)
    return b.view(np.float32)


def keep_to_k(keep: float, n_kc: int) -> int:
    """Number of kept key clusters for a keep fraction: ceil(keep * n_kc), at least 1."""
    return max(1, min(n_kc, int(math.ceil(keep * n_kc - 1e-9))))


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    heads: int
    n: int
    d: int
    dtype: str  # "f32" or "bf16"
    c: tuple  # cluster sizes to run
    keeps: tuple  # keep fractions (k = ceil(keep * n_kc))
    recipe: str
    params: dict = field(default_factory=dict)


CONFIGS = {
    1: Config(1, "mixture8-n1024-d64-f32", 1, 1024, 64, "f32", (64,), (0.25, 1.0), "mixture",
              dict(centres=8, sigma=0.3, weights="uniform")),
    2: Config(2, "tabular-8h-n65536-d64-bf16", 8, 65536, 64, "bf16", (128,), (1 / 8,), "mixture",
              dict(centres=64, sigma=0.5, weights="dirichlet")),
    3: Config(3, "tabular-16h-n262144-d64-bf16", 16, 262144, 64, "bf16", (128,), (1 / 16, 1 / 4),
              "mixture", dict(centres=256, weights="uniform", aniso=(0.1, 1.0), outliers=0.05)),
    4: Config(4, "video480p-40h-n32760-d128-bf16", 40, 32760, 128, "bf16", (64,), (1 / 4,), "field",
              dict(grid=(21, 30, 52), corr_len=4.0, noise=0.2)),
    5: Config(5, "video720p-40h-n75600-d128-bf16", 40, 75600, 128, "bf16", (64, 128),
              (1 / 4, 1 / 8, 1 / 16), "field", dict(grid=(21, 45, 80), corr_len=4.0, noise=0.2)),
}


def _mixture_head(rng, n, d, centres, sigma=None, weights="uniform", aniso=None, outliers=0.0):
    mu = rng.standard_normal((centres, d))
    if weights == "dirichlet":
        pi = rng.dirichlet(np.ones(centres))
    else:
        pi = np.full(centres, 1.0 / centres)
    if aniso is not None:
        lo, hi = aniso
        var = np.exp(rng.uniform(math.log(lo), math.log(hi), size=(centres, d)))
        scale = np.sqrt(var)
    else:
        scale = np.full((centres, d), float(sigma))

    def draw():
        z = rng.choice(centres, size=n, p=pi)
        x = mu[z] + scale[z] * rng.standard_normal((n, d))
        if outliers > 0:
            m = int(round(outliers * n))
            rows = rng.choice(n, size=m, replace=False)
            x[rows] = rng.uniform(-3.0, 3.0, size=(m, d))
        return x

    q = draw()
    k = draw()
    v = rng.standard_normal((n, d))
    return q, k, v


def _field_head(rng, grid, d, corr_len, noise):
    T, H, W = grid
    n = T * H * W
    # White noise per channel, filtered by a periodic Gaussian kernel of std
    # corr_len / sqrt(2), so the field's correlation is exp(-r^2 / (2 corr_len^2)).
    sig = corr_len / math.sqrt(2.0)
    white = rng.standard_normal((T, H, W, d))
    spec = np.fft.rfftn(white, axes=(0, 1, 2))
    ft = np.fft.fftfreq(T)[:, None, None]
    fh = np.fft.fftfreq(H)[None, :, None]
    fw = np.fft.rfftfreq(W)[None, None, :]
    g = np.exp(-2.0 * (math.pi ** 2) * (sig ** 2) * (ft ** 2 + fh ** 2 + fw ** 2))
    f = np.fft.irfftn(spec * g[..., None], s=(T, H, W), axes=(0, 1, 2)).reshape(n, d)
    f = (f - f.mean(axis=0)) / f.std(axis=0)
    q = f + noise * rng.standard_normal((n, d))
    k = f + noise * rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    p = rng.permutation(n)
    return q[p], k[p], v[p]


def _finish(arrs, dtype):
    out = []
    for a in arrs:
        a = np.asarray(a, dtype=np.float32)
        out.append(bf16_round(a) if dtype == "bf16" else a)
    return out


def mixture_inputs(seed, heads, n, d, dtype="bf16", centres=16, sigma=0.5, weights="uniform",
                   aniso=None, outliers=0.0):
    """Gaussian-mixture Q/K/V of shape [heads, n, d] for arbitrary (test) sizes."""
    qs, ks, vs = [], [], []
    for h in range(heads):
        rng = np.random.default_rng([int(seed), h])
        q, k, v = _mixture_head(rng, n, d, centres, sigma, weights, aniso, outliers)
        q, k, v = _finish((q, k, v), dtype)
        qs.append(q), ks.append(k), vs.append(v)
    return np.stack(qs), np.stack(ks), np.stack(vs)


def field_inputs(seed, heads, grid, d, dtype="bf16", corr_len=4.0, noise=0.2):
    """Random-field Q/K/V of shape [heads, T*H*W, d] (video-shaped workloads)."""
    qs, ks, vs = [], [], []
    for h in range(heads):
        rng = np.random.default_rng([int(seed), h])
        q, k, v = _field_head(rng, grid, d, corr_len, noise)
        q, k, v = _finish((q, k, v), dtype)
        qs.append(q), ks.append(k), vs.append(v)
    return np.stack(qs), np.stack(ks), np.stack(vs)


def _config_head(cid, h):
    cfg = CONFIGS[cid]
    rng = np.random.default_rng([cid, int(h)])
    p = cfg.params
    if cfg.recipe == "mixture":
        q, k, v = _mixture_head(rng, cfg.n, cfg.d, p["centres"], p.get("sigma"),
                                p.get("weights", "uniform"), p.get("aniso"),
                                p.get("outliers", 0.0))
    else:
        q, k, v = _field_head(rng, p["grid"], cfg.d, p["corr_len"], p["noise"])
    return _finish((q, k, v), cfg.dtype)


def _config_head_star(args):
    return _config_head(*args)


def make_config(cid, heads=None, workers=1):
    """Inputs of a named workload. ``heads`` selects a subset of head indices
    (default: all); each head's draw depends only on (config id, head index),
    so ``workers`` > 1 draws heads in that many forked processes with the same
    result. Fork before anything initialises a GPU in the calling process."""
    cfg = CONFIGS[cid]
    hs = list(range(cfg.heads) if heads is None else heads)
    if workers > 1 and len(hs) > 1:
        import multiprocessing as mp
        with mp.get_context("fork").Pool(min(workers, len(hs))) as pool:
            parts = pool.map(_config_head_star, [(cid, h) for h in hs])
    else:
        parts = [_config_head(cid, h) for h in hs]
    return tuple(np.stack([pt[i] for pt in parts]) for i in range(3))
