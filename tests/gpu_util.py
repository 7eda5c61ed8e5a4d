"""Helpers for the GPU parity tests: move seeded host inputs to the device and
lay them out as the C ABI expects. No method arithmetic lives here."""
import numpy as np
import torch

TOL = {"f32": 1e-5, "bf16": 2e-2}


def tdtype(dt):
    return torch.float32 if dt == "f32" else torch.bfloat16


def dev(x, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(dtype)


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def permuted_rows(X, perm, c, dtype):
    """[BH, n, d] -> [BH, n_pad, d] rows in cluster order, zero pad rows."""
    BH, n, d = X.shape
    nc = -(-n // c)
    out = np.zeros((BH, nc * c, d), np.float32)
    for b in range(BH):
        out[b, :n] = X[b, perm[b]]
    return dev(out, dtype)


def value_tiles(V, perm, c, dtype):
    """[BH, n, d] -> [BH, nc, d, c]: each key cluster's value rows, transposed."""
    BH, n, d = V.shape
    nc = -(-n // c)
    rows = np.zeros((BH, nc * c, d), np.float32)
    for b in range(BH):
        rows[b, :n] = V[b, perm[b]]
    tiles = rows.reshape(BH, nc, c, d).transpose(0, 1, 3, 2)
    return dev(tiles, dtype)


def counts(n, c):
    return np.array([min(c, n - a * c) for a in range(-(-n // c))], np.int32)


def random_lists(rng, BH, nqc, nkc, k):
    L = np.zeros((BH, nqc, k), np.int32)
    for b in range(BH):
        for a in range(nqc):
            L[b, a] = np.sort(rng.choice(nkc, size=k, replace=False))
    return L


def flush(msg):
    print(msg, flush=True)
