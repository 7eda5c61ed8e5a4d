"""Pins of the oracle's dense, sparse and compensated attention against what the
paper and the mathematics fix: brute force, a library routine on the dense
case, the error identities of the paper, the closed-form special cases and a
hand-worked example."""
import json
import math
import os

import numpy as np
import pytest

from oracle import ref

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rand(seed, n, d, scale=1.0):
    rng = np.random.default_rng(seed)
    return [scale * rng.standard_normal((n, d)) for _ in range(3)]


def test_dense_matches_bruteforce_loops():
    """Preliminaries: o = sum_i w_i v_i with w the softmax of the logits."""
    Q, K, V = _rand(1, 9, 5)
    tau = 0.7
    o, lse = ref.dense_attention(Q, K, V, tau)
    for i in range(9):
        logits = [tau * sum(Q[i, t] * K[j, t] for t in range(5)) for j in range(9)]
        z = sum(math.exp(x) for x in logits)
        for t in range(5):
            want = sum(math.exp(logits[j]) * V[j, t] for j in range(9)) / z
            assert abs(o[i, t] - want) < 1e-12
        assert abs(lse[i] - math.log(z)) < 1e-12


def test_dense_matches_torch_sdpa_fp64():
    torch = pytest.importorskip("torch")
    Q, K, V = _rand(2, 40, 16, scale=2.0)
    o, _ = ref.dense_attention(Q, K, V, 1.0 / 4.0)
    t = torch.nn.functional.scaled_dot_product_attention(
        *(torch.from_numpy(x)[None, None] for x in (Q, K, V)))
    assert np.abs(o - t[0, 0].numpy()).max() < 1e-12


def _clusters(n, c):
    counts = np.array([min(c, n - a * c) for a in range(-(-n // c))])
    return counts


def test_all_clusters_kept_equals_dense():
    """With every key cluster selected the method is exactly dense attention,
    compensation or not (Preliminaries: sparse attention over the full set)."""
    Q, K, V = _rand(3, 70, 8, scale=1.5)
    for mode in ("none", "pca", "metric"):
        r = ref.forward(Q, K, V, 16, 16, 5, mode)  # 70 keys -> 5 clusters, all kept
        o, lse = ref.dense_attention(Q, K, V, 1 / math.sqrt(8))
        assert np.abs(r["out"] - o).max() < 1e-12
        assert np.abs(r["lse"] - lse).max() < 1e-12
        assert r["lists"].shape == (5, 5)


def test_hand_worked_compensation():
    g = json.load(open(os.path.join(GOLD, "smc_hand.json")))
    e = math.e
    Q, K, V = (np.array(g[x]) for x in ("q", "k", "v"))
    r = ref.forward(Q, K, V, 1, g["ck"], 1, tau=g["tau"], perm_q=np.array([0]),
                    perm_k=np.arange(4), lists=np.array(g["lists"]))
    assert np.allclose(r["o_s"][0], [1 / (1 + e), e / (1 + e)], atol=1e-15)
    assert abs(r["lse_s"][0] - math.log(1 + e)) < 1e-15
    assert np.allclose(r["out"][0], [(1 + 2 * e) / (1 + 3 * e), 3 * e / (1 + 3 * e)], atol=1e-15)
    assert abs(r["lse"][0] - math.log(1 + 3 * e)) < 1e-15
    o, _ = ref.dense_attention(Q, K, V, 1.0)
    z = 2 + e + e * e
    assert np.allclose(o[0], [(1 + 2 * e * e) / z, (e + 2 * e * e) / z], atol=1e-15)
    r0 = ref.forward(Q, K, V, 1, g["ck"], 1, enable_comp=False, tau=g["tau"],
                     perm_q=np.array([0]), perm_k=np.arange(4), lists=np.array(g["lists"]))
    assert np.allclose(r0["out"], r0["o_s"])


def _setup_partition(seed=4, n=64, d=8, c=8, keep=(0, 3)):
    Q, K, V = _rand(seed, n, d)
    rng = np.random.default_rng(seed + 100)
    perm_k = rng.permutation(n)
    counts = _clusters(n, c)
    lists = np.array([list(keep)] * (-(-n // c)))
    return Q, K, V, perm_k, counts, lists


def _weights(Q, K, tau):
    L = tau * Q @ K.T
    W = np.exp(L - L.max(axis=1, keepdims=True))
    return W / W.sum(axis=1, keepdims=True)


def test_error_identity_uncompensated():
    """Preliminaries: o - o_S = (1 - w_S)(o_Sbar - o_S) for every query."""
    Q, K, V, perm_k, counts, lists = _setup_partition()
    tau = 0.5
    n, c = Q.shape[0], 8
    r = ref.forward(Q, K, V, c, c, 2, "none", enable_comp=False, tau=tau,
                    perm_q=np.arange(n), perm_k=perm_k, lists=lists)
    o, _ = ref.dense_attention(Q, K, V, tau)
    W = _weights(Q, K, tau)
    mem = ref.cluster_members(perm_k, counts)
    S = np.concatenate([mem[b] for b in lists[0]])
    Sbar = np.setdiff1d(np.arange(n), S)
    wS = W[:, S].sum(axis=1)
    o_sbar = (W[:, Sbar] @ V[Sbar]) / W[:, Sbar].sum(axis=1, keepdims=True)
    lhs = o - r["o_s"]
    rhs = (1 - wS)[:, None] * (o_sbar - r["o_s"])
    assert np.abs(lhs - rhs).max() < 1e-14


def test_error_identity_compensated():
    """App. A: with w the dense softmax weights, w_c = exp(tau q.kbar_c)/Z, delta_c =
    mean_c(w) - w_c and Cov_c(w, v) the in-cluster covariance,
      o - o_hat = sum_c |c| (delta_c (vbar_c - o_hat) + Cov_c(w, v))            (exact form)
      o - o_hat = (1/d_hat) sum_c |c| (delta_c (vbar_c - o) + Cov_c(w, v))      (second form)
    with d_hat = w_S + sum_c |c| w_c; also delta_c >= 0 (Jensen). This pins the
    size weighting and the centroid value of the compensation."""
    Q, K, V, perm_k, counts, lists = _setup_partition(seed=5)
    tau = 0.5
    n, c = Q.shape[0], 8
    r = ref.forward(Q, K, V, c, c, 2, "none", tau=tau, perm_q=np.arange(n), perm_k=perm_k,
                    lists=lists)
    o, _ = ref.dense_attention(Q, K, V, tau)
    L = tau * Q @ K.T
    Z = np.exp(L).sum(axis=1)
    W = np.exp(L) / Z[:, None]
    mem = ref.cluster_members(perm_k, counts)
    excl = [b for b in range(len(mem)) if b not in lists[0]]
    S = np.concatenate([mem[b] for b in lists[0]])
    d_hat = W[:, S].sum(axis=1)
    exact = np.zeros_like(o)
    second = np.zeros_like(o)
    for b in excl:
        idx = mem[b]
        kbar, vbar = K[idx].mean(axis=0), V[idx].mean(axis=0)
        w_c = np.exp(tau * Q @ kbar) / Z
        wbar = W[:, idx].mean(axis=1)
        delta = wbar - w_c
        assert (delta >= -1e-15).all()
        cov = ((W[:, idx] - wbar[:, None])[:, :, None] * (V[idx] - vbar)[None]).mean(axis=1)
        d_hat = d_hat + len(idx) * w_c
        exact += len(idx) * (delta[:, None] * (vbar[None] - r["out"]) + cov)
        second += len(idx) * (delta[:, None] * (vbar[None] - o) + cov)
    assert np.abs((o - r["out"]) - exact).max() < 1e-14
    assert np.abs((o - r["out"]) - second / d_hat[:, None]).max() < 1e-14


def test_identical_keys_make_compensation_exact():
    """Preliminaries: with every key of each excluded cluster identical the Jensen
    and covariance terms vanish, so compensated sparse attention equals dense."""
    rng = np.random.default_rng(6)
    n, d, c = 64, 8, 8
    Q = rng.standard_normal((n, d))
    V = rng.standard_normal((n, d))
    K = np.repeat(rng.standard_normal((n // c, d)), c, axis=0)  # cluster b: rows b*c..b*c+7 equal
    lists = np.array([[0, 3]] * (n // c))
    r = ref.forward(Q, K, V, c, c, 2, "none", tau=0.4, perm_q=np.arange(n), perm_k=np.arange(n),
                    lists=lists)
    o, lse = ref.dense_attention(Q, K, V, 0.4)
    assert np.abs(r["out"] - o).max() < 1e-14
    assert np.abs(r["lse"] - lse).max() < 1e-13
    assert np.abs(r["o_s"] - o).max() > 1e-3  # the uncompensated part alone is not exact


def test_key_shift_leaves_outputs_unchanged():
    """Softmax shift invariance: adding one vector to every key changes each
    query's logits by a constant, so with fixed clusters and lists the dense,
    sparse and compensated outputs are unchanged."""
    Q, K, V, perm_k, counts, lists = _setup_partition(seed=7)
    shift = np.random.default_rng(8).standard_normal(Q.shape[1])
    kw = dict(tau=0.5, perm_q=np.arange(64), perm_k=perm_k, lists=lists)
    a = ref.forward(Q, K, V, 8, 8, 2, "none", **kw)
    b = ref.forward(Q, K + shift, V, 8, 8, 2, "none", **kw)
    assert np.abs(a["out"] - b["out"]).max() < 1e-13
    assert np.abs(a["o_s"] - b["o_s"]).max() < 1e-13


def test_sparse_part_ignores_unselected_keys():
    """Block-sparse attention reads only the selected clusters: perturbing the
    keys and values of an unselected cluster leaves o_S unchanged."""
    Q, K, V, perm_k, counts, lists = _setup_partition(seed=9)
    kw = dict(tau=0.5, perm_q=np.arange(64), perm_k=perm_k, lists=lists)
    a = ref.forward(Q, K, V, 8, 8, 2, "none", **kw)
    mem = ref.cluster_members(perm_k, counts)
    K2, V2 = K.copy(), V.copy()
    K2[mem[5]] += 3.0
    V2[mem[5]] -= 2.0
    b = ref.forward(Q, K2, V2, 8, 8, 2, "none", **kw)
    assert np.array_equal(a["o_s"], b["o_s"])
    assert np.abs(a["out"] - b["out"]).max() > 1e-6
