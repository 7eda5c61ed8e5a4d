"""Pins of the oracle's centroids, scores and top-k selection (Method: cluster
assignment)."""
import itertools

import numpy as np
import pytest

from oracle import ref


def test_centroid_score_is_mean_pairwise_logit():
    """Method, scoring: qbar . kbar equals the average of q . k over all pairs."""
    rng = np.random.default_rng(0)
    Q = rng.standard_normal((37, 6))
    K = rng.standard_normal((29, 6))
    perm_q, perm_k = rng.permutation(37), rng.permutation(29)
    cq = np.array([8, 8, 8, 8, 5])
    ck = np.array([8, 8, 8, 5])
    S = ref.centroid_scores(ref.centroids(Q, perm_q, cq), ref.centroids(K, perm_k, ck))
    qm, km = ref.cluster_members(perm_q, cq), ref.cluster_members(perm_k, ck)
    for a in range(5):
        for b in range(4):
            want = np.mean([Q[i] @ K[j] for i in qm[a] for j in km[b]])
            assert abs(S[a, b] - want) < 1e-13


def test_centroids_use_real_members_only():
    X = np.arange(12, dtype=float).reshape(6, 2)
    c = ref.centroids(X, np.array([5, 0, 3, 1, 2, 4]), np.array([4, 2]))
    assert np.allclose(c, [X[[5, 0, 3, 1]].mean(0), X[[2, 4]].mean(0)])


@pytest.mark.parametrize("seed", range(20))
def test_topk_bruteforce(seed):
    """Top-k: the k-subset with the largest scores; among equally good subsets
    (ties) the lexicographically smallest index set; listed ascending."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 11))
    k = int(rng.integers(1, n + 1))
    S = rng.integers(-3, 4, size=(3, n)).astype(float)  # many ties
    got = ref.topk(S, k)
    for a in range(3):
        best = None
        for sub in itertools.combinations(range(n), k):
            key = (sorted((-S[a, j] for j in sub)), sub)
            if best is None or key < best:
                best = key
        assert got[a].tolist() == list(best[1])


def test_topk_real_valued():
    rng = np.random.default_rng(9)
    S = rng.standard_normal((50, 40))
    got = ref.topk(S, 7)
    for a in range(50):
        assert set(got[a]) == set(np.argsort(S[a])[-7:])
        assert (np.diff(got[a]) > 0).all()
