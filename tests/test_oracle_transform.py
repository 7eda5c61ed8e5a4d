"""Pins of the oracle's split spaces (Method: transforms; App. B) against the
properties the paper derives for them."""
import numpy as np
import pytest

from oracle import ref


def _mix(seed, n=400, d=6, low_rank=False):
    rng = np.random.default_rng(seed)
    cen = rng.standard_normal((5, d)) * 2
    Q = cen[rng.integers(0, 5, n)] + 0.5 * rng.standard_normal((n, d)) + 0.7
    K = cen[rng.integers(0, 5, n)] + 0.5 * rng.standard_normal((n, d)) - 0.3
    if low_rank:
        Q[:, -2:] = 0.0  # queries span a subspace: M is singular
    return Q, K


@pytest.mark.parametrize("low_rank", [False, True])
def test_key_metric_distances(low_rank):
    """Method, key clustering: |y_a - y_b|^2 = (k_a - k_b)^T (Q^T Q / n) (k_a - k_b),
    i.e. the mean squared difference of the two keys' logits over all queries."""
    Q, K = _mix(0, low_rank=low_rank)
    Y = ref.key_split_space(Q, K, "metric")
    rng = np.random.default_rng(1)
    for _ in range(50):
        a, b = rng.integers(0, len(K), 2)
        want = ((Q @ (K[a] - K[b])) ** 2).mean()
        got = ((Y[a] - Y[b]) ** 2).sum()
        assert abs(got - want) <= 1e-10 * max(1.0, want)


def test_query_representation_properties():
    """App. B.2: r(q) = R_k q / |R_k q| with R_k^T R_k = K_c^T K_c: unit norm, and
    r_a . r_b = q_a^T C q_b / sqrt(q_a^T C q_a q_b^T C q_b), C the key covariance."""
    Q, K = _mix(2)
    R = ref.query_representation(Q, K)
    C = np.cov(K.T, bias=True)
    assert np.abs((R * R).sum(axis=1) - 1).max() < 1e-12
    G = Q @ C @ Q.T
    nrm = np.sqrt(np.diag(G))
    assert np.abs(R @ R.T - G / np.outer(nrm, nrm)).max() < 1e-11
    Y = ref.query_split_space(Q, K, "metric")
    assert np.abs(Y @ Y.T - R @ R.T).max() < 1e-11  # rotation only


def test_zero_query_maps_to_zero():
    Q, K = _mix(3)
    Q[7] = 0.0
    assert (ref.query_representation(Q, K)[7] == 0).all()


def test_pairwise_difference_gram_is_2n_covariance():
    """App. B.2: D^T D = 2n K_c^T K_c for D the matrix of all ordered key differences."""
    rng = np.random.default_rng(4)
    K = rng.standard_normal((30, 4)) + 1.5
    n = len(K)
    D = (K[:, None, :] - K[None, :, :]).reshape(n * n, -1)
    assert np.abs(D.T @ D - 2 * n * n * ref.centred_cov(K)).max() < 1e-10


@pytest.mark.parametrize("mode", ["pca", "metric", "adaptive"])
def test_split_space_is_decorrelated_sorted_and_oriented(mode):
    """Diagonalized splitting works on principal coordinates: the covariance of
    Y is diagonal with non-increasing variances, and (orientation reading) every
    coordinate has a non-negative mean."""
    Q, K = _mix(5)
    for Y in (ref.key_split_space(Q, K, mode), ref.query_split_space(Q, K, mode)):
        C = np.cov(Y.T, bias=True)
        off = C - np.diag(np.diag(C))
        assert np.abs(off).max() < 1e-10 * np.abs(C).max()
        assert (np.diff(np.diag(C)) <= 1e-12).all()
        assert (Y.mean(axis=0) >= -1e-12).all()


def test_query_space_is_invariant_to_key_shift():
    """App. B.1/B.2: the centred key metric quotients out the softmax shift, so
    shifting every key by one vector leaves the query split space unchanged."""
    Q, K = _mix(6)
    a = ref.query_split_space(Q, K, "metric")
    b = ref.query_split_space(Q, K + np.array([3.0, -1, 2, 0.5, 0, 1]), "metric")
    assert np.abs(a - b).max() < 1e-9


def test_adaptive_representation_distances():
    """App. B.1: for adaptive assignment the queries live in the metric
    K_c^T K_c / n, i.e. |r(q1) - r(q2)|^2 = |K_c (q1 - q2)|^2 / n, written out
    here with the centred key matrix itself."""
    Q, K = _mix(7)
    R = ref.query_representation_adaptive(Q, K)
    Kc = K - K.mean(axis=0)
    rng = np.random.default_rng(7)
    for a, b in rng.integers(0, len(Q), size=(40, 2)):
        want = ((Kc @ (Q[a] - Q[b])) ** 2).sum() / len(K)
        got = ((R[a] - R[b]) ** 2).sum()
        assert abs(got - want) <= 1e-10 * max(1.0, want)


def test_adaptive_representation_quotients_softmax_shift():
    """App. B.1: queries whose logits differ by a constant over all keys (the
    softmax's invariance) get the same representation, and so do queries that
    differ along a direction in which the keys do not vary; the top-k
    representation normalises, the adaptive one does not (scaling q scales r)."""
    rng = np.random.default_rng(8)
    K = rng.standard_normal((50, 5))
    K[:, 4] = 2.5  # every key has the same last coordinate
    Q = rng.standard_normal((20, 5))
    delta = np.array([0, 0, 0, 0, 3.0])
    a = ref.query_representation_adaptive(Q, K)
    b = ref.query_representation_adaptive(Q + delta, K)
    assert np.abs(a - b).max() < 1e-12
    assert np.allclose(ref.query_representation_adaptive(2 * Q, K), 2 * a, atol=1e-12)
    # same attention distribution => same point: logits K q1 and K q2 differ by a constant
    assert np.allclose(np.diff(K @ (Q[0] + delta) - K @ Q[0]), 0.0)


def test_adaptive_key_space_equals_metric():
    Q, K = _mix(9)
    assert np.array_equal(ref.key_split_space(Q, K, "adaptive"), ref.key_split_space(Q, K, "metric"))


def test_metric_key_space_independent_of_root_choice():
    """Any factor S with S S^T = M gives the same split coordinates (up to the
    orientation rule): compare E sqrt(L) with the symmetric root E sqrt(L) E^T."""
    Q, K = _mix(7)
    M = ref.second_moment(Q)
    lam, E = np.linalg.eigh(M)
    Rsym = E @ np.diag(np.sqrt(np.maximum(lam, 0))) @ E.T
    Z = K @ Rsym
    Ysym = Z @ ref.pca_basis(Z)
    assert np.abs(Ysym - ref.key_split_space(Q, K, "metric")).max() < 1e-10


def test_none_mode_is_identity():
    Q, K = _mix(8)
    assert np.array_equal(ref.key_split_space(Q, K, "none"), K)
    assert np.array_equal(ref.query_split_space(Q, K, "none"), Q)


def test_clamped_root_of_indefinite_matrix():
    """Method, key clustering: negative eigenvalues are clamped to zero."""
    rng = np.random.default_rng(10)
    E, _ = np.linalg.qr(rng.standard_normal((3, 3)))
    A = E @ np.diag([4.0, 1.0, -0.25]) @ E.T
    S = ref.psd_root(A)
    want = E @ np.diag([4.0, 1.0, 0.0]) @ E.T
    assert np.abs(S @ S.T - want).max() < 1e-13


def test_splitmix64_published_outputs():
    """The generator behind the random-cluster control: its first outputs from
    state 0 as published with splitmix64."""
    out = ref.splitmix64(np.arange(3))
    assert [int(x) for x in out] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_random_split_space():
    """Coordinates are 24-bit fractions in [0, 1), differ between heads and
    sides, look uniform, and splitting on them gives valid clusters whose
    membership does not follow the data."""
    Y = ref.random_split_space(5000, 16, head=3, side=1)
    assert Y.shape == (5000, 16) and Y.min() >= 0.0 and Y.max() < 1.0
    assert np.array_equal(Y * 2 ** 24, np.floor(Y * 2 ** 24))
    assert abs(Y.mean() - 0.5) < 0.01 and abs(Y.var() - 1 / 12) < 0.005
    assert not np.array_equal(Y, ref.random_split_space(5000, 16, head=3, side=0))
    assert not np.array_equal(Y, ref.random_split_space(5000, 16, head=4, side=1))
    c = ref.random_split_space(1, 4, head=0, side=0)[0]
    want = (ref.splitmix64(np.arange(4)) >> np.uint64(40)).astype(float) * 2.0 ** -24
    assert np.array_equal(c, want)  # head 0, queries, token 0: outputs 0..3
    Q, K = _mix(10)
    yq = ref.query_split_space(Q, K, "random", head=2)
    perm, cid, counts = ref.split(yq, 16)
    assert sorted(perm) == list(range(len(Q)))
    # clusters of random coordinates ignore the data: cluster means of Q stay
    # near the global mean (a data-driven split would separate them)
    means = ref.centroids(Q, perm, counts)
    assert np.abs(means - Q.mean(axis=0)).max() < 6 * Q.std(axis=0).max() / np.sqrt(16)
