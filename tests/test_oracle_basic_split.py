"""Pins of the oracle's basic recursive splitting (Method: recursive splitting,
basic; a PDDP variation with power iteration)."""
import numpy as np
import pytest

from oracle import ref


def test_irwin_hall_normal_moments():
    """Sum of 12 uniforms minus 6: values in [-6, 6), mean 0 and variance 1
    (12 x 1/12), light tails (|x| > 4 is rare)."""
    x = ref.irwin_hall_normal(np.arange(200000)).astype(float)
    assert x.min() >= -6.0 and x.max() < 6.0
    assert abs(x.mean()) < 0.01 and abs(x.var() - 1.0) < 0.01
    assert (np.abs(x) > 4).mean() < 1e-3
    # each value is (an integer) / 2^24 - 6 rounded once to float32
    u = (ref.splitmix64(np.arange(12, dtype=np.uint64)) >> np.uint64(40)).astype(np.int64).sum()
    assert ref.irwin_hall_normal([0])[0] == np.float32(u * 2.0 ** -24 - 6.0)


def test_basic_noise_differs_per_node():
    a = ref.basic_noise(16, 0, 0, 2, 3)
    assert not np.array_equal(a, ref.basic_noise(16, 0, 0, 2, 2))
    assert not np.array_equal(a, ref.basic_noise(16, 0, 0, 3, 3))
    assert not np.array_equal(a, ref.basic_noise(16, 0, 1, 2, 3))
    assert not np.array_equal(a, ref.basic_noise(16, 1, 0, 2, 3))
    assert np.array_equal(a, ref.basic_noise(16, 0, 0, 2, 3))


def test_power_direction_converges_to_top_eigenvector():
    """With many iterations the direction is the leading eigenvector of the
    subsample's centred covariance (numpy eigh in fp64)."""
    rng = np.random.default_rng(1)
    X = rng.standard_normal((64, 12)) @ np.diag(np.linspace(3, 0.5, 12)) + 2.0
    X = X @ np.linalg.qr(rng.standard_normal((12, 12)))[0]
    v = ref.power_direction(X, rng.standard_normal(12), iters=300).astype(float)
    Xc = X - X.mean(axis=0)
    lam, U = np.linalg.eigh(Xc.T @ Xc)
    u = U[:, -1]
    assert abs(abs(v @ u) - 1.0) < 1e-5
    assert abs(np.linalg.norm(v) - 1.0) < 1e-6


def test_power_direction_dominant_axis_and_degenerate():
    rng = np.random.default_rng(2)
    axis = np.array([0.6, 0.0, -0.8, 0.0])
    X = np.outer(rng.standard_normal(40) * 10, axis) + 0.01 * rng.standard_normal((40, 4))
    v = ref.power_direction(X, ref.basic_noise(4, 0, 0, 0, 0)).astype(float)
    assert abs(abs(v @ axis) - 1.0) < 1e-4
    # all rows equal: no variance, the start vector is kept
    v0 = np.array([1.0, 2.0, 3.0, 4.0], np.float32)
    assert np.array_equal(ref.power_direction(np.ones((8, 4)), v0), v0)


def test_warm_start():
    """Root: the noise itself. Otherwise the mean of the parent estimate and the
    noise rescaled to the parent's norm (compared with the same formula in
    fp64)."""
    rng = np.random.default_rng(3)
    r = rng.standard_normal(10).astype(np.float32)
    assert np.array_equal(ref.warm_start(None, r), r)
    vp = rng.standard_normal(10).astype(np.float32)
    v0 = ref.warm_start(vp, r).astype(float)
    want = 0.5 * (vp + r * np.linalg.norm(vp) / np.linalg.norm(r))
    assert np.abs(v0 - want).max() < 1e-6


@pytest.mark.parametrize("n,d,c", [(1000, 8, 32), (777, 16, 64), (4096, 6, 16), (130, 4, 128)])
def test_basic_split_structure(n, d, c):
    """Valid permutation with the split tree's cluster sizes; every split is a
    threshold split along its direction (the largest projection sent left is at
    most the smallest sent right, projections recomputed in fp64), the left
    part has left_size members, and children keep ascending index order."""
    rng = np.random.default_rng(n)
    Y = (rng.standard_normal((n, d)) * np.linspace(2, 0.2, d)).astype(np.float32)
    trace = []
    perm, cid, counts = ref.basic_split(Y, c, head=1, side=0, trace=trace)
    assert sorted(perm) == list(range(n))
    sizes = []
    s, rest = n, []

    def tree(s):
        if s <= c:
            sizes.append(s)
            return
        mL = ref.left_size(s, c)
        tree(mL)
        tree(s - mL)
    tree(n)
    assert counts.tolist() == sizes
    for members, v, left, right in trace:
        assert len(left) == ref.left_size(len(members), c)
        assert (np.diff(left) > 0).all() and (np.diff(right) > 0).all()
        proj = Y[members].astype(float) @ v.astype(float)
        pl = proj[np.isin(members, left)]
        pr = proj[np.isin(members, right)]
        scale = np.abs(proj).max() + 1e-30
        assert pl.max() <= pr.min() + 1e-5 * scale


def test_basic_split_separates_two_groups():
    """Two groups far apart along one axis: the first split puts them on
    different sides (PDDP's principal direction)."""
    rng = np.random.default_rng(4)
    n = 512
    lab = rng.integers(0, 2, n)
    lab[:256], lab[256:] = 0, 1
    rng.shuffle(lab)
    Y = rng.standard_normal((n, 6)) * 0.3
    Y[:, 3] += np.where(lab == 1, 8.0, -8.0)
    trace = []
    ref.basic_split(Y, 64, trace=trace)
    members, v, left, right = trace[0]
    assert len(set(lab[left])) == 1 and len(set(lab[right])) == 1


def test_basic_split_noise_matters_only_through_the_start():
    """Same head: identical results. On strongly anisotropic data another
    head's noise finds the same first split, up to the sign of the direction
    (which swaps the children)."""
    rng = np.random.default_rng(5)
    Y = (rng.standard_normal((600, 5)) * np.array([10, 5, 2, 1, 0.5])).astype(np.float32)
    a = ref.basic_split(Y, 32, head=0)[0]
    assert np.array_equal(a, ref.basic_split(Y, 32, head=0)[0])
    ta, tb = [], []
    ref.basic_split(Y, 32, head=0, iters=60, trace=ta)
    ref.basic_split(Y, 32, head=7, iters=60, trace=tb)
    sa = {frozenset(ta[0][2].tolist()), frozenset(ta[0][3].tolist())}
    sb = {frozenset(tb[0][2].tolist()), frozenset(tb[0][3].tolist())}
    assert sa == sb or abs(float(ta[0][1] @ tb[0][1])) > 0.999


def test_default_iterations_reach_the_direction():
    """With the default number of iterations and an eigenvalue ratio of 4
    between the two leading directions of the subsample, the estimate is within
    1e-3 of the leading eigenvector from a random start."""
    rng = np.random.default_rng(6)
    Q = np.linalg.qr(rng.standard_normal((8, 8)))[0]
    X = (rng.standard_normal((64, 8)) * np.array([4, 2, 1, 1, 0.5, 0.5, 0.3, 0.2])) @ Q.T
    Xc = X - X.mean(axis=0)
    lam, U = np.linalg.eigh(Xc.T @ Xc)
    assert lam[-1] / lam[-2] > 3
    v = ref.power_direction(X.astype(np.float32), ref.basic_noise(8, 0, 0, 0, 0)).astype(float)
    assert 1.0 - abs(v @ U[:, -1]) < 1e-3
