"""Pins of the oracle's diagonalized recursive splitting (Method: recursive
splitting): a hand-worked example, structural invariants re-derived by plain
sorting, and exhaustive brute force with exact rational variances on tiny
inputs."""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import ref

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_split():
    g = json.load(open(os.path.join(GOLD, "split_hand.json")))
    Y = np.array(g["y"], dtype=np.float64)
    assert np.signbit(Y[5, 0]) and not np.signbit(Y[2, 0])  # the fixture keeps -0.0
    trace = []
    perm, cid, counts = ref.split(Y, g["c"], trace)
    assert perm.tolist() == g["perm"]
    assert counts.tolist() == g["counts"]
    assert cid.tolist() == g["cid"]
    assert [t[1] for t in trace] == g["jstars"]


@pytest.mark.parametrize("c", [1, 2, 4, 8, 64, 128])
def test_left_size_is_nearest_multiple_of_c_to_half(c):
    """The part below the threshold is the multiple of c closest to s/2; on a
    tie the smaller one; the remainder always lands in the right part."""
    for s in range(c + 1, 40 * c + 7):
        mL = ref.left_size(s, c)
        mults = [j * c for j in range(0, s // c + 1)]
        best = min(mults, key=lambda m: (abs(2 * m - s), m))
        assert mL == best, (s, c)
        assert 0 < mL < s
        assert (s - mL) % c == s % c


def _structure_checks(Y, c, perm, cid, counts, trace):
    n = Y.shape[0]
    assert sorted(perm.tolist()) == list(range(n))
    nc = -(-n // c)
    assert len(counts) == nc
    assert (counts[:-1] == c).all() and 1 <= counts[-1] <= c
    assert counts.sum() == n
    starts = np.concatenate([[0], np.cumsum(counts)[:-1]])
    for a, (s0, m) in enumerate(zip(starts, counts)):
        seg = perm[s0:s0 + m]
        assert (np.diff(seg) > 0).all()  # ascending original index inside a cluster
        assert (cid[seg] == a).all()
    for members, jstar, mL, left, right in trace:
        # re-derive the two children by plain sorting of (value, index) pairs
        pairs = sorted((float(Y[i, jstar]) + 0.0, int(i)) for i in members)
        want_left = sorted(i for _, i in pairs[:mL])
        assert left.tolist() == want_left
        assert right.tolist() == sorted(set(members.tolist()) - set(want_left))
        # the chosen coordinate has the largest exact subsample variance
        s = len(members)
        m = min(Y.shape[1], s)
        rows = Y[members[ref.subsample_positions(s, m)]]
        ex = [_exact_pvar(rows[:, t]) for t in range(Y.shape[1])]
        assert ex[jstar] == max(ex) or abs(float(ex[jstar]) - float(max(ex))) <= 1e-12 * float(max(ex))


def _exact_pvar(col):
    vals = [Fraction(float(x)) for x in col]
    mean = sum(vals) / len(vals)
    return sum((v - mean) ** 2 for v in vals) / len(vals)


@pytest.mark.parametrize("seed,n,d,c", [(0, 100, 8, 8), (1, 257, 5, 16), (2, 512, 16, 64),
                                        (3, 1000, 3, 32), (4, 130, 64, 128)])
def test_split_structure_and_rederived_nodes(seed, n, d, c):
    Y = np.random.default_rng(seed).standard_normal((n, d)).astype(np.float32).astype(np.float64)
    trace = []
    perm, cid, counts = ref.split(Y, c, trace)
    _structure_checks(Y, c, perm, cid, counts, trace)


def test_split_with_many_ties():
    """Heavily tied coordinates (small integers): ties go by original index."""
    Y = np.random.default_rng(5).integers(-2, 3, size=(300, 4)).astype(np.float64)
    Y[Y == 0] = np.where(np.random.default_rng(6).random((Y == 0).sum()) < 0.5, -0.0, 0.0)
    trace = []
    perm, cid, counts = ref.split(Y, 16, trace)
    _structure_checks(Y, 16, perm, cid, counts, trace)


def _brute_split(Y, c):
    """Independent brute force: exact rational variances over the whole node
    (d >= n, so the subsample is the node), exhaustive search over every subset
    of the left size for the one whose (value, index) keys all precede the rest."""
    n, d = Y.shape
    leaves = []

    def rec(members):
        s = len(members)
        if s <= c:
            leaves.append(list(members))
            return
        var = [_exact_pvar([Y[i, t] for i in members]) for t in range(d)]
        j = var.index(max(var))
        mL = c * ((-(-s // c)) // 2)
        key = {i: (float(Y[i, j]) + 0.0, i) for i in members}
        found = None
        for sub in itertools.combinations(members, mL):
            rest = [i for i in members if i not in sub]
            if max(key[i] for i in sub) < min(key[i] for i in rest):
                assert found is None
                found = list(sub)
        rec(sorted(found))
        rec(sorted(set(members) - set(found)))

    rec(list(range(n)))
    return leaves


@pytest.mark.parametrize("seed", range(12))
def test_tiny_split_bruteforce(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 13))
    c = int(rng.choice([1, 2, 4]))
    d = 12  # d >= n: the subsample is every member
    Y = rng.standard_normal((n, d)).astype(np.float32).astype(np.float64)
    perm, cid, counts = ref.split(Y, c)
    leaves = _brute_split(Y, c)
    assert perm.tolist() == [i for leaf in leaves for i in leaf]
    assert counts.tolist() == [len(x) for x in leaves]


def test_subsample_positions():
    assert ref.subsample_positions(5, 5) == [0, 1, 2, 3, 4]
    for s in range(1, 300):
        for m in range(1, min(s, 70) + 1):
            p = ref.subsample_positions(s, m)
            assert len(set(p)) == m and p == sorted(p) and 0 <= p[0] and p[-1] < s


def test_sequential_variance_exact_cases():
    rows = np.array([[1.0, 2.0, 5.0], [3.0, 2.0, -5.0]])
    assert ref.sequential_variance(rows).tolist() == [1.0, 0.0, 25.0]
    rng = np.random.default_rng(3)
    R = rng.standard_normal((64, 10)).astype(np.float32).astype(np.float64)
    v = ref.sequential_variance(R)
    for t in range(10):
        assert abs(v[t] - float(_exact_pvar(R[:, t]))) <= 1e-14 * float(_exact_pvar(R[:, t]))
