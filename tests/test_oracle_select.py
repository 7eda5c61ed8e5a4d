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


# ---------------------------------------------------------------------------
# The two-pass histogram selection (Method: selection)
# ---------------------------------------------------------------------------


def _hist_bruteforce(S, counts, tau, min_count, mass_recall):
    """The selection restated without the two passes: scan every edge of the
    128 x 128 grid from the top and take the first whose upper set holds both
    thresholds."""
    n = len(S)
    g = ref.hist_grid_index(S)
    if g is None or min_count >= n:
        return np.arange(n)
    mass = ref.hist_mass_units(S, counts, tau)
    need = min(int(np.ceil(float(mass_recall) * float(mass.sum()))), int(mass.sum()))
    for G in range(ref.HIST_GRID - 1, -1, -1):
        up = g >= G
        if up.sum() >= min_count and mass[up].sum() >= need:
            return np.nonzero(up)[0]
    return np.arange(n)


def _rows(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 300))
    kind = seed % 4
    if kind == 0:
        S = rng.standard_normal(n) * rng.uniform(0.1, 30)
    elif kind == 1:
        S = rng.integers(-5, 6, size=n).astype(float)  # many exact ties
    elif kind == 2:
        S = np.concatenate([rng.standard_normal(n - 3), [50.0, 49.0, -40.0]])  # outliers
    else:
        S = rng.exponential(3.0, n)
    counts = rng.integers(1, 129, size=n)
    return S, counts


@pytest.mark.parametrize("seed", range(24))
def test_hist_select_matches_grid_bruteforce(seed):
    S, counts = _rows(seed)
    n = len(S)
    rng = np.random.default_rng(100 + seed)
    for min_count, mass_recall in ((1, 0.0), (int(rng.integers(1, n + 1)), 0.0), (16, 0.9),
                                   (1, 0.5), (3, 0.99), (16, 1.0), (n + 5, 0.3)):
        got = ref.hist_select(S, counts, 0.125, min_count, mass_recall)
        want = _hist_bruteforce(S, counts, 0.125, min_count, mass_recall)
        assert np.array_equal(got, want), (seed, min_count, mass_recall)


@pytest.mark.parametrize("seed", range(12))
def test_hist_topk_mode_contains_topk_and_is_upper_set(seed):
    """Top-k through the histogram (mass threshold 0): at least k clusters, all
    k best among them, and every cluster scoring above a selected one is
    selected; the smallest grid edge that keeps k clusters."""
    S, counts = _rows(seed)
    n = len(S)
    k = int(np.random.default_rng(seed).integers(1, n + 1))
    sel = ref.hist_select(S, counts, 0.125, k, 0.0)
    assert len(sel) >= k
    assert set(ref.topk(S[None], k)[0]) <= set(sel)
    assert (np.diff(sel) > 0).all()
    lowest = S[sel].min()
    assert set(np.nonzero(S > lowest)[0]) <= set(sel)
    g = ref.hist_grid_index(S)
    if g is not None and k < n:
        edge = g[sel].min()
        assert (g >= edge + 1).sum() < k  # one grid step higher keeps fewer than k


@pytest.mark.parametrize("seed", range(12))
def test_hist_mass_recall_reached_and_minimal(seed):
    """Adaptive selection: the estimated mass sum(count_b exp(tau S_b)) of the
    selection reaches the recall fraction of the total (in exact arithmetic,
    up to the 2^-32 rounding of each term), and one grid step higher it would
    not (unless the count floor binds)."""
    S, counts = _rows(seed)
    tau = 0.2
    m = counts * np.exp(tau * (S - S.max()))
    for recall in (0.5, 0.8, 0.95):
        sel = ref.hist_select(S, counts, tau, 1, recall)
        assert m[sel].sum() >= recall * m.sum() - len(S) * 2.0 ** -32
        g = ref.hist_grid_index(S)
        if g is None:
            continue
        edge = g[sel].min()
        higher = g >= edge + 1
        assert m[higher].sum() < recall * m.sum() + len(S) * 2.0 ** -32


def test_hist_degenerate_rows():
    """All scores equal: no range to bin, everything is selected; a single
    cluster is always selected; min_count above the row selects all."""
    assert np.array_equal(ref.hist_select(np.full(7, 2.5), np.ones(7), 0.1, 1, 0.0), np.arange(7))
    assert np.array_equal(ref.hist_select(np.array([3.0]), np.array([5]), 0.1, 1, 0.9), [0])
    S = np.array([1.0, 5.0, 2.0])
    assert np.array_equal(ref.hist_select(S, np.ones(3), 0.1, 9, 0.0), [0, 1, 2])
    assert np.array_equal(ref.hist_select(S, np.ones(3), 0.1, 1, 0.0), [1])


def test_hist_grid_index():
    """g runs from 0 at the lowest score to 16383 at the highest and does not
    decrease with the score; scores on the grid's steps land on their step
    (within one, for float32 rounding)."""
    rng = np.random.default_rng(3)
    S = rng.standard_normal(1000)
    g = ref.hist_grid_index(S)
    order = np.argsort(S, kind="stable")
    assert (np.diff(g[order]) >= 0).all()
    assert g[S.argmin()] == 0 and g[S.argmax()] == ref.HIST_GRID - 1
    lo, hi = -2.0, 6.0
    steps = np.arange(0, ref.HIST_GRID, 37)
    T = np.concatenate([[lo, hi], lo + steps * (hi - lo) / ref.HIST_GRID])
    gt = ref.hist_grid_index(T)
    assert np.abs(gt[2:] - steps).max() <= 1


def test_hist_forward_lists_vary_in_length():
    """forward(select="hist") feeds ragged lists through sparse attention and
    compensation; with recall 1 every cluster with a real key is kept and the
    result is dense attention."""
    rng = np.random.default_rng(5)
    Q, K, V = (rng.standard_normal((200, 8)) for _ in range(3))
    r = ref.forward(Q, K, V, 32, 32, 2, mode="metric", select="hist", mass_recall=0.5)
    lens = [len(x) for x in r["lists"]]
    assert min(lens) >= 2 and len(set(lens)) >= 1
    r1 = ref.forward(Q, K, V, 32, 32, 2, mode="metric", select="hist", mass_recall=1.0)
    o, _ = ref.dense_attention(Q, K, V, 1 / np.sqrt(8))
    assert np.abs(r1["out"] - o).max() < 1e-12
