"""ClusterAttention oracle: a plain, slow, fp64 CPU implementation of the method.

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports this module; only
the tests, the smoke check and the bench's CPU-baseline leg may call it. It
shares no code with the HIP library.

Every function works on one attention head (2-D arrays, rows = tokens) in fp64
and cites the passage of the paper it follows. Where the paper leaves a choice
open, the reading taken is stated in the docstring. Inputs are the exact
values the GPU receives (float32 or bf16-representable), upcast to fp64.

Pins: see tests/test_oracle_*.py. Parts with no independent pin are marked
"parity unpinned" below (none at present).
"""
from __future__ import annotations

import numpy as np

F64 = np.float64

# ---------------------------------------------------------------------------
# Dense attention (Preliminaries: error in sparse attention, o = sum_i w_i v_i)
# ---------------------------------------------------------------------------


def dense_attention(Q, K, V, tau):
    """o_i = sum_j softmax_j(tau q_i.k_j) v_j, and lse_i = log sum_j exp(tau q_i.k_j).

    Preliminaries (error in sparse attention): the output of a query is the
    attention-weighted sum of all values.
    """
    Q, K, V = (np.asarray(x, F64) for x in (Q, K, V))
    S = tau * (Q @ K.T)
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    l = E.sum(axis=1, keepdims=True)
    return (E @ V) / l, (m + np.log(l))[:, 0]


# ---------------------------------------------------------------------------
# Moments, eigendecompositions and the split spaces (Method: Transforms;
# Method: Diagonalized recursive splitting; App. B.2)
# ---------------------------------------------------------------------------


def second_moment(X):
    """M = X^T X / n (Method, key clustering: the metric matrix Q^T Q / n)."""
    X = np.asarray(X, F64)
    return X.T @ X / X.shape[0]


def centred_cov(X):
    """X_c^T X_c / n with X_c the column-centred matrix (Method, query clustering;
    App. B: the covariance of the keys)."""
    X = np.asarray(X, F64)
    Xc = X - X.mean(axis=0)
    return Xc.T @ Xc / X.shape[0]


def eigh_desc(A):
    """Eigenpairs of a symmetric matrix, eigenvalues in descending order."""
    lam, U = np.linalg.eigh(np.asarray(A, F64))
    order = np.argsort(-lam, kind="stable")
    return lam[order], U[:, order]


def psd_root(A):
    """Root factor S = E diag(sqrt(max(lambda, 0))) of a PSD matrix, so that
    S S^T = A with negative eigenvalues clamped to zero (Method, key clustering:
    small negative eigenvalues are clamped to 0; x^T A y = (x S).(y S))."""
    lam, E = eigh_desc(A)
    return E * np.sqrt(np.maximum(lam, 0.0))[None, :]


def orient(U, mean_row):
    """Flip each column u_j of U so that mean_row . u_j >= 0 (the mean of the
    projected coordinate is non-negative; exactly 0 keeps the sign). The paper
    does not fix eigenvector signs; this reading makes the split coordinates
    independent of the eigensolver's arbitrary sign choice."""
    s = np.asarray(mean_row, F64) @ U
    return U * np.where(s < 0.0, -1.0, 1.0)[None, :]


def pca_basis(X):
    """Principal axes of X: eigenvectors of the centred covariance, descending,
    oriented by the data mean (Method: diagonalized recursive splitting
    projects the data onto its principal components)."""
    X = np.asarray(X, F64)
    _, U = eigh_desc(centred_cov(X))
    return orient(U, X.mean(axis=0))


SPLITMIX_GAMMA = 0x9E3779B97F4A7C15


def splitmix64(c):
    """Output number c (counting from 0) of splitmix64 started at state 0, the
    generator published by S. Vigna: the state after c + 1 increments by the
    golden-ratio constant, passed through the published mixing function.
    Vectorised over uint64 arrays (arithmetic modulo 2^64)."""
    z = (np.asarray(c, dtype=np.uint64) + np.uint64(1)) * np.uint64(SPLITMIX_GAMMA)
    z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def random_split_space(n, d, head, side):
    """Split coordinates of the random-cluster control (Experiments:
    baselines, random clusters with top-k routing through centroid scores):
    y[i][j] = (top 24 bits of splitmix64 output c) / 2^24, c = (((2 head +
    side) << 22 | i) << 7) | j, side 0 for queries and 1 for keys. Splitting
    on these coordinates partitions the tokens into clusters at random.
    Reading: the paper does not say how its random assignment is drawn; a
    counter-based generator makes it reproducible on both sides."""
    i = np.arange(n, dtype=np.uint64)[:, None]
    j = np.arange(d, dtype=np.uint64)[None, :]
    c = (((np.uint64(2 * head + side) << np.uint64(22)) | i) << np.uint64(7)) | j
    return (splitmix64(c) >> np.uint64(40)).astype(F64) * 2.0 ** -24


def key_split_space(Q, K, mode, head=0):
    """Split coordinates Y_K of the keys.

    none:     Y_K = K.
    pca:      Y_K = K U, U the principal axes of K.
    metric:   keys are mapped into the query-aware metric M = Q^T Q / n (Method,
              key clustering): K -> K S_q with S_q S_q^T = M, then projected on
              the principal axes of K S_q (diagonalized splitting). The
              principal axes of K S_q are the eigenvectors of S_q^T C_K S_q.
    adaptive: as metric (the key side does not depend on the selection mode).
    random:   pseudo-random coordinates (random_split_space, side 1).
    metric_root: K S_q without the principal axes (basic splitting finds its
              own directions: "the metric injected", no eigendecomposition).
    """
    Q, K = np.asarray(Q, F64), np.asarray(K, F64)
    if mode == "none":
        return K.copy()
    if mode == "random":
        return random_split_space(K.shape[0], K.shape[1], head, 1)
    if mode == "pca":
        return K @ pca_basis(K)
    if mode == "metric_root":
        return K @ psd_root(second_moment(Q))
    if mode in ("metric", "adaptive"):
        S_q = psd_root(second_moment(Q))
        Z = K @ S_q
        return Z @ pca_basis(Z)
    raise ValueError(mode)


def query_representation(Q, K):
    """r(q) = q S_k / |q S_k| with S_k S_k^T = K_c^T K_c / n (Method, query
    clustering for top-k selection; App. B.2). A query with |q S_k| = 0 maps
    to r = 0 (the paper leaves this case open)."""
    Q, K = np.asarray(Q, F64), np.asarray(K, F64)
    S_k = psd_root(centred_cov(K))
    rho = Q @ S_k
    nrm = np.sqrt((rho * rho).sum(axis=1))
    safe = np.where(nrm > 0.0, nrm, 1.0)
    return np.where(nrm[:, None] > 0.0, rho / safe[:, None], 0.0)


def query_representation_adaptive(Q, K):
    """r(q) = q S_k with S_k S_k^T = K_c^T K_c / n, not normalised (Method,
    query clustering, the adaptive-assignment case; App. B.1: the
    representation K_c q / sqrt(n), whose distances are those of the metric
    K_c^T K_c / n; the root factor gives the same distances in d coordinates).
    Queries with the same attention distribution over the keys map to the
    same point: K_c removes the shift invariance of the softmax."""
    Q, K = np.asarray(Q, F64), np.asarray(K, F64)
    return Q @ psd_root(centred_cov(K))


def query_split_space(Q, K, mode, head=0):
    """Split coordinates Y_Q of the queries: none -> Q; pca -> Q on its principal
    axes; metric -> r(q) (top-k representation) on its principal axes;
    adaptive -> the unnormalised centred-key representation on its principal
    axes; random -> pseudo-random coordinates (side 0)."""
    Q = np.asarray(Q, F64)
    if mode == "none":
        return Q.copy()
    if mode == "random":
        return random_split_space(Q.shape[0], Q.shape[1], head, 0)
    if mode == "pca":
        return Q @ pca_basis(Q)
    if mode == "metric":
        R = query_representation(Q, K)
        return R @ pca_basis(R)
    if mode == "metric_root":
        return query_representation(Q, K)
    if mode == "adaptive":
        R = query_representation_adaptive(Q, K)
        return R @ pca_basis(R)
    raise ValueError(mode)


# ---------------------------------------------------------------------------
# Diagonalized recursive splitting (Method: recursive splitting; App. D.2)
# ---------------------------------------------------------------------------


def subsample_positions(s, m):
    """Positions of the m-point subsample inside a node of s members (in the
    node's order): p_j = floor((2j + 1) s / (2m)). The paper samples
    min(a d, |S|) points with a = 1 but gives no sampling rule; this evenly
    strided, deterministic rule is the reading taken. For m = s it is every
    member."""
    return [((2 * j + 1) * s) // (2 * m) for j in range(m)]


def sequential_variance(rows):
    """Population variance of each column of ``rows`` (m x d), fp64, two passes,
    rows summed strictly in order, no fused multiply-add: the mean first, then
    the mean of squared deviations. (The paper asks for the highest-variance
    coordinate without fixing an estimator; this exact order is the reading.)"""
    rows = np.asarray(rows, F64)
    m = rows.shape[0]
    acc = np.zeros(rows.shape[1], F64)
    for j in range(m):
        acc = acc + rows[j]
    mean = acc / F64(m)
    acc = np.zeros(rows.shape[1], F64)
    for j in range(m):
        dev = rows[j] - mean
        acc = acc + dev * dev
    return acc / F64(m)


def left_size(s, c):
    """Members sent left when splitting s points with cluster size c: the
    multiple of c closest to half of s, taking the smaller one on a tie, i.e.
    c * floor(ceil(s / c) / 2) (Method: basic recursive splitting)."""
    return c * ((-(-s // c)) // 2)


def split(Y, c, trace=None):
    """Diagonalized recursive splitting of the rows of Y into clusters of size c.

    Method: recursive splitting (basic: split so the part below the threshold
    is the multiple of c closest to half; diagonalized: at each split pick the
    global principal coordinate of highest variance on a subsample of min(d, s)
    points). A node of s <= c points is a leaf. Otherwise:

      1. subsample m = min(d, s) members at ``subsample_positions``;
      2. j* = argmax of ``sequential_variance`` (ties -> lowest coordinate);
      3. the left child gets the ``left_size(s, c)`` members with the smallest
         (Y[i, j*], i) pairs (-0.0 counts as +0.0; equal values go by original
         index), the right child the rest; both keep ascending index order;
      4. recurse on the left child, then on the right child.

    Returns (perm, cid, counts): perm lists the original token indices cluster
    by cluster (leaves left to right, ascending index inside a leaf); cid[i] is
    the cluster of token i; counts[a] the size of cluster a. If ``trace`` is a
    list, one (members, j_star, m_left, left, right) tuple per split is
    appended.
    """
    Y = np.asarray(Y, F64)
    n, d = Y.shape
    if c < 1:
        raise ValueError("cluster size must be positive")
    leaves = []

    def rec(members):
        s = len(members)
        if s <= c:
            leaves.append(members)
            return
        m = min(d, s)
        sub = Y[members[subsample_positions(s, m)]]
        jstar = int(np.argmax(sequential_variance(sub)))
        mL = left_size(s, c)
        vals = Y[members, jstar] + 0.0  # -0.0 -> +0.0
        order = np.argsort(vals, kind="stable")  # members are in ascending index order
        left = np.sort(members[order[:mL]])
        right = np.sort(members[order[mL:]])
        if trace is not None:
            trace.append((members, jstar, mL, left, right))
        rec(left)
        rec(right)

    rec(np.arange(n, dtype=np.int64))
    perm = np.concatenate(leaves)
    counts = np.array([len(x) for x in leaves], dtype=np.int64)
    cid = np.empty(n, dtype=np.int64)
    for a, x in enumerate(leaves):
        cid[x] = a
    return perm, cid, counts


# ---------------------------------------------------------------------------
# Basic recursive splitting (Method: recursive splitting, basic: a PDDP
# variant with power iteration)
# ---------------------------------------------------------------------------

BASIC_POWER_ITERS = 8


def irwin_hall_normal(counters):
    """Approximately standard normal values, one per counter: the sum of 12
    uniforms on [0, 1) minus 6 (the Irwin-Hall approximation of N(0, 1)),
    uniform u of counter c being the top 24 bits of splitmix64 output
    16 c + u. The 24-bit integers are summed exactly, scaled in fp64 and
    rounded once to fp32, so the values are reproducible bit for bit."""
    c = np.asarray(counters, dtype=np.uint64)[..., None] * np.uint64(16) + \
        np.arange(12, dtype=np.uint64)
    u = (splitmix64(c) >> np.uint64(40)).astype(np.int64).sum(axis=-1)
    return (u.astype(F64) * 2.0 ** -24 - 6.0).astype(np.float32)


def basic_noise(d, head, side, level, node):
    """Warm-start noise of the split at slot `node` of tree level `level`
    (the slot numbering of the split tree: a node's children are 2 node and
    2 node + 1 one level down): irwin_hall_normal at counters
    ((((2 head + side) << 5 | level) << 20 | node) << 7) | k, k < d."""
    base = ((((np.uint64(2 * head + side) << np.uint64(5)) | np.uint64(level))
             << np.uint64(20) | np.uint64(node)) << np.uint64(7))
    return irwin_hall_normal(base | np.arange(d, dtype=np.uint64))


def f32_dot_rows(X, v):
    """X v row by row in fp32, summed over the coordinates in order (a
    rounded product and a rounded sum per step, no fused multiply-add)."""
    X = np.asarray(X, np.float32)
    v = np.asarray(v, np.float32)
    acc = np.zeros(X.shape[0], np.float32)
    for k in range(X.shape[1]):
        acc = (acc + X[:, k] * v[k]).astype(np.float32)
    return acc


def power_direction(sub, v0, iters=BASIC_POWER_ITERS):
    """First principal direction of the subsample rows (m x d) by power
    iteration on their centred covariance, started at v0 (Method: basic
    recursive splitting: the first principal component of the subset is
    estimated with power iteration). fp32 in a fixed order: the mean (rows
    summed in order, divided by m), centred rows, then per iteration
    t_j = (x_j - mu) . v (f32_dot_rows), w = sum_j t_j (x_j - mu) (rows in
    order), v = w / sqrt(|w|^2) (|w|^2 summed in order; a zero w keeps v).
    The 1/m of the covariance cancels in the normalisation. Reading: the
    paper does not give the number of iterations; BASIC_POWER_ITERS."""
    sub = np.asarray(sub, np.float32)
    m, d = sub.shape
    mu = np.zeros(d, np.float32)
    for j in range(m):
        mu = (mu + sub[j]).astype(np.float32)
    mu = (mu / np.float32(m)).astype(np.float32)
    D = (sub - mu).astype(np.float32)
    v = np.asarray(v0, np.float32).copy()
    for _ in range(iters):
        t = f32_dot_rows(D, v)
        w = np.zeros(d, np.float32)
        for j in range(m):
            w = (w + t[j] * D[j]).astype(np.float32)
        nn = np.float32(0.0)
        for k in range(d):
            nn = np.float32(nn + np.float32(w[k] * w[k]))
        if nn > 0:
            v = (w / np.sqrt(nn)).astype(np.float32)
    return v


def warm_start(v_parent, noise):
    """Start of a node's power iteration (Method: basic recursive splitting):
    the mean of the parent's estimate and a random normal vector rescaled to
    the parent estimate's norm, in fp32: v0 = (v_p + r * (|v_p| / |r|)) / 2
    (squared norms summed in order). The root starts from the noise alone."""
    if v_parent is None:
        return np.asarray(noise, np.float32)
    vp = np.asarray(v_parent, np.float32)
    r = np.asarray(noise, np.float32)
    nv = np.float32(0.0)
    nr = np.float32(0.0)
    for k in range(len(vp)):
        nv = np.float32(nv + np.float32(vp[k] * vp[k]))
        nr = np.float32(nr + np.float32(r[k] * r[k]))
    sc = np.float32(np.sqrt(nv) / np.sqrt(nr))
    return ((vp + (r * sc).astype(np.float32)).astype(np.float32) * np.float32(0.5)).astype(
        np.float32)


def basic_split(Y, c, head=0, side=0, iters=BASIC_POWER_ITERS, trace=None):
    """Basic recursive splitting of the rows of Y into clusters of size c
    (Method: recursive splitting, basic; a variation of principal direction
    divisive partitioning). A node of s <= c points is a leaf. Otherwise:

      1. subsample m = min(d, s) members at ``subsample_positions``;
      2. v = ``power_direction`` of the subsample from ``warm_start`` (the
         parent's direction and ``basic_noise`` of this node);
      3. project every member on v (``f32_dot_rows``) and send the
         ``left_size(s, c)`` smallest (projection, original index) pairs left
         (-0.0 counts as +0.0), the rest right, both in ascending index order;
      4. recurse on the children, passing v down.

    Y is used in fp32 (the split coordinates the GPU works on). Returns
    (perm, cid, counts) as ``split``; ``trace`` collects (members, v, left,
    right) per split."""
    Y32 = np.asarray(Y, np.float32)
    n, d = Y32.shape
    leaves = []

    def rec(members, level, node, v_parent):
        s = len(members)
        if s <= c:
            leaves.append(members)
            return
        m = min(d, s)
        sub = Y32[members[subsample_positions(s, m)]]
        v0 = warm_start(v_parent, basic_noise(d, head, side, level, node))
        v = power_direction(sub, v0, iters)
        keys = f32_dot_rows(Y32[members], v).astype(F64) + 0.0
        mL = left_size(s, c)
        order = np.argsort(keys, kind="stable")
        left = np.sort(members[order[:mL]])
        right = np.sort(members[order[mL:]])
        if trace is not None:
            trace.append((members, v, left, right))
        rec(left, level + 1, 2 * node, v)
        rec(right, level + 1, 2 * node + 1, v)

    rec(np.arange(n, dtype=np.int64), 0, 0, None)
    perm = np.concatenate(leaves)
    counts = np.array([len(x) for x in leaves], dtype=np.int64)
    cid = np.empty(n, dtype=np.int64)
    for a, x in enumerate(leaves):
        cid[x] = a
    return perm, cid, counts


# ---------------------------------------------------------------------------
# Centroids, scoring, selection (Method: cluster assignment)
# ---------------------------------------------------------------------------


def cluster_members(perm, counts):
    starts = np.concatenate([[0], np.cumsum(counts)[:-1]])
    return [perm[s:s + n] for s, n in zip(starts, counts)]


def centroids(X, perm, counts):
    """Mean of the original (untransformed) vectors of each cluster's real
    members (Method, scoring: centroid of a cluster; App. A: centroid keys and
    values)."""
    X = np.asarray(X, F64)
    return np.stack([X[mem].mean(axis=0) for mem in cluster_members(perm, counts)])


def centroid_scores(qbar, kbar):
    """score(a, b) = qbar_a . kbar_b, the average logit between the two clusters
    (Method: scoring). The 1/sqrt(d) factor does not change the ranking and is
    left out."""
    return np.asarray(qbar, F64) @ np.asarray(kbar, F64).T


def topk(S, k):
    """For each query cluster, the k key clusters with the largest score (ties
    to the lower index), listed in ascending order (Method: selection, top-k)."""
    S = np.asarray(S, F64)
    out = np.empty((S.shape[0], k), dtype=np.int64)
    for a in range(S.shape[0]):
        order = np.argsort(-S[a], kind="stable")
        out[a] = np.sort(order[:k])
    return out


HIST_BINS = 128            # bins of each of the two histogram passes
HIST_GRID = HIST_BINS * HIST_BINS
MASS_ONE = float(2 ** 32)  # fixed-point unit of the estimated attention mass


def hist_grid_index(S_row):
    """Grid position of every score of one query cluster's row (Method:
    selection, the 128-bin histogram from the lowest to the highest
    cluster-interaction score, refined by 128 bins inside one bin).

    Reading: the refinement splits a bin into 128 equal parts, so the two
    passes work on one grid of 128 x 128 steps over [lo, hi]; g =
    floor((S - lo) * (16384 / (hi - lo))) in float32 arithmetic (the kernel's
    precision, so that both sides bin identically), clamped to 16383; the
    coarse bin is g // 128 and the fine bin g % 128. Returns None when every
    score is equal (no range to bin: everything is selected)."""
    S32 = np.asarray(S_row, dtype=np.float32)
    lo, hi = S32.min(), S32.max()
    if not hi > lo:
        return None
    inv = np.float32(HIST_GRID) / np.float32(hi - lo)
    g = np.floor((S32 - lo) * inv).astype(np.int64)
    return np.clip(g, 0, HIST_GRID - 1)


def hist_mass_units(S_row, counts_k, tau):
    """Estimated attention mass of each key cluster for the query cluster,
    count_b * exp(tau * (S_b - max S)), in integer units of 2^-32 (Method:
    scoring and selection: the unnormalised attention score of the centroid
    pair, weighted by the cluster size, is the estimate of the mass the
    cluster receives; by Jensen's inequality it underestimates the true mass).
    Reading: the fixed point makes the running sums exact and independent of
    summation order; the common factor exp(tau * max S) cancels in the
    recall fraction."""
    S = np.asarray(S_row, F64)
    m = np.asarray(counts_k, F64) * np.exp(tau * (S - S.max()))
    return np.floor(m * MASS_ONE + 0.5).astype(np.int64)


def hist_select(S_row, counts_k, tau, min_count, mass_recall):
    """Key clusters selected for one query cluster by the two-pass histogram
    (Method: selection): thresholds on the number of selected clusters
    (min_count) and on the fraction of the estimated attention mass
    (mass_recall); the coarse bin in which the first of them to need it is
    passed (scanning from the highest scores down) is refined by a second
    histogram, and every cluster at or above the lower edge of the refinement
    bin where both thresholds hold is selected. Top-k assignment is
    mass_recall = 0 (returns at least k clusters, the ties inside the edge's
    bin included); adaptive assignment uses min_count = 16.

    Reading: the count threshold counts clusters (so that top-k's k is the
    same k as in exact top-k); the mass threshold is ceil(mass_recall *
    total) in the fixed-point units of hist_mass_units, at most the total.
    Returns the selected indices in ascending order."""
    S_row = np.asarray(S_row)
    n = S_row.shape[0]
    g = hist_grid_index(S_row)
    if g is None or min_count >= n:
        return np.arange(n)
    mass = hist_mass_units(S_row, counts_k, tau)
    total = int(mass.sum())
    # never above the total (the product is rounded in fp64 for large totals)
    need_mass = min(int(np.ceil(float(mass_recall) * float(total))), total)
    coarse, fine = g // HIST_BINS, g % HIST_BINS

    def crossing(cnt, ms, cnt_above, mass_above):
        # highest bin whose lower edge already holds both thresholds
        c, m = cnt_above, mass_above
        for b in range(HIST_BINS - 1, -1, -1):
            c += cnt[b]
            m += ms[b]
            if c >= min_count and m >= need_mass:
                return b
        return 0

    # pass 1: coarse histogram of counts and masses
    cnt1 = np.bincount(coarse, minlength=HIST_BINS)
    ms1 = np.bincount(coarse, weights=mass, minlength=HIST_BINS).astype(np.int64)
    B = crossing(cnt1, ms1, 0, 0)
    # pass 2: the refinement inside coarse bin B
    inside = coarse == B
    above = coarse > B
    cnt2 = np.bincount(fine[inside], minlength=HIST_BINS)
    ms2 = np.zeros(HIST_BINS, dtype=np.int64)
    np.add.at(ms2, fine[inside], mass[inside])
    j = crossing(cnt2, ms2, int(above.sum()), int(mass[above].sum()))
    return np.nonzero(g >= B * HIST_BINS + j)[0]


# ---------------------------------------------------------------------------
# Block-sparse attention and striped mean-compensation (Method: overview;
# Preliminaries: error in sparse attention; App. A)
# ---------------------------------------------------------------------------


def sparse_attention(Q, K, V, perm_q, counts_q, perm_k, counts_k, lists, tau):
    """o_S and lse_S for every query: softmax attention restricted to the real
    keys of the selected key clusters of the query's cluster (Method: overview,
    the attention step returns the output and the softmax denominator).
    Returned in original query order."""
    Q, K, V = (np.asarray(x, F64) for x in (Q, K, V))
    qmem = cluster_members(perm_q, counts_q)
    kmem = cluster_members(perm_k, counts_k)
    o = np.zeros_like(Q)
    lse = np.zeros(Q.shape[0])
    for a, rows in enumerate(qmem):
        keys = np.concatenate([kmem[b] for b in lists[a]])
        o[rows], lse[rows] = dense_attention(Q[rows], K[keys], V[keys], tau)
    return o, lse


def compensate(Q, kbar, vbar, counts_k, perm_q, counts_q, lists, o_s, lse_s, tau, enable=True):
    """Striped mean-compensation (Preliminaries: error in sparse attention; App. A).

    Each key cluster b not selected for the query's cluster enters the
    query's softmax through its centroid key and value, weighted by its size:
    logit tau q.kbar_b + ln|b|, value vbar_b. Merged with the sparse part in
    log-sum-exp form this equals
        (sum_{i in S} w_i v_i + sum_b |b| w_b vbar_b) / (w_S + sum_b |b| w_b).
    With compensation off, or all clusters selected, the output is o_S.
    """
    Q = np.asarray(Q, F64)
    kbar, vbar = np.asarray(kbar, F64), np.asarray(vbar, F64)
    out = np.array(o_s, F64, copy=True)
    lse = np.array(lse_s, F64, copy=True)
    if not enable:
        return out, lse
    n_kc = kbar.shape[0]
    logc = np.log(np.asarray(counts_k, F64))
    for a, rows in enumerate(cluster_members(perm_q, counts_q)):
        excl = np.setdiff1d(np.arange(n_kc), lists[a])
        if excl.size == 0:
            continue
        t = tau * (Q[rows] @ kbar[excl].T) + logc[excl][None, :]
        m = t.max(axis=1, keepdims=True)
        e = np.exp(t - m)
        l = e.sum(axis=1, keepdims=True)
        o_c = (e @ vbar[excl]) / l
        lse_c = (m + np.log(l))[:, 0]
        both = np.logaddexp(lse[rows], lse_c)
        out[rows] = (np.exp(lse[rows] - both)[:, None] * out[rows]
                     + np.exp(lse_c - both)[:, None] * o_c)
        lse[rows] = both
    return out, lse


# ---------------------------------------------------------------------------
# The whole forward pass of one head
# ---------------------------------------------------------------------------


def forward(Q, K, V, cq, ck, k, mode="metric", enable_comp=True, tau=None,
            perm_q=None, perm_k=None, lists=None, scores=None, select="topk",
            mass_recall=0.0, head=0):
    """ClusterAttention for one head: clustering -> centroids -> scores ->
    selection -> block-sparse attention -> compensation (Method: overview).

    select="topk": exact top-k; select="hist": the two-pass histogram with
    min_count = k and the given mass_recall (lists then have varying length).
    perm_q / perm_k / scores / lists may be supplied from outside (parity hooks:
    the checker then follows the given permutation or ranking instead of its
    own). Returns a dict with every intermediate; ``out`` and ``lse`` are in
    original query order.
    """
    Q, K, V = (np.asarray(x, F64) for x in (Q, K, V))
    d = Q.shape[1]
    tau = 1.0 / np.sqrt(d) if tau is None else tau
    r = {}
    if perm_q is None:
        r["yq"] = query_split_space(Q, K, mode, head)
        perm_q, _, _ = split(r["yq"], cq)
    if perm_k is None:
        r["yk"] = key_split_space(Q, K, mode, head)
        perm_k, _, _ = split(r["yk"], ck)
    nq, nk = Q.shape[0], K.shape[0]
    counts_q = np.array([min(cq, nq - a * cq) for a in range(-(-nq // cq))])
    counts_k = np.array([min(ck, nk - b * ck) for b in range(-(-nk // ck))])
    r.update(perm_q=np.asarray(perm_q), perm_k=np.asarray(perm_k),
             counts_q=counts_q, counts_k=counts_k)
    r["qbar"] = centroids(Q, perm_q, counts_q)
    r["kbar"] = centroids(K, perm_k, counts_k)
    r["vbar"] = centroids(V, perm_k, counts_k)
    r["scores"] = centroid_scores(r["qbar"], r["kbar"]) if scores is None else np.asarray(scores, F64)
    if lists is not None:
        r["lists"] = lists
    elif select == "topk":
        r["lists"] = topk(r["scores"], k)
    elif select == "hist":
        r["lists"] = [hist_select(row, counts_k, tau, k, mass_recall) for row in r["scores"]]
    else:
        raise ValueError(select)
    o_s, lse_s = sparse_attention(Q, K, V, perm_q, counts_q, perm_k, counts_k, r["lists"], tau)
    r["o_s"], r["lse_s"] = o_s, lse_s
    r["out"], r["lse"] = compensate(Q, r["kbar"], r["vbar"], counts_k, perm_q, counts_q,
                                    r["lists"], o_s, lse_s, tau, enable_comp)
    return r
