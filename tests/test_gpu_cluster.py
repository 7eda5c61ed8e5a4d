"""GPU parity of ca_cluster.

* Raw-coordinate mode: the permutation is compared end to end with the
  oracle's split of the same inputs, bit for bit.
* PCA / metric modes: the split coordinates are exported; the permutation must
  equal the oracle's split of exactly those coordinates, and the coordinates
  themselves must satisfy the properties the paper gives for the split spaces
  (metric distances, unit-norm query representation, decorrelated and
  descending principal coordinates with non-negative means) to fp32 accuracy.
* Permuted copies, value tiles, counts, cluster ids and centroids are checked
  against the permutation.
"""
import numpy as np
import pytest

from oracle import ref
from synth import mixture_inputs

pytestmark = pytest.mark.gpu

SPLIT_CASES = [
    # dtype, n, d, c, transform
    ("f32", 1024, 64, 64, "none"),
    ("bf16", 1000, 64, 64, "none"),
    ("bf16", 5000, 32, 16, "none"),
    ("bf16", 20000, 64, 128, "none"),
    ("f32", 9000, 16, 32, "none"),
    ("bf16", 3001, 128, 64, "none"),
    ("f32", 1024, 64, 64, "pca"),
    ("bf16", 6000, 64, 128, "pca"),
    ("f32", 1024, 64, 64, "metric"),
    ("bf16", 20000, 64, 128, "metric"),
    ("bf16", 12345, 128, 64, "metric"),
    ("bf16", 100, 64, 128, "metric"),
    # d below the eigensolver's padded size (64 or 128)
    ("f32", 2000, 40, 32, "metric"),
    ("bf16", 4000, 100, 64, "pca"),
    # queries in the centred-key metric (adaptive assignment)
    ("bf16", 20000, 64, 128, "adaptive"),
    ("bf16", 6000, 128, 64, "adaptive"),
    ("f32", 1500, 48, 32, "adaptive"),
    # the random-cluster control
    ("bf16", 20000, 64, 128, "random"),
    ("f32", 3000, 32, 64, "random"),
]


def _run(dt, n, d, c, xf, seed=0, heads=2, layout="bhnd"):
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    Q, K, V = mixture_inputs(seed, heads, n, d, dt, centres=12, sigma=0.5)
    p = ca.Problem(1, heads, n, n, d, c, c, G.tdtype(dt), xf, layout)
    if layout == "bhnd":
        tq, tk, tv = (G.dev(x[None], G.tdtype(dt)) for x in (Q, K, V))
    else:
        tq, tk, tv = (G.dev(x[None].transpose(0, 2, 1, 3), G.tdtype(dt)) for x in (Q, K, V))
    r = ca.cluster(p, tq, tk, tv, export_y=True)
    torch.cuda.synchronize()
    return Q, K, V, p, {k: v.cpu() for k, v in r.items()}


def _check_copies(X, perm, cnt, cent, xp, c, dt):
    from tests import gpu_util as G
    n = X.shape[0]
    assert cnt.tolist() == G.counts(n, c).tolist()
    xp = xp.float().numpy()
    assert np.array_equal(xp[:n], X[perm].astype(np.float32))
    assert (xp[n:] == 0).all()
    want = ref.centroids(X, perm, cnt)
    assert np.abs(cent.numpy() - want).max() <= 1e-5 * max(1.0, np.abs(want).max())


@pytest.mark.parametrize("dt,n,d,c,xf", SPLIT_CASES)
def test_cluster_parity(dt, n, d, c, xf):
    from tests import gpu_util as G
    G.flush(f"cluster case dt={dt} n={n} d={d} c={c} xf={xf}")
    Q, K, V, p, r = _run(dt, n, d, c, xf)
    for h in range(Q.shape[0]):
        yq = r["yq"][h].numpy().astype(np.float64)
        yk = r["yk"][h].numpy().astype(np.float64)
        if xf == "none":
            assert np.array_equal(yq, Q[h]) and np.array_equal(yk, K[h])
        if xf == "random":  # the generator is exact on both sides
            assert np.array_equal(yq, ref.random_split_space(n, d, h, 0))
            assert np.array_equal(yk, ref.random_split_space(n, d, h, 1))
        pq, cidq, cntq = ref.split(yq, c)
        pk, cidk, cntk = ref.split(yk, c)
        assert np.array_equal(r["perm_q"][h].numpy(), pq), "query permutation"
        assert np.array_equal(r["perm_k"][h].numpy(), pk), "key permutation"
        assert np.array_equal(r["cid_q"][h].numpy(), cidq)
        assert np.array_equal(r["cid_k"][h].numpy(), cidk)
        _check_copies(Q[h], pq, r["count_q"][h], r["cent_q"][h], r["qp"][h], c, dt)
        _check_copies(K[h], pk, r["count_k"][h], r["cent_k"][h], r["kp"][h], c, dt)
        # value tiles follow the key permutation, transposed per cluster
        nkc = p.nkc
        rows = np.zeros((nkc * c, d))
        rows[:n] = V[h][pk]
        tiles = rows.reshape(nkc, c, d).transpose(0, 2, 1)
        assert np.array_equal(r["vp"][h].float().numpy(), tiles.astype(np.float32))
        wantv = ref.centroids(V[h], pk, cntk)
        assert np.abs(r["cent_v"][h].numpy() - wantv).max() <= 1e-5 * max(1, np.abs(wantv).max())
        if xf not in ("none", "random"):
            _check_split_space(Q[h], K[h], yq, yk, xf)


def _check_split_space(Q, K, yq, yk, xf):
    """Properties of the split coordinates that do not depend on the
    eigensolver's basis choice."""
    rtol = 2e-4
    for Y in (yq, yk):
        C = np.cov(Y.T, bias=True)
        scale = np.abs(C).max()
        off = C - np.diag(np.diag(C))
        assert np.abs(off).max() <= 5e-4 * scale, "decorrelated"
        dg = np.diag(C)
        assert (np.diff(dg) <= 1e-4 * scale).all(), "descending variances"
        assert (Y.mean(axis=0) >= -1e-4 * np.sqrt(scale)).all(), "oriented"
    rng = np.random.default_rng(0)
    pairs = rng.integers(0, len(K), size=(200, 2))
    if xf == "adaptive":
        for a, b in pairs:
            want = ((Q @ (K[a] - K[b])) ** 2).mean()
            got = ((yk[a] - yk[b]) ** 2).sum()
            assert abs(got - want) <= rtol * ((yk[a] ** 2).sum() + (yk[b] ** 2).sum()) + 1e-9
        # queries: |y_a - y_b|^2 = (q_a - q_b)^T C_K (q_a - q_b), C_K the key covariance
        C = ref.centred_cov(K)
        qpairs = rng.integers(0, len(Q), size=(200, 2))
        for a, b in qpairs:
            dq = Q[a] - Q[b]
            want = dq @ C @ dq
            got = ((yq[a] - yq[b]) ** 2).sum()
            assert abs(got - want) <= rtol * ((yq[a] ** 2).sum() + (yq[b] ** 2).sum()) + 1e-9
    elif xf == "metric":
        for a, b in pairs:
            want = ((Q @ (K[a] - K[b])) ** 2).mean()
            got = ((yk[a] - yk[b]) ** 2).sum()
            assert abs(got - want) <= rtol * ((yk[a] ** 2).sum() + (yk[b] ** 2).sum()) + 1e-9
        R = ref.query_representation(Q, K)
        assert np.abs((yq * yq).sum(axis=1) - (R * R).sum(axis=1)).max() <= 1e-4
        G1 = yq[pairs[:, 0]] * yq[pairs[:, 1]]
        G2 = R[pairs[:, 0]] * R[pairs[:, 1]]
        assert np.abs(G1.sum(axis=1) - G2.sum(axis=1)).max() <= 1e-4
    else:
        for X, Y in ((Q, yq), (K, yk)):
            for a, b in pairs:
                want = ((X[a] - X[b]) ** 2).sum()
                got = ((Y[a] - Y[b]) ** 2).sum()
                assert abs(got - want) <= rtol * ((X[a] ** 2).sum() + (X[b] ** 2).sum()) + 1e-9


def test_layout_bnhd_matches_bhnd():
    from tests import gpu_util as G
    Q, K, V, p, r1 = _run("bf16", 3000, 64, 64, "metric", layout="bhnd")
    _, _, _, _, r2 = _run("bf16", 3000, 64, 64, "metric", layout="bnhd")
    for key in ("perm_q", "perm_k", "qp", "kp", "vp", "cent_q", "cent_k", "yq", "yk"):
        assert np.array_equal(r1[key].float().numpy(), r2[key].float().numpy()), key


def test_cluster_deterministic():
    _, _, _, _, r1 = _run("bf16", 20000, 64, 128, "metric", seed=4)
    _, _, _, _, r2 = _run("bf16", 20000, 64, 128, "metric", seed=4)
    for key in r1:
        assert np.array_equal(r1[key].float().numpy(), r2[key].float().numpy()), key


def test_single_cluster_and_tiny():
    """n <= c: one cluster, identity order; n = 1."""
    for n in (1, 37, 64):
        Q, K, V, p, r = _run("f32", n, 16, 64, "pca", seed=n)
        for h in range(2):
            assert r["perm_q"][h].tolist() == list(range(n))
            assert r["count_k"][h].tolist() == [n]


BASIC_CASES = [
    # dtype, n, d, c, transform
    ("f32", 3000, 16, 64, "none"),
    ("bf16", 20000, 64, 128, "none"),
    ("bf16", 20000, 64, 128, "metric"),
    ("f32", 5000, 128, 64, "metric"),
    ("bf16", 9000, 32, 16, "none"),
    ("bf16", 700, 64, 64, "metric"),
    # nodes smaller than d (samples of m < d rows) at d = 64 and d = 128
    ("bf16", 3000, 64, 16, "metric"),
    ("bf16", 4000, 128, 32, "none"),
]


@pytest.mark.parametrize("dt,n,d,c,xf", BASIC_CASES)
def test_basic_split_parity(dt, n, d, c, xf):
    """Basic recursive splitting (power iteration per node): permutations
    bit-exact against the oracle's basic split of the exported split
    coordinates (the directions, projections and noise are reproduced bit for
    bit); permuted copies and centroids as for the diagonalized split; in the
    metric root space the key distances are the query-induced metric's and
    the query representations have unit norm."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"basic split case dt={dt} n={n} d={d} c={c} xf={xf}")
    heads = 2
    Q, K, V = mixture_inputs(41, heads, n, d, dt, centres=12, sigma=0.5)
    p = ca.Problem(1, heads, n, n, d, c, c, G.tdtype(dt), xf, "bhnd", split="basic")
    tq, tk, tv = (G.dev(x[None], G.tdtype(dt)) for x in (Q, K, V))
    r = ca.cluster(p, tq, tk, tv, export_y=True)
    torch.cuda.synchronize()
    r = {k: v.cpu() for k, v in r.items()}
    for h in range(heads):
        yq = r["yq"][h].numpy()
        yk = r["yk"][h].numpy()
        if xf == "none":
            assert np.array_equal(yq, Q[h].astype(np.float32))
        pq, cidq, _ = ref.basic_split(yq, c, head=h, side=0)
        pk, cidk, _ = ref.basic_split(yk, c, head=h, side=1)
        assert np.array_equal(r["perm_q"][h].numpy(), pq), "query permutation"
        assert np.array_equal(r["perm_k"][h].numpy(), pk), "key permutation"
        assert np.array_equal(r["cid_q"][h].numpy(), cidq)
        _check_copies(Q[h], pq, r["count_q"][h], r["cent_q"][h], r["qp"][h], c, dt)
        _check_copies(K[h], pk, r["count_k"][h], r["cent_k"][h], r["kp"][h], c, dt)
        if xf == "metric":
            yk64, yq64 = yk.astype(np.float64), yq.astype(np.float64)
            rng = np.random.default_rng(h)
            for a, b in rng.integers(0, n, size=(100, 2)):
                want = ((Q[h] @ (K[h][a] - K[h][b])) ** 2).mean()
                got = ((yk64[a] - yk64[b]) ** 2).sum()
                assert abs(got - want) <= 2e-4 * ((yk64[a] ** 2).sum() + (yk64[b] ** 2).sum()) + 1e-9
            nrm = np.sqrt((yq64 ** 2).sum(axis=1))
            assert np.abs(nrm[nrm > 0] - 1.0).max() < 1e-4


# Inputs whose multi-block split levels take the select pass's fallback
# paths. "duplicates": 60% of the queries and 70% of the keys are one repeated
# row, so at the root the wanted rank falls inside a run of more than 8192
# equal keys (a run of D equal values covers rank r whatever its position when
# D > max(r, s - r)); that linear bin overflows the select pass's candidate
# buffer and the threshold is found by streaming the node's keys from memory.
# "flat_root_sample": the root's subsample rows are all equal, so its spread
# is zero and every key lands in one bin (and streams). "all_identical": every
# node of every level is in that case, and the order is decided by the
# original index alone.
DEGENERATE = [
    # kind, n, transform, split
    ("duplicates", 40000, "none", "diag"),
    ("duplicates", 40000, "metric", "diag"),
    ("flat_root_sample", 40000, "none", "diag"),
    ("flat_root_sample", 40000, "metric", "diag"),
    ("all_identical", 33000, "none", "diag"),
    ("all_identical", 33000, "metric", "diag"),
    ("duplicates", 40000, "none", "basic"),
    ("flat_root_sample", 40000, "metric", "basic"),
    ("all_identical", 33000, "metric", "basic"),
]


def _degenerate_inputs(kind, n, d, seed):
    Q, K, V = mixture_inputs(seed, 1, n, d, "bf16", centres=12, sigma=0.5)
    rng = np.random.default_rng([seed, 1])
    for X, frac in ((Q[0], 0.6), (K[0], 0.7)):
        row = X[rng.integers(n)].copy()
        if kind == "duplicates":
            X[rng.choice(n, int(frac * n), replace=False)] = row
        elif kind == "flat_root_sample":
            X[ref.subsample_positions(n, min(d, n))] = row
        else:
            X[:] = row
    return Q, K, V


def _reaches_fallback(kind, Y, c):
    """The exported split coordinates really put the root on the fallback
    path: a long enough run of equal rows, or a subsample without spread."""
    n, d = Y.shape
    if kind == "flat_root_sample":
        sub = Y[ref.subsample_positions(n, min(d, n))]
        return bool((sub == sub[0]).all())
    _, dup = np.unique(Y, axis=0, return_counts=True)
    mL = ref.left_size(n, c)
    return dup.max() > max(8192, mL - 1, n - mL + 1)


@pytest.mark.parametrize("kind,n,xf,split", DEGENERATE)
def test_split_select_fallbacks(kind, n, xf, split):
    """Permutations bit-exact against the oracle's split of the exported
    coordinates on inputs with long runs of equal split keys and subsamples
    without spread (padding rows, repeated tokens), which take the select
    pass's streaming and one-bin paths; permuted copies, counts and centroids
    as in the other cluster tests."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    d, c = 64, 128
    G.flush(f"split fallback case kind={kind} n={n} xf={xf} split={split}")
    Q, K, V = _degenerate_inputs(kind, n, d, seed=n)
    p = ca.Problem(1, 1, n, n, d, c, c, torch.bfloat16, xf, "bhnd", split=split)
    tq, tk, tv = (G.dev(x[None], torch.bfloat16) for x in (Q, K, V))
    r = ca.cluster(p, tq, tk, tv, export_y=True)
    torch.cuda.synchronize()
    r = {key: val.cpu() for key, val in r.items()}
    yq = r["yq"][0].numpy().astype(np.float64)
    yk = r["yk"][0].numpy().astype(np.float64)
    for side, Y in (("query", yq), ("key", yk)):
        assert _reaches_fallback(kind, Y, c), f"{side} input does not reach the fallback path"
    if split == "basic":
        pq, cidq, _ = ref.basic_split(yq, c, head=0, side=0)
        pk, cidk, _ = ref.basic_split(yk, c, head=0, side=1)
    else:
        pq, cidq, _ = ref.split(yq, c)
        pk, cidk, _ = ref.split(yk, c)
    if kind == "all_identical" and split == "diag":
        assert np.array_equal(pq, np.arange(n)) and np.array_equal(pk, np.arange(n))
    assert np.array_equal(r["perm_q"][0].numpy(), pq), "query permutation"
    assert np.array_equal(r["perm_k"][0].numpy(), pk), "key permutation"
    assert np.array_equal(r["cid_q"][0].numpy(), cidq)
    assert np.array_equal(r["cid_k"][0].numpy(), cidk)
    _check_copies(Q[0], pq, r["count_q"][0], r["cent_q"][0], r["qp"][0], c, "bf16")
    _check_copies(K[0], pk, r["count_k"][0], r["cent_k"][0], r["kp"][0], c, "bf16")


@pytest.mark.parametrize("seed", [0, 3])
def test_split_column_copy_and_fallback(seed):
    """The multi-block keys pass reads a node's coordinate from the
    coordinate-major copy of the first 16 split coordinates, and from the
    row-major coordinates for any later one. Input chosen so that, on the
    exported coordinates, nodes above the tail size choose both kinds (checked
    on the oracle's trace of those coordinates); permutations bit-exact."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    n, d, c = 20000, 64, 128
    G.flush(f"column copy and fallback, seed={seed}")
    Q, K, V = mixture_inputs(seed, 1, n, d, "bf16", centres=2, sigma=1.0)
    p = ca.Problem(1, 1, n, n, d, c, c, torch.bfloat16, "metric")
    tq, tk, tv = (G.dev(x[None], torch.bfloat16) for x in (Q, K, V))
    r = ca.cluster(p, tq, tk, tv, export_y=True)
    torch.cuda.synchronize()
    chosen = []
    for side, key in ((0, "yq"), (1, "yk")):
        Y = r[key][0].double().cpu().numpy()
        trace = []
        perm, cid, _ = ref.split(Y, c, trace=trace)
        chosen += [j for (mem, j, _, _, _) in trace if len(mem) > 2048]
        got = r["perm_q" if side == 0 else "perm_k"][0].cpu().numpy()
        assert np.array_equal(got, perm), f"side {side} permutation"
    assert min(chosen) < 16 <= max(chosen), f"multi-block choices {chosen}"
