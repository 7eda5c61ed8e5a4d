"""GPU parity of the attention calls against the oracle, through the C ABI.

Inputs are seeded synthetic mixtures; permutations and selection lists are
drawn at random so that the attention kernels are checked on their own
(independently of the clustering). Sizes span several tiles and a ragged last
cluster."""
import math

import numpy as np
import pytest

from oracle import ref
from synth import mixture_inputs

pytestmark = pytest.mark.gpu

CASES = [
    # dtype, d, cq, ck, n, k
    ("bf16", 64, 128, 128, 1000, 3),
    ("bf16", 64, 64, 64, 700, 5),
    ("bf16", 128, 64, 64, 650, 4),
    ("bf16", 128, 128, 128, 1111, 2),
    ("bf16", 64, 128, 64, 900, 6),
    ("bf16", 128, 64, 128, 777, 7),
    # query clusters of 64 with lists long enough for the two-wavefront kernel
    # (their selected tiles exceed 4 MiB)
    ("bf16", 128, 64, 64, 9000, 130),
    ("bf16", 64, 64, 128, 33000, 130),
    ("f32", 64, 64, 64, 1000, 4),
    ("f32", 32, 32, 16, 333, 5),
    ("f32", 128, 16, 64, 300, 2),
    # fp32 query clusters of 128 and 256: two and one key parts per query
    ("f32", 64, 128, 64, 700, 3),
    ("f32", 32, 256, 32, 600, 4),
]


def _setup(dt, d, cq, ck, n, k, seed=0, heads=2):
    from tests import gpu_util as G
    Q, K, V = mixture_inputs(seed, heads, n, d, dt, centres=8, sigma=0.4)
    rng = np.random.default_rng(seed + 1)
    perm_q = np.stack([rng.permutation(n) for _ in range(heads)]).astype(np.int32)
    perm_k = np.stack([rng.permutation(n) for _ in range(heads)]).astype(np.int32)
    nqc, nkc = -(-n // cq), -(-n // ck)
    k = min(k, nkc)
    lists = G.random_lists(rng, heads, nqc, nkc, k)
    return Q, K, V, perm_q, perm_k, lists, k


@pytest.mark.parametrize("dt,d,cq,ck,n,k", CASES)
def test_block_sparse_attention_parity(dt, d, cq, ck, n, k):
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"attn case dt={dt} d={d} cq={cq} ck={ck} n={n} k={k}")
    Q, K, V, perm_q, perm_k, lists, k = _setup(dt, d, cq, ck, n, k)
    H = Q.shape[0]
    p = ca.Problem(1, H, n, n, d, cq, ck, G.tdtype(dt))
    tq = G.permuted_rows(Q, perm_q, cq, G.tdtype(dt))
    tk = G.permuted_rows(K, perm_k, ck, G.tdtype(dt))
    tv = G.value_tiles(V, perm_k, ck, G.tdtype(dt))
    cnt = G.dev(np.stack([G.counts(n, ck)] * H), torch.int32)
    op, lse = ca.block_sparse_attn(p, tq, tk, tv, cnt, G.dev(lists, torch.int32), k)
    torch.cuda.synchronize()
    op, lse = G.host(op), G.host(lse)
    tau = 1 / math.sqrt(d)
    worst = 0.0
    for h in range(H):
        o, l = ref.sparse_attention(Q[h], K[h], V[h], perm_q[h], G.counts(n, cq), perm_k[h],
                                    G.counts(n, ck), lists[h], tau)
        got = op[h, :n]
        want = o[perm_q[h]]
        err = np.abs(got - want).max()
        worst = max(worst, err)
        assert err <= G.TOL[dt], (h, err)
        lerr = np.abs(lse[h, :n] - l[perm_q[h]]).max()
        assert lerr <= (1e-5 if dt == "f32" else 1e-3) * max(1.0, np.abs(l).max()), lerr
    G.flush(f"  max abs err {worst:.3g}")


JUMP = [
    # d, cq, ck, n, k
    (64, 128, 128, 1000, 3),
    (128, 64, 64, 650, 4),
    (64, 64, 128, 900, 3),
    (128, 128, 128, 1111, 2),
]


@pytest.mark.parametrize("d,cq,ck,n,k", JUMP)
def test_logit_jump_after_first_stage(d, cq, ck, n, k):
    """bf16 attention where some logits exceed the first stage's maximum by
    far more than the exponent range: every query has 3 on axis 0 and the
    keys of the last key cluster 400 there, so that cluster's logits lie
    about 2^7.2 to 2^7.6 (log2 units) above the others'. Every list holds that
    cluster and never first (lists are in ascending order), so exponentials
    taken against the first stage's maximum overflow and the kernel has to
    settle stage by stage instead. The lse carries the rounding of the
    pre-scaled queries (bf16, unit roundoff 2^-8), at most 2^-8 of
    tau sum |q_i k_i| (a common shift of the large logits that the outputs do
    not see)."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    from synth import bf16_round
    G.flush(f"logit jump case d={d} cq={cq} ck={ck} n={n} k={k}")
    Q, K, V, perm_q, perm_k, lists, k = _setup("bf16", d, cq, ck, n, k, seed=11)
    H = Q.shape[0]
    nkc = -(-n // ck)
    Q[:, :, 0] = 3.0
    for h in range(H):
        K[h, perm_k[h][(nkc - 1) * ck:], 0] = 400.0
        for a in range(lists.shape[1]):
            if lists[h, a, -1] != nkc - 1:
                lists[h, a, -1] = nkc - 1
    Q, K = bf16_round(Q.astype(np.float32)).astype(np.float64), bf16_round(K.astype(np.float32)).astype(np.float64)
    p = ca.Problem(1, H, n, n, d, cq, ck, torch.bfloat16)
    tq = G.permuted_rows(Q, perm_q, cq, torch.bfloat16)
    tk = G.permuted_rows(K, perm_k, ck, torch.bfloat16)
    tv = G.value_tiles(V, perm_k, ck, torch.bfloat16)
    cnt = G.dev(np.stack([G.counts(n, ck)] * H), torch.int32)
    op, lse = ca.block_sparse_attn(p, tq, tk, tv, cnt, G.dev(lists, torch.int32), k)
    torch.cuda.synchronize()
    op, lse = G.host(op), G.host(lse)
    tau = 1 / math.sqrt(d)
    for h in range(H):
        o, l = ref.sparse_attention(Q[h], K[h], V[h], perm_q[h], G.counts(n, cq), perm_k[h],
                                    G.counts(n, ck), lists[h], tau)
        got, want = op[h, :n], o[perm_q[h]]
        assert np.isfinite(got).all() and np.isfinite(lse[h, :n]).all(), h
        err = np.abs(got - want).max()
        assert err <= G.TOL["bf16"], (h, err)
        slack = 2.0 ** -8 * tau * (np.abs(Q[h]) @ np.abs(K[h]).T).max(axis=1)
        lerr = np.abs(lse[h, :n] - l[perm_q[h]]) - slack[perm_q[h]]
        assert lerr.max() <= 1e-3 * max(1.0, np.abs(l).max()), lerr.max()
        G.flush(f"  head {h}: max abs err {err:.3g}")


SHORT_FIRST = [
    # d, cq, ck, n, k: the last key cluster holds n % ck <= 32 keys
    (128, 64, 64, 650, 4),
    (128, 64, 128, 777, 4),
    (64, 128, 128, 918, 4),
    (64, 64, 64, 980, 4),
    (128, 64, 64, 8970, 130),  # the two-wavefront kernel for 64-query clusters
]


@pytest.mark.parametrize("d,cq,ck,n,k", SHORT_FIRST)
def test_short_cluster_first(d, cq, ck, n, k):
    """The last key cluster (at most 32 real keys, so the second 32-key row
    tile of its first stage is all padding) comes first in every list: every
    third query cluster uses it alone (list length 1), the others follow it
    with k - 1 more clusters, in both calls against the oracle. Where a
    wavefront takes half of a stage's keys, one half then sees only padding in
    its first stage, or in every stage."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"short cluster first d={d} cq={cq} ck={ck} n={n} k={k}")
    H = 2
    Q, K, V = mixture_inputs(41, H, n, d, "bf16", centres=8, sigma=0.4)
    rng = np.random.default_rng(42)
    p = ca.Problem(1, H, n, n, d, cq, ck, torch.bfloat16)
    perm_q = np.stack([rng.permutation(n) for _ in range(H)]).astype(np.int32)
    perm_k = np.stack([rng.permutation(n) for _ in range(H)]).astype(np.int32)
    nkc, cq_n, ck_n = p.nkc, G.counts(n, cq), G.counts(n, ck)
    assert ck_n[-1] <= 32 and nkc > k
    L = np.zeros((H, p.nqc, k), np.int32)
    lens = np.full((H, p.nqc), k, np.int32)
    lens[:, ::3] = 1
    ragged = []
    for h in range(H):
        rows = []
        for a in range(p.nqc):
            L[h, a, 0] = nkc - 1
            L[h, a, 1:] = rng.choice(nkc - 1, size=k - 1, replace=False)
            rows.append(L[h, a, :lens[h, a]].copy())
        ragged.append(rows)
    tau = 1 / math.sqrt(d)
    tq = G.permuted_rows(Q, perm_q, cq, torch.bfloat16)
    tk = G.permuted_rows(K, perm_k, ck, torch.bfloat16)
    tv = G.value_tiles(V, perm_k, ck, torch.bfloat16)
    cnt = G.dev(np.stack([ck_n] * H), torch.int32)
    dL, dN = G.dev(L, torch.int32), G.dev(lens, torch.int32)
    kbar = np.stack([ref.centroids(K[h], perm_k[h], ck_n) for h in range(H)]).astype(np.float32)
    vbar = np.stack([ref.centroids(V[h], perm_k[h], ck_n) for h in range(H)]).astype(np.float32)
    op, lse = ca.block_sparse_attn(p, tq, tk, tv, cnt, dL, k, lens=dN)
    out, lse_out = ca.attn_compensated(p, tq, tk, tv, G.dev(kbar), G.dev(vbar), cnt, dL, k,
                                       G.dev(perm_q, torch.int32), want_lse=True, lens=dN)
    torch.cuda.synchronize()
    op, lse = G.host(op), G.host(lse)
    out, lse_out = G.host(out)[0], G.host(lse_out)
    for h in range(H):
        o, l = ref.sparse_attention(Q[h], K[h], V[h], perm_q[h], cq_n, perm_k[h], ck_n, ragged[h],
                                    tau)
        assert np.isfinite(op[h, :n]).all() and np.isfinite(lse[h, :n]).all(), h
        err = np.abs(op[h, :n] - o[perm_q[h]]).max()
        assert err <= G.TOL["bf16"], (h, err)
        assert np.abs(lse[h, :n] - l[perm_q[h]]).max() <= 1e-3 * max(1.0, np.abs(l).max())
        o_w, l_w = ref.compensate(Q[h], kbar[h], vbar[h], ck_n, perm_q[h], cq_n, ragged[h], o, l,
                                  tau)
        assert np.isfinite(out[h]).all() and np.isfinite(lse_out[h]).all(), h
        ferr = np.abs(out[h] - o_w).max()
        assert ferr <= G.TOL["bf16"], (h, ferr)
        assert np.abs(lse_out[h] - l_w).max() <= 1e-3 * max(1.0, np.abs(l_w).max())
        G.flush(f"  head {h}: max abs err {err:.3g} (two calls), {ferr:.3g} (one pass)")


@pytest.mark.parametrize("dt,d,cq,ck,n,k", CASES)
@pytest.mark.parametrize("enable", [True, False])
def test_compensation_parity(dt, d, cq, ck, n, k, enable):
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"comp case dt={dt} d={d} cq={cq} ck={ck} n={n} k={k} enable={enable}")
    Q, K, V, perm_q, perm_k, lists, k = _setup(dt, d, cq, ck, n, k, seed=3)
    H = Q.shape[0]
    p = ca.Problem(1, H, n, n, d, cq, ck, G.tdtype(dt))
    tau = 1 / math.sqrt(d)
    cq_n, ck_n = G.counts(n, cq), G.counts(n, ck)
    # sparse part from the oracle, handed over in the GPU's storage precision
    op = np.zeros((H, p.nq_pad, d), np.float32)
    lse = np.zeros((H, p.nq_pad), np.float32)
    kbar = np.zeros((H, p.nkc, d), np.float32)
    vbar = np.zeros((H, p.nkc, d), np.float32)
    want = []
    for h in range(H):
        o, l = ref.sparse_attention(Q[h], K[h], V[h], perm_q[h], cq_n, perm_k[h], ck_n, lists[h],
                                    tau)
        if dt == "bf16":
            from synth import bf16_round
            o = bf16_round(o.astype(np.float32)).astype(np.float64)
        op[h, :n] = o[perm_q[h]]
        lse[h, :n] = l[perm_q[h]]
        kb = ref.centroids(K[h], perm_k[h], ck_n).astype(np.float32)
        vb = ref.centroids(V[h], perm_k[h], ck_n).astype(np.float32)
        kbar[h], vbar[h] = kb, vb
        want.append(ref.compensate(Q[h], kb, vb, ck_n, perm_q[h], cq_n, lists[h], o,
                                   lse[h, :n][np.argsort(perm_q[h])].astype(np.float64), tau,
                                   enable))
    tq = G.permuted_rows(Q, perm_q, cq, G.tdtype(dt))
    out, lse_out = ca.compensate(p, tq, G.dev(kbar), G.dev(vbar),
                                 G.dev(np.stack([ck_n] * H), torch.int32),
                                 G.dev(lists, torch.int32), k, G.dev(op, G.tdtype(dt)),
                                 G.dev(lse), G.dev(perm_q, torch.int32), enable=enable,
                                 want_lse=True)
    torch.cuda.synchronize()
    out, lse_out = G.host(out)[0], G.host(lse_out)
    for h in range(H):
        o_w, l_w = want[h]
        err = np.abs(out[h] - o_w).max()
        assert err <= G.TOL[dt], (h, err)
        assert np.abs(lse_out[h] - l_w).max() <= 1e-4 * max(1.0, np.abs(l_w).max())


MULTI = [
    # dtype, d, cq, ck, n, k, whole_tile: every other query cluster selects all
    # of centroids [128, 256), a 128-centroid tile the bf16 kernel must skip
    ("bf16", 64, 128, 64, 20000, 140, True),
    ("bf16", 128, 64, 64, 9000, 10, False),
    ("bf16", 64, 64, 128, 40000, 20, False),
    ("f32", 64, 64, 64, 20000, 140, True),
]


@pytest.mark.parametrize("dt,d,cq,ck,n,k,whole_tile", MULTI)
def test_compensation_multi_tile(dt, d, cq, ck, n, k, whole_tile):
    """Compensation over several 128-centroid tiles with a ragged last tile.
    The sparse part is synthetic (it only enters through the merge)."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    from synth import bf16_round
    G.flush(f"comp multi-tile dt={dt} d={d} cq={cq} ck={ck} n={n} k={k} whole={whole_tile}")
    H = 2
    Q, K, V = mixture_inputs(21, H, n, d, dt, centres=8, sigma=0.4)
    rng = np.random.default_rng(22)
    p = ca.Problem(1, H, n, n, d, cq, ck, G.tdtype(dt))
    perm_q = np.stack([rng.permutation(n) for _ in range(H)]).astype(np.int32)
    perm_k = np.stack([rng.permutation(n) for _ in range(H)]).astype(np.int32)
    lists = G.random_lists(rng, H, p.nqc, p.nkc, k)
    if whole_tile:
        assert p.nkc > 256 and k >= 128
        for b in range(H):
            for a in range(0, p.nqc, 2):
                rest = np.setdiff1d(np.arange(p.nkc), np.arange(128, 256))
                extra = rng.choice(rest, size=k - 128, replace=False)
                lists[b, a] = np.sort(np.concatenate([np.arange(128, 256), extra]))
    cq_n, ck_n = G.counts(n, cq), G.counts(n, ck)
    tau = 1 / math.sqrt(d)
    op = np.zeros((H, p.nq_pad, d), np.float32)
    lse = np.zeros((H, p.nq_pad), np.float32)
    kbar = np.zeros((H, p.nkc, d), np.float32)
    vbar = np.zeros((H, p.nkc, d), np.float32)
    want = []
    for h in range(H):
        o = rng.standard_normal((n, d)) * 0.5
        if dt == "bf16":
            o = bf16_round(o.astype(np.float32)).astype(np.float64)
        ls = rng.uniform(8.0, 12.0, n).astype(np.float32).astype(np.float64)
        op[h, :n] = o[perm_q[h]]
        lse[h, :n] = ls[perm_q[h]]
        kbar[h] = ref.centroids(K[h], perm_k[h], ck_n).astype(np.float32)
        vbar[h] = ref.centroids(V[h], perm_k[h], ck_n).astype(np.float32)
        want.append(ref.compensate(Q[h], kbar[h], vbar[h], ck_n, perm_q[h], cq_n, lists[h], o,
                                   ls, tau))
    tq = G.permuted_rows(Q, perm_q, cq, G.tdtype(dt))
    out, lse_out = ca.compensate(p, tq, G.dev(kbar), G.dev(vbar),
                                 G.dev(np.stack([ck_n] * H), torch.int32),
                                 G.dev(lists, torch.int32), k, G.dev(op, G.tdtype(dt)),
                                 G.dev(lse), G.dev(perm_q, torch.int32), want_lse=True)
    torch.cuda.synchronize()
    out, lse_out = G.host(out)[0], G.host(lse_out)
    worst = 0.0
    for h in range(H):
        o_w, l_w = want[h]
        err = np.abs(out[h] - o_w).max()
        worst = max(worst, err)
        assert err <= G.TOL[dt], (h, err)
        assert np.abs(lse_out[h] - l_w).max() <= 1e-4 * max(1.0, np.abs(l_w).max())
    G.flush(f"  max abs err {worst:.3g}")


LENS_CASES = [
    # dtype, d, cq, ck, n
    ("bf16", 64, 128, 128, 20000),
    ("bf16", 128, 64, 64, 5000),
    ("bf16", 64, 64, 128, 9000),
    ("f32", 64, 64, 64, 3000),
]


@pytest.mark.parametrize("dt,d,cq,ck,n", LENS_CASES)
def test_attention_and_compensation_with_lengths(dt, d, cq, ck, n):
    """Lists of varying length (histogram selection): row a uses its first
    lens[a] entries (list stride nkc; the rest of the row holds garbage that
    must not be read), from a single cluster to all of them."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"lens case dt={dt} d={d} cq={cq} ck={ck} n={n}")
    H = 2
    Q, K, V = mixture_inputs(31, H, n, d, dt, centres=8, sigma=0.4)
    rng = np.random.default_rng(32)
    p = ca.Problem(1, H, n, n, d, cq, ck, G.tdtype(dt))
    perm_q = np.stack([rng.permutation(n) for _ in range(H)]).astype(np.int32)
    perm_k = np.stack([rng.permutation(n) for _ in range(H)]).astype(np.int32)
    nkc = p.nkc
    lens = rng.integers(1, nkc + 1, size=(H, p.nqc)).astype(np.int32)
    lens[0, 0], lens[-1, -1] = 1, nkc
    L = np.full((H, p.nqc, nkc), 10 ** 6, np.int32)  # garbage past each length
    ragged = []
    for h in range(H):
        rows = []
        for a in range(p.nqc):
            sel = np.sort(rng.choice(nkc, size=lens[h, a], replace=False)).astype(np.int32)
            L[h, a, :lens[h, a]] = sel
            rows.append(sel)
        ragged.append(rows)
    tau = 1 / math.sqrt(d)
    cq_n, ck_n = G.counts(n, cq), G.counts(n, ck)
    tq = G.permuted_rows(Q, perm_q, cq, G.tdtype(dt))
    cnt = G.dev(np.stack([ck_n] * H), torch.int32)
    dL, dN = G.dev(L, torch.int32), G.dev(lens, torch.int32)
    op, lse = ca.block_sparse_attn(p, tq, G.permuted_rows(K, perm_k, ck, G.tdtype(dt)),
                                   G.value_tiles(V, perm_k, ck, G.tdtype(dt)), cnt, dL, nkc,
                                   lens=dN)
    kbar = np.stack([ref.centroids(K[h], perm_k[h], ck_n) for h in range(H)]).astype(np.float32)
    vbar = np.stack([ref.centroids(V[h], perm_k[h], ck_n) for h in range(H)]).astype(np.float32)
    out, lse_out = ca.compensate(p, tq, G.dev(kbar), G.dev(vbar), cnt, dL, nkc, op, lse,
                                 G.dev(perm_q, torch.int32), want_lse=True, lens=dN)
    torch.cuda.synchronize()
    op_h, lse_h = G.host(op), G.host(lse)
    out_h, lse_out_h = G.host(out)[0], G.host(lse_out)
    for h in range(H):
        o, l = ref.sparse_attention(Q[h], K[h], V[h], perm_q[h], cq_n, perm_k[h], ck_n, ragged[h],
                                    tau)
        assert np.abs(op_h[h, :n] - o[perm_q[h]]).max() <= G.TOL[dt]
        assert np.abs(lse_h[h, :n] - l[perm_q[h]]).max() <= (1e-5 if dt == "f32" else 1e-3) * max(
            1.0, np.abs(l).max())
        # compensation from the GPU's own sparse part (in its storage precision)
        o_s = op_h[h, :n][np.argsort(perm_q[h])]
        l_s = lse_h[h, :n][np.argsort(perm_q[h])]
        o_w, l_w = ref.compensate(Q[h], kbar[h], vbar[h], ck_n, perm_q[h], cq_n, ragged[h], o_s,
                                  l_s, tau)
        assert np.abs(out_h[h] - o_w).max() <= G.TOL[dt]
        assert np.abs(lse_out_h[h] - l_w).max() <= 1e-4 * max(1.0, np.abs(l_w).max())


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_all_kept_equals_dense(dt):
    """Every key cluster selected: the two calls give dense attention."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    d, c, n = 64, 64, 1000
    Q, K, V = mixture_inputs(11, 1, n, d, dt, centres=8, sigma=0.4)
    rng = np.random.default_rng(5)
    perm_q = rng.permutation(n)[None].astype(np.int32)
    perm_k = rng.permutation(n)[None].astype(np.int32)
    p = ca.Problem(1, 1, n, n, d, c, c, G.tdtype(dt))
    k = p.nkc
    lists = np.arange(k, dtype=np.int32)[None, None].repeat(p.nqc, 1)
    tq = G.permuted_rows(Q, perm_q, c, G.tdtype(dt))
    cnt = G.dev(G.counts(n, c)[None], torch.int32)
    L = G.dev(lists, torch.int32)
    op, lse = ca.block_sparse_attn(p, tq, G.permuted_rows(K, perm_k, c, G.tdtype(dt)),
                                   G.value_tiles(V, perm_k, c, G.tdtype(dt)), cnt, L, k)
    kbar = np.zeros((1, p.nkc, d), np.float32)
    out, _ = ca.compensate(p, tq, G.dev(kbar), G.dev(kbar), cnt, L, k, op, lse,
                           G.dev(perm_q, torch.int32))
    torch.cuda.synchronize()
    o, _ = ref.dense_attention(Q[0], K[0], V[0], 1 / 8)
    assert np.abs(G.host(out)[0, 0] - o).max() <= G.TOL[dt]


@pytest.mark.parametrize("pattern", ["ones", "full", "one_long", "ramp"])
def test_scheduled_launch_matches_index_order(pattern):
    """Lists of different lengths run in the longest-first schedule (workspace
    given) and in index order (no workspace): identical outputs and LSE,
    whatever the length pattern. Every length 1; every length k; one full
    list among single-cluster ones; and a ramp sorted by length, whose
    work-balanced ranges would exceed the per-XCD item cap."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"scheduled launch pattern={pattern}")
    H, n, d, c = 3, 30000, 64, 128
    Q, K, V = mixture_inputs(41, H, n, d, "bf16", centres=8, sigma=0.4)
    rng = np.random.default_rng(43)
    p = ca.Problem(1, H, n, n, d, c, c, torch.bfloat16)
    nkc, nqc = p.nkc, p.nqc
    if pattern == "ones":
        lens = np.ones((H, nqc), np.int32)
    elif pattern == "full":
        lens = np.full((H, nqc), nkc, np.int32)
    elif pattern == "one_long":
        lens = np.ones((H, nqc), np.int32)
        lens[1, nqc // 2] = nkc
    else:
        lens = np.sort(rng.integers(1, nkc + 1, size=H * nqc)).reshape(H, nqc).astype(np.int32)
    L = np.stack([np.stack([np.sort(rng.permutation(nkc)).astype(np.int32) for _ in range(nqc)])
                  for _ in range(H)])
    for h in range(H):
        for a in range(nqc):
            L[h, a, :lens[h, a]] = np.sort(rng.choice(nkc, size=lens[h, a], replace=False))
    perm_k = np.stack([rng.permutation(n) for _ in range(H)]).astype(np.int32)
    perm_q = np.stack([rng.permutation(n) for _ in range(H)]).astype(np.int32)
    ck_n = G.counts(n, c)
    args = (G.permuted_rows(Q, perm_q, c, torch.bfloat16),
            G.permuted_rows(K, perm_k, c, torch.bfloat16),
            G.value_tiles(V, perm_k, c, torch.bfloat16),
            G.dev(np.stack([ck_n] * H), torch.int32), G.dev(L, torch.int32))
    dN = G.dev(lens, torch.int32)
    ws = ca.workspace(p, args[0].device, nkc)
    op1, lse1 = ca.block_sparse_attn(p, *args, nkc, lens=dN, ws=ws)
    op0, lse0 = ca.block_sparse_attn(p, *args, nkc, lens=dN)
    torch.cuda.synchronize()
    assert torch.equal(op1, op0) and torch.equal(lse1, lse0)
    assert torch.isfinite(lse1[:, :n]).all()
