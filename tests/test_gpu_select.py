"""GPU parity of ca_select: centroid scores within 1e-5 of the oracle's (fp32
rounding, or the three-term bf16 split on the matrix cores for bf16 problems
with d = 64 or 128), and lists bit-exact against the oracle's top-k of the
very same scores."""
import numpy as np
import pytest

from oracle import ref

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nqc,nkc,d,k", [(16, 16, 64, 4), (50, 130, 64, 13), (33, 300, 128, 300),
                                         (7, 1000, 32, 1), (200, 77, 64, 76), (4, 8192, 64, 64),
                                         (3, 5000, 64, 820)])
def test_scores_and_topk(nqc, nkc, d, k):
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"select case nqc={nqc} nkc={nkc} d={d} k={k}")
    rng = np.random.default_rng(nqc * 1000 + nkc)
    H = 2
    cq = rng.standard_normal((H, nqc, d)).astype(np.float32)
    ck = rng.standard_normal((H, nkc, d)).astype(np.float32)
    p = ca.Problem(1, H, nqc * 64, nkc * 64, d, 64, 64, torch.bfloat16)
    lists, scores = ca.select(p, G.dev(cq), G.dev(ck), k, export_scores=True)
    torch.cuda.synchronize()
    S = G.host(scores)
    L = lists.cpu().numpy()
    for h in range(H):
        want = ref.centroid_scores(cq[h], ck[h])
        assert np.abs(S[h] - want).max() <= 1e-5 * max(1.0, np.abs(want).max())
        assert np.array_equal(L[h], ref.topk(S[h], k))


@pytest.mark.parametrize("k", [1, 5, 17, 40])
def test_topk_with_ties_given_scores(k):
    """Integer-valued scores with many ties, including -0.0 / +0.0: lists must
    equal the oracle's (ties to the lower index) exactly."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    rng = np.random.default_rng(k)
    H, nqc, nkc = 3, 20, 40
    S = rng.integers(-3, 4, size=(H, nqc, nkc)).astype(np.float32)
    S[S == 0] = np.where(rng.random((S == 0).sum()) < 0.5, -0.0, 0.0)
    S[1, 2] = 0.5  # a row of equal scores
    S[2, 3] = np.linspace(1.0, 1.0 + 1e-5, nkc, dtype=np.float32)  # a very narrow range
    p = ca.Problem(1, H, nqc * 16, nkc * 16, 8, 16, 16, torch.float32)
    lists, _ = ca.select(p, None, None, k, scores_in=G.dev(S))
    torch.cuda.synchronize()
    L = lists.cpu().numpy()
    for h in range(H):
        assert np.array_equal(L[h], ref.topk(S[h].astype(np.float64), k))


@pytest.mark.parametrize("nkc,k", [(2049, 2049), (3000, 64), (4096, 100), (5000, 64),
                                   (8192, 820), (8192, 64), (4097, 4097), (6001, 3),
                                   (7999, 2000), (1001, 500), (1000, 1), (9000, 64),
                                   (257, 257)])
def test_topk_long_rows_with_ties(nkc, k):
    """Rows of up to 2048 scores (one row per wavefront), up to 8192 (one row
    per block of four wavefronts) and beyond (one per block of 256 threads),
    with heavy ties (so the threshold's bin overflows the
    candidate list), a constant row, a range a few subnormals wide, and row
    lengths that are not multiples of four: lists equal the oracle's."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"long-row top-k nkc={nkc} k={k}")
    rng = np.random.default_rng(nkc + k)
    H, nqc = 2, 6
    S = rng.integers(-3, 4, size=(H, nqc, nkc)).astype(np.float32)
    S[0, 1] = rng.standard_normal(nkc).astype(np.float32)
    S[0, 2] = 2.5
    S[1, 0] = (np.arange(nkc) % 7).astype(np.float32) * np.float32(1e-44)
    S[1, 1] = rng.standard_normal(nkc).astype(np.float32) * 1e3
    S[1, 1, ::97] = -1e30  # far outliers stretch the linear bins
    p = ca.Problem(1, H, nqc * 16, nkc * 16, 8, 16, 16, torch.float32)
    lists, _ = ca.select(p, None, None, k, scores_in=G.dev(S))
    torch.cuda.synchronize()
    L = lists.cpu().numpy()
    for h in range(H):
        for a in range(nqc):
            assert np.array_equal(L[h, a], ref.topk(S[h, a:a + 1].astype(np.float64), k)[0]), (h, a)


@pytest.mark.gpu
@pytest.mark.parametrize("nkc,k", [(4096, 100), (8192, 64), (8192, 819), (6000, 3), (2052, 2052)])
def test_topk_many_long_rows(nkc, k):
    """A thousand rows of 2049-8192 scores (more rows than workgroups fit on
    the device at once, one row per block of four wavefronts). Rows mix
    continuous values, heavy ties, constant rows, subnormal ranges and far
    outliers; every list equals the oracle's."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"many long-row top-k nkc={nkc} k={k}")
    rng = np.random.default_rng(3 * nkc + k)
    H, nqc = 2, 500
    S = rng.standard_normal((H, nqc, nkc)).astype(np.float32)
    S[:, 1::5] = rng.integers(-3, 4, size=(H, len(range(1, nqc, 5)), nkc))
    S[:, 2::5] = 0.75
    S[:, 3::5] = (np.arange(nkc) % 7).astype(np.float32) * np.float32(1e-44)
    S[:, 4::5, ::97] = -1e30
    p = ca.Problem(1, H, nqc * 16, nkc * 16, 8, 16, 16, torch.float32)
    lists, _ = ca.select(p, None, None, k, scores_in=G.dev(S))
    torch.cuda.synchronize()
    L = lists.cpu().numpy()
    for h in range(H):
        for a in range(nqc):
            assert np.array_equal(L[h, a], ref.topk(S[h, a:a + 1].astype(np.float64), k)[0]), (h, a)


HIST_CASES = [
    # nqc, nkc, d, min_count, mass_recall
    (16, 16, 64, 4, 0.0),
    (50, 130, 64, 13, 0.0),
    (50, 130, 64, 16, 0.9),
    (33, 300, 128, 16, 0.5),
    (7, 1000, 32, 1, 0.99),
    (200, 77, 64, 76, 0.0),
    (64, 512, 64, 64, 0.0),   # one head of the tabular workload: top-k through the histogram
    (64, 512, 64, 16, 0.9),   # ... and adaptive assignment
    (5, 3000, 64, 16, 1.0),
]


@pytest.mark.parametrize("nqc,nkc,d,min_count,recall", HIST_CASES)
def test_hist_select(nqc, nkc, d, min_count, recall):
    """Two-pass histogram selection: lists and lengths equal the oracle's on
    the GPU's own scores (count-only mode is integer work on fp32 grid
    positions; the mass mode sums fp64 estimates in fixed point)."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"hist select nqc={nqc} nkc={nkc} d={d} min_count={min_count} recall={recall}")
    rng = np.random.default_rng(nqc * 7 + nkc)
    H = 2
    cq = (rng.standard_normal((H, nqc, d)) * 0.7).astype(np.float32)
    ck = (rng.standard_normal((H, nkc, d)) * 0.7).astype(np.float32)
    cnt = rng.integers(1, 129, size=(H, nkc)).astype(np.int32)
    p = ca.Problem(1, H, nqc * 64, nkc * 64, d, 64, 64, torch.bfloat16)
    scale = np.float32(1.0 / np.sqrt(d))
    lists, lens, scores = ca.select_hist(p, G.dev(cq), G.dev(ck), G.dev(cnt, torch.int32),
                                         min_count, recall, float(scale), export_scores=True)
    torch.cuda.synchronize()
    S = scores.cpu().numpy().astype(np.float64)
    L, N = lists.cpu().numpy(), lens.cpu().numpy()
    worst = 0
    for h in range(H):
        for a in range(nqc):
            want = ref.hist_select(S[h, a], cnt[h], float(scale), min_count,
                                   float(np.float32(recall)))
            assert N[h, a] == len(want), (h, a, N[h, a], len(want))
            assert np.array_equal(L[h, a, :N[h, a]], want), (h, a)
            worst = max(worst, len(want))
    G.flush(f"  longest list {worst} of {nkc}")


@pytest.mark.parametrize("min_count,recall", [(5, 0.0), (1, 0.7), (16, 0.95)])
def test_hist_select_ties_and_degenerate_rows(min_count, recall):
    """Integer scores with many exact ties (-0.0 and +0.0 among them), rows
    whose scores are all equal, and a row of one distinct value plus one
    outlier, given through scores_in."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    rng = np.random.default_rng(min_count)
    H, nqc, nkc = 2, 12, 40
    S = rng.integers(-3, 4, size=(H, nqc, nkc)).astype(np.float32)
    S[S == 0] = np.where(rng.random((S == 0).sum()) < 0.5, -0.0, 0.0)
    S[0, 3] = 1.5                      # all equal
    S[1, 5] = 2.0
    S[1, 5, 17] = 9.0                  # one outlier
    cnt = rng.integers(1, 65, size=(H, nkc)).astype(np.int32)
    p = ca.Problem(1, H, nqc * 16, nkc * 16, 8, 16, 16, torch.float32)
    lists, lens, _ = ca.select_hist(p, None, None, G.dev(cnt, torch.int32), min_count, recall,
                                    0.25, scores_in=G.dev(S))
    torch.cuda.synchronize()
    L, N = lists.cpu().numpy(), lens.cpu().numpy()
    for h in range(H):
        for a in range(nqc):
            want = ref.hist_select(S[h, a].astype(np.float64), cnt[h], 0.25, min_count,
                                   float(np.float32(recall)))
            assert N[h, a] == len(want) and np.array_equal(L[h, a, :N[h, a]], want), (h, a)
    assert N[0, 3] == nkc
