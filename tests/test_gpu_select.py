"""GPU parity of ca_select: centroid scores within fp32 rounding of the oracle,
and lists bit-exact against the oracle's top-k of the very same scores."""
import numpy as np
import pytest

from oracle import ref

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nqc,nkc,d,k", [(16, 16, 64, 4), (50, 130, 64, 13), (33, 300, 128, 300),
                                         (7, 1000, 32, 1), (200, 77, 64, 76)])
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
    p = ca.Problem(1, H, nqc * 16, nkc * 16, 8, 16, 16, torch.float32)
    lists, _ = ca.select(p, None, None, k, scores_in=G.dev(S))
    torch.cuda.synchronize()
    L = lists.cpu().numpy()
    for h in range(H):
        assert np.array_equal(L[h], ref.topk(S[h].astype(np.float64), k))
