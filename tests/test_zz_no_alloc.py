"""ca_attn_compensated_noalloc (steps 3 and 4 in one pass, no workspace: the
centroid tiles and the launch schedule live in the library's per-device
scratch array) against ca_attn_compensated with a caller workspace, through
the C ABI. The same kernels run, so outputs and lse must agree bit for bit.

Every case makes two calls in a row on the same device, the second with a
smaller problem, so the second call runs on scratch that still holds the
first call's tiles and schedule: exact top-k lists (tiles), adaptive lists of
different lengths (tiles and schedule), compensation off and every cluster
kept (no scratch needed)."""
import math

import pytest

pytestmark = pytest.mark.gpu


def _layer(H, n, d, c, seed, xf):
    import torch
    import paper_2608_26965_amd as ca
    g = torch.Generator(device="cpu").manual_seed(seed)
    q, k, v = (torch.randn(1, H, n, d, generator=g).to("cuda").to(torch.bfloat16)
               for _ in range(3))
    p = ca.Problem(1, H, n, n, d, c, c, torch.bfloat16, xf)
    return p, ca.cluster(p, q, k, v)


def _lists(p, r, mode):
    import paper_2608_26965_amd as ca
    if mode == "adaptive":
        lists, lens, _ = ca.select_hist(p, r["cent_q"], r["cent_k"], r["count_k"], 4, 0.9,
                                        1.0 / math.sqrt(p.d))
        return lists, lens, p.nkc
    k = p.nkc if mode == "all" else ca.keep_to_k(0.2, p.nkc)
    lists, _ = ca.select(p, r["cent_q"], r["cent_k"], k)
    return lists, None, k


def _compare(p, r, mode, enable):
    import torch
    import paper_2608_26965_amd as ca
    lists, lens, k = _lists(p, r, mode)
    args = (p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"], r["count_k"], lists, k,
            r["perm_q"])
    ws = ca.workspace(p, lists.device, k)
    a_out, a_lse = ca.attn_compensated(*args, enable=enable, want_lse=True, ws=ws, lens=lens)
    b_out, b_lse = ca.attn_compensated_noalloc(*args, enable=enable, want_lse=True, lens=lens)
    torch.cuda.synchronize()
    assert torch.equal(a_out, b_out), f"{mode}: outputs differ"
    assert torch.equal(a_lse, b_lse), f"{mode}: lse differ"


@pytest.mark.parametrize("mode,enable", [("topk", True), ("adaptive", True), ("topk", False),
                                         ("all", True)])
@pytest.mark.parametrize("first,second", [((4, 9000, 64, 128), (2, 3000, 64, 128)),
                                          ((3, 6000, 128, 64), (1, 2500, 128, 64))])
def test_noalloc_matches_workspace_call(mode, enable, first, second):
    from tests import gpu_util as G
    xf = "adaptive" if mode == "adaptive" else "metric"
    for (H, n, d, c), seed in ((first, 1), (second, 2)):
        G.flush(f"noalloc: mode={mode} enable={enable} H={H} n={n} d={d} c={c}")
        p, r = _layer(H, n, d, c, seed, xf)
        _compare(p, r, mode, enable)

