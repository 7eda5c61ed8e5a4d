"""ca_attn_compensated (steps 3 and 4 in one pass) against ca_block_sparse_attn
followed by ca_compensate on the same clusters and lists: ragged sizes, both
layouts, every supported (d, c_q, c_k), compensation off, every cluster kept,
and list lengths from adaptive assignment (with and without the scheduled
launch). The separate path rounds the sparse part to bf16 before the merge;
the one-pass path does not, so the two agree to about one bf16 unit of the
outputs."""
import math

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _setup(H, n, d, cq, ck, layout="bhnd", seed=0, xf="metric"):
    import torch
    import paper_2608_26965_amd as ca
    g = torch.Generator(device="cpu").manual_seed(seed)
    shape = (1, H, n, d) if layout == "bhnd" else (1, n, H, d)
    q, k, v = (torch.randn(shape, generator=g).to("cuda").to(torch.bfloat16) for _ in range(3))
    p = ca.Problem(1, H, n, n, d, cq, ck, torch.bfloat16, xf, layout)
    r = ca.cluster(p, q, k, v)
    return p, r


def _separate(p, r, lists, k, comp, lens=None, ws=None):
    import paper_2608_26965_amd as ca
    op, lse = ca.block_sparse_attn(p, r["qp"], r["kp"], r["vp"], r["count_k"], lists, k,
                                   lens=lens, ws=ws)
    return ca.compensate(p, r["qp"], r["cent_k"], r["cent_v"], r["count_k"], lists, k, op, lse,
                         r["perm_q"], enable=comp, want_lse=True, lens=lens, ws=ws)


def _fused(p, r, lists, k, comp, lens=None, ws=None):
    import paper_2608_26965_amd as ca
    return ca.attn_compensated(p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"],
                               r["count_k"], lists, k, r["perm_q"], enable=comp, want_lse=True,
                               lens=lens, ws=ws)


def _compare(a, b, what):
    import torch
    torch.cuda.synchronize()
    oa, la = a
    ob, lb = b
    assert torch.isfinite(oa.float()).all() and torch.isfinite(la).all(), what
    d = (oa.float() - ob.float()).abs()
    scale = ob.float().abs().clamp_min(1.0)
    assert (d / scale).max().item() <= 2e-2, f"{what}: output {d.max().item()}"
    assert d.mean().item() <= 2e-3, f"{what}: mean output difference {d.mean().item()}"
    # Both paths sum probabilities rounded to bf16 (relative error at most
    # 2^-9 each), so each lse is within ln(1 + 2^-9) < 2e-3 of the exact one.
    assert (la - lb).abs().max().item() <= 4e-3, f"{what}: lse {(la - lb).abs().max().item()}"


@pytest.mark.parametrize("d,cq,ck,n,keep", [
    (64, 128, 128, 3000, 0.2), (64, 64, 64, 2500, 0.25), (64, 64, 128, 2900, 0.3),
    (64, 128, 64, 3100, 0.2), (128, 64, 64, 2600, 0.25), (128, 128, 128, 4100, 0.3),
    (128, 64, 128, 3000, 0.2), (128, 128, 64, 3300, 0.25),
    # lists long enough for the two-wavefront kernel of 64-query clusters
    (128, 64, 64, 12000, 0.75), (64, 64, 128, 20000, 0.9)])
def test_fused_matches_separate(d, cq, ck, n, keep):
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"fused vs separate d={d} cq={cq} ck={ck} n={n} keep={keep}")
    p, r = _setup(2, n, d, cq, ck, seed=d + cq + ck)
    k = ca.keep_to_k(keep, p.nkc)
    lists, _ = ca.select(p, r["cent_q"], r["cent_k"], k)
    _compare(_fused(p, r, lists, k, True), _separate(p, r, lists, k, True), "compensated")
    _compare(_fused(p, r, lists, k, False), _separate(p, r, lists, k, False), "no compensation")


@pytest.mark.parametrize("d,cq,ck,n", [(64, 128, 128, 3000), (128, 64, 64, 2600),
                                        (128, 128, 128, 4100)])
def test_fused_logit_jump(d, cq, ck, n):
    """Logits far above the first stage's maximum (queries with 3 on axis 0,
    3% of the keys with 400 there): the one-pass call, whose exponentials
    against the first stage's maximum overflow for many query clusters, must
    still agree with the separate calls."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"fused logit jump d={d} cq={cq} ck={ck} n={n}")
    H = 2
    g = torch.Generator(device="cpu").manual_seed(d + n)
    q, k, v = (torch.randn((1, H, n, d), generator=g) for _ in range(3))
    q[..., 0] = 3.0
    out = torch.rand((1, H, n), generator=g) < 0.03
    k[..., 0] = torch.where(out, torch.full_like(k[..., 0], 400.0), k[..., 0])
    q, k, v = (t.to("cuda").to(torch.bfloat16) for t in (q, k, v))
    p = ca.Problem(1, H, n, n, d, cq, ck, torch.bfloat16, "metric")
    r = ca.cluster(p, q, k, v)
    kk = ca.keep_to_k(0.2, p.nkc)
    lists, _ = ca.select(p, r["cent_q"], r["cent_k"], kk)
    _compare(_fused(p, r, lists, kk, True), _separate(p, r, lists, kk, True), "compensated")
    _compare(_fused(p, r, lists, kk, False), _separate(p, r, lists, kk, False), "no compensation")


def test_fused_bnhd_layout_and_all_kept():
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush("fused: BNHD layout; every cluster kept")
    p, r = _setup(3, 2200, 64, 64, 64, layout="bnhd", seed=5)
    k = ca.keep_to_k(0.25, p.nkc)
    lists, _ = ca.select(p, r["cent_q"], r["cent_k"], k)
    _compare(_fused(p, r, lists, k, True), _separate(p, r, lists, k, True), "bnhd")
    lists, _ = ca.select(p, r["cent_q"], r["cent_k"], p.nkc)
    a = _fused(p, r, lists, p.nkc, True)
    _compare(a, _separate(p, r, lists, p.nkc, True), "all kept")
    _compare(a, _fused(p, r, lists, p.nkc, False), "all kept: compensation has nothing to add")


@pytest.mark.parametrize("scheduled", [False, True])
def test_fused_adaptive_lists(scheduled):
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"fused: adaptive list lengths, scheduled={scheduled}")
    p, r = _setup(2, 6000, 64, 128, 128, seed=11, xf="adaptive")
    lists, lens, _ = ca.select_hist(p, r["cent_q"], r["cent_k"], r["count_k"], 4, 0.9,
                                    1.0 / math.sqrt(p.d))
    ws = ca.workspace(p, lists.device, p.nkc) if scheduled else None
    n = lens.cpu().numpy()
    assert n.min() < n.max() or n.min() < p.nkc
    _compare(_fused(p, r, lists, p.nkc, True, lens=lens, ws=ws),
             _separate(p, r, lists, p.nkc, True, lens=lens, ws=ws), "adaptive")


@pytest.mark.parametrize("select,transform", [("topk", "metric"), ("adaptive", "adaptive")])
def test_forward_one_pass_matches_two_calls(select, transform):
    """The layer API: bf16 layers take the one-pass call by default."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"forward: one pass vs two calls, select={select}")
    g = torch.Generator(device="cpu").manual_seed(3)
    q, k, v = (torch.randn(1, 2, 3500, 64, generator=g).to("cuda").to(torch.bfloat16)
               for _ in range(3))
    kw = dict(cq=128, keep=0.2, transform=transform, select=select, min_count=4)
    a = ca.forward(q, k, v, **kw)
    b, parts = ca.forward(q, k, v, return_parts=True, **kw)
    c = ca.forward(q, k, v, one_pass=False, **kw)
    torch.cuda.synchronize()
    assert torch.equal(b, c)
    d = (a.float() - c.float()).abs()
    assert (d / c.float().abs().clamp_min(1.0)).max().item() <= 2e-2
    assert d.mean().item() <= 2e-3
