"""CA_LAYOUT_STRIDED: q, k and v read in place as views of one fused
[B, N, 3, H, d] projection, and the output written into a slice of a wider
tensor, against the same problem on dense BHND copies. Only the addressing
differs, so clusters, lists and outputs must agree bit for bit; the rest of
the wider output tensor must stay untouched."""
import pytest

pytestmark = pytest.mark.gpu


def _fused_views(B, N, H, d, dtype, seed):
    import torch
    g = torch.Generator(device="cpu").manual_seed(seed)
    qkv = torch.randn(B, N, 3, H, d, generator=g).to("cuda").to(dtype)
    return qkv, [qkv[:, :, j].permute(0, 2, 1, 3) for j in range(3)]


@pytest.mark.parametrize("dtype_name,d,c,n", [("bf16", 64, 128, 3000), ("bf16", 128, 64, 2500),
                                              ("f32", 32, 64, 1500)])
def test_strided_views_match_dense(dtype_name, d, c, n):
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush(f"strided: {dtype_name} d={d} c={c} n={n}")
    dtype = G.tdtype(dtype_name)
    B, H = 2, 2
    _, (q, k, v) = _fused_views(B, n, H, d, dtype, seed=d + c)
    assert not q.is_contiguous()
    qd, kd, vd = (x.contiguous() for x in (q, k, v))
    wide = torch.zeros(B, n, H, 3 * d, dtype=dtype, device="cuda")
    out_view = wide[..., d:2 * d].permute(0, 2, 1, 3)  # [B,H,N,d] view, rows 3d apart
    ps = ca.Problem(B, H, n, n, d, c, c, dtype, "metric", "strided", q_stride=ca.bhnd_strides(q),
                    k_stride=ca.bhnd_strides(k), v_stride=ca.bhnd_strides(v),
                    out_stride=ca.bhnd_strides(out_view))
    pd = ca.Problem(B, H, n, n, d, c, c, dtype, "metric", "bhnd")
    rs = ca.cluster(ps, q, k, v)
    rd = ca.cluster(pd, qd, kd, vd)
    kk = ca.keep_to_k(0.25, pd.nkc)
    ls, _ = ca.select(ps, rs["cent_q"], rs["cent_k"], kk)
    ld, _ = ca.select(pd, rd["cent_q"], rd["cent_k"], kk)
    if dtype == torch.bfloat16:
        ca.attn_compensated(ps, rs["qp"], rs["kp"], rs["vp"], rs["cent_k"], rs["cent_v"],
                            rs["count_k"], ls, kk, rs["perm_q"], out=out_view)
        od, _ = ca.attn_compensated(pd, rd["qp"], rd["kp"], rd["vp"], rd["cent_k"],
                                    rd["cent_v"], rd["count_k"], ld, kk, rd["perm_q"])
    else:
        op, lse = ca.block_sparse_attn(ps, rs["qp"], rs["kp"], rs["vp"], rs["count_k"], ls, kk)
        ca.compensate(ps, rs["qp"], rs["cent_k"], rs["cent_v"], rs["count_k"], ls, kk, op, lse,
                      rs["perm_q"], out=out_view)
        op, lse = ca.block_sparse_attn(pd, rd["qp"], rd["kp"], rd["vp"], rd["count_k"], ld, kk)
        od, _ = ca.compensate(pd, rd["qp"], rd["cent_k"], rd["cent_v"], rd["count_k"], ld, kk,
                              op, lse, rd["perm_q"])
    torch.cuda.synchronize()
    for key in rd:
        assert torch.equal(rs[key], rd[key]), key
    # the permuted copies are the input rows in cluster order (both paths
    # read the right rows, not merely the same ones)
    for bh in range(B * H):
        b, h = divmod(bh, H)
        for x, xp, perm in ((q, "qp", "perm_q"), (k, "kp", "perm_k")):
            got = rs[xp][bh, :n]
            assert torch.equal(got, x[b, h][rs[perm][bh].long()]), xp
    assert torch.equal(ls, ld), "lists"
    assert torch.equal(out_view, od), "outputs"
    assert (wide[..., :d] == 0).all() and (wide[..., 2 * d:] == 0).all(), "wrote outside the view"


def test_forward_strided_views():
    """The layer API reads a fused projection's views in place."""
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    G.flush("strided: forward()")
    _, (q, k, v) = _fused_views(1, 4000, 2, 64, torch.bfloat16, seed=9)
    a = ca.forward(q, k, v, cq=128, keep=0.2, layout="strided")
    b = ca.forward(q.contiguous(), k.contiguous(), v.contiguous(), cq=128, keep=0.2)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("dtype_name", ["bf16", "f32"])
def test_check_finite_flags(dtype_name):
    """Checked mode flags exactly the tensors holding a NaN or an infinity,
    in a dense and in a strided layout, and forward(checked=True) raises."""
    import math
    import torch
    import paper_2608_26965_amd as ca
    from paper_2608_26965_amd import _lib as L
    from tests import gpu_util as G
    dtype = G.tdtype(dtype_name)
    B, H, n, d = 1, 3, 700, 32
    g = torch.Generator(device="cpu").manual_seed(5)
    q, k, v = (torch.randn(B, H, n, d, generator=g).to("cuda").to(dtype) for _ in range(3))
    p = ca.Problem(B, H, n, n, d, 64, 64, dtype)
    assert ca.check_finite(p, q, k, v) == 0
    k[0, 2, 699, 31] = math.inf
    v[0, 1, 5, 0] = math.nan
    assert ca.check_finite(p, q, k, v, raise_error=False) == 6
    assert ca.check_finite(p, q, k, None, raise_error=False) == 2
    with pytest.raises(ca.CAError) as e:
        ca.forward(q, k, v, cq=64, keep=0.5, checked=True)
    assert e.value.status == L.CA_E_NONFINITE
    # strided views: the non-finite value outside the view is not seen
    qkv, (qs, ks, vs) = _fused_views(1, 500, 2, 32, dtype, seed=6)
    ps = ca.Problem(1, 2, 500, 500, 32, 64, 64, dtype, "metric", "strided",
                    q_stride=ca.bhnd_strides(qs), k_stride=ca.bhnd_strides(ks),
                    v_stride=ca.bhnd_strides(vs), out_stride=(2 * 500 * 32, 500 * 32, 32))
    assert ca.check_finite(ps, qs, ks, vs) == 0
    qkv[0, 499, 2, 1, 31] = -math.inf  # v of head 1, last token
    assert ca.check_finite(ps, qs, ks, vs, raise_error=False) == 4
