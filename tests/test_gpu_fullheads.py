"""The timed layers at their full head counts, checked against the oracle.

The bench and the configuration table time ca_cluster -> ca_select ->
ca_attn_compensated (and the two calls ca_block_sparse_attn +
ca_compensate) over every head of a layer. Here the same calls run at the
same sizes and head counts: the 16-head tabular layer of 262,144 tokens
(d = 64, clusters of 128, keep 1/16 and 1/4) and the 40-head video layers of
32,760 tokens (d = 128, clusters of 64, keep 1/4) and 75,600 tokens (d = 128,
clusters of 64 and 128, keep 1/4, 1/8 and 1/16, compensation on and off). So
the per-head workspace offsets, the multi-GB buffers and the XCD renumbering
of the attention launch run exactly as timed.

Two distinct heads are generated per configuration and repeated to the
layer's head count (head h is generated head h mod 2), as in the timed runs.
Heads 0 and H - 1 are checked against the oracle: permutations bit-exact
against its split of the exported coordinates, lists bit-exact against its
top-k of the exported scores, and the outputs and merged lse of sampled query
clusters (the last, ragged one always among them) within the bf16 tolerance of
its compensated sparse attention given the GPU's permutations and lists, for
the one-pass call and for the two calls. Every other head must reproduce its
generated head's permutations, lists, outputs and lse bit for bit (the calls
are deterministic and heads are independent), which covers the rest of the
launch."""
import numpy as np
import pytest

from synth import CONFIGS, keep_to_k, make_config
from tests.oracle_check import check_head

pytestmark = pytest.mark.gpu

GEN = 2  # distinct heads generated per configuration

# (configuration, cluster size, [(keep fraction, compensation)])
LAYERS = [
    (3, 128, [(1 / 16, True), (1 / 4, True)]),
    (4, 64, [(1 / 4, True)]),
    (5, 64, [(kp, cm) for kp in (1 / 4, 1 / 8, 1 / 16) for cm in (True, False)]),
    (5, 128, [(kp, cm) for kp in (1 / 4, 1 / 8, 1 / 16) for cm in (True, False)]),
]

_CACHE = {}


def _inputs(cid):
    if cid not in _CACHE:
        _CACHE.clear()
        _CACHE[cid] = make_config(cid, heads=list(range(GEN)))
    return _CACHE[cid]


def _same_as_source(t, H, what):
    """Head h of t equals head h mod GEN (t: [H, ...] or [1, H, ...])."""
    import torch
    if t.dim() >= 2 and t.shape[0] == 1 and t.shape[1] == H:
        t = t[0]
    for h in range(GEN, H):
        assert torch.equal(t[h], t[h % GEN]), f"{what}: head {h} differs from head {h % GEN}"


@pytest.mark.parametrize("cid,c,runs", LAYERS, ids=[f"cfg{a}-c{b}" for a, b, _ in LAYERS])
def test_full_layer(cid, c, runs):
    import torch
    import paper_2608_26965_amd as ca
    from tests import gpu_util as G
    cfg = CONFIGS[cid]
    H, n, d = cfg.heads, cfg.n, cfg.d
    G.flush(f"full layer config {cid}: heads={H} n={n} d={d} c={c}")
    Q, K, V = _inputs(cid)
    rep = -(-H // GEN)
    tq, tk, tv = (G.dev(x, torch.bfloat16).repeat(rep, 1, 1)[:H][None].contiguous()
                  for x in (Q, K, V))
    p = ca.Problem(1, H, n, n, d, c, c, torch.bfloat16, "metric")
    ws = ca.workspace(p, tq.device, p.nkc)
    r = ca.cluster(p, tq, tk, tv, export_y=True, ws=ws)
    torch.cuda.synchronize()
    for key in ("perm_q", "perm_k", "count_q", "count_k", "cent_q", "cent_k", "cent_v", "qp", "kp",
                "vp"):
        _same_as_source(r[key], H, key)
    check = (0, H - 1)
    for keep, comp in runs:
        k = keep_to_k(keep, p.nkc)
        G.flush(f"  keep={keep:.4g} (k={k} of {p.nkc}) compensation={comp}")
        lists, scores = ca.select(p, r["cent_q"], r["cent_k"], k, export_scores=True, ws=ws)
        out1, lse1 = ca.attn_compensated(p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"],
                                         r["count_k"], lists, k, r["perm_q"], enable=comp,
                                         want_lse=True, ws=ws)
        op, lse = ca.block_sparse_attn(p, r["qp"], r["kp"], r["vp"], r["count_k"], lists, k)
        out2, lse2 = ca.compensate(p, r["qp"], r["cent_k"], r["cent_v"], r["count_k"], lists, k,
                                   op, lse, r["perm_q"], enable=comp, want_lse=True, ws=ws)
        torch.cuda.synchronize()
        for t, what in ((lists, "lists"), (out1, "one-pass output"), (lse1, "one-pass lse"),
                        (out2, "two-call output"), (lse2, "two-call lse")):
            _same_as_source(t, H, what)
        for out, lse_o, what in ((out1, lse1, "one pass"), (out2, lse2, "two calls")):
            outh = {h: G.host(out[0, h]) for h in check}
            lseh = {h: G.host(lse_o[h]) for h in check}
            worst = 0.0
            for h in check:
                g = h % GEN
                worst = max(worst, check_head(Q[g], K[g], V[g], r, lists, scores, outh, h, c, k,
                                              "bf16", 6, comp, seed=cid * 1000 + h, lse=lseh))
            G.flush(f"    {what}: worst sampled error {worst:.3g}")
        del lists, scores, out1, lse1, op, lse, out2, lse2
