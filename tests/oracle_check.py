"""Per-head oracle checks of a whole layer's GPU results, shared by the
end-to-end parity tests.

check_head: permutations bit-exact against the oracle's split of the exported
split coordinates; lists bit-exact against the oracle's top-k of the exported
scores; scores within fp32 rounding of the oracle's centroid scores; outputs
(and, when given, the merged lse) of sampled query clusters within the
tolerance of the oracle's compensated sparse attention given the GPU's
permutations and lists (the last, possibly ragged, query cluster is always
sampled)."""
import math

import numpy as np

from oracle import ref
from tests import gpu_util as G

# The merged log-sum-exp of the bf16 path sums probabilities rounded to bf16
# (relative error at most 2^-9 each, so at most ln(1 + 2^-9) < 2e-3 in lse);
# the fp32 path rounds only the fp32 sums. The tolerances are those of the
# outputs.
LSE_TOL = G.TOL


def sample_clusters(nqc, nsample, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[nqc - 1],
                                     rng.choice(nqc, min(nsample, nqc), replace=False)]))


def oracle_rows(Q, K, V, perm_q, perm_k, cq, ck, lists, sample, tau, comp):
    """The oracle's output and lse for the query rows of the sampled clusters
    (original indices, cluster by cluster), given the permutations and the
    lists of every query cluster."""
    n_q, n_k = Q.shape[0], K.shape[0]
    cq_n, ck_n = G.counts(n_q, cq), G.counts(n_k, ck)
    kbar = ref.centroids(K, perm_k, ck_n)
    vbar = ref.centroids(V, perm_k, ck_n)
    mem = ref.cluster_members(perm_q, cq_n)
    rows = np.concatenate([mem[a] for a in sample])
    sub_counts = cq_n[sample]
    sub_perm = np.arange(len(rows))
    sub_lists = [lists[a] for a in sample]
    o_s, l_s = ref.sparse_attention(Q[rows], K, V, sub_perm, sub_counts, perm_k, ck_n, sub_lists,
                                    tau)
    o, l = ref.compensate(Q[rows], kbar, vbar, ck_n, sub_perm, sub_counts, sub_lists, o_s, l_s,
                          tau, comp)
    return rows, o, l


def check_head(Q, K, V, r, lists, scores, out, h, c, k, dt, nsample, comp, seed, split="diag",
               lse=None, ck=None):
    """Check head h of a layer (see the module docstring). r: the cluster
    outputs (with exported coordinates yq/yk), lists/scores: device tensors of
    the layer, out: host array [BH, nq, d] of outputs in original order, lse:
    optional host array [BH, nq]. c is the query cluster size, ck the key
    cluster size (default c). Returns the worst output error."""
    ck = c if ck is None else ck
    n_q, d = Q.shape
    n_k = K.shape[0]
    tau = 1 / math.sqrt(d)
    yq = r["yq"][h].double().cpu().numpy()
    yk = r["yk"][h].double().cpu().numpy()
    perm_q = r["perm_q"][h].cpu().numpy()
    perm_k = r["perm_k"][h].cpu().numpy()
    if split == "basic":
        want_q = ref.basic_split(yq, c, head=h, side=0)[0]
        want_k = ref.basic_split(yk, ck, head=h, side=1)[0]
    else:
        want_q, want_k = ref.split(yq, c)[0], ref.split(yk, ck)[0]
    assert np.array_equal(perm_q, want_q), f"head {h}: query permutation"
    assert np.array_equal(perm_k, want_k), f"head {h}: key permutation"
    cq_n, ck_n = G.counts(n_q, c), G.counts(n_k, ck)
    S = scores[h].double().cpu().numpy()
    L = lists[h].cpu().numpy()
    assert np.array_equal(L, ref.topk(S, k)), f"head {h}: lists"
    qbar = ref.centroids(Q, perm_q, cq_n)
    kbar = ref.centroids(K, perm_k, ck_n)
    S_or = ref.centroid_scores(qbar, kbar)
    assert np.abs(S - S_or).max() <= 1e-4 * max(1.0, np.abs(S_or).max()), f"head {h}: scores"
    sample = sample_clusters(len(cq_n), nsample, seed)
    rows, o, l = oracle_rows(Q, K, V, perm_q, perm_k, c, ck, L, sample, tau, comp)
    err = np.abs(out[h][rows] - o).max()
    assert err <= G.TOL[dt], f"head {h}: output error {err}"
    if lse is not None:
        lerr = np.abs(lse[h][rows] - l).max()
        assert lerr <= LSE_TOL[dt], f"head {h}: lse error {lerr}"
    return err
