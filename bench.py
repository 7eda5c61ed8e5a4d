#!/usr/bin/env python3
"""Throughput of the ClusterAttention hot path on one MI355X.

One step = one whole layer: ca_cluster -> ca_select -> ca_attn_compensated
(block-sparse attention and the striped mean compensation in one pass) over
all heads of the large tabular-attention workload (batch 1, 16 heads, 262,144
tokens, d = 64, bf16, clusters of 128, top 1/16 of key clusters, compensation
on, metric transform, exact top-k), inputs resident in HBM.

Reported value: dense-equivalent attention TFLOP/s = 4 * heads * N^2 * d /
(end-to-end time per layer). Alongside: ms per layer, per-call ms from HIP
events, the same layer keeping 1/4 of the key clusters, the dense baseline
(this library's attention with every key cluster kept) and the layer's
speedup over it, the roofline position of the dominant kernel (the attention
kernel with its centroid stages, bf16 MFMA) and of the clustering call (HBM),
the same layer with the two calls ca_block_sparse_attn and ca_compensate, the
selection modes, and the CPU oracle timed on a bounded sample of one head.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
       [--no-modes] [--headline-only] [--configs] [--sweep] [--quality]
       [--copy-calibration]
"""
from __future__ import annotations

import argparse
import gc
import json
import math
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = dict(cfg=3, name="tabular-16h-n262144-d64-bf16-c128-keep1/16", heads=16, n=262144,
                d=64, c=128, keep=1 / 16, keep2=1 / 4)
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
# HBM bytes per launch from rocprofv3 FETCH_SIZE and WRITE_SIZE, scaled by a
# plain-copy calibration (FETCH_SIZE x 2, WRITE_SIZE x 1; the traffic summaries
# under profiles/ give the commands), valid for the kernel sources with the
# given fingerprint only (else reported as null).
ATTN_TRAFFIC = {"fingerprint": "4e609afc1da9508f", "bytes": 8.4878e10}
CLUSTER_TRAFFIC = {"fingerprint": "ee7b6a8dec29e18b", "bytes": 1.8445e10}


def _fingerprint(files):
    """sha256 over the given csrc files in order (first 16 hex digits)."""
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2608_26965_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def attn_fingerprint():
    return _fingerprint(("k_attn.hip", "attn_tile.h", "common.h"))


def cluster_fingerprint():
    return _fingerprint(("k_cluster.hip", "common.h"))


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cluster_bytes(heads, n, d, e, c):
    """Algorithmic HBM bytes of one ca_cluster call (both sides, all heads):
    per head and token, moments 2de (q, k read), query representation de,
    projection 2de read + 8d (fp32 split coordinates written, both sides),
    4 + 4 + 4 bytes per split level and side (key and index read, index
    written), permute/gather 6de (q, k, v read and written), permutation and
    cluster ids 16."""
    levels = max(0, math.ceil(math.log2(-(-n // c))))
    return float(heads) * n * (11 * d * e + 8 * d + 24 * levels + 16)


def time_oracle_sample(Q, K, V, c, k, every=2):
    """The oracle, as it stands, on a bounded sample of one head: the whole
    clustering (split spaces and recursive splits of both sides), centroids,
    scores and top-k, then the block-sparse attention and the compensation of
    every ``every``-th query cluster. Returns (measured seconds, estimated
    seconds for the whole head = clustering and selection + every x the
    sampled attention and compensation, threads, sampled clusters)."""
    from oracle import ref
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    Q, K, V = (np.asarray(x, np.float64) for x in (Q, K, V))
    n, d = Q.shape
    tau = 1.0 / math.sqrt(d)
    t0 = time.perf_counter()
    yq = ref.query_split_space(Q, K, "metric")
    yk = ref.key_split_space(Q, K, "metric")
    perm_q, _, cnt_q = ref.split(yq, c)
    perm_k, _, cnt_k = ref.split(yk, c)
    kbar = ref.centroids(K, perm_k, cnt_k)
    vbar = ref.centroids(V, perm_k, cnt_k)
    lists = ref.topk(ref.centroid_scores(ref.centroids(Q, perm_q, cnt_q), kbar), k)
    t1 = time.perf_counter()
    sample = np.arange(0, len(cnt_q), every)
    mem = ref.cluster_members(perm_q, cnt_q)
    rows = np.concatenate([mem[a] for a in sample])
    sub = np.arange(len(rows))
    o_s, l_s = ref.sparse_attention(Q[rows], K, V, sub, cnt_q[sample], perm_k, cnt_k,
                                    lists[sample], tau)
    ref.compensate(Q[rows], kbar, vbar, cnt_k, sub, cnt_q[sample], lists[sample], o_s, l_s, tau)
    t2 = time.perf_counter()
    est = (t1 - t0) + (t2 - t1) * len(cnt_q) / len(sample)
    return t2 - t0, est, threads, len(sample)


def _timed(torch, step, n_ev, steps, warmup):
    """Run step() warmup times, then steps times with n_ev HIP events each
    (recorded by step on the stream the calls are enqueued on); returns (ms
    per step by the host clock between two synchronisations, mean ms between
    consecutive events). Python's garbage collector is run before and kept
    off during the timed steps, so that no collection pause (the host issues
    every launch) lands inside the timed region."""
    for _ in range(warmup):
        step()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(steps)]
    gc.collect()
    gc_was_on = gc.isenabled()
    gc.disable()
    try:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            step(evs[s])
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
    finally:
        if gc_was_on:
            gc.enable()
    calls = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(n_ev - 1)] for e in evs])
    return ms, calls.mean(axis=0)


def time_selection_modes(ca, torch, p, q, k, v, keep_k, out, args):
    """The same layer in the other modes, timed after (and apart from) the
    headline run: top-k through the two-pass histogram (at least keep_k
    clusters, metric transform), adaptive assignment (90% of the estimated
    attention mass, at least 16 clusters, adaptive transform), the
    random-cluster control (random clusters, exact top-k of keep_k) and basic
    recursive splitting (power-iteration directions in the metric root space,
    exact top-k of keep_k); steps 3 and 4 in one pass. Per call ms (HIP
    events, mean over the timed steps), ms per layer and the mean number of
    selected key clusters per query cluster."""
    res = {}
    for name, xf, floor, recall, split in (
            ("hist_topk", "metric", keep_k, 0.0, "diag"),
            ("adaptive_mass0.9_min16", "adaptive", 16, 0.9, "diag"),
            ("random_clusters_topk", "random", keep_k, None, "diag"),
            ("basic_split_topk", "metric", keep_k, None, "basic")):
        pm = ca.Problem(p.batch, p.heads, p.nq, p.nk, p.d, p.cq, p.ck, p.dtype, xf, p.layout,
                        split=split)
        ws = ca.workspace(pm, q.device, keep_k)
        seen = {}

        def step(ev=None):
            if ev:
                ev[0].record()
            r = ca.cluster(pm, q, k, v, ws=ws)
            if ev:
                ev[1].record()
            if recall is None:  # exact top-k
                lists, _ = ca.select(pm, r["cent_q"], r["cent_k"], floor, ws=ws)
                lens, stride = None, floor
            else:
                lists, lens, _ = ca.select_hist(pm, r["cent_q"], r["cent_k"], r["count_k"], floor,
                                                recall, ws=ws)
                stride = pm.nkc
            if ev:
                ev[2].record()
            ca.attn_compensated(pm, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"],
                                r["count_k"], lists, stride, r["perm_q"], out=out, ws=ws,
                                lens=lens)
            if ev:
                ev[3].record()
            seen["lens"] = lens

        ms, calls = _timed(torch, step, 4, max(3, args.steps // 2), args.warmup)
        lens = seen["lens"]
        res[name] = {"transform": xf, "split": split, "min_count": floor,
                     "mass_recall": recall if recall is not None else "exact top-k",
                     "ms_per_step": round(ms, 4),
                     "breakdown_ms": {"cluster": round(calls[0], 4), "select": round(calls[1], 4),
                                      "attn_compensated": round(calls[2], 4)},
                     "mean_clusters": (round(float(lens.float().mean()), 2) if lens is not None
                                       else float(floor))}
        del ws
    return res


SWEEP_N = (8192, 16384, 32768, 65536, 131072, 262144, 524288, 1048576)


def latency_sweep(args):
    """Latency scaling with the number of tokens (the paper's latency-scaling
    experiment): 8 heads, d = 64, bf16, c = 128, metric transform, exact top-k,
    compensation on; k fixed to 64 clusters (8192 keys) or set to 10% of the
    key clusters; and, with k fixed, basic recursive splitting in the metric
    root space (power iteration per node, no eigendecomposition). Inputs: the tabular recipe (per head 64 mixture centres
    N(0, I), Dirichlet(1) weights, queries and keys drawn from the mixture
    with sigma 0.5 and independent labels, values N(0, 1)), drawn on the GPU
    with torch's generator seeded by N (the host generator would take minutes
    at a million tokens), rounded to bf16. Per call ms: HIP events, mean over
    the timed steps after the warm-up."""
    import torch
    import paper_2608_26965_amd as ca
    H, d, c = 8, 64, 128
    dev = torch.device("cuda:0")
    steps, warmup = max(2, min(args.steps, 5)), max(1, min(args.warmup, 2))

    def mixture(n, g):
        mu = torch.randn(H, 64, d, device=dev, generator=g)
        w = -torch.log(torch.rand(H, 64, device=dev, generator=g))  # Dirichlet(1) via Exp(1)
        w = w / w.sum(dim=1, keepdim=True)
        xs = []
        for _ in range(2):  # queries, keys: independent labels, shared centres
            lab = torch.multinomial(w, n, replacement=True, generator=g)
            x = torch.gather(mu, 1, lab[..., None].expand(H, n, d))
            xs.append((x + 0.5 * torch.randn(H, n, d, device=dev, generator=g))
                      .to(torch.bfloat16)[None].contiguous())
        v = torch.randn(H, n, d, device=dev, generator=g).to(torch.bfloat16)[None].contiguous()
        return xs[0], xs[1], v

    for n in (args.sweep_sizes or SWEEP_N):
        g = torch.Generator(device=dev)
        g.manual_seed(n)
        q, k, v = mixture(n, g)
        out = None
        for rule, split in (("k64", "diag"), ("keep10pct", "diag"), ("k64", "basic")):
            p = ca.Problem(1, H, n, n, d, c, c, torch.bfloat16, "metric", "bhnd", split=split)
            if out is None:
                out = torch.empty(p.shape(n), dtype=torch.bfloat16, device=dev)
            keep_k = min(64, p.nkc) if rule == "k64" else ca.keep_to_k(0.1, p.nkc)
            ws = ca.workspace(p, dev, keep_k)

            def step(ev=None):
                if ev:
                    ev[0].record()
                r = ca.cluster(p, q, k, v, ws=ws)
                if ev:
                    ev[1].record()
                lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
                if ev:
                    ev[2].record()
                op, lse = ca.block_sparse_attn(p, r["qp"], r["kp"], r["vp"], r["count_k"], lists,
                                               keep_k)
                if ev:
                    ev[3].record()
                ca.compensate(p, r["qp"], r["cent_k"], r["cent_v"], r["count_k"], lists, keep_k,
                              op, lse, r["perm_q"], out=out, ws=ws)
                if ev:
                    ev[4].record()

            for _ in range(warmup):
                step()
            evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(steps):
                step(evs[i])
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3 / steps
            calls = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(4)]
                              for e in evs]).mean(0)
            f_dense = 4.0 * H * n * n * d

            # the same layer with steps 3 and 4 in one pass (ca_attn_compensated)
            def step1(ev=None):
                r = ca.cluster(p, q, k, v, ws=ws)
                lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
                if ev:
                    ev[0].record()
                ca.attn_compensated(p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"],
                                    r["count_k"], lists, keep_k, r["perm_q"], out=out, ws=ws)
                if ev:
                    ev[1].record()

            for _ in range(warmup):
                step1()
            ev1 = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            for i in range(steps):
                step1(ev1[i])
            torch.cuda.synchronize()
            one_pass = {"ms_per_layer": round((time.perf_counter() - t1) * 1e3 / steps, 4),
                        "attn_compensated_ms": round(float(np.mean(
                            [e[0].elapsed_time(e[1]) for e in ev1])), 4)}
            print(json.dumps({"sweep": "latency_scaling", "n": n, "rule": rule, "split": split,
                              "one_pass": one_pass,
                              "kept_clusters":
                              keep_k, "key_clusters": p.nkc, "ms_per_layer": round(ms, 4),
                              "cluster_ms": round(calls[0], 4), "select_ms": round(calls[1], 4),
                              "attention_ms": round(calls[2], 4),
                              "compensation_ms": round(calls[3], 4),
                              "dense_equiv_tflops": round(f_dense / (ms * 1e-3) / 1e12, 1)}),
                  flush=True)
            del ws
        del q, k, v, out
        torch.cuda.empty_cache()


# Rows of the per-configuration table: (config, query cluster size, key
# cluster size, keep fraction, compensation). Every head of a configuration
# is generated (in parallel processes, before the GPU is used).
CONFIG_ROWS = (
    [(1, 64, 64, 0.25, True), (1, 64, 64, 1.0, True), (2, 128, 128, 0.125, True),
     (3, 128, 128, 0.0625, True), (3, 128, 128, 0.25, True), (4, 64, 64, 0.25, True)]
    + [(5, c, c, keep, comp) for c in (64, 128) for keep in (0.25, 0.125, 0.0625)
       for comp in (True, False)]
    # the paper's evaluated tile shape: query clusters of 64, key clusters of 128
    + [(2, 64, 128, 0.125, True), (5, 64, 128, 0.125, True)])


def config_table(args):
    """One JSON line per row of CONFIG_ROWS: the whole layer (metric
    transform, exact top-k) timed with HIP events, mean over the timed steps
    after the warm-ups, with steps 3 and 4 as two calls and (bf16) as the one
    pass; dense-equivalent TFLOP/s; the attention kernel's TFLOP/s on the
    computed interactions (4 d c_q c_k per query-cluster / selected
    key-cluster pair) against the bf16 MFMA peak."""
    from synth import CONFIGS, make_config
    workers = min(16, os.cpu_count() or 1)
    host = {}
    for cid in sorted({row[0] for row in CONFIG_ROWS}):
        host[cid] = make_config(cid, workers=workers)
    import torch
    import paper_2608_26965_amd as ca
    dev = torch.device("cuda:0")
    steps, warmup = max(3, min(args.steps, 10)), max(1, min(args.warmup, 3))
    cache = {}
    for cid, cq, ck, keep, comp in CONFIG_ROWS:
        cfg = CONFIGS[cid]
        if cid not in cache:
            cache.clear()
            torch.cuda.empty_cache()
            dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
            cache[cid] = tuple(torch.from_numpy(x[None]).to(dev).to(dt) for x in host[cid])
        q, k, v = cache[cid]
        H, n, d = q.shape[1:]
        p = ca.Problem(1, H, n, n, d, cq, ck, q.dtype, "metric", "bhnd")
        keep_k = ca.keep_to_k(keep, p.nkc)
        ws = ca.workspace(p, dev, keep_k)
        out = torch.empty(p.shape(n), dtype=q.dtype, device=dev)

        def step(ev=None):
            if ev:
                ev[0].record()
            r = ca.cluster(p, q, k, v, ws=ws)
            if ev:
                ev[1].record()
            lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
            if ev:
                ev[2].record()
            op, lse = ca.block_sparse_attn(p, r["qp"], r["kp"], r["vp"], r["count_k"], lists,
                                           keep_k)
            if ev:
                ev[3].record()
            ca.compensate(p, r["qp"], r["cent_k"], r["cent_v"], r["count_k"], lists, keep_k, op,
                          lse, r["perm_q"], enable=comp, out=out, ws=ws)
            if ev:
                ev[4].record()

        ms, calls = _timed(torch, step, 5, steps, warmup)
        f_dense = 4.0 * H * n * n * d
        f_attn = 4.0 * d * cq * ck * keep_k * p.nqc * H
        attn_tf = f_attn / (calls[2] * 1e-3) / 1e12
        one_pass = None
        if cfg.dtype == "bf16":
            def step1(ev=None):
                r = ca.cluster(p, q, k, v, ws=ws)
                lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
                if ev:
                    ev[0].record()
                ca.attn_compensated(p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"],
                                    r["count_k"], lists, keep_k, r["perm_q"], enable=comp,
                                    out=out, ws=ws)
                if ev:
                    ev[1].record()

            ms1, c1 = _timed(torch, step1, 2, steps, warmup)
            one_pass = {"ms_per_layer": round(ms1, 4), "attn_compensated_ms": round(c1[0], 4)}
        print(json.dumps({"table": "configs", "config": cfg.name, "heads": H, "n": n, "d": d,
                          "dtype": cfg.dtype, "cq": cq, "ck": ck, "keep": keep,
                          "kept_clusters": keep_k, "key_clusters": p.nkc, "compensation": comp,
                          "distinct_heads_generated": H, "ms_per_layer": round(ms, 4),
                          "cluster_ms": round(calls[0], 4), "select_ms": round(calls[1], 4),
                          "attention_ms": round(calls[2], 4), "compensation_ms": round(calls[3], 4),
                          "dense_equiv_tflops": round(f_dense / (ms * 1e-3) / 1e12, 1),
                          "attention_tflops": round(attn_tf, 1),
                          "attention_mfma_frac": (round(attn_tf / PEAK_BF16_TFLOPS, 4)
                                                  if cfg.dtype == "bf16" else None),
                          "one_pass": one_pass}),
              flush=True)
        del ws, out


# Rows of the quality table: (config, cluster size, keep fraction, transform).
QUALITY_ROWS = (
    [(2, 128, 1 / 8, "metric"), (2, 128, 1 / 8, "random"),
     (3, 128, 1 / 16, "metric"), (3, 128, 1 / 4, "metric"), (3, 128, 1 / 16, "random"),
     (4, 64, 1 / 4, "metric"), (4, 64, 1 / 4, "random")]
    + [(5, c, keep, "metric") for c in (64, 128) for keep in (1 / 4, 1 / 8, 1 / 16)]
    + [(5, 128, 1 / 8, "random")])


def quality_table(args):
    """How close the layer's output is to dense attention (the paper's
    measure of the approximation: output similarity to the exact softmax
    attention). Per row of QUALITY_ROWS, two generated heads run through the
    layer (exact top-k, steps 3 and 4 in one pass) with compensation on and
    off; for 512 sampled queries per head the exact dense attention output is
    formed in fp32 on the GPU (scores against every key, softmax, values),
    and the JSON line gives the relative L2 error ||o - o_dense|| /
    ||o_dense|| over the sampled rows, the mean per-row relative error and
    the mean cosine similarity of the rows."""
    from synth import CONFIGS, make_config
    import torch
    import paper_2608_26965_amd as ca
    dev = torch.device("cuda:0")
    cache = {}
    for cid, c, keep, xf in QUALITY_ROWS:
        if cid not in cache:
            cache.clear()
            torch.cuda.empty_cache()
            cache[cid] = tuple(torch.from_numpy(x[None]).to(dev).to(torch.bfloat16)
                               for x in make_config(cid, heads=[0, 1]))
        q, k, v = cache[cid]
        H, n, d = q.shape[1:]
        p = ca.Problem(1, H, n, n, d, c, c, torch.bfloat16, xf, "bhnd")
        keep_k = ca.keep_to_k(keep, p.nkc)
        ws = ca.workspace(p, dev, keep_k)
        r = ca.cluster(p, q, k, v, ws=ws)
        lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
        g = torch.Generator(device="cpu").manual_seed(cid * 1000 + c)
        rows = torch.randint(0, n, (H, 512), generator=g).to(dev)
        dense = []
        for h in range(H):
            qs = q[0, h, rows[h]].float()
            s = (qs @ k[0, h].float().T) / math.sqrt(d)
            dense.append(torch.softmax(s, dim=1) @ v[0, h].float())
        dense = torch.stack(dense)
        res = {}
        for comp in (True, False):
            out, _ = ca.attn_compensated(p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"],
                                         r["count_k"], lists, keep_k, r["perm_q"], enable=comp,
                                         ws=ws)
            got = torch.stack([out[0, h, rows[h]].float() for h in range(H)])
            err = (got - dense).flatten(0, 1)
            ref_rows = dense.flatten(0, 1)
            got_rows = got.flatten(0, 1)
            res["compensated" if comp else "uncompensated"] = {
                "rel_l2": round(float(err.norm() / ref_rows.norm()), 5),
                "mean_row_rel_l2": round(float((err.norm(dim=1) / ref_rows.norm(dim=1)).mean()), 5),
                "mean_cosine": round(float(torch.nn.functional.cosine_similarity(
                    got_rows, ref_rows, dim=1).mean()), 5)}
        print(json.dumps({"table": "quality_vs_dense", "config": CONFIGS[cid].name, "n": n,
                          "d": d, "c": c, "keep": keep, "kept_clusters": keep_k,
                          "key_clusters": p.nkc, "transform": xf, "heads_sampled": H,
                          "rows_per_head": 512, **res}), flush=True)
        del ws, r, lists


def copy_calibration():
    """A plain device copy of 256 MiB (fp32), three launches."""
    import torch
    n = 256 * 1024 * 1024 // 4
    src = torch.randn(n, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {n * 4 // 1024} KiB per launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", action="store_true",
                    help="latency scaling with the token count instead of the headline run: one "
                         "JSON line per (N, rule), k = 64 clusters or 10%% of the key clusters")
    ap.add_argument("--sweep-sizes", type=lambda x: [int(t) for t in x.split(",")], default=None,
                    help="token counts of the sweep (comma-separated; default: 8192 to 1048576)")
    ap.add_argument("--configs", action="store_true",
                    help="every workload configuration (cluster sizes, keep fractions, "
                         "compensation on/off) instead of the headline run: one JSON line each")
    ap.add_argument("--no-modes", action="store_true",
                    help="skip the selection modes timed after the headline run")
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the headline layer (no keep-1/4 layer, dense baseline, "
                         "two-call layer, modes or CPU baseline): the profiling runs use it, so "
                         "that the attention kernel's launches are all the headline's")
    ap.add_argument("--quality", action="store_true",
                    help="output quality against dense attention per configuration instead of "
                         "the headline run: one JSON line each")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy three times: the known-size "
                         "reference that scales the FETCH_SIZE / WRITE_SIZE counters")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.sweep:
        latency_sweep(args)
        return
    if args.configs:
        config_table(args)
        return
    if args.quality:
        quality_table(args)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: ClusterAttention's heads are independent, so a "
              "multi-GPU layer shards heads with no communication; run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    from synth import make_config
    W = WORKLOAD
    H, n, d, c = W["heads"], W["n"], W["d"], W["c"]
    # Every head drawn on the host (forked workers, before anything touches the GPU).
    t_gen = time.perf_counter()
    Qh, Kh, Vh = make_config(W["cfg"], workers=min(16, os.cpu_count() or 1))
    t_gen = time.perf_counter() - t_gen
    print(f"inputs: {H} heads drawn in {t_gen:.1f} s", file=sys.stderr, flush=True)

    import torch
    import paper_2608_26965_amd as ca

    dev = torch.device("cuda:0")
    q, k, v = (torch.from_numpy(x[None]).to(dev).to(torch.bfloat16) for x in (Qh, Kh, Vh))
    head0 = (Qh[0].copy(), Kh[0].copy(), Vh[0].copy())
    del Qh, Kh, Vh
    p = ca.Problem(1, H, n, n, d, c, c, torch.bfloat16, "metric", "bhnd")
    ws = ca.workspace(p, dev, p.nkc)
    out = torch.empty(p.shape(n), dtype=torch.bfloat16, device=dev)
    f_dense = 4.0 * H * n * n * d

    def layer(keep_k):
        def step(ev=None):
            if ev:
                ev[0].record()
            r = ca.cluster(p, q, k, v, ws=ws)
            if ev:
                ev[1].record()
            lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
            if ev:
                ev[2].record()
            ca.attn_compensated(p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"],
                                r["count_k"], lists, keep_k, r["perm_q"], out=out, ws=ws)
            if ev:
                ev[3].record()
        return step

    def attn_flops(keep_k):
        # algorithmic flops of the attention launch: the selected keys, then
        # the unselected clusters' centroids (4 d per query and key either way)
        return (4.0 * d * c * c * keep_k * p.nqc * H
                + 4.0 * d * c * (p.nkc - keep_k) * p.nqc * H)

    keep_k = ca.keep_to_k(W["keep"], p.nkc)
    # headline: warm-up, then exactly K timed steps between two synchronisations
    ms_step, call_ms = _timed(torch, layer(keep_k), 4, args.steps, args.warmup)
    print(f"headline: {ms_step:.3f} ms per layer", file=sys.stderr, flush=True)
    value = f_dense / (ms_step * 1e-3) / 1e12
    attn_tflops = attn_flops(keep_k) / (call_ms[2] * 1e-3) / 1e12
    cl_bytes = cluster_bytes(H, n, d, 2, c)
    cl_gbs = cl_bytes / (call_ms[0] * 1e-3) / 1e9
    rec = {
        "metric": "dense-equivalent attention TFLOP/s + end-to-end ms/layer (clustering incl.)",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": W["name"], "batch": 1, "heads": H, "seq_len": n, "head_dim": d,
                   "cluster_size": c, "keep": W["keep"], "kept_clusters": keep_k,
                   "key_clusters": p.nkc, "transform": "metric", "selection": "exact top-k",
                   "compensation": True},
        "breakdown_ms": {"cluster": round(call_ms[0], 4), "select": round(call_ms[1], 4),
                         "attn_compensated": round(call_ms[2], 4)},
        "roofline": {"kernel": "attn_bf16_kernel<64,128,128,fused>", "bound": "mfma",
                     "achieved": round(attn_tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": (ATTN_TRAFFIC["bytes"]
                                 if attn_fingerprint() == ATTN_TRAFFIC["fingerprint"] else None)},
        "cluster_roofline": {"call": "ca_cluster", "bound": "hbm", "algorithmic_bytes": cl_bytes,
                             "achieved": round(cl_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                             "frac": round(cl_gbs / PEAK_HBM_GBS, 4),
                             "traffic": (CLUSTER_TRAFFIC["bytes"]
                                         if cluster_fingerprint() == CLUSTER_TRAFFIC["fingerprint"]
                                         else None)},
    }
    if not args.headline_only:
        # the same layer keeping 1/4 of the key clusters
        keep2 = ca.keep_to_k(W["keep2"], p.nkc)
        ms2, c2 = _timed(torch, layer(keep2), 4, max(3, args.steps // 2), 1)
        a2 = attn_flops(keep2) / (c2[2] * 1e-3) / 1e12
        rec["keep_1/4"] = {"kept_clusters": keep2, "ms_per_layer": round(ms2, 4),
                           "dense_equiv_tflops": round(f_dense / (ms2 * 1e-3) / 1e12, 2),
                           "breakdown_ms": {"cluster": round(c2[0], 4), "select": round(c2[1], 4),
                                            "attn_compensated": round(c2[2], 4)},
                           "attention_tflops": round(a2, 2),
                           "attention_mfma_frac": round(a2 / PEAK_BF16_TFLOPS, 4)}
        # dense baseline: this library's attention with every key cluster kept
        # (the exact dense softmax; compensation has nothing to add), on the
        # clustered layout, no clustering or selection
        r = ca.cluster(p, q, k, v, ws=ws)
        all_lists = torch.arange(p.nkc, dtype=torch.int32, device=dev).expand(
            H, p.nqc, p.nkc).contiguous()

        def dense_step(ev=None):
            if ev:
                ev[0].record()
            ca.attn_compensated(p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"],
                                r["count_k"], all_lists, p.nkc, r["perm_q"], out=out, ws=ws)
            if ev:
                ev[1].record()

        ms_d, c_d = _timed(torch, dense_step, 2, 3, 1)
        f_all = 4.0 * d * c * c * p.nkc * p.nqc * H
        rec["dense_baseline"] = {
            "what": "ca_attn_compensated with all key clusters kept (exact dense attention)",
            "ms_per_layer": round(c_d[0], 4),
            "dense_tflops": round(f_dense / (c_d[0] * 1e-3) / 1e12, 2),
            "attention_mfma_frac": round(f_all / (c_d[0] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "speedup_keep_1/16": round(c_d[0] / ms_step, 3),
            "speedup_keep_1/4": round(c_d[0] / ms2, 3)}
        del all_lists, r
        # steps 3 and 4 as the two calls ca_block_sparse_attn + ca_compensate
        def step_separate(ev=None):
            r = ca.cluster(p, q, k, v, ws=ws)
            lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
            if ev:
                ev[0].record()
            op, lse = ca.block_sparse_attn(p, r["qp"], r["kp"], r["vp"], r["count_k"], lists,
                                           keep_k)
            if ev:
                ev[1].record()
            ca.compensate(p, r["qp"], r["cent_k"], r["cent_v"], r["count_k"], lists, keep_k, op,
                          lse, r["perm_q"], out=out, ws=ws)
            if ev:
                ev[2].record()

        _, sep = _timed(torch, step_separate, 3, min(args.steps, 10), 2)
        rec["separate_calls_ms"] = {"block_sparse_attn": round(sep[0], 4),
                                    "compensate": round(sep[1], 4),
                                    "sum": round(sep[0] + sep[1], 4)}
        if not args.no_modes:
            rec["modes"] = time_selection_modes(ca, torch, p, q, k, v, keep_k, out, args)
        if not args.no_cpu_baseline:
            measured, est, threads, ns = time_oracle_sample(*head0, c, keep_k)
            rec["cpu_baseline"] = {
                "value": round(4.0 * n * n * d / est / 1e12, 5), "unit": "TFLOP/s",
                "cores": threads, "kind": "oracle",
                "sample": (f"head 0 of {H}: whole clustering (split spaces and splits of both "
                           f"sides), centroids, scores and top-k, then block-sparse attention and "
                           f"compensation of every 2nd query cluster ({ns} of {p.nqc}), fp64 "
                           f"NumPy; {measured:.1f} s measured, {est:.1f} s estimated for the "
                           f"whole head (attention and compensation scaled x{p.nqc / ns:g}); "
                           f"value = 4 n^2 d of one head / that estimate; {cpu_model()}")}
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
