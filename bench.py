#!/usr/bin/env python3
"""Throughput of the ClusterAttention hot path on one MI355X.

One step = one whole layer: ca_cluster -> ca_select -> ca_attn_compensated
(block-sparse attention and the striped mean compensation in one pass) over
all heads of the tabular-attention workload (batch 1, 8 heads, 65,536 tokens,
d = 64, bf16, clusters of 128, top 1/8 of key clusters, compensation on),
inputs resident in HBM.

Reported value: dense-equivalent attention TFLOP/s = 4 * heads * N^2 * d /
(end-to-end time per layer). Alongside: ms per layer, per-call ms from HIP
events, the roofline position of the dominant kernel (the attention kernel
with its centroid stages, bf16 MFMA), the same layer with the two calls
ca_block_sparse_attn and ca_compensate, and the CPU oracle timed on one head.
The selection modes and the --configs and --sweep tables time the two separate
calls.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = dict(cfg=2, name="tabular-8h-n65536-d64-bf16-c128-keep1/8", heads=8, n=65536, d=64,
                c=128, keep=1 / 8)
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
# HBM bytes per launch of the attention kernel from rocprofv3 FETCH_SIZE and
# WRITE_SIZE, scaled by a plain-copy calibration (see the traffic summary under
# profiles/), valid for the kernel source with this fingerprint only.
ATTN_TRAFFIC = {"fingerprint": "b30eb1a42825b6c0", "bytes": 1.607e+09}


def attn_fingerprint():
    """sha256 over k_attn.hip then attn_tile.h (first 16 hex digits)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("k_attn.hip", "attn_tile.h"):
        with open(os.path.join(ROOT, "paper_2608_26965_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def time_oracle(Q, K, V, c, k):
    """The oracle, as it stands, on one head of the workload (full pipeline)."""
    from oracle import ref
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    t0 = time.perf_counter()
    ref.forward(Q, K, V, c, c, k, "metric", True)
    dt = time.perf_counter() - t0
    return dt, threads


def time_selection_modes(ca, torch, p, q, k, v, keep_k, out, args):
    """The same layer in the other modes, timed after (and apart from) the
    headline run: top-k through the two-pass histogram (at least keep_k
    clusters, metric transform), adaptive assignment (90% of the estimated
    attention mass, at least 16 clusters, adaptive transform) and the
    random-cluster control (random clusters, exact top-k of keep_k) and basic
    recursive splitting (power-iteration directions in the metric root space,
    exact top-k of keep_k). Per call ms (HIP events, mean over the timed
    steps), ms per layer and the mean number of selected key clusters per
    query cluster."""
    res = {}
    for name, xf, floor, recall, split in (
            ("hist_topk", "metric", keep_k, 0.0, "diag"),
            ("adaptive_mass0.9_min16", "adaptive", 16, 0.9, "diag"),
            ("random_clusters_topk", "random", keep_k, None, "diag"),
            ("basic_split_topk", "metric", keep_k, None, "basic")):
        pm = ca.Problem(p.batch, p.heads, p.nq, p.nk, p.d, p.cq, p.ck, p.dtype, xf, p.layout,
                        split=split)
        ws = ca.workspace(pm, q.device, keep_k)
        lens_seen = []

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
            op, lse = ca.block_sparse_attn(pm, r["qp"], r["kp"], r["vp"], r["count_k"], lists,
                                           stride, lens=lens, ws=ws)
            if ev:
                ev[3].record()
            ca.compensate(pm, r["qp"], r["cent_k"], r["cent_v"], r["count_k"], lists, stride, op,
                          lse, r["perm_q"], out=out, ws=ws, lens=lens)
            if ev:
                ev[4].record()
            return lens

        for _ in range(args.warmup):
            step()
        steps = max(3, args.steps // 2)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            lens = step(evs[s])
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        calls = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(4)] for e in evs]).mean(0)
        res[name] = {"transform": xf, "split": split, "min_count": floor,
                     "mass_recall": recall if recall is not None else "exact top-k",
                     "ms_per_step": round(ms, 4),
                     "breakdown_ms": {"cluster": round(calls[0], 4), "select": round(calls[1], 4),
                                      "block_sparse_attn": round(calls[2], 4),
                                      "compensate": round(calls[3], 4)},
                     "mean_clusters": (round(float(lens.float().mean()), 2) if lens is not None
                                       else float(floor))}
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

    for n in SWEEP_N:
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


# Rows of the per-configuration table: (config, cluster size, keep fraction,
# compensation, distinct heads generated). The generated heads are repeated up
# to the configuration's head count (heads are independent units of the
# method, so the work and its shape are those of the full layer; generating
# every head on the host would take minutes).
CONFIG_ROWS = (
    [(1, 64, 0.25, True, 1), (1, 64, 1.0, True, 1), (2, 128, 0.125, True, 8),
     (3, 128, 0.0625, True, 2), (3, 128, 0.25, True, 2), (4, 64, 0.25, True, 4)]
    + [(5, c, keep, comp, 4) for c in (64, 128) for keep in (0.25, 0.125, 0.0625)
       for comp in (True, False)])


def config_table(args):
    """One JSON line per row of CONFIG_ROWS: the whole layer (metric
    transform, exact top-k) timed with HIP events, mean over the timed steps
    after the warm-ups; dense-equivalent TFLOP/s; the attention kernel's
    TFLOP/s on the computed interactions (4 d c_q c_k per query-cluster /
    selected-key-cluster pair) against the bf16 MFMA peak."""
    import torch
    import paper_2608_26965_amd as ca
    from synth import CONFIGS, make_config
    dev = torch.device("cuda:0")
    steps, warmup = max(3, min(args.steps, 10)), max(1, min(args.warmup, 3))
    cache = {}
    for cid, c, keep, comp, gen in CONFIG_ROWS:
        cfg = CONFIGS[cid]
        if cid not in cache:
            cache.clear()
            torch.cuda.empty_cache()
            Qh, Kh, Vh = make_config(cid, heads=list(range(gen)))
            rep = -(-cfg.heads // gen)
            dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
            cache[cid] = tuple(torch.from_numpy(x).to(dev).to(dt).repeat(rep, 1, 1)[:cfg.heads][None]
                               .contiguous() for x in (Qh, Kh, Vh))
        q, k, v = cache[cid]
        H, n, d = q.shape[1:]
        p = ca.Problem(1, H, n, n, d, c, c, q.dtype, "metric", "bhnd")
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

        for _ in range(warmup):
            step()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            step(evs[i])
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        calls = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(4)] for e in evs]).mean(0)
        f_dense = 4.0 * H * n * n * d
        f_attn = 4.0 * d * c * c * keep_k * p.nqc * H
        attn_tf = f_attn / (calls[2] * 1e-3) / 1e12
        # bf16: the same layer with steps 3 and 4 in one pass (ca_attn_compensated)
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
        print(json.dumps({"table": "configs", "config": cfg.name, "heads": H, "n": n, "d": d,
                          "dtype": cfg.dtype, "c": c, "keep": keep, "kept_clusters": keep_k,
                          "key_clusters": p.nkc, "compensation": comp,
                          "distinct_heads_generated": gen, "ms_per_layer": round(ms, 4),
                          "cluster_ms": round(calls[0], 4), "select_ms": round(calls[1], 4),
                          "attention_ms": round(calls[2], 4), "compensation_ms": round(calls[3], 4),
                          "dense_equiv_tflops": round(f_dense / (ms * 1e-3) / 1e12, 1),
                          "attention_tflops": round(attn_tf, 1),
                          "attention_mfma_frac": (round(attn_tf / PEAK_BF16_TFLOPS, 4)
                                                  if cfg.dtype == "bf16" else None),
                          "one_pass": one_pass}),
              flush=True)
        del ws, out


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
    ap.add_argument("--configs", action="store_true",
                    help="every workload configuration (cluster sizes, keep fractions, "
                         "compensation on/off) instead of the headline run: one JSON line each")
    ap.add_argument("--no-modes", action="store_true",
                    help="skip the histogram-selection modes timed after the headline run")
    ap.add_argument("--no-separate", action="store_true",
                    help="skip the two-call layer (ca_block_sparse_attn + ca_compensate) timed "
                         "after the headline run")
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
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: ClusterAttention's heads are independent, so a "
              "multi-GPU layer shards heads with no communication; run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_26965_amd as ca
    from synth import make_config

    W = WORKLOAD
    H, n, d, c = W["heads"], W["n"], W["d"], W["c"]
    Qh, Kh, Vh = make_config(W["cfg"])
    dev = torch.device("cuda:0")
    q = torch.from_numpy(Qh[None]).to(dev).to(torch.bfloat16)
    k = torch.from_numpy(Kh[None]).to(dev).to(torch.bfloat16)
    v = torch.from_numpy(Vh[None]).to(dev).to(torch.bfloat16)
    p = ca.Problem(1, H, n, n, d, c, c, torch.bfloat16, "metric", "bhnd")
    keep_k = ca.keep_to_k(W["keep"], p.nkc)
    ws = ca.workspace(p, dev, keep_k)
    out = torch.empty(p.shape(n), dtype=torch.bfloat16, device=dev)

    def step(ev=None):
        if ev:
            ev[0].record()
        r = ca.cluster(p, q, k, v, ws=ws)
        if ev:
            ev[1].record()
        lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
        if ev:
            ev[2].record()
        ca.attn_compensated(p, r["qp"], r["kp"], r["vp"], r["cent_k"], r["cent_v"], r["count_k"],
                            lists, keep_k, r["perm_q"], out=out, ws=ws)
        if ev:
            ev[3].record()

    def step_separate(ev=None):
        r = ca.cluster(p, q, k, v, ws=ws)
        lists, _ = ca.select(p, r["cent_q"], r["cent_k"], keep_k, ws=ws)
        if ev:
            ev[0].record()
        op, lse = ca.block_sparse_attn(p, r["qp"], r["kp"], r["vp"], r["count_k"], lists, keep_k)
        if ev:
            ev[1].record()
        ca.compensate(p, r["qp"], r["cent_k"], r["cent_v"], r["count_k"], lists, keep_k, op, lse,
                      r["perm_q"], out=out, ws=ws)
        if ev:
            ev[2].record()

    for _ in range(args.warmup):
        step()
    # HIP events on the stream the calls are enqueued on (torch's current
    # stream), one set per step, read back after the timed region.
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    calls = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(3)] for e in evs])
    call_ms = calls.mean(axis=0)
    # the same layer with steps 3 and 4 as two calls (after the timed region)
    sep_ms = None
    if not args.no_separate:
        sep_steps = min(args.steps, 10)
        for _ in range(2):
            step_separate()
        sevs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(sep_steps)]
        for s in range(sep_steps):
            step_separate(sevs[s])
        torch.cuda.synchronize()
        sep_ms = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(2)] for e in sevs]).mean(0)

    f_dense = 4.0 * H * n * n * d
    value = f_dense / (ms_step * 1e-3) / 1e12
    # algorithmic flops of the attention launch: the selected keys, then the
    # unselected clusters' centroids (4 d per query and key either way)
    f_attn = 4.0 * d * c * c * keep_k * p.nqc * H
    f_cent = 4.0 * d * c * (p.nkc - keep_k) * p.nqc * H
    attn_tflops = (f_attn + f_cent) / (call_ms[2] * 1e-3) / 1e12
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
                   "transform": "metric", "compensation": True},
        "breakdown_ms": {"cluster": round(call_ms[0], 4), "select": round(call_ms[1], 4),
                         "attn_compensated": round(call_ms[2], 4)},
        "roofline": {"kernel": "attn_bf16_kernel<64,128,128,fused>", "bound": "mfma",
                     "achieved": round(attn_tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": (ATTN_TRAFFIC["bytes"]
                                 if attn_fingerprint() == ATTN_TRAFFIC["fingerprint"] else None)},
    }
    if sep_ms is not None:
        rec["separate_calls_ms"] = {"block_sparse_attn": round(sep_ms[0], 4),
                                    "compensate": round(sep_ms[1], 4),
                                    "sum": round(sep_ms[0] + sep_ms[1], 4)}
    if not args.no_modes:
        rec["modes"] = time_selection_modes(ca, torch, p, q, k, v, keep_k, out, args)
    if not args.no_cpu_baseline:
        t_head, threads = time_oracle(Qh[0], Kh[0], Vh[0], c, keep_k)
        rec["cpu_baseline"] = {
            "value": round(4.0 * n * n * d / t_head / 1e12, 5), "unit": "TFLOP/s",
            "cores": threads, "kind": "oracle",
            "sample": f"head 0 of {H}, full pipeline (clustering, selection, sparse attention, "
                      f"compensation), fp64 NumPy, {t_head:.1f} s; {cpu_model()}"}
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
