#!/usr/bin/env python3
"""Benchmark of cluster-level sparse prefill (the Similarity Chunk Rolling hot path) on one MI355X.

One step = one whole layer through the C ABI: representative keys -> cluster selection (anchor
fingerprints, logits, soft-voting top-k) -> block-sparse attention, over synthetic
topic-structured inputs already resident in HBM. The default workload is one Llama-3-8B-shaped
attention layer (32 query / 8 KV heads, head dim 128) at a 131072-token context, KV blocks of
128, sub-chunks of 512, clusters of 8 sub-chunks, top-32 blocks + 128 sink tokens + a 4096-token
local window.

Prints ONE JSON line (rank 0) with the throughput, the roofline of the dominant kernel
(attention, bf16 MFMA), HBM rates of the selection kernels, retrieval-call counts and the fp64
oracle timed on a bounded sample on the host's cores.

Other modes (one JSON line each, no CPU baseline unless stated): --sweep over cluster sizes,
--theta / --theta-sweep with clusters formed on the GPU by anchor-based clustering, --tokens K
for token-level selection with a budget of K tokens, and the selection variants --rep-bounds,
--kv-sets and --score-scale.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sparse-prefill tokens/s at 128K ctx (1 GPU); MFMA util %; retrieval calls"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
PEAK_FP64_TFLOPS = 78.6       # MI355X fp64 vector

# The paper's own figures for this step (Sec. 6.1: the prefill stage breakdown and the RULER
# time-to-first-token table). Whole-model, token-level selection, real data, other hardware:
# context for the reader, not a target of this measurement.
PAPER_CONTEXT = {
    "hardware": "1x NVIDIA H100 80GB HBM3, bf16, SGLang + FlashInfer; Qwen2-7B-Instruct (28 layers), "
                "token-level TokenSelect selection, L_outer 8192, sub-chunk 512, SCR theta 0.95, L_max 4096",
    "retrieval_calls": {"per_sub_chunk": 8959, "scr": 1165, "workload": "InfiniteBench R.KV, 30 samples"},
    "retrieval_time_s": {"per_sub_chunk": 4.5, "scr": 0.9, "workload": "InfiniteBench R.KV, per sample"},
    "ttft_s": {"per_sub_chunk": 13.1, "scr": 8.3, "workload": "InfiniteBench R.KV, instrumented run"},
    "ruler_128k_ttft_s": {"per_sub_chunk": 9.89, "scr": 6.64, "workload": "RULER 128K, 8 NIAH tasks x 100 samples"},
    "note": "context only: whole-model TTFT on other hardware; this bench times the attention path of one layer",
}


# Default warm-up: enough steps for about half a second of GPU work. The clocks of a GPU that has
# just started working settle within a few hundred milliseconds; a timed region that starts
# earlier measures the ramp.
WARMUP_S = 0.5


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed warm-up steps (default: at least 3, and at least %.1f s of them)" % WARMUP_S)
    ap.add_argument("--workload", default="llama128k")
    ap.add_argument("--cluster", type=int, default=0, help="cluster size in sub-chunks (0: the workload's)")
    ap.add_argument("--sweep", default="", help="comma-separated cluster sizes; one JSON line each")
    ap.add_argument("--theta", type=float, default=None,
                    help="form the clusters on the GPU by anchor-based similarity clustering at this threshold "
                         "(each step) instead of fixed runs of --cluster sub-chunks")
    ap.add_argument("--theta-sweep", default="", help="comma-separated thresholds; one JSON line each")
    ap.add_argument("--l-max", type=int, default=0, help="cluster cap in tokens for --theta (0: 8 sub-chunks)")
    ap.add_argument("--outer", type=int, default=0, help="outer chunk in sub-chunks for --theta (0: whole context)")
    ap.add_argument("--overlap", action="store_true",
                    help="also report the top-k overlap ratio (Eq. 7) of the clusters against per-sub-chunk selection")
    ap.add_argument("--tokens", type=int, default=0,
                    help="token-level selection with this budget in tokens (0: block-level selection)")
    ap.add_argument("--rep-bounds", action="store_true",
                    help="score blocks by their channel-wise key bounds (min / max) instead of the mean key")
    ap.add_argument("--kv-sets", action="store_true", help="one selected set per (cluster, KV head)")
    ap.add_argument("--score-scale", type=float, default=0.0, help="selection logit scale sigma (0: 1)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-tiles", type=int, default=2,
                    help="least row chunks (the oracle's own 512-row chunks of a cluster) in its attention sample")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="the oracle's attention sample grows by tiles until it has run this long")
    ap.add_argument("--cpu-full", action="store_true",
                    help="time the oracle on the whole layer instead of a bounded sample (about 100 s for the "
                         "128K layer on 16 cores)")
    ap.add_argument("--out-bf16", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only copy 1 GiB device to device (reference for HBM byte counters) and exit")
    ap.add_argument("--gemm-probe", type=float, default=0.0, metavar="SECONDS",
                    help="only run a dense 8192^3 bf16 library GEMM for SECONDS and print its TFLOP/s (the "
                         "MFMA rate the chip sustains at its power limit, a reference for the attention "
                         "roofline) and exit")
    return ap.parse_args(argv)


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "attention_traffic_llama128k.md")
COUNTER_PROFILE = os.path.join(ROOT, "profiles", "attention_counters_llama128k.md")
POWER_PROFILE = os.path.join(ROOT, "profiles", "clock_power_mi355x.md")
ORACLE_FULL_PROFILE = os.path.join(ROOT, "profiles", "oracle_full_layer_llama128k.md")


def profile_block(path):
    """The JSON block of a committed rocprofv3 summary (taken on the default 128K layer), or None
    when the file is missing or the counters were taken on other kernel source."""
    import hashlib
    import re

    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    block = json.loads(m.group(1))
    if "kernel_source" not in block:
        return block
    src = os.path.join(ROOT, block["kernel_source"])
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != block["kernel_source_sha256"]:
        return None
    return block


def measured_traffic():
    """HBM bytes per attention launch from the FETCH_SIZE / WRITE_SIZE summary, scaled by the
    copy-probe factors."""
    block = profile_block(TRAFFIC_PROFILE)
    return int(block["traffic_bytes"]) if block else None


def library_gemm_reference(achieved):
    """The bf16 rate a dense library GEMM sustains on this part at its power limit (committed
    measurement, `--gemm-probe`), and the attention rate as a fraction of it: context for the
    nominal-peak fraction, not a replacement for it."""
    block = profile_block(POWER_PROFILE)
    if not block:
        return None
    ref = float(block["library_gemm_tflops"])
    return {"tflops": ref, "frac": round(achieved / ref, 4), "what": block["library_gemm"],
            "clock_mhz": block["library_gemm_clock_mhz"],
            "source": os.path.relpath(POWER_PROFILE, ROOT)}


def counted_mfma(alg_flops, launch_ms):
    """Executed MFMA work per attention launch from the SQ counter summary: FLOPs from
    SQ_INSTS_MFMA (masked and padded products included), their ratio to the algorithmic FLOPs,
    and their rate over the live launch time against the bf16 peak."""
    block = profile_block(COUNTER_PROFILE)
    if not block or launch_ms <= 0:
        return None
    flops = float(block["mfma_flops_per_dispatch"])
    return {"flops": flops, "per_algorithmic": round(flops / alg_flops, 4),
            "frac": round(flops / (launch_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "mfma_busy": block["mfma_busy_fraction"], "clock_ghz": block["clock_ghz"]}


def counters_apply(args, w, c, theta, tokens):
    """The committed counter summaries describe the default attention launch of the 128K layer
    only: block-level selection with fixed clusters of the workload's size, mean representative
    keys, one set per cluster, σ = 1 and fp32 output."""
    import gen

    return (w.name == "llama128k" and theta is None and not tokens and not args.kv_sets and not args.rep_bounds
            and not args.score_scale and not args.out_bf16 and c == gen.WORKLOADS[w.name].cluster)


def geometry_work(w, geo, tokens=False, bounds=False):
    """Algorithmic attention FLOPs and the selection-side bytes from the cluster geometry.

    Attention: 4 d Hq per (query row, visible key) pair (two products of 2 d FLOP), over
    exactly the keys of Eq. 10 -- masked pairs are not work. With token-level selection, n_cand
    and sel_cnt count tokens.
    """
    B, d, Hq, Hkv = w.block_size, w.head_dim, w.num_q_heads, w.num_kv_heads
    pairs = 0
    for s, e, lo_blk, sink_eff, n_cand, sel_cnt in geo.tolist():
        rows = e - s
        fixed = sink_eff * B + sel_cnt * (1 if tokens else B)
        base = lo_blk * B
        pairs += rows * fixed + (sum(range(s - base + 1, e - base + 1)))
    n_clusters = len(geo)
    nb = w.n_tokens // B
    anchor_rows = sum(min(e, s + w.sub_chunk) - s for s, e, *_ in geo.tolist())
    n_cand = int(geo[:, 4].sum())
    if tokens:
        max_cand = int(geo[:, 4].max()) if len(geo) else 0
        n_sel = int(geo[:, 5].sum())
        return {
            "attention_flops": 4.0 * d * Hq * pairs,
            "pairs": pairs,
            "fingerprint_bytes": anchor_rows * Hq * d * 2 + n_clusters * Hq * d * 4,
            # every candidate key read once, and one logit (2 d FLOP) per (cluster, head, token)
            "token_logits_bytes": max_cand * Hkv * d * 2,
            "token_logits_flops": 2.0 * d * Hq * n_cand,
            "vote_bytes": n_cand * Hkv * 4,
            "gather_bytes": 2 * 2 * n_sel * Hkv * d * 2,
        }
    rep = 2 if bounds else 1        # bound form: channel-wise minimum and maximum per block
    return {
        "attention_flops": 4.0 * d * Hq * pairs,
        "pairs": pairs,
        "rep_keys_bytes": w.n_tokens * Hkv * d * 2 + rep * nb * Hkv * d * 4,
        "fingerprint_bytes": anchor_rows * Hq * d * 2 + n_clusters * Hq * d * 4,
        "logits_bytes": rep * n_cand * Hkv * d * 4 + n_cand * Hq * 4 + n_clusters * Hq * d * 4,
        "logits_flops": 2.0 * d * Hq * n_cand * rep,
        "vote_bytes": n_cand * Hq * 4,
    }


ORACLE_CHUNK = 512   # rows per call of the oracle's own full-layer attention (its cluster_attention)


def cpu_full_layer(w, data, cs):
    """The fp64 oracle as it stands on the whole of layer 0 (every cluster's selection and every
    row's attention, oracle.prefill), timed end to end; multiplied by the layer count."""
    import threadpoolctl

    import oracle

    info = threadpoolctl.threadpool_info()
    cores = max([i.get("num_threads", 1) for i in info] or [1])
    t0 = time.perf_counter()
    oracle.prefill(data["q"], data["k_pages"], data["v_pages"], data["block_table"], w.n_tokens,
                   sub_chunk=w.sub_chunk, block_size=w.block_size, top_k=w.top_k, sink_tokens=w.sink_tokens,
                   local_window=w.local_window, cluster_start=cs)
    t = time.perf_counter() - t0
    return {
        "value": w.n_tokens / (t * w.layers),
        "unit": "tokens/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"full layer: fp64 numpy oracle on every cluster and every row of layer 0 ({w.n_tokens} tokens), "
                  f"x{w.layers} layers",
        "seconds_measured": round(t, 2),
    }


def cpu_baseline(w, data, cs, geo, min_tiles, min_seconds, n_sel_clusters=32, seed=0):
    """The fp64 oracle as it stands, timed on a bounded sample of one layer and scaled to the
    workload: representative keys of the blocks the sampled clusters score (scaled by block
    count), selection for up to `n_sel_clusters` clusters (all of them when there are no more;
    else the first, the last and random ones, scaled by anchor rows + candidates, the two terms
    its cost is linear in), and attention for random row chunks of the sampled clusters, each one
    of the oracle's own chunks (up to 512 rows from the cluster start, as its full-layer pass
    takes them; scaled by visible (row, key) pairs): at least `min_tiles` chunks, and more until
    the attention sample has run `min_seconds`, so the sample is seconds of CPU work on any host.
    Every layer has the same geometry, so the layer time is multiplied by the layer count."""
    import numpy as np
    import threadpoolctl

    import oracle

    info = threadpoolctl.threadpool_info()
    cores = max([i.get("num_threads", 1) for i in info] or [1])
    rng = np.random.default_rng(seed)
    B, Hkv = w.block_size, w.num_kv_heads
    G = oracle.geometry(w.n_tokens, w.sub_chunk, B, w.sink_tokens, w.local_window, w.top_k, cs)
    J = len(G)
    if J <= n_sel_clusters:
        sample = list(range(J))
    else:
        rest = rng.choice(np.arange(1, J - 1), size=n_sel_clusters - 2, replace=False)
        sample = sorted({0, J - 1, *rest.tolist()})
    n_rep = max(G[j].sink_blk + G[j].n_cand for j in sample)

    t0 = time.perf_counter()
    k_rep = oracle.rep_keys(data["k_pages"], data["block_table"], w.n_tokens, B, blocks=np.arange(n_rep))
    t_rep = (time.perf_counter() - t0) * (w.n_tokens // B) / max(n_rep, 1)

    sels = {}
    t1 = time.perf_counter()
    for j in sample:
        g = G[j]
        v = oracle.anchor_fingerprint(data["q"], g.s, g.anchor_end)
        x = oracle.block_logits(v, k_rep[g.sink_blk:g.sink_blk + g.n_cand], Hkv)
        sels[j], _ = oracle.select_topk(oracle.soft_vote(x), g.sink_blk, w.top_k)
    cost = [(g.anchor_end - g.s) + g.n_cand for g in G]
    t_sel = (time.perf_counter() - t1) * sum(cost) / max(sum(cost[j] for j in sample), 1)

    sampled_pairs = 0
    n_tiles = 0
    t2 = time.perf_counter()
    while n_tiles < min_tiles or time.perf_counter() - t2 < min_seconds:
        n_tiles += 1
        j = sample[int(rng.integers(0, len(sample)))]
        g = G[j]
        p0 = g.s + ORACLE_CHUNK * int(rng.integers(0, max(1, -(-(g.e - g.s) // ORACLE_CHUNK))))
        rows = np.arange(p0, min(p0 + ORACLE_CHUNK, g.e))
        oracle.attention_rows(data["q"], data["k_pages"], data["v_pages"], data["block_table"], g, sels[j], rows, B)
        sampled_pairs += len(rows) * (g.sink_eff + g.sel_cnt) * B + int(sum(p - g.lo_blk * B + 1 for p in rows))
    t_att_raw = time.perf_counter() - t2
    total_pairs = geometry_work(w, geo)["pairs"]
    t_layer = t_rep + t_sel + t_att_raw * total_pairs / max(sampled_pairs, 1)
    measured = time.perf_counter() - t0
    return {
        "value": w.n_tokens / (t_layer * w.layers),
        "unit": "tokens/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"fp64 numpy oracle on layer 0: representative keys of {n_rep} of {w.n_tokens // B} blocks, "
                   f"selection of {len(sample)} of {J} clusters, attention of {n_tiles} random {ORACLE_CHUNK}-row chunks x "
                   f"{w.num_q_heads} heads ({sampled_pairs} of {total_pairs} visible (row, key) pairs); each part "
                   f"scaled to the layer, x{w.layers} layers"),
        "seconds_measured": round(measured, 2),
    }


def time_path(args, w, c, layers, dev, theta=None):
    """Times `args.steps` steps of the whole path (every layer) for cluster size c, or, with
    `theta`, with the clusters formed on the GPU by the anchor-based clustering at every step;
    returns the result dict without the CPU baseline."""
    import gen
    import paper_2609_31568_amd as pk
    import torch

    l_max = args.l_max or 8 * w.sub_chunk
    max_clusters = w.n_sub_chunks if theta is not None else len(gen.cluster_starts(w.n_sub_chunks, c)) - 1
    tokens = args.tokens > 0
    cfg = pk.config_for(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                        block_size=w.block_size, sub_chunk=w.sub_chunk, top_k=args.tokens if tokens else w.top_k,
                        sink_tokens=w.sink_tokens, local_window=w.local_window, max_tokens=w.n_tokens,
                        max_clusters=max_clusters, out_bf16=args.out_bf16, select_tokens=tokens,
                        rep_bounds=args.rep_bounds, kv_head_sets=args.kv_sets, score_scale=args.score_scale)
    h = pk.Scale(cfg)
    if theta is None:
        cs = gen.cluster_starts(w.n_sub_chunks, c)
        layer_cs = [cs] * len(layers)
    else:
        layer_cs = [h.cluster_subchunks(q, w.n_tokens, theta, l_max, args.outer) for q, *_ in layers]
        cs = layer_cs[0]
    geo = pk.scale_cluster_geometry(cfg, w.n_tokens, cs)
    work = geometry_work(w, geo, tokens, bounds=args.rep_bounds)
    # one set of outputs shared by the layers: each layer's output is complete when its attention
    # call ends, and the next layer's calls are ordered after it on the stream
    bufs = pk.LayerBuffers(cfg, w.n_tokens, max_clusters, device=dev)

    def step():
        for (q, kp, vp, bt), lcs in zip(layers, layer_cs):
            if theta is not None:
                lcs = h.cluster_subchunks(q, w.n_tokens, theta, l_max, args.outer)
                if tokens:
                    h.select_cluster_tokens(q, w.n_tokens, kp, bt, lcs, bufs.sel_idx, bufs.sel_cnt)
                else:
                    h.rep_keys(kp, bt, w.n_tokens, bufs.k_rep)
                    h.select_cluster(q, w.n_tokens, bufs.k_rep, lcs, bufs.sel_idx, bufs.sel_cnt)
                h.sparse_prefill(q, kp, vp, bt, w.n_tokens, lcs, bufs.sel_idx, bufs.sel_cnt, bufs.out)
            else:
                pk.run_layer(h, q, kp, vp, bt, w.n_tokens, lcs, bufs)

    n_warm = 0
    t_warm = time.perf_counter()
    while (n_warm < args.warmup if args.warmup is not None
           else n_warm < 3 or time.perf_counter() - t_warm < WARMUP_S):
        step()
        n_warm += 1
        torch.cuda.synchronize()
    # Inside the timed region only the attention launches are bracketed by events (the roofline's
    # launch time); an event pair around every stage would sit between launches that otherwise run
    # back to back.
    h.enable_stage_timing(("attention",))
    h.stage_times(reset=True)
    calls0 = h.retrieval_calls()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    timed = h.stage_times(reset=True)
    calls = (h.retrieval_calls() - calls0) // max(args.steps, 1)
    # the same steps again, one at a time, outside the timed region, every stage timed: the other
    # stages' launch times and the per-launch spread of attention
    h.enable_timing(True)
    per_step = []
    stages = {k: (0.0, 0) for k in timed}
    for _ in range(args.steps):
        step()
        st = h.stage_times(reset=True)
        per_step.append(st["attention"][0] / max(st["attention"][1], 1))
        stages = {k: (stages[k][0] + st[k][0], stages[k][1] + st[k][1]) for k in stages}
    per_step.sort()
    stages["attention"] = timed["attention"]
    overlap = overlap_stats(h, bufs, w, layers[0], cs) if args.overlap and not tokens and not args.kv_sets else None
    h.close()
    del bufs

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    tokens_per_s = w.n_tokens / (ms_per_step / 1e3)
    per_launch = {k: (ms / n if n else 0.0) for k, (ms, n) in stages.items()}
    att_ms = per_launch["attention"]
    achieved = work["attention_flops"] / (att_ms * 1e-3) / 1e12 if att_ms > 0 else 0.0
    profiled = counters_apply(args, w, c, theta, tokens)

    def gbs(nbytes, ms):
        return round(nbytes / (ms * 1e-3) / 1e9, 1) if ms > 0 else None

    if tokens:
        lg_ms = per_launch["logits"]
        hbm = {
            "fingerprint": {"GB/s": gbs(work["fingerprint_bytes"], per_launch["fingerprint"]),
                            "bytes": work["fingerprint_bytes"]},
            "token_logits": {"GB/s": gbs(work["token_logits_bytes"], lg_ms), "bytes": work["token_logits_bytes"],
                             "TFLOP/s": round(work["token_logits_flops"] / (lg_ms * 1e-3) / 1e12, 2) if lg_ms else None,
                             "flops": work["token_logits_flops"],
                             "note": "split + stats pass + log-normaliser + scores pass; bytes = one read of every "
                                     "candidate key, flops = one logit per (cluster, head, candidate token)"},
            "vote_topk": {"GB/s": gbs(work["vote_bytes"], per_launch["vote_topk"]), "bytes": work["vote_bytes"]},
            "gather": {"GB/s": gbs(work["gather_bytes"], per_launch["gather"]), "bytes": work["gather_bytes"]},
            "peak_GB/s": PEAK_HBM_GBS,
        }
    else:
        hbm = None
    hbm = hbm or {
        "rep_keys": {"GB/s": gbs(work["rep_keys_bytes"], per_launch["rep_keys"]), "bytes": work["rep_keys_bytes"]},
        "fingerprint": {"GB/s": gbs(work["fingerprint_bytes"], per_launch["fingerprint"]),
                        "bytes": work["fingerprint_bytes"]},
        "logits": {"GB/s": gbs(work["logits_bytes"], per_launch["logits"]), "bytes": work["logits_bytes"],
                   "fp64_TFLOP/s": (round(work["logits_flops"] / (per_launch["logits"] * 1e-3) / 1e12, 2)
                                    if per_launch["logits"] > 0 else None),
                   "fp64_peak_TFLOP/s": PEAK_FP64_TFLOPS,
                   "note": "effective: k_rep bytes counted once per cluster that scores them (the per-call cost "
                           "model); the kernel stages each k_rep tile once for up to 64 (cluster, head) rows, "
                           "so large cluster counts run above the HBM rate; fp64 FLOPs = 2 d per "
                           "(cluster, query head, candidate)"},
        "vote_topk": {"GB/s": gbs(work["vote_bytes"], per_launch["vote_topk"]), "bytes": work["vote_bytes"],
                      "bound": "latency",
                      "note": "one work-group per output row: soft-voting sums, then three radix passes and an "
                              "ordered compaction over the row's scores, each a handful of work-group barriers; "
                              "a few MB per launch, so the launch time is latency, not bandwidth"},
        "peak_GB/s": PEAK_HBM_GBS,
    }
    shape = {32: "Llama-3-8B-shaped attention layer", 28: "Qwen2-7B-shaped attention stack",
             8: "four-way KV-head shard (8 query / 2 KV heads) of a Llama-3-8B-shaped attention layer"}.get(
                 w.num_q_heads, f"{w.num_q_heads} query / {w.num_kv_heads} KV head attention layer")
    return {
        "metric": METRIC,
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": n_warm,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded topic-structured Q/K/V, bf16)",
        "config": {
            "workload": f"{w.name}: {w.layers} x {shape}, {w.n_tokens} tokens",
            "n_tokens": w.n_tokens, "layers": w.layers, "num_q_heads": w.num_q_heads,
            "num_kv_heads": w.num_kv_heads, "head_dim": w.head_dim, "block_size": w.block_size,
            "sub_chunk": w.sub_chunk, "cluster": c if theta is None else f"anchor clustering, theta {theta}",
            "top_k": w.top_k if not tokens else None,
            "select_tokens": args.tokens if tokens else None, "sink_tokens": w.sink_tokens,
            "rep_keys": "channel-wise bounds" if args.rep_bounds else "mean",
            "index_sets": "per KV head" if args.kv_sets else "per cluster",
            "score_scale": args.score_scale or 1.0,
            "local_window": w.local_window, "out_dtype": "bf16" if args.out_bf16 else "fp32",
            "seed": w.seed,
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "sparse_attention",
            "achieved": round(achieved, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic() if profiled else None,
            "flops_per_launch": work["attention_flops"],
            "avg_launch_ms": round(att_ms, 4),
            "median_launch_ms": round(per_step[len(per_step) // 2], 4),
            "min_launch_ms": round(per_step[0], 4),
            "library_gemm": library_gemm_reference(achieved),
        },
        "mfma_util_pct": round(100 * achieved / PEAK_BF16_TFLOPS, 2),
        "mfma_counted": counted_mfma(work["attention_flops"], att_ms) if profiled else None,
        "layer_tokens_per_s": round(w.n_tokens * w.layers / (ms_per_step / 1e3), 1),
        "stage_ms_per_layer": {k: round(v, 4) for k, v in per_launch.items()},
        "hbm": hbm,
        "retrieval_calls": {"per_step": int(calls), "per_layer": len(cs) - 1, "clusters": len(cs) - 1,
                            "per_sub_chunk_baseline": w.n_sub_chunks * w.layers,
                            "reduction": round(w.n_sub_chunks * w.layers / max(calls, 1), 2)},
        "paper_context": PAPER_CONTEXT,
        **({"clustering": _cluster_stats(cs, theta, l_max, args.outer, w)} if theta is not None else {}),
        **({"topk_overlap": overlap} if overlap is not None else {}),
    }, cs, geo


def overlap_stats(h, bufs, w, layer, cs):
    """Eq. 7 for every cluster of layer 0: the cluster's selected blocks against the union of its
    member sub-chunks' own selections (each over its single-sub-chunk candidate range), from two
    selection calls on the GPU; min / median / mean / max over the clusters with a selection."""
    import numpy as np
    import torch

    q, kp, vp, bt = layer
    h.rep_keys(kp, bt, w.n_tokens, bufs.k_rep)
    k = len(cs) - 1
    h.select_cluster(q, w.n_tokens, bufs.k_rep, cs, bufs.sel_idx[:k], bufs.sel_cnt[:k])
    torch.cuda.synchronize()
    idx, cnt = bufs.sel_idx.cpu().numpy(), bufs.sel_cnt.cpu().numpy()
    sel_c = [set(idx[j, :cnt[j]].tolist()) for j in range(k)]
    m = w.n_sub_chunks
    if bufs.sel_idx.shape[0] < m:
        return {"note": "needs max_clusters >= the sub-chunk count (run with --theta or --cluster 1)"}
    h.select_cluster(q, w.n_tokens, bufs.k_rep, np.arange(m + 1, dtype=np.int32), bufs.sel_idx, bufs.sel_cnt)
    torch.cuda.synchronize()
    idx, cnt = bufs.sel_idx.cpu().numpy(), bufs.sel_cnt.cpu().numpy()
    rho = []
    for j in range(k):
        if not sel_c[j]:
            continue
        union = set()
        for i in range(cs[j], cs[j + 1]):
            union |= set(idx[i, :cnt[i]].tolist())
        rho.append(len(sel_c[j] & union) / len(sel_c[j]))
    rho = np.asarray(rho)
    return {"clusters": int(len(rho)), "min": round(float(rho.min()), 4), "median": round(float(np.median(rho)), 4),
            "mean": round(float(rho.mean()), 4), "max": round(float(rho.max()), 4)}


def _cluster_stats(cs, theta, l_max, outer, w):
    import numpy as np

    sizes = np.diff(np.asarray(cs))
    cap = -(-l_max // w.sub_chunk)
    hist = np.bincount(sizes, minlength=cap + 1)[1:cap + 1]
    return {"theta": theta, "l_max_tokens": l_max, "outer_subchunks": outer, "clusters": int(len(sizes)),
            "mean_size_tokens": round(float(sizes.mean() * w.sub_chunk), 1),
            "size_fraction": {str(i + 1): round(float(x) / len(sizes), 4) for i, x in enumerate(hist)}}


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (it measures the path "
              f"on one GPU's share of the work)", file=sys.stderr)
        sys.exit(2)
    rank = int(os.environ.get("RANK", "0"))

    import numpy as np
    import torch

    import gen

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_probe:
        a = torch.ones(1 << 28, dtype=torch.int32, device=dev)     # 1 GiB
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": a.numel() * 4, "copy_probe_bytes_written": b.numel() * 4}))
        return
    if args.gemm_probe > 0:
        n = 8192
        a = torch.randn(n, n, dtype=torch.bfloat16, device=dev)
        b = torch.randn(n, n, dtype=torch.bfloat16, device=dev)
        for _ in range(5):
            c = a @ b
        torch.cuda.synchronize()
        done, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < args.gemm_probe:
            for _ in range(50):
                c = a @ b
            torch.cuda.synchronize()
            done += 50
        dt = time.perf_counter() - t0
        print(json.dumps({"gemm_probe": f"{n}^3 bf16 torch.matmul", "launches": done, "seconds": round(dt, 2),
                          "tflops": round(2 * n ** 3 * done / dt / 1e12, 1), "checksum": float(c[0, 0])}))
        return
    w = gen.WORKLOADS[args.workload]
    sweep = [int(x) for x in args.sweep.split(",")] if args.sweep else [args.cluster or w.cluster]

    def up(a):
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    t_gen = time.perf_counter()
    layers, host0 = [], None
    for layer in range(w.layers):
        print(f"[bench] generating {w.name} layer {layer}: N={w.n_tokens} Hq={w.num_q_heads} Hkv={w.num_kv_heads} "
              f"d={w.head_dim} B={w.block_size} L={w.sub_chunk} k={w.top_k}", file=sys.stderr, flush=True)
        data = gen.make_layer(w, layer)
        layers.append((up(data["q"]), up(data["k_pages"]), up(data["v_pages"]), up(data["block_table"])))
        if layer == 0:
            host0 = data
        del data
    print(f"[bench] inputs ready in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr, flush=True)

    thetas = [float(x) for x in args.theta_sweep.split(",")] if args.theta_sweep else (
        [args.theta] if args.theta is not None else [])
    runs = [(w.cluster, t) for t in thetas] if thetas else [(c, None) for c in sweep]
    for c, theta in runs:
        wc = w.with_(cluster=c)
        print(f"[bench] timing " + (f"theta={theta}" if theta is not None else f"c={c}"), file=sys.stderr, flush=True)
        result, cs, geo = time_path(args, wc, c, layers, dev, theta=theta)
        variant = args.tokens or args.rep_bounds or args.kv_sets or args.score_scale
        if rank == 0 and not args.no_cpu_baseline and not variant:
            if args.cpu_full:
                print("[bench] timing the oracle on the whole layer", file=sys.stderr, flush=True)
                result["cpu_baseline"] = cpu_full_layer(wc, host0, cs)
            else:
                print("[bench] timing the oracle on a sample", file=sys.stderr, flush=True)
                result["cpu_baseline"] = cpu_baseline(wc, host0, cs, geo, args.cpu_tiles, args.cpu_seconds)
                full = profile_block(ORACLE_FULL_PROFILE)
                if full and full.get("workload") == wc.name and full.get("cluster") == c and theta is None:
                    # the committed whole-layer timing of the same oracle on the same workload
                    result["cpu_baseline"]["full_layer_measured"] = {
                        k: full[k] for k in ("value", "seconds", "cores", "host") if k in full}
                    result["cpu_baseline"]["full_layer_measured"]["source"] = os.path.relpath(ORACLE_FULL_PROFILE,
                                                                                              ROOT)
        if rank == 0:
            print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
