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


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama128k")
    ap.add_argument("--cluster", type=int, default=0, help="cluster size in sub-chunks (0: the workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-tiles", type=int, default=48, help="32-row tiles the oracle attends in its sample")
    ap.add_argument("--out-bf16", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only copy 1 GiB device to device (reference for HBM byte counters) and exit")
    return ap.parse_args()


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "attention_traffic_llama128k.md")


def measured_traffic(workload_name):
    """HBM bytes per attention launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary,
    scaled by the copy-probe factors, or None when the counters were taken on other kernel source
    or another workload."""
    import hashlib
    import re

    if workload_name != "llama128k" or not os.path.exists(TRAFFIC_PROFILE):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(TRAFFIC_PROFILE).read(), re.S)
    if not m:
        return None
    block = json.loads(m.group(1))
    src = os.path.join(ROOT, block["kernel_source"])
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != block["kernel_source_sha256"]:
        return None
    return int(block["traffic_bytes"])


def geometry_work(w, geo):
    """Algorithmic attention FLOPs and the selection-side bytes from the cluster geometry.

    Attention: 4 d Hq per (query row, visible key) pair (two products of 2 d FLOP), over
    exactly the keys of Eq. 10 -- masked pairs are not work.
    """
    B, d, Hq, Hkv = w.block_size, w.head_dim, w.num_q_heads, w.num_kv_heads
    pairs = 0
    for s, e, lo_blk, sink_eff, n_cand, sel_cnt in geo.tolist():
        rows = e - s
        fixed = (sink_eff + sel_cnt) * B
        base = lo_blk * B
        pairs += rows * fixed + (sum(range(s - base + 1, e - base + 1)))
    n_clusters = len(geo)
    nb = w.n_tokens // B
    anchor_rows = sum(min(e, s + w.sub_chunk) - s for s, e, *_ in geo.tolist())
    n_cand = int(geo[:, 4].sum())
    return {
        "attention_flops": 4.0 * d * Hq * pairs,
        "pairs": pairs,
        "rep_keys_bytes": w.n_tokens * Hkv * d * 2 + nb * Hkv * d * 4,
        "fingerprint_bytes": anchor_rows * Hq * d * 2 + n_clusters * Hq * d * 4,
        "logits_bytes": n_cand * Hkv * d * 4 + n_cand * Hq * 4 + n_clusters * Hq * d * 4,
        "vote_bytes": n_cand * Hq * 4,
    }


def cpu_baseline(w, data, cs, geo, n_tiles, seed=0):
    """The fp64 oracle as it stands, on a bounded sample: the whole selection (all clusters) plus
    attention for `n_tiles` random 32-row tiles; the attention time is scaled to the layer by
    visible-pair count (the oracle's cost is linear in it)."""
    import numpy as np
    import threadpoolctl

    import oracle

    info = threadpoolctl.threadpool_info()
    cores = max([i.get("num_threads", 1) for i in info] or [1])
    t0 = time.perf_counter()
    ref = oracle.prefill(data["q"], data["k_pages"], data["v_pages"], data["block_table"], w.n_tokens,
                         sub_chunk=w.sub_chunk, block_size=w.block_size, top_k=w.top_k,
                         sink_tokens=w.sink_tokens, local_window=w.local_window, cluster_start=cs,
                         with_output=False)
    t_sel = time.perf_counter() - t0
    rng = np.random.default_rng(seed)
    B = w.block_size
    sampled_pairs = 0
    t1 = time.perf_counter()
    for _ in range(n_tiles):
        j = int(rng.integers(0, len(ref["geometry"])))
        g = ref["geometry"][j]
        p0 = g.s + 32 * int(rng.integers(0, max(1, (g.e - g.s) // 32)))
        rows = np.arange(p0, min(p0 + 32, g.e))
        oracle.attention_rows(data["q"], data["k_pages"], data["v_pages"], data["block_table"], g,
                              ref["selections"][j], rows, B)
        sampled_pairs += len(rows) * (g.sink_eff + g.sel_cnt) * B + int(sum(p - g.lo_blk * B + 1 for p in rows))
    t_att = time.perf_counter() - t1
    total_pairs = geometry_work(w, geo)["pairs"]
    t_layer = t_sel + t_att * total_pairs / max(sampled_pairs, 1)
    return {
        "value": w.n_tokens * w.layers / t_layer,
        "unit": "tokens/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"fp64 numpy oracle: selection for all {len(cs) - 1} clusters ({t_sel:.1f} s) + attention of "
                   f"{n_tiles} random 32-row tiles x {w.num_q_heads} heads ({t_att:.1f} s), scaled to the layer "
                   f"by visible (row, key) pairs ({sampled_pairs} of {total_pairs})"),
        "seconds_measured": round(t_sel + t_att, 2),
    }


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (the kernel on one "
              f"GPU's share is what this build measures)", file=sys.stderr)
        sys.exit(2)
    rank = int(os.environ.get("RANK", "0"))

    import numpy as np
    import torch

    import gen
    import paper_2609_31568_amd as pk

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
    w = gen.WORKLOADS[args.workload]
    c = args.cluster or w.cluster
    w = w.with_(cluster=c)
    print(f"[bench] generating {w.name}: N={w.n_tokens} Hq={w.num_q_heads} Hkv={w.num_kv_heads} d={w.head_dim} "
          f"B={w.block_size} L={w.sub_chunk} c={c} k={w.top_k}", file=sys.stderr, flush=True)
    t_gen = time.perf_counter()
    data = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    print(f"[bench] inputs ready in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr, flush=True)

    def up(a):
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    q, kp, vp, bt = up(data["q"]), up(data["k_pages"]), up(data["v_pages"]), up(data["block_table"])
    cfg = pk.config_for(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                        block_size=w.block_size, sub_chunk=w.sub_chunk, top_k=w.top_k, sink_tokens=w.sink_tokens,
                        local_window=w.local_window, max_tokens=w.n_tokens, max_clusters=len(cs) - 1,
                        out_bf16=args.out_bf16)
    geo = pk.scale_cluster_geometry(cfg, w.n_tokens, cs)
    work = geometry_work(w, geo)
    h = pk.Scale(cfg)
    bufs = pk.LayerBuffers(cfg, w.n_tokens, len(cs) - 1, device=dev)

    for _ in range(args.warmup):
        pk.run_layer(h, q, kp, vp, bt, w.n_tokens, cs, bufs)
    torch.cuda.synchronize()
    h.enable_timing(True)
    h.stage_times(reset=True)
    calls0 = h.retrieval_calls()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        pk.run_layer(h, q, kp, vp, bt, w.n_tokens, cs, bufs)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    stages = h.stage_times(reset=True)
    calls = (h.retrieval_calls() - calls0) // max(args.steps, 1)
    h.close()

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    tokens_per_s = w.n_tokens * w.layers / (ms_per_step / 1e3)
    per_launch = {k: (ms / n if n else 0.0) for k, (ms, n) in stages.items()}
    att_ms = per_launch["attention"]
    achieved = work["attention_flops"] / (att_ms * 1e-3) / 1e12 if att_ms > 0 else 0.0

    def gbs(nbytes, ms):
        return round(nbytes / (ms * 1e-3) / 1e9, 1) if ms > 0 else None

    hbm = {
        "rep_keys": {"GB/s": gbs(work["rep_keys_bytes"], per_launch["rep_keys"]), "bytes": work["rep_keys_bytes"]},
        "fingerprint": {"GB/s": gbs(work["fingerprint_bytes"], per_launch["fingerprint"]),
                        "bytes": work["fingerprint_bytes"]},
        "logits": {"GB/s": gbs(work["logits_bytes"], per_launch["logits"]), "bytes": work["logits_bytes"],
                   "note": "k_rep re-read per cluster; largely L2/MALL resident at this size"},
        "vote_topk": {"GB/s": gbs(work["vote_bytes"], per_launch["vote_topk"]), "bytes": work["vote_bytes"]},
        "peak_GB/s": PEAK_HBM_GBS,
    }
    result = {
        "metric": METRIC,
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded topic-structured Q/K/V, bf16)",
        "config": {
            "workload": f"{w.name}: one Llama-3-8B-shaped attention layer, {w.n_tokens} tokens",
            "n_tokens": w.n_tokens, "layers": w.layers, "num_q_heads": w.num_q_heads,
            "num_kv_heads": w.num_kv_heads, "head_dim": w.head_dim, "block_size": w.block_size,
            "sub_chunk": w.sub_chunk, "cluster": c, "top_k": w.top_k, "sink_tokens": w.sink_tokens,
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
            "traffic": measured_traffic(w.name),
            "flops_per_launch": work["attention_flops"],
            "avg_launch_ms": round(att_ms, 4),
        },
        "mfma_util_pct": round(100 * achieved / PEAK_BF16_TFLOPS, 2),
        "stage_ms_per_step": {k: round(v, 4) for k, v in per_launch.items()},
        "hbm": hbm,
        "retrieval_calls": {"per_step": int(calls), "clusters": len(cs) - 1, "per_sub_chunk_baseline": w.n_sub_chunks,
                            "reduction": round(w.n_sub_chunks / max(calls, 1), 2)},
    }
    if rank == 0 and not args.no_cpu_baseline:
        print("[bench] timing the oracle on a sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(w, data, cs, geo, args.cpu_tiles)
    if rank == 0:
        print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
