"""Host-side checks of bench.py: the algorithmic work it divides by, the committed counter block,
and the one-GPU contract (no GPU needed)."""
import os
import subprocess
import sys

import numpy as np

import gen
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_attention_flops_match_key_sets():
    """4 d Hq per (row, visible key) pair, summed over the exact key sets of Eq. 10."""
    import paper_2609_31568_amd as pk

    for name, c in (("tiny", 4), ("tiny", 1)):
        w = gen.WORKLOADS[name].with_(cluster=c)
        cs = gen.cluster_starts(w.n_sub_chunks, c)
        cfg = pk.config_for(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                            block_size=w.block_size, sub_chunk=w.sub_chunk, top_k=w.top_k,
                            sink_tokens=w.sink_tokens, local_window=w.local_window, max_tokens=w.n_tokens,
                            max_clusters=len(cs) - 1)
        geo = pk.scale_cluster_geometry(cfg, w.n_tokens, cs)
        work = bench.geometry_work(w, geo)
        pairs = 0
        for g in oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, w.top_k, cs):
            sel = np.arange(g.sink_blk, g.sink_blk + g.sel_cnt)        # any sel_cnt distinct candidates
            for p in range(g.s, g.e):
                pairs += len(oracle.key_positions(g, sel, p, w.block_size))
        assert work["pairs"] == pairs
        assert work["attention_flops"] == 4.0 * w.head_dim * w.num_q_heads * pairs


def test_headline_attention_flops():
    """13.178 TFLOP for the 128K Llama layer (the figure the roofline divides by)."""
    import paper_2609_31568_amd as pk

    w = gen.WORKLOADS["llama128k"]
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    cfg = pk.config_for(num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=128, sub_chunk=512, top_k=32,
                        sink_tokens=128, local_window=4096, max_tokens=w.n_tokens, max_clusters=len(cs) - 1)
    work = bench.geometry_work(w, pk.scale_cluster_geometry(cfg, w.n_tokens, cs))
    assert abs(work["attention_flops"] / 1e12 - 13.178) < 1e-3


def test_counter_blocks_parse():
    t = bench.measured_traffic()
    assert t is None or t > 3.5 * 2**30       # at least the minimum Q + K + V + O bytes
    alg = 13178033405952.0
    m = bench.counted_mfma(alg, 12.5)
    if m is not None:
        assert 1.0 <= m["per_algorithmic"] < 1.05          # executed MFMA work covers the visible pairs
        assert abs(m["frac"] - m["flops"] / 12.5e-3 / 2.5e15) < 1e-3
    assert bench.counted_mfma(alg, 0.0) is None


def test_counters_apply_to_the_default_launch_only():
    args = bench.parse_args([])
    w = gen.WORKLOADS["llama128k"]
    assert bench.counters_apply(args, w, w.cluster, None, False)
    assert not bench.counters_apply(args, w, 1, None, False)                  # another cluster size
    assert not bench.counters_apply(args, w, w.cluster, 0.95, False)          # threshold clustering
    assert not bench.counters_apply(args, w, w.cluster, None, True)           # token-level selection
    assert not bench.counters_apply(args, gen.WORKLOADS["llama32k"], 8, None, False)
    for flag in (["--kv-sets"], ["--rep-bounds"], ["--out-bf16"], ["--score-scale", "0.088"]):
        assert not bench.counters_apply(bench.parse_args(flag), w, w.cluster, None, False), flag


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
