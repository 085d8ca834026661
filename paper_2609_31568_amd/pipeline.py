"""One layer of cluster-level sparse prefill through the C ABI: rep keys -> select -> attention
(block-level selection), or token selection -> attention (token-level selection).

torch allocates the device buffers; the work runs in libscale's kernels.
"""
from __future__ import annotations

import numpy as np

from .binding import SCALE_OUT_BF16, SCALE_REP_BOUNDS, Scale, make_config


def config_for(*, num_q_heads, num_kv_heads, head_dim, block_size, sub_chunk, top_k, sink_tokens, local_window,
               max_tokens, max_clusters, out_bf16=False, softmax_scale=0.0, score_scale=0.0, select_tokens=False,
               rep_bounds=False, kv_head_sets=False):
    return make_config(num_q_heads=num_q_heads, num_kv_heads=num_kv_heads, head_dim=head_dim,
                       block_size=block_size, sub_chunk=sub_chunk, top_k=top_k, sink_tokens=sink_tokens,
                       local_window=local_window, max_tokens=max_tokens, max_clusters=max_clusters,
                       softmax_scale=softmax_scale, score_scale=score_scale,
                       out_dtype=SCALE_OUT_BF16 if out_bf16 else 0, select_tokens=select_tokens,
                       rep_kind=SCALE_REP_BOUNDS if rep_bounds else 0, kv_head_sets=kv_head_sets)


class LayerBuffers:
    """Device outputs of one layer, allocated once and reused across calls."""

    def __init__(self, cfg, n_tokens: int, n_clusters: int, device="cuda", with_scores=False):
        import torch

        nb = n_tokens // cfg.block_size
        rep = (2, cfg.head_dim) if cfg.rep_kind == SCALE_REP_BOUNDS else (cfg.head_dim,)
        self.k_rep = torch.empty((nb, cfg.num_kv_heads, *rep), dtype=torch.float32, device=device)
        rows = n_clusters * (cfg.num_kv_heads if cfg.kv_head_sets else 1)   # selection rows
        self.sel_idx = torch.empty((rows, max(cfg.top_k, 1)), dtype=torch.int32, device=device)
        self.sel_cnt = torch.empty((rows,), dtype=torch.int32, device=device)
        odt = torch.bfloat16 if cfg.out_dtype == SCALE_OUT_BF16 else torch.float32
        self.out = torch.empty((n_tokens, cfg.num_q_heads, cfg.head_dim), dtype=odt, device=device)
        n_score = n_tokens if cfg.select_tokens else nb
        self.scores = torch.empty((rows, n_score), dtype=torch.float32, device=device) if with_scores else None
        self.fingerprints = (torch.empty((n_clusters, cfg.num_q_heads, cfg.head_dim), dtype=torch.float32,
                                         device=device) if with_scores else None)


def run_layer(h: Scale, q, k_pages, v_pages, block_table, n_tokens: int, cluster_start, bufs: LayerBuffers):
    """Enqueue the whole hot path of one layer on the handle's stream (no synchronisation)."""
    cs = np.asarray(cluster_start, dtype=np.int32)
    if h.cfg.select_tokens:
        h.select_cluster_tokens(q, n_tokens, k_pages, block_table, cs, bufs.sel_idx, bufs.sel_cnt, bufs.scores)
    else:
        h.rep_keys(k_pages, block_table, n_tokens, bufs.k_rep)
        h.select_cluster(q, n_tokens, bufs.k_rep, cs, bufs.sel_idx, bufs.sel_cnt, bufs.scores)
    if bufs.fingerprints is not None:
        h.fingerprints(bufs.fingerprints, len(cs) - 1)
    h.sparse_prefill(q, k_pages, v_pages, block_table, n_tokens, cs, bufs.sel_idx, bufs.sel_cnt, bufs.out)
    return bufs
