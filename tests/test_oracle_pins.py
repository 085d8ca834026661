"""Pins of the fp64 oracle against what the paper and the mathematics fix (CPU only).

Each pin is independent of the oracle's own code: a library routine (torch's causal
scaled-dot-product attention), brute-force enumeration on tiny inputs (tests/brute.py),
closed forms, or invariants. A plausible slip in the oracle -- a dropped key group, a wrong
window bound, a transposed head map, a wrong softmax domain, a cluster mean in place of the
anchor -- fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

import gen
import oracle
from tests import brute


def _run_oracle(d, w, n_tokens=None, cs=None, **over):
    n = w.n_tokens if n_tokens is None else n_tokens
    kw = dict(sub_chunk=w.sub_chunk, block_size=w.block_size, top_k=w.top_k, sink_tokens=w.sink_tokens,
              local_window=w.local_window)
    kw.update(over)
    if cs is None:
        cs = gen.cluster_starts(-(-n // kw["sub_chunk"]), w.cluster)
    return oracle.prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], n, cluster_start=cs, **kw)


def _sdpa_causal(q_bits, k_pages, v_pages, n):
    """Library reference: textbook causal attention (Eq. 1 + causal mask) via torch, fp64."""
    q = torch.from_numpy(oracle.bf16_to_f64(q_bits[:n]))                 # [N, Hq, d]
    K = torch.from_numpy(oracle.logical_kv(k_pages, np.arange(k_pages.shape[0]), np.arange(k_pages.shape[0])))[:n]
    V = torch.from_numpy(oracle.logical_kv(v_pages, np.arange(v_pages.shape[0]), np.arange(v_pages.shape[0])))[:n]
    G = q.shape[1] // K.shape[1]
    K = K.repeat_interleave(G, dim=1)
    V = V.repeat_interleave(G, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(
        q.transpose(0, 1), K.transpose(0, 1), V.transpose(0, 1), is_causal=True)
    return o.transpose(0, 1).numpy()


SMALL = {
    "tiny": gen.WORKLOADS["tiny"],
    # GQA 4:1 with two KV heads, cluster size 3 does not divide M = 8
    "gqa": gen.Workload("gqa", 1, 8, 2, 32, 1024, 32, 128, 3, 3, 32, 128, 6, 1, 3, 11),
    # group size 7 (Qwen-like), ragged last cluster
    "g7": gen.Workload("g7", 1, 7, 1, 32, 768, 32, 64, 5, 2, 64, 96, 5, 1, 4, 12),
    # a window (100) and a sink (40) off the block grid (32): with one sub-chunk (64 rows) per
    # cluster the window starts inside a block and is rounded down (R10), the sink rounds up (R11)
    "offgrid": gen.Workload("offgrid", 1, 4, 1, 32, 1024, 32, 64, 1, 3, 40, 100, 6, 1, 3, 13),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_dense_reduction_matches_library_sdpa(name):
    """k >= every candidate count: sink + candidates + local = all earlier keys, so Eq. 10 is dense
    causal attention (P1)."""
    w = SMALL[name]
    d = gen.make_layer(w)
    r = _run_oracle(d, w, top_k=w.n_blocks)
    ref = _sdpa_causal(d["q"], d["k_pages"], d["v_pages"], w.n_tokens)
    assert np.max(np.abs(r["output"] - ref)) < 1e-12


def test_wide_window_is_dense():
    w = SMALL["gqa"]
    d = gen.make_layer(w)
    r = _run_oracle(d, w, top_k=0, local_window=w.n_tokens)
    ref = _sdpa_causal(d["q"], d["k_pages"], d["v_pages"], w.n_tokens)
    assert np.max(np.abs(r["output"] - ref)) < 1e-12


@pytest.mark.parametrize("name,c", [("tiny", 4), ("tiny", 1), ("gqa", 3), ("gqa", 1), ("g7", 5), ("offgrid", 1)])
def test_brute_force_selection_and_attention(name, c):
    """Selection = best-total-score k-subset, attention = masked dense softmax (P2 at c=1, P3)."""
    w = SMALL[name].with_(cluster=c)
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    r = _run_oracle(d, w, cs=cs)
    b = brute.brute_prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, w.sub_chunk,
                            w.block_size, w.sink_tokens, w.local_window, w.top_k, cs)
    assert len(r["selections"]) == len(b["selections"])
    for sel_o, sel_b, sc_o, sc_b, g in zip(r["selections"], b["selections"], r["scores"], b["scores"],
                                           r["geometry"]):
        assert tuple(int(x) for x in sel_o) == tuple(sel_b)
        cand = list(range(g.sink_blk, g.sink_blk + g.n_cand))
        assert sorted(sc_b) == cand
        for i, blk in enumerate(cand):
            assert abs(sc_o[i] - sc_b[blk]) < 1e-12
    assert np.max(np.abs(r["output"] - b["output"])) < 1e-12


def test_ragged_tail_matches_brute_force():
    """n_tokens not a multiple of the block or sub-chunk size: short last sub-chunk and block."""
    w = SMALL["gqa"]
    d = gen.make_layer(w)
    n = 1000
    cs = gen.cluster_starts(-(-n // w.sub_chunk), 3)
    r = _run_oracle(d, w, n_tokens=n, cs=cs)
    b = brute.brute_prefill(d["q"][:n], d["k_pages"], d["v_pages"], d["block_table"], n, w.sub_chunk,
                            w.block_size, w.sink_tokens, w.local_window, w.top_k, cs)
    for sel_o, sel_b in zip(r["selections"], b["selections"]):
        assert tuple(int(x) for x in sel_o) == tuple(sel_b)
    assert np.max(np.abs(r["output"] - b["output"])) < 1e-12
    # partial last block: its representative key averages the 8 valid tokens only
    K = brute.unpage(d["k_pages"], d["block_table"])
    last = r["k_rep"][-1]
    assert np.allclose(last, K[992:1000].mean(axis=0), rtol=0, atol=1e-15)


def test_exact_ties_resolve_to_lowest_index():
    """Duplicated K blocks have identical scores; the lowest block indices win (R12), and brute-force
    subset enumeration with the lexicographic rule agrees."""
    w = SMALL["gqa"].with_(top_k=2, cluster=8)
    d = gen.make_layer(w)
    cs = np.array([0, 6, 8], dtype=np.int32)          # the second cluster has 23 candidates
    r0 = _run_oracle(d, w, cs=cs)
    g = r0["geometry"][1]
    best = int(r0["selections"][1][np.argmax([r0["scores"][1][b - g.sink_blk] for b in r0["selections"][1]])])
    dups = [blk for blk in range(g.sink_blk, g.sink_blk + g.n_cand) if blk != best][:3]
    for blk in dups:
        d["k_pages"][blk] = d["k_pages"][best]
    r = _run_oracle(d, w, cs=cs)
    tied = sorted(dups + [best])
    assert list(r["selections"][1]) == tied[:2]
    assert r["margins"][1] == 0.0
    b = brute.brute_prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, w.sub_chunk,
                            w.block_size, w.sink_tokens, w.local_window, 2, cs)
    assert tuple(b["selections"][1]) == tuple(tied[:2])


def test_soft_vote_closed_form():
    """Two heads, three candidates, logits chosen so each softmax is known in closed form."""
    x = np.array([[0.0, math.log(3.0), 0.0],
                  [math.log(2.0), 0.0, 0.0]])
    s = oracle.soft_vote(x)
    assert np.allclose(s, [1 / 5 + 2 / 4, 3 / 5 + 1 / 4, 1 / 5 + 1 / 4], rtol=0, atol=1e-15)
    # logits of a single head: sigma * v . k_rep, with the consecutive-heads GQA map (R5, R6)
    v = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0], [2.0, 0.0]])        # Hq = 4
    k_rep = np.array([[[1.0, 2.0], [3.0, 5.0]]])                          # 1 block, Hkv = 2
    lg = oracle.block_logits(v, k_rep, num_kv_heads=2, score_scale=0.5)
    assert np.allclose(lg[:, 0], [0.5 * 1, 0.5 * 2, 0.5 * 8, 0.5 * 6])


def test_score_invariants():
    w = SMALL["gqa"].with_(cluster=1)
    d = gen.make_layer(w)
    r = _run_oracle(d, w, cs=gen.cluster_starts(w.n_sub_chunks, 1))
    for sc, g in zip(r["scores"], r["geometry"]):
        if g.n_cand:
            assert abs(sc.sum() - w.num_q_heads) < 1e-12
            assert sc.min() >= 0 and sc.max() <= w.num_q_heads


def test_rep_keys_token_loop():
    w = SMALL["tiny"]
    d = gen.make_layer(w)
    kr = oracle.rep_keys(d["k_pages"], d["block_table"], w.n_tokens, w.block_size)
    for b in (0, 7, 31):
        for g in range(w.num_kv_heads):
            acc = [0.0] * w.head_dim
            for t in range(w.block_size):
                row = oracle.bf16_to_f64(d["k_pages"][b, g, t])
                for c in range(w.head_dim):
                    acc[c] += float(row[c])
            assert np.allclose(kr[b, g], np.array(acc) / w.block_size, rtol=0, atol=1e-14)


def test_selection_depends_only_on_anchor_rows():
    """Eq. 9: the cluster query is the anchor fingerprint, so changing non-anchor rows changes no
    selection (a cluster-mean query would)."""
    w = SMALL["tiny"].with_(cluster=4, n_topics=3)
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 4)
    r0 = _run_oracle(d, w, cs=cs)
    q2 = d["q"].copy()
    for g in r0["geometry"]:
        q2[g.anchor_end:g.e] = d["q"][::-1][: g.e - g.anchor_end]       # scramble non-anchor rows
    r1 = _run_oracle(dict(d, q=q2), w, cs=cs)
    for a, b in zip(r0["selections"], r1["selections"]):
        assert np.array_equal(a, b)
    for a, b in zip(r0["scores"], r1["scores"]):
        assert np.array_equal(a, b)
    # ... while changing an anchor row does move the scores
    q3 = d["q"].copy()
    g = r0["geometry"][1]
    q3[g.s:g.anchor_end] = d["q"][0:g.anchor_end - g.s]
    r2 = _run_oracle(dict(d, q=q3), w, cs=cs)
    assert not np.array_equal(r0["scores"][1], r2["scores"][1])


def test_output_convexity_and_first_row():
    w = SMALL["gqa"]
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    r = _run_oracle(d, w, cs=cs)
    b = brute.brute_prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, w.sub_chunk,
                            w.block_size, w.sink_tokens, w.local_window, w.top_k, cs)
    V = brute.unpage(d["v_pages"], d["block_table"])
    G = w.num_q_heads // w.num_kv_heads
    for p in range(0, w.n_tokens, 37):
        keys = np.nonzero(b["mask"][p])[0]
        for h in range(w.num_q_heads):
            vv = V[keys, h // G, :]
            assert np.all(r["output"][p, h] >= vv.min(axis=0) - 1e-12)
            assert np.all(r["output"][p, h] <= vv.max(axis=0) + 1e-12)
    # row 0 sees only key 0: the output is V[0] exactly
    for h in range(w.num_q_heads):
        assert np.array_equal(r["output"][0, h], V[0, h // G])


def test_selection_order_and_page_permutation_invariance():
    w = SMALL["gqa"]
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    r = _run_oracle(d, w, cs=cs)
    rev = [s[::-1].copy() for s in r["selections"]]
    out_rev = np.concatenate([oracle.cluster_attention(d["q"], d["k_pages"], d["v_pages"], d["block_table"], g,
                                                       s, w.block_size) for g, s in zip(r["geometry"], rev)])
    assert np.max(np.abs(out_rev - r["output"])) < 1e-12
    rng = np.random.default_rng(5)
    perm = rng.permutation(w.n_blocks)                 # logical block b lives on page perm[b]
    kp = np.empty_like(d["k_pages"])
    vp = np.empty_like(d["v_pages"])
    kp[perm] = d["k_pages"]
    vp[perm] = d["v_pages"]
    r_p = _run_oracle(dict(d, k_pages=kp, v_pages=vp, block_table=perm.astype(np.int32)), w, cs=cs)
    assert np.array_equal(r_p["output"], r["output"])
    for a, b in zip(r_p["selections"], r["selections"]):
        assert np.array_equal(a, b)


def _read_golden_calls():
    rows = []
    with open(__file__.replace("test_oracle_pins.py", "golden/retrieval_calls.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                name, c, calls, calls_c1 = line.split()
                rows.append((name, int(c), int(calls), int(calls_c1)))
    return rows


@pytest.mark.parametrize("name,c,calls,calls_c1", _read_golden_calls())
def test_retrieval_call_counts(name, c, calls, calls_c1):
    """Closed form: one selection call per cluster per layer, ceil(M / c) per layer."""
    w = gen.WORKLOADS[name]
    M = w.n_sub_chunks
    per_layer = len(oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window,
                                    w.top_k, gen.cluster_starts(M, c)))
    per_layer_c1 = len(oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window,
                                       w.top_k, gen.cluster_starts(M, 1)))
    assert oracle.retrieval_calls([per_layer] * w.layers) == calls
    assert oracle.retrieval_calls([per_layer_c1] * w.layers) == calls_c1


def test_geometry_headline_closed_form():
    """128K context, B 128, L 512, c 8, S 128, W 4096: cluster j >= 1 starts at 4096 j, its window
    starts at its own first row, so it has 32 j - 1 candidate blocks; cluster 0 has none."""
    w = gen.WORKLOADS["llama128k"]
    geo = oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, w.top_k,
                          gen.cluster_starts(w.n_sub_chunks, 8))
    assert len(geo) == 32
    assert geo[0].n_cand == 0 and geo[0].sink_eff == 0 and geo[0].lo_blk == 0
    for j, g in enumerate(geo[1:], start=1):
        assert (g.s, g.e, g.anchor_end, g.lo_blk, g.sink_eff) == (4096 * j, 4096 * (j + 1), 4096 * j + 512, 32 * j, 1)
        assert g.n_cand == 32 * j - 1 and g.sel_cnt == min(32, 32 * j - 1)
    assert sum(1 for g in geo if g.n_cand <= w.top_k) == 2
    # Qwen shape: cluster of 4096 rows inside an 8192-token window reaches 4096 tokens back
    q = gen.WORKLOADS["qwen256k"]
    gq = oracle.geometry(q.n_tokens, q.sub_chunk, q.block_size, q.sink_tokens, q.local_window, q.top_k,
                         gen.cluster_starts(q.n_sub_chunks, 4))
    assert gq[3].s == 12288 and gq[3].lo_blk == (12288 + 4096 - 8192) // 128 and gq[1].lo_blk == 0


def test_topic_matched_blocks_rank_first():
    """P7 (statistical): candidates sharing the anchor's topic should be selected first."""
    w = gen.Workload("stat", 1, 8, 2, 128, 32768, 128, 512, 1, 8, 128, 1024, 48, 2, 6, 21)
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 1)
    r = oracle.prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, sub_chunk=w.sub_chunk,
                       block_size=w.block_size, top_k=w.top_k, sink_tokens=w.sink_tokens,
                       local_window=w.local_window, cluster_start=cs, with_output=False)
    hits = total = 0
    for g, sel in zip(r["geometry"], r["selections"]):
        topic = d["qtopic"][g.s // w.sub_chunk]
        matched = [b for b in range(g.sink_blk, g.sink_blk + g.n_cand) if d["kvtopic"][b] == topic]
        if 0 < len(matched) <= w.top_k:
            hits += len(set(matched) & set(int(x) for x in sel))
            total += len(matched)
    assert total > 10 and hits / total >= 0.9


@pytest.mark.parametrize("scores,k,sel,margin", [
    # distinct scores: order 3.0 (13), 2.0 (11), 1.25 (12), 1.0 (14), 0.5 (10); the gap below the
    # k-th is 2.0 - 1.25 (the gaps next to it, 1.0 and 0.25, would be the off-by-one readings)
    ([0.5, 2.0, 1.25, 3.0, 1.0], 2, [11, 13], 0.75),
    ([0.5, 2.0, 1.25, 3.0, 1.0], 1, [13], 1.0),
    ([0.5, 2.0, 1.25, 3.0, 1.0], 4, [11, 12, 13, 14], 0.5),
    # one candidate more than k: the gap to the only unselected one
    ([1.0, 4.0, 2.5], 2, [11, 12], 1.5),
    # a tie straddling position k: the lower index of the two 2.0s is taken, and the margin is 0
    ([2.0, 1.0, 2.0, 3.0], 2, [10, 13], 0.0),
    # a tie inside the top-k does not make the margin 0
    ([3.0, 3.0, 1.0], 2, [10, 11], 2.0),
    # no budget, or every candidate selected: nothing is decided, the margin is infinite
    ([0.5, 2.0, 1.25], 0, [], math.inf),
    ([0.5, 2.0, 1.25], 3, [10, 11, 12], math.inf),
    ([0.5, 2.0, 1.25], 7, [10, 11, 12], math.inf),
])
def test_topk_margin_closed_form(scores, k, sel, margin):
    """R12 on hand-picked scores (candidates start at block 10): the selection and the margin
    score_(k) - score_(k+1) in (score desc, index asc) order, which decides where the GPU's indices
    must equal the oracle's."""
    got, m = oracle.select_topk(np.asarray(scores, dtype=np.float64), 10, k)
    assert got.tolist() == sel
    assert m == margin
