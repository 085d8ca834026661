"""GPU parity of token-level selection (paper Sec. 5.1.3, Eq. 9 over single tokens; Eq. 10 over
the selected tokens): the HIP path through the C ABI against the fp64 oracle on the same seeded
inputs -- scores within their error bound, the exact top-k of the GPU's own scores, oracle-equal
selections above the margin, and the attention output under the GPU's selection."""
import numpy as np
import pytest

import gen
import oracle
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_31568_amd  # noqa: F401  (fails loudly if the library is missing)

    return torch.device("cuda:0")


def _oracle(w, d, cs, k, with_output=True, external_sel=None):
    return oracle.prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, sub_chunk=w.sub_chunk,
                          block_size=w.block_size, top_k=k, sink_tokens=w.sink_tokens, local_window=w.local_window,
                          cluster_start=cs, with_output=with_output, external_sel=external_sel, select_tokens=True)


def _run(w, d, cs, dev, k, **over):
    return gu.run_gpu(w, d, cs, dev, top_k=k, select_tokens=True, **over)


SHAPES = {
    # name: (workload, cluster size, token budget); budgets off the 64-row tile exercise the
    # padding mask of the last gathered tile
    "tiny_c4": (gen.WORKLOADS["tiny"], 4, 300),
    "tiny_c1": (gen.WORKLOADS["tiny"], 1, 64),
    "gqa128": (gen.Workload("gqa128", 1, 8, 2, 128, 8192, 128, 512, 3, 5, 128, 1024, 12, 1, 4, 31), 3, 603),
    "g7": (gen.Workload("g7", 1, 14, 2, 128, 4096, 64, 256, 4, 6, 64, 512, 8, 1, 3, 32), 4, 333),
    "g1": (gen.Workload("g1", 1, 2, 2, 64, 4096, 128, 512, 2, 3, 0, 700, 6, 1, 3, 33), 2, 200),
    "g8": (gen.Workload("g8", 1, 8, 1, 64, 2048, 64, 128, 5, 4, 130, 100, 6, 1, 5, 34), 5, 130),
    # group sizes 2, 3, 5, 6 (fingerprint rows padded to 2, 4, 8, 8 per cluster)
    "g2": (gen.Workload("g2", 1, 4, 2, 128, 4096, 128, 512, 2, 4, 128, 600, 8, 1, 3, 36), 2, 250),
    "g3": (gen.Workload("g3", 1, 6, 2, 128, 4096, 64, 256, 3, 6, 64, 512, 8, 1, 3, 37), 3, 190),
    "g5": (gen.Workload("g5", 1, 5, 1, 128, 4096, 128, 512, 2, 3, 128, 900, 6, 1, 3, 38), 2, 77),
    "g6": (gen.Workload("g6", 1, 12, 2, 64, 3072, 128, 256, 4, 5, 128, 512, 8, 1, 3, 39), 4, 129),
    "g2d64": (gen.Workload("g2d64", 1, 4, 2, 64, 4096, 64, 256, 3, 5, 64, 700, 8, 1, 3, 40), 3, 160),
    "g3d64": (gen.Workload("g3d64", 1, 3, 1, 64, 3072, 128, 512, 2, 3, 128, 600, 6, 1, 3, 42), 2, 300),
    "g5d64": (gen.Workload("g5d64", 1, 10, 2, 64, 4096, 128, 512, 2, 4, 128, 1000, 6, 1, 3, 43), 2, 200),
}


def _check_all(name, w, d, cs, k, res, ref):
    B = w.block_size
    cands = gu.token_candidates(d, ref["geometry"], B)
    bounds = gu.token_score_bounds(ref, cands, w.num_kv_heads)
    gu.check_rounding(res["fingerprints"], np.stack(ref["fingerprints"]), "fingerprints")
    worst = gu.check_token_scores(res["scores"], ref, bounds, B, name)
    # sel_idx rows hold k entries (the buffer keeps one column when k = 0)
    n_exact = gu.check_token_selection(res["sel_idx"][:, :k], res["sel_cnt"], res["scores"], ref, bounds, B, name)
    assert res["calls"] == len(cs) - 1
    sels = gu.gpu_selections(res, len(cs) - 1)
    own = _oracle(w, d, cs, k, external_sel=sels)
    mx, rel = gu.check_output(res["out"], own["output"], f"{name} output")
    gu.log(f"[tokens] {name}: worst relative score error {worst:.2e}; {n_exact} of {len(cs) - 1} clusters above "
           f"the margin; output max-abs {mx:.2e} rel-L2 {rel:.2e}")
    for j, g in enumerate(ref["geometry"]):
        if np.array_equal(sels[j], ref["selections"][j]):
            gu.check_output(res["out"][g.s:g.e], ref["output"][g.s:g.e], f"{name} cluster {j}")


@pytest.mark.parametrize("name", list(SHAPES))
def test_token_small_shapes_full_parity(dev, name):
    w, c, k = SHAPES[name]
    gu.log(f"[tokens] {name} k={k}")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    res = _run(w, d, cs, dev, k)
    ref = _oracle(w, d, cs, k)
    _check_all(name, w, d, cs, k, res, ref)


@pytest.mark.parametrize("k", [0, 1, 63, 65, 10 ** 6])
def test_token_budget_edges(dev, k):
    """Empty selection (sinks and window only), a single token (63 padding rows masked), budgets
    one below and one above a tile, and the dense limit (every candidate selected)."""
    w, c, _ = SHAPES["gqa128"]
    gu.log(f"[tokens] budget {k}")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    res = _run(w, d, cs, dev, k)
    ref = _oracle(w, d, cs, k)
    if k >= 10 ** 6:
        assert all(g.sel_cnt == g.n_cand for g in ref["geometry"])
    _check_all(f"budget {k}", w, d, cs, k, res, ref)


def test_token_mode_on_block_constant_keys_selects_whole_blocks(dev):
    """Keys constant inside each block: every token of a block has the same score (bit for bit on
    the GPU), so a budget of kb * B tokens takes whole blocks -- the blocks block-level selection
    takes wherever its margin is clear -- and the two paths give the same attention."""
    w, c, _ = SHAPES["gqa128"]
    kb = 3
    gu.log("[tokens] block-constant keys")
    d = gen.make_layer(w)
    d["k_pages"] = np.ascontiguousarray(np.broadcast_to(d["k_pages"][:, :, :1, :], d["k_pages"].shape))
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    tok = _run(w, d, cs, dev, kb * w.block_size)
    blk = gu.run_gpu(w.with_(top_k=kb), d, cs, dev)
    ref_blk = oracle.prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, sub_chunk=w.sub_chunk,
                             block_size=w.block_size, top_k=kb, sink_tokens=w.sink_tokens,
                             local_window=w.local_window, cluster_start=cs, with_output=False)
    n_same = 0
    for j, g in enumerate(ref_blk["geometry"]):
        st = tok["sel_idx"][j, :tok["sel_cnt"][j]].astype(np.int64)
        first = g.sink_blk * w.block_size
        row = tok["scores"][j, first:first + g.n_cand * w.block_size].reshape(-1, w.block_size)
        assert np.all(row == row[:, :1]), f"cluster {j}: token scores differ inside a block"
        assert len(st) % w.block_size == 0 and np.all(np.diff(st.reshape(-1, w.block_size), axis=1) == 1)
        if ref_blk["margins"][j] > gu.MARGIN:
            sb = blk["sel_idx"][j, :blk["sel_cnt"][j]].astype(np.int64)
            assert np.array_equal(st, oracle.selected_positions(g, sb, w.block_size))   # g: block geometry
            gu.check_output(tok["out"][g.s:g.e], blk["out"][g.s:g.e], f"cluster {j} token vs block")
            n_same += 1
    assert n_same >= 1
    gu.log(f"[tokens] block-constant keys: {n_same} of {len(cs) - 1} clusters compared")


def test_token_deterministic_and_page_permutation(dev):
    w, c, k = SHAPES["g7"]
    gu.log("[tokens] determinism + paging")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    a = _run(w, d, cs, dev, k)
    b = _run(w, d, cs, dev, k)
    for key in ("sel_idx", "sel_cnt", "out", "scores", "fingerprints"):
        assert np.array_equal(a[key], b[key]), key
    perm = np.random.default_rng(4).permutation(w.n_blocks)
    kp = np.empty_like(d["k_pages"])
    vp = np.empty_like(d["v_pages"])
    kp[perm] = d["k_pages"]
    vp[perm] = d["v_pages"]
    p = _run(w, dict(d, k_pages=kp, v_pages=vp, block_table=perm.astype(np.int32)), cs, dev, k)
    for key in ("sel_idx", "sel_cnt", "out", "scores"):
        assert np.array_equal(a[key], p[key]), key


def test_token_exact_ties_pick_lowest_position(dev):
    """Copies of the best token's key (all KV heads) score identically; the lowest positions win."""
    w, _, _ = SHAPES["gqa128"]
    k = 2
    gu.log("[tokens] exact ties")
    d = gen.make_layer(w)
    cs = np.array([0, 12, 16], dtype=np.int32)
    ref0 = _oracle(w, d, cs, k, with_output=False)
    g = ref0["geometry"][1]
    B = w.block_size
    first = g.sink_blk * B
    best = first + int(np.argmax(ref0["scores"][1]))
    rng = np.random.default_rng(5)
    dups = sorted(int(t) for t in rng.choice([t for t in range(first, first + g.n_cand) if t != best], 3,
                                             replace=False))
    src = d["k_pages"][d["block_table"][best // B], :, best % B, :].copy()
    for t in dups:
        d["k_pages"][d["block_table"][t // B], :, t % B, :] = src
    res = _run(w, d, cs, dev, k)
    ref = _oracle(w, d, cs, k, with_output=False)
    tied = sorted(dups + [best])
    assert list(ref["selections"][1]) == tied[:2]
    assert list(res["sel_idx"][1, :2]) == tied[:2]


@pytest.mark.parametrize("name,c", [("llama128k", 8), ("llama32k", 1)])
def test_token_full_size(dev, name, c):
    """Llama-3-8B-shaped layers at full context with a budget of 32 blocks' worth of tokens: the
    GPU runs the whole layer; every cluster is checked against the oracle (fingerprints, scores,
    selection) and every row of the attention output under the GPU's selection."""
    w = gen.WORKLOADS[name].with_(cluster=c)
    k = 32 * w.block_size
    gu.log(f"[tokens] {name} c={c}: generating")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    J = len(cs) - 1
    geo = oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, k, cs,
                          select_tokens=True)
    gu.log(f"[tokens] {name}: GPU, {J} clusters")
    res = _run(w, d, cs, dev, k)
    assert res["calls"] == J
    B = w.block_size
    n_max = max(g.sink_blk * B + g.n_cand for g in geo)
    K_all = oracle.logical_rows(d["k_pages"], d["block_table"], np.arange(n_max), B)
    ref = {"geometry": [], "fingerprints": [], "scores": [], "selections": []}
    for g in geo:
        v = oracle.anchor_fingerprint(d["q"], g.s, g.anchor_end)
        sc = oracle.soft_vote(oracle.block_logits(v, K_all[g.sink_blk * B:g.sink_blk * B + g.n_cand], w.num_kv_heads))
        sel, _ = oracle.select_topk(sc, g.sink_blk * B, k)
        for key, val in (("geometry", g), ("fingerprints", v), ("scores", sc), ("selections", sel)):
            ref[key].append(val)
    gu.log(f"[tokens] {name}: oracle selection of {J} clusters")
    cands = [K_all[g.sink_blk * B:g.sink_blk * B + g.n_cand] for g in geo]
    bounds = gu.token_score_bounds(ref, cands, w.num_kv_heads)
    del cands, K_all
    gu.check_rounding(res["fingerprints"], np.stack(ref["fingerprints"]), "fingerprints")
    worst = gu.check_token_scores(res["scores"], ref, bounds, B, name)
    n_exact = gu.check_token_selection(res["sel_idx"], res["sel_cnt"], res["scores"], ref, bounds, B, name)
    gu.log(f"[tokens] {name}: worst relative score error {worst:.2e}; {n_exact} of {J} clusters above the margin")
    sels = gu.gpu_selections(res, J)
    worst = (0.0, 0.0)
    for j, g in enumerate(geo):
        o_ref = oracle.cluster_attention(d["q"], d["k_pages"], d["v_pages"], d["block_table"], g, sels[j], B)
        mx, rel = gu.check_output(res["out"][g.s:g.e], o_ref, f"{name} cluster {j}")
        worst = (max(worst[0], mx), max(worst[1], rel))
        if j % 8 == 7 or j == J - 1:
            gu.log(f"[tokens] {name}: clusters up to {j} every row, worst max-abs {worst[0]:.2e} rel-L2 {worst[1]:.2e}")


def test_token_128k_one_call_per_subchunk_sampled(dev):
    """Token-level selection on the 128K layer with clusters of one sub-chunk (256 selection calls,
    the c = 1 end of the token sweep): the GPU runs the whole layer; 12 sampled clusters are checked
    against the oracle (fingerprints, scores, selection) and their first, last and two random
    32-row tiles of attention output under the GPU's selection."""
    w = gen.WORKLOADS["llama128k"].with_(cluster=1)
    k = 32 * w.block_size
    B = w.block_size
    gu.log("[tokens] llama128k c=1: generating")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 1)
    J = len(cs) - 1
    geo = oracle.geometry(w.n_tokens, w.sub_chunk, B, w.sink_tokens, w.local_window, k, cs, select_tokens=True)
    rng = np.random.default_rng(17)
    clusters = sorted({0, J - 1, *(int(x) for x in rng.choice(np.arange(1, J - 1), size=10, replace=False))})
    rows = gu.sample_rows([geo[j] for j in clusters], rng, tiles_per_cluster=2)
    gu.log(f"[tokens] llama128k c=1: GPU, {J} clusters")
    res = _run(w, d, cs, dev, k, out_rows=np.concatenate(rows))
    assert res["calls"] == J
    n_max = max(geo[j].sink_blk * B + geo[j].n_cand for j in clusters)
    K_all = oracle.logical_rows(d["k_pages"], d["block_table"], np.arange(n_max), B)
    ref = {"geometry": [], "fingerprints": [], "scores": [], "selections": []}
    cands = []
    for j in clusters:
        g = geo[j]
        v = oracle.anchor_fingerprint(d["q"], g.s, g.anchor_end)
        cand = K_all[g.sink_blk * B:g.sink_blk * B + g.n_cand]
        sc = oracle.soft_vote(oracle.block_logits(v, cand, w.num_kv_heads))
        sel, _ = oracle.select_topk(sc, g.sink_blk * B, k)
        for key, val in (("geometry", g), ("fingerprints", v), ("scores", sc), ("selections", sel)):
            ref[key].append(val)
        cands.append(cand)
    gu.log(f"[tokens] llama128k c=1: oracle selection of {len(clusters)} clusters")
    bounds = gu.token_score_bounds(ref, cands, w.num_kv_heads)
    del cands, K_all
    gu.check_rounding(res["fingerprints"][clusters], np.stack(ref["fingerprints"]), "fingerprints")
    worst = gu.check_token_scores(res["scores"][clusters], ref, bounds, B, "llama128k c=1")
    n_exact = gu.check_token_selection(res["sel_idx"][clusters], res["sel_cnt"][clusters], res["scores"][clusters],
                                       ref, bounds, B, "llama128k c=1")
    gu.log(f"[tokens] llama128k c=1: worst relative score error {worst:.2e}; {n_exact} of {len(clusters)} sampled "
           f"clusters above the margin")
    sels = gu.gpu_selections(res, J)
    at = 0
    for i, j in enumerate(clusters):
        o_ref = oracle.attention_rows(d["q"], d["k_pages"], d["v_pages"], d["block_table"], geo[j], sels[j], rows[i], B)
        gu.check_output(res["out"][at:at + len(rows[i])], o_ref, f"llama128k c=1 cluster {j}")
        at += len(rows[i])


def test_token_short_last_subchunk(dev):
    """n_tokens = 2368: nine sub-chunks of 256 and a last one of 64; clusters of 4; a budget off the
    tile."""
    w = gen.WORKLOADS["tiny"].with_(n_tokens=2368)
    k = 200
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 4)
    assert cs[-1] == 10
    res = _run(w, d, cs, dev, k)
    ref = _oracle(w, d, cs, k)
    _check_all("token short tail", w, d, cs, k, res, ref)


def test_token_incremental_prefill_equals_one_shot(dev):
    """The outer-chunk loop with token-level selection: each outer chunk of 16 sub-chunks selects
    tokens and attends against the cache so far; the result equals the one-shot run bit for bit."""
    import torch

    import paper_2609_31568_amd as pk

    w = gen.WORKLOADS["llama32k"]
    k = 2048
    d = gen.make_layer(w)
    outer = 16
    cs_full = gen.cluster_starts(w.n_sub_chunks, 8)        # 8 divides 16: no cluster straddles
    cfg = gu.config(w, len(cs_full) - 1, top_k=k, select_tokens=True)
    q, kp, vp, bt = (gu.to_dev(d[x], dev) for x in ("q", "k_pages", "v_pages", "block_table"))
    with pk.Scale(cfg) as h:
        one = pk.LayerBuffers(cfg, w.n_tokens, len(cs_full) - 1, device=dev)
        pk.run_layer(h, q, kp, vp, bt, w.n_tokens, cs_full, one)
        inc = pk.LayerBuffers(cfg, w.n_tokens, len(cs_full) - 1, device=dev)
        inc.out.fill_(float("nan"))
        sel_rows = []
        for o in range(w.n_sub_chunks // outer):
            n = (o + 1) * outer * w.sub_chunk
            cs = cs_full[(cs_full >= o * outer) & (cs_full <= (o + 1) * outer)]
            m = len(cs) - 1
            h.select_cluster_tokens(q, n, kp, bt, cs, inc.sel_idx[:m], inc.sel_cnt[:m])
            h.sparse_prefill(q, kp, vp, bt, n, cs, inc.sel_idx[:m], inc.sel_cnt[:m], inc.out)
            torch.cuda.synchronize()
            sel_rows.append(inc.sel_idx[:m].clone())
        torch.cuda.synchronize()
    assert torch.equal(torch.cat(sel_rows), one.sel_idx)
    assert torch.equal(one.out, inc.out)
    gu.log(f"[tokens] incremental = one-shot over {w.n_sub_chunks // outer} outer chunks")
