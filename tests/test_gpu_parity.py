"""GPU parity: the HIP path, called through the C ABI, against the fp64 oracle on the same seeded
inputs. Small shapes and the full-size Llama layers are compared on every selection and every
attention row; the larger workloads on sampled clusters and rows."""
import numpy as np
import pytest

import gen
import oracle
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

# eps of the eps-valid top-k check: ten times the score tolerance (gpu_util.SCORE_ATOL, 1e-6 absolute)
# and far below typical score gaps.
EPS_VALID = 1e-5


@pytest.fixture(scope="module")
def dev():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_31568_amd  # noqa: F401  (fails loudly if the library is missing)

    return torch.device("cuda:0")


def _oracle(w, d, cs, n=None, with_output=True, external_sel=None):
    n = w.n_tokens if n is None else n
    return oracle.prefill(d["q"][:n], d["k_pages"], d["v_pages"], d["block_table"], n, sub_chunk=w.sub_chunk,
                          block_size=w.block_size, top_k=w.top_k, sink_tokens=w.sink_tokens,
                          local_window=w.local_window, cluster_start=cs, with_output=with_output,
                          external_sel=external_sel)


SHAPES = {
    # name: (workload, cluster size)
    "tiny_c4": (gen.WORKLOADS["tiny"], 4),
    "tiny_c1": (gen.WORKLOADS["tiny"], 1),
    # GQA 4:1, d 128, B 128, cluster 3 of M = 16 (ragged last cluster), cluster longer than W
    "gqa128": (gen.Workload("gqa128", 1, 8, 2, 128, 8192, 128, 512, 3, 5, 128, 1024, 12, 1, 4, 31), 3),
    # group of 7 query heads, d 128, B 64
    "g7": (gen.Workload("g7", 1, 14, 2, 128, 4096, 64, 256, 4, 6, 64, 512, 8, 1, 3, 32), 4),
    # MHA (group 1), d 64, B 128, no sink, window not a block multiple
    "g1": (gen.Workload("g1", 1, 2, 2, 64, 4096, 128, 512, 2, 3, 0, 700, 6, 1, 3, 33), 2),
    # group 8, sink rounded up to 3 blocks, short window
    "g8": (gen.Workload("g8", 1, 8, 1, 64, 2048, 64, 128, 5, 4, 130, 100, 6, 1, 5, 34), 5),
    # the remaining group sizes: 2 (4 row blocks), and 3, 5, 6, whose work-groups (384, 320, 384
    # threads) do not divide the tile's 16-byte chunks evenly
    "g2": (gen.Workload("g2", 1, 4, 2, 128, 4096, 128, 512, 2, 4, 128, 600, 8, 1, 3, 36), 2),
    "g3": (gen.Workload("g3", 1, 6, 2, 128, 4096, 64, 256, 3, 6, 64, 512, 8, 1, 3, 37), 3),
    "g5": (gen.Workload("g5", 1, 5, 1, 128, 4096, 128, 512, 2, 3, 128, 900, 6, 1, 3, 38), 2),
    "g6": (gen.Workload("g6", 1, 12, 2, 64, 3072, 128, 256, 4, 5, 128, 512, 8, 1, 3, 39), 4),
    # d 64 work-groups of 6 x 2, 4 x 3 and 2 x 5 waves (three waves per SIMD where they fit)
    "g2d64": (gen.Workload("g2d64", 1, 4, 2, 64, 4096, 64, 256, 3, 5, 64, 700, 8, 1, 3, 40), 3),
    "g3d64": (gen.Workload("g3d64", 1, 3, 1, 64, 3072, 128, 512, 2, 3, 128, 600, 6, 1, 3, 42), 2),
    "g5d64": (gen.Workload("g5d64", 1, 10, 2, 64, 4096, 128, 512, 2, 4, 128, 1000, 6, 1, 3, 43), 2),
}


@pytest.mark.parametrize("name", list(SHAPES))
def test_small_shapes_full_parity(dev, name):
    w, c = SHAPES[name]
    gu.log(f"[parity] {name}")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    res = gu.run_gpu(w, d, cs, dev)
    ref = _oracle(w, d, cs)
    gu.check_rounding(res["k_rep"], ref["k_rep"], "k_rep")
    gu.check_rounding(res["fingerprints"], np.stack(ref["fingerprints"]), "fingerprints")
    gu.check_scores(res["scores"], ref, name)
    gu.check_selection(res["sel_idx"], res["sel_cnt"], ref, EPS_VALID)
    assert res["calls"] == len(cs) - 1
    # attention under the GPU's own selection, every row and head
    own = _oracle(w, d, cs, external_sel=gu.gpu_selections(res, len(cs) - 1))
    mx, rel = gu.check_output(res["out"], own["output"], f"{name} output")
    gu.log(f"[parity] {name}: max-abs {mx:.2e} rel-L2 {rel:.2e}")
    # and under the oracle's selection on clusters where both agree
    for j, g in enumerate(ref["geometry"]):
        if np.array_equal(gu.gpu_selections(res, len(cs) - 1)[j], ref["selections"][j]):
            gu.check_output(res["out"][g.s:g.e], ref["output"][g.s:g.e], f"{name} cluster {j}")


def test_dense_reduction_on_gpu(dev):
    """top_k >= every candidate count: the GPU output must be dense causal attention."""
    w = SHAPES["gqa128"][0].with_(top_k=64)
    gu.log("[parity] dense reduction")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 3)
    res = gu.run_gpu(w, d, cs, dev)
    ref = _oracle(w, d, cs)
    assert all(g.sel_cnt == g.n_cand for g in ref["geometry"])
    gu.check_output(res["out"], ref["output"], "dense")


def test_short_last_subchunk(dev):
    """n_tokens = 2368: nine sub-chunks of 256 and a last one of 64; clusters of 4."""
    w = gen.WORKLOADS["tiny"].with_(n_tokens=2368)
    gu.log("[parity] short last sub-chunk")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 4)
    assert cs[-1] == 10
    res = gu.run_gpu(w, d, cs, dev)
    ref = _oracle(w, d, cs)
    gu.check_selection(res["sel_idx"], res["sel_cnt"], ref, EPS_VALID)
    own = _oracle(w, d, cs, external_sel=gu.gpu_selections(res, len(cs) - 1))
    gu.check_output(res["out"], own["output"], "short tail")


@pytest.mark.parametrize("name,over", [
    ("gqa128", {}),                                  # d 128, four heads per work-group
    ("g7", {}),                                      # d 128, one head x 8 row blocks
    ("g2d64", {}),                                   # d 64, 12-wave work-groups
    ("gqa128", {"select_tokens": True, "top_k": 603}),   # token-level, padded last gathered tile
    ("g5d64", {"select_tokens": True, "top_k": 200}),
], ids=["gqa128", "g7", "g2d64", "gqa128-tokens", "g5d64-tokens"])
def test_bf16_output_is_rne_of_fp32(dev, name, over):
    """The bf16 epilogue of every kernel shape rounds the fp32 result to nearest even, bit for bit."""
    w, c = SHAPES[name]
    gu.log(f"[parity] bf16 epilogue {name} {over}")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    r32 = gu.run_gpu(w, d, cs, dev, **over)
    r16 = gu.run_gpu(w, d, cs, dev, out_bf16=True, **over)
    assert np.array_equal(r16["sel_idx"], r32["sel_idx"])
    assert np.array_equal(r16["out"].view(np.uint16), gu.bf16_rne(r32["out"]))


def test_cluster_sets_change_between_calls(dev):
    """One handle, a sequence of layers whose clusters change, return and repeat (the handle keeps
    the device geometry and work list of the last cluster set and uploads or rebuilds them only
    when the set changes): every layer must give the bits of a fresh handle for its own set, and
    the sets' calls must each select from the set they were given."""
    import torch

    import paper_2609_31568_amd as pk

    w = SHAPES["gqa128"][0]
    d = gen.make_layer(w)
    q, kp, vp, bt = gu.upload(d, dev)
    n_short = w.n_tokens - w.sub_chunk
    cs_a = gen.cluster_starts(w.n_sub_chunks, 3)
    cs_b = gen.cluster_starts(w.n_sub_chunks, 5)
    cs_c = gen.cluster_starts(w.n_sub_chunks - 1, 3)     # the same starts as cs_a, one sub-chunk shorter
    runs = [("a", cs_a, w.n_tokens), ("b", cs_b, w.n_tokens), ("a", cs_a, w.n_tokens), ("a", cs_a, w.n_tokens),
            ("c", cs_c, n_short), ("a", cs_a, w.n_tokens)]
    fresh = {}
    for name, cs, n in runs:
        if name not in fresh:
            fresh[name] = gu.run_gpu(w, d, cs, dev, n_tokens=n, dev_data=(q[:n], kp, vp, bt))
    cfg = gu.config(w, max(len(cs) - 1 for _, cs, _ in runs))
    gu.log("[parity] cluster sets changing between calls on one handle")
    with pk.Scale(cfg) as h:
        for name, cs, n in runs:
            bufs = pk.LayerBuffers(cfg, n, len(cs) - 1, device=dev, with_scores=True)
            pk.run_layer(h, q[:n], kp, vp, bt, n, cs, bufs)
            torch.cuda.synchronize()
            ref = fresh[name]
            assert np.array_equal(bufs.sel_cnt.cpu().numpy(), ref["sel_cnt"]), name
            assert np.array_equal(bufs.sel_idx.cpu().numpy(), ref["sel_idx"]), name
            assert np.array_equal(bufs.scores.cpu().numpy(), ref["scores"]), name
            assert np.array_equal(bufs.out.cpu().numpy(), ref["out"]), name


def test_work_item_counts_alternate_on_one_handle(dev):
    """Attention work-groups take their items from per-XCD queues whose counters the last
    work-group clears for the next launch. Alternate launches with fewer items than the eight
    queues, as many, a few more and many on one handle: every launch must give the bits of a fresh
    handle, so no counter is left set and no item is skipped or taken twice."""
    import torch

    import paper_2609_31568_amd as pk

    w = SHAPES["gqa128"][0]     # d 128, 2 KV heads of 4 query heads: 64-row items per KV head
    d = gen.make_layer(w)
    q, kp, vp, bt = gu.upload(d, dev)
    full = gen.cluster_starts(w.n_sub_chunks, 3)
    # (context length, cluster starts): 128 tokens -> 2 row tiles x 2 KV heads = 4 items; 256 -> 8;
    # 384 -> 12; the full context -> 256 items
    runs = [(128, [0, 1]), (w.n_tokens, full), (256, [0, 1]), (384, [0, 1]), (w.n_tokens, full), (128, [0, 1])]
    fresh = {}
    for n, cs in runs:
        if n not in fresh:
            fresh[n] = gu.run_gpu(w, d, np.asarray(cs, dtype=np.int32), dev, n_tokens=n,
                                  dev_data=(q[:n], kp, vp, bt))
    cfg = gu.config(w, len(full) - 1)
    gu.log("[parity] work-item counts alternating on one handle")
    with pk.Scale(cfg) as h:
        for n, cs in runs:
            cs = np.asarray(cs, dtype=np.int32)
            bufs = pk.LayerBuffers(cfg, n, len(cs) - 1, device=dev, with_scores=True)
            pk.run_layer(h, q[:n], kp, vp, bt, n, cs, bufs)
            torch.cuda.synchronize()
            assert np.array_equal(bufs.out.float().cpu().numpy(), fresh[n]["out"]), n
    for n in (128, 384):
        ref = _oracle(w, d, np.asarray([0, 1], dtype=np.int32), n=n)
        gu.check_output(fresh[n]["out"], ref["output"], f"{n}-token context")


def test_deterministic_and_page_permutation(dev):
    w, c = SHAPES["g7"]
    gu.log("[parity] determinism + paging")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    a = gu.run_gpu(w, d, cs, dev)
    b = gu.run_gpu(w, d, cs, dev)
    for key in ("k_rep", "sel_idx", "sel_cnt", "out", "scores", "fingerprints"):
        assert np.array_equal(a[key], b[key]), key
    perm = np.random.default_rng(3).permutation(w.n_blocks)
    kp = np.empty_like(d["k_pages"])
    vp = np.empty_like(d["v_pages"])
    kp[perm] = d["k_pages"]
    vp[perm] = d["v_pages"]
    p = gu.run_gpu(w, dict(d, k_pages=kp, v_pages=vp, block_table=perm.astype(np.int32)), cs, dev)
    for key in ("k_rep", "sel_idx", "sel_cnt", "out", "scores"):
        assert np.array_equal(a[key], p[key]), key


@pytest.mark.parametrize("over", [{}, {"select_tokens": True, "top_k": 333}], ids=["blocks", "tokens"])
def test_null_block_table_is_identity(dev, over):
    """A NULL block table maps logical block b to page b: bit-identical to passing the identity table
    (representative keys, the token gather and attention all read pages through it)."""
    w, c = SHAPES["g7"]
    gu.log(f"[parity] NULL block table {over}")
    d = gen.make_layer(w)
    assert np.array_equal(d["block_table"], np.arange(w.n_blocks))
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    a = gu.run_gpu(w, d, cs, dev, **over)
    q, kp, vp, _ = gu.upload(d, dev)
    b = gu.run_gpu(w, d, cs, dev, dev_data=(q, kp, vp, None), **over)
    keys = ("sel_idx", "sel_cnt", "out", "scores") + (() if over else ("k_rep",))
    for key in keys:
        assert np.array_equal(a[key], b[key]), key


def test_exact_ties_pick_lowest_index(dev):
    """Duplicated K blocks give identical scores on the GPU too; the lowest indices win."""
    w = SHAPES["gqa128"][0].with_(top_k=2)
    gu.log("[parity] exact ties")
    d = gen.make_layer(w)
    cs = np.array([0, 12, 16], dtype=np.int32)
    ref0 = _oracle(w, d, cs, with_output=False)
    g = ref0["geometry"][1]
    sc = ref0["scores"][1]
    best = g.sink_blk + int(np.argmax(sc))
    dups = [b for b in range(g.sink_blk, g.sink_blk + g.n_cand) if b != best][:3]
    for b in dups:
        d["k_pages"][b] = d["k_pages"][best]
    res = gu.run_gpu(w, d, cs, dev)
    ref = _oracle(w, d, cs, with_output=False)
    tied = sorted(dups + [best])
    assert list(ref["selections"][1]) == tied[:2]
    assert list(res["sel_idx"][1, :2]) == tied[:2]


def test_items_with_more_than_256_tiles(dev):
    """A window of 18000 tokens: late work items walk more than 256 key tiles, so the kernel's tile
    table is refilled mid-item. Checked on sampled rows of every cluster."""
    w = gen.Workload("wide", 1, 4, 1, 64, 20480, 64, 512, 2, 4, 64, 18000, 10, 1, 3, 41)
    gu.log("[parity] wide window")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 2)
    res = gu.run_gpu(w, d, cs, dev)
    ref = _oracle(w, d, cs, with_output=False)
    gu.check_selection(res["sel_idx"], res["sel_cnt"], ref, EPS_VALID)
    last = ref["geometry"][-1]
    assert (last.e - last.lo_blk * w.block_size) // 64 > 256
    rows = gu.sample_rows(ref["geometry"], np.random.default_rng(9), tiles_per_cluster=2)
    sels = gu.gpu_selections(res, len(cs) - 1)
    for j, g in enumerate(ref["geometry"]):
        o_ref = oracle.attention_rows(d["q"], d["k_pages"], d["v_pages"], d["block_table"], g, sels[j], rows[j],
                                      w.block_size)
        gu.check_output(res["out"][rows[j]], o_ref, f"wide cluster {j}")


@pytest.mark.parametrize("name,seed_rows,every_row", [("llama32k", 5, True), ("llama128k", 6, True)])
def test_full_size_llama(dev, name, seed_rows, every_row):
    """Full Llama-3-8B-layer workloads: every selection, and attention on every row of every
    cluster against the fp64 oracle on the GPU's own selection (2.1 and 13.2 TFLOP of oracle work)."""
    w = gen.WORKLOADS[name]
    gu.log(f"[parity] {name}: generating")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    gu.log(f"[parity] {name}: GPU")
    res = gu.run_gpu(w, d, cs, dev)
    gu.log(f"[parity] {name}: oracle selection")
    ref = _oracle(w, d, cs, with_output=False)
    gu.check_rounding(res["k_rep"], ref["k_rep"], "k_rep")
    gu.check_rounding(res["fingerprints"], np.stack(ref["fingerprints"]), "fingerprints")
    worst = gu.check_scores(res["scores"], ref, name)
    gu.log(f"[parity] {name}: worst score error {worst:.2e}")
    n_exact = gu.check_selection(res["sel_idx"], res["sel_cnt"], ref, EPS_VALID)
    gu.log(f"[parity] {name}: {n_exact} of {len(cs) - 1} clusters above the margin, all equal")
    assert res["calls"] == len(cs) - 1
    rng = np.random.default_rng(seed_rows)
    rows = ([np.arange(g.s, g.e) for g in ref["geometry"]] if every_row else gu.sample_rows(ref["geometry"], rng))
    sels = gu.gpu_selections(res, len(cs) - 1)
    worst = (0.0, 0.0)
    for j, g in enumerate(ref["geometry"]):
        if every_row:
            o_ref = oracle.cluster_attention(d["q"], d["k_pages"], d["v_pages"], d["block_table"], g, sels[j],
                                             w.block_size)
        else:
            o_ref = oracle.attention_rows(d["q"], d["k_pages"], d["v_pages"], d["block_table"], g, sels[j],
                                          rows[j], w.block_size)
        mx, rel = gu.check_output(res["out"][rows[j]], o_ref, f"{name} cluster {j}")
        worst = (max(worst[0], mx), max(worst[1], rel))
        if every_row:
            gu.log(f"[parity] {name}: cluster {j} every row, max-abs {mx:.2e} rel-L2 {rel:.2e}")
    gu.log(f"[parity] {name}: {'every-row' if every_row else 'sampled'} attention worst max-abs {worst[0]:.2e} "
           f"rel-L2 {worst[1]:.2e}")


def _oracle_clusters(w, d, cs, clusters, k_rep=None):
    """The oracle's selection (Alg. 2's per-cluster steps) for the listed clusters only, with the
    representative keys of every block they score (or the given ones); the same layout as
    oracle.prefill's result."""
    geo = oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, w.top_k, cs)
    n_rep = max(geo[j].sink_blk + geo[j].n_cand for j in clusters)
    if k_rep is None:
        k_rep = oracle.rep_keys(d["k_pages"], d["block_table"], w.n_tokens, w.block_size, blocks=np.arange(n_rep))
    k_rep = k_rep[:n_rep]
    ref = {"geometry": [], "fingerprints": [], "scores": [], "selections": [], "margins": [], "k_rep": k_rep}
    for j in clusters:
        g = geo[j]
        v = oracle.anchor_fingerprint(d["q"], g.s, g.anchor_end)
        sc = oracle.soft_vote(oracle.block_logits(v, k_rep[g.sink_blk:g.sink_blk + g.n_cand], w.num_kv_heads))
        sel, margin = oracle.select_topk(sc, g.sink_blk, w.top_k)
        for key, val in (("geometry", g), ("fingerprints", v), ("scores", sc), ("selections", sel),
                         ("margins", margin)):
            ref[key].append(val)
    return ref


def _sampled_layer(dev, w, d, cs, clusters, rng, name, dev_data=None, k_rep=None):
    """The GPU runs the whole layer; the listed clusters are checked against the oracle --
    representative keys, fingerprints, scores, selection -- and attention on each cluster's first
    and last 32-row tiles plus two random ones, on the GPU's own selection."""
    J = len(cs) - 1
    geo = oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, w.top_k, cs)
    rows = gu.sample_rows([geo[j] for j in clusters], rng, tiles_per_cluster=2)
    gu.log(f"[parity] {name}: GPU, {J} clusters")
    res = gu.run_gpu(w, d, cs, dev, out_rows=np.concatenate(rows), dev_data=dev_data)
    assert res["calls"] == J
    gu.log(f"[parity] {name}: oracle on {len(clusters)} clusters")
    ref = _oracle_clusters(w, d, cs, clusters, k_rep=k_rep)
    gu.check_rounding(res["k_rep"][:len(ref["k_rep"])], ref["k_rep"], "k_rep")
    gu.check_rounding(res["fingerprints"][clusters], np.stack(ref["fingerprints"]), "fingerprints")
    worst = gu.check_scores(res["scores"][clusters], ref, name)
    n_exact = gu.check_selection(res["sel_idx"][clusters], res["sel_cnt"][clusters], ref, EPS_VALID)
    gu.log(f"[parity] {name}: worst score error {worst:.2e}; {n_exact} of {len(clusters)} sampled clusters above "
           f"the margin, all equal")
    sels = gu.gpu_selections(res, J)
    worst, at = (0.0, 0.0), 0
    for i, j in enumerate(clusters):
        o_ref = oracle.attention_rows(d["q"], d["k_pages"], d["v_pages"], d["block_table"], geo[j], sels[j], rows[i],
                                      w.block_size)
        mx, rel = gu.check_output(res["out"][at:at + len(rows[i])], o_ref, f"{name} cluster {j}")
        at += len(rows[i])
        worst = (max(worst[0], mx), max(worst[1], rel))
    gu.log(f"[parity] {name}: sampled attention ({sum(len(r) for r in rows)} rows) worst max-abs {worst[0]:.2e} "
           f"rel-L2 {worst[1]:.2e}")
    return ref


def _sample_clusters(J, n_sample, rng, always=()):
    """First, last, the `always` ones and random others, n_sample in all."""
    fixed = {0, J - 1, *always}
    rest = [j for j in range(1, J - 1) if j not in fixed]
    extra = rng.choice(np.asarray(rest), size=max(0, min(len(rest), n_sample - len(fixed))), replace=False)
    return sorted(fixed | set(int(x) for x in extra))


@pytest.fixture(scope="module")
def stress1m(dev):
    """The 1M-token Llama-shaped layer, generated and uploaded once, with the oracle's
    representative keys of every block."""
    import torch

    w = gen.WORKLOADS["stress1m"]
    gu.log("[parity] stress1m: generating")
    d = gen.make_layer(w)
    dev_data = gu.upload(d, dev)
    gu.log("[parity] stress1m: oracle representative keys")
    k_rep = oracle.rep_keys(d["k_pages"], d["block_table"], w.n_tokens, w.block_size)
    yield w, d, dev_data, k_rep
    del dev_data
    torch.cuda.empty_cache()


@pytest.mark.parametrize("c,n_sample,seed", [(1, 16, 8), (2, 12, 9), (4, 12, 10), (8, 12, 11), (16, 10, 12)])
def test_stress1m_sampled(dev, stress1m, c, n_sample, seed):
    """The 1M context at every cluster size of the sweep; at c = 16 a cluster (8192 rows) is longer
    than the base window, so the local window spans the cluster (Eq. 10)."""
    w, d, dev_data, k_rep = stress1m
    w = w.with_(cluster=c)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    rng = np.random.default_rng(seed)
    clusters = _sample_clusters(len(cs) - 1, n_sample, rng)
    ref = _sampled_layer(dev, w, d, cs, clusters, rng, f"stress1m c={c}", dev_data=dev_data, k_rep=k_rep)
    if c == 16:
        assert all(g.e - g.s > w.local_window and g.lo_blk * w.block_size == g.s for g in ref["geometry"])


@pytest.mark.parametrize("layer,seed", [(0, 7), (13, 13), (27, 14)])
def test_qwen256k_layer_sampled(dev, layer, seed):
    """Layers of the Qwen2-7B-shaped stack at 256K (G = 7, independent per-layer inputs)."""
    w = gen.WORKLOADS["qwen256k"]
    gu.log(f"[parity] qwen256k layer {layer}: generating")
    d = gen.make_layer(w, layer)
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    rng = np.random.default_rng(seed)
    clusters = _sample_clusters(len(cs) - 1, 10, rng)
    _sampled_layer(dev, w, d, cs, clusters, rng, f"qwen256k layer {layer}")


def test_kv_head_shard_sampled(dev):
    """The 128K layer's four-way KV-head shard (8 query / 2 KV heads per GPU): 4096 work items,
    16 per CU, so the queues run dry four times sooner than at the full layer."""
    w = gen.WORKLOADS["llama128k_tp4"]
    gu.log("[parity] llama128k_tp4: generating")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    rng = np.random.default_rng(16)
    clusters = _sample_clusters(len(cs) - 1, 10, rng)
    _sampled_layer(dev, w, d, cs, clusters, rng, "llama128k_tp4")


def test_topk_spill_path(dev):
    """More candidates than the top-k keeps in LDS (8192): a 640K context in blocks of 64 gives up to
    10175 candidates, so the last clusters' scores go through the global spill row, and their heads'
    softmax partials span 160 chunks."""
    w = gen.Workload("spill", 1, 4, 1, 64, 655360, 64, 512, 8, 16, 64, 4096, 512, 1, 8, 44)
    gu.log("[parity] spill: generating")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    J = len(cs) - 1
    rng = np.random.default_rng(15)
    geo = oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, w.top_k, cs)
    spilled = [j for j in range(J) if geo[j].n_cand > 8192]
    assert len(spilled) > 20
    clusters = _sample_clusters(J, 10, rng, always=(spilled[0], spilled[len(spilled) // 2], J - 2))
    _sampled_layer(dev, w, d, cs, clusters, rng, "spill")


def test_abi_errors_on_device(dev):
    """Invalid calls on a live handle return their status and launch nothing."""
    import ctypes

    import torch

    import paper_2609_31568_amd as pk

    w = gen.WORKLOADS["tiny"]
    cfg = gu.config(w, 2)
    with pk.Scale(cfg) as h:
        lib = pk.lib
        buf = torch.zeros(1 << 20, dtype=torch.int32, device=dev)
        p = buf.data_ptr()
        cs = np.array([0, 4, 8], dtype=np.int32)
        assert lib.scale_rep_keys(h.handle, p, None, 2048 + 64, p) == pk.SCALE_ERR_CAPACITY
        assert lib.scale_rep_keys(h.handle, p, None, 100, p) == pk.SCALE_ERR_UNSUPPORTED
        assert lib.scale_rep_keys(h.handle, None, None, 2048, p) == pk.SCALE_ERR_INVALID_ARG
        big = np.array([0, 1, 2, 8], dtype=np.int32)
        assert lib.scale_select_cluster(h.handle, p, 2048, p, big.ctypes.data, 3, p, p, None) == \
            pk.SCALE_ERR_CAPACITY
        bad = np.array([0, 5, 4], dtype=np.int32)
        assert lib.scale_select_cluster(h.handle, p, 2048, p, bad.ctypes.data, 2, p, p, None) == \
            pk.SCALE_ERR_INVALID_ARG
        assert lib.scale_sparse_prefill(h.handle, p, p, p, None, 2048, cs.ctypes.data, 2, p, None, p) == \
            pk.SCALE_ERR_INVALID_ARG
        # tensors that do not start on a 16-byte boundary (the kernels' vector width)
        assert lib.scale_rep_keys(h.handle, p + 2, None, 2048, p) == pk.SCALE_ERR_INVALID_ARG
        assert lib.scale_rep_keys_range(h.handle, p + 8, None, 0, 2048, p) == pk.SCALE_ERR_INVALID_ARG
        assert lib.scale_select_cluster(h.handle, p + 2, 2048, p, cs.ctypes.data, 2, p, p, None) == \
            pk.SCALE_ERR_INVALID_ARG
        assert lib.scale_select_cluster(h.handle, p, 2048, p + 4, cs.ctypes.data, 2, p, p, None) == \
            pk.SCALE_ERR_INVALID_ARG
        for args in [(p + 2, p, p), (p, p + 2, p), (p, p, p + 2)]:
            assert lib.scale_sparse_prefill(h.handle, *args, None, 2048, cs.ctypes.data, 2, p, p, p) == \
                pk.SCALE_ERR_INVALID_ARG
        assert lib.scale_sparse_prefill(h.handle, p, p, p, None, 2048, cs.ctypes.data, 2, p, p, p + 8) == \
            pk.SCALE_ERR_INVALID_ARG
        cs_out = np.zeros(9, dtype=np.int32)
        n_cl = ctypes.c_int32()
        assert lib.scale_cluster_subchunks(h.handle, p + 2, 2048, 0, 0.9, 1024, 0, cs_out.ctypes.data,
                                           ctypes.byref(n_cl), None) == pk.SCALE_ERR_INVALID_ARG
        assert lib.scale_select_cluster_static(ctypes.byref(cfg.base), None, p + 2, 2048, p, cs.ctypes.data, 2, p, p,
                                               None) == pk.SCALE_ERR_INVALID_ARG
        n = ctypes.c_int64()
        assert lib.scale_retrieval_calls(h.handle, ctypes.byref(n)) == 0 and n.value == 0
        torch.cuda.synchronize()
        assert int(buf.abs().sum()) == 0


def test_abi_selection_mode_mismatch(dev):
    """The block-level selection call refuses a token-level handle and the token-level call a
    block-level one, with SCALE_ERR_UNSUPPORTED, counting no call and launching nothing."""
    import ctypes

    import torch

    import paper_2609_31568_amd as pk

    w = gen.WORKLOADS["tiny"]
    buf = torch.zeros(1 << 20, dtype=torch.int32, device=dev)
    p = buf.data_ptr()
    cs = np.array([0, 4, 8], dtype=np.int32)
    n = ctypes.c_int64()
    with pk.Scale(gu.config(w, 2, select_tokens=True)) as h:
        assert pk.lib.scale_select_cluster(h.handle, p, 2048, p, cs.ctypes.data, 2, p, p, None) == \
            pk.SCALE_ERR_UNSUPPORTED
        assert pk.lib.scale_retrieval_calls(h.handle, ctypes.byref(n)) == 0 and n.value == 0
    with pk.Scale(gu.config(w, 2)) as h:
        assert pk.lib.scale_select_cluster_tokens(h.handle, p, 2048, p, None, cs.ctypes.data, 2, p, p, None) == \
            pk.SCALE_ERR_UNSUPPORTED
        assert pk.lib.scale_retrieval_calls(h.handle, ctypes.byref(n)) == 0 and n.value == 0
    torch.cuda.synchronize()
    assert int(buf.abs().sum()) == 0


@pytest.mark.parametrize("name,w,cs", [
    # one block and one short sub-chunk: no candidates, no sinks, dense causal attention
    ("one_block", gen.WORKLOADS["tiny"].with_(n_tokens=64), [0, 1]),
    # a context shorter than one sub-chunk
    ("short_ctx", gen.WORKLOADS["tiny"].with_(n_tokens=192), [0, 1]),
    # no budget: sinks and the local window only
    ("k0", gen.WORKLOADS["tiny"].with_(top_k=0), gen.cluster_starts(8, 2)),
    # no sink tokens and a zero base window: the window is the cluster itself
    ("s0_w0", gen.WORKLOADS["tiny"].with_(sink_tokens=0, local_window=0), gen.cluster_starts(8, 4)),
    # one cluster of every sub-chunk
    ("one_cluster", gen.WORKLOADS["tiny"], [0, 8]),
])
def test_degenerate_shapes(dev, name, w, cs):
    gu.log(f"[parity] degenerate {name}")
    d = gen.make_layer(w)
    cs = np.asarray(cs, dtype=np.int32)
    res = gu.run_gpu(w, d, cs, dev)
    ref = _oracle(w, d, cs)
    gu.check_selection(res["sel_idx"][:, :w.top_k], res["sel_cnt"], ref, EPS_VALID)   # rows hold top_k entries
    gu.check_output(res["out"], ref["output"], f"degenerate {name}")
    assert res["calls"] == len(cs) - 1
