"""GPU parity of the selection variants against the fp64 oracle: channel-wise min/max bound
representative keys (the page criticality of Quest, cited in paper Sec. 2), one index set per KV
head voted by its own query heads, and the selection logit scale sigma = 1/sqrt(d), in block and
token mode."""
import math

import numpy as np
import pytest

import gen
import oracle
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

EPS_VALID = 1e-5


@pytest.fixture(scope="module")
def dev():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_31568_amd  # noqa: F401  (fails loudly if the library is missing)

    return torch.device("cuda:0")


GQA = gen.Workload("gqa128", 1, 8, 2, 128, 8192, 128, 512, 3, 5, 128, 1024, 12, 1, 4, 31)
G7 = gen.Workload("g7", 1, 14, 2, 128, 4096, 64, 256, 4, 6, 64, 512, 8, 1, 3, 32)
G8 = gen.Workload("g8", 1, 8, 1, 64, 2048, 64, 128, 5, 4, 130, 100, 6, 1, 5, 34)


def _oracle(w, d, cs, **kw):
    base = dict(sub_chunk=w.sub_chunk, block_size=w.block_size, top_k=w.top_k, sink_tokens=w.sink_tokens,
                local_window=w.local_window)
    base.update(kw)
    return oracle.prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, cluster_start=cs, **base)


def _group_view(ref, g, Hkv, G, k_rep=None):
    """The per-KV-head result of KV head g as a one-KV-head result (its query heads only)."""
    out = {"geometry": ref["geometry"], "fingerprints": [v[g * G:(g + 1) * G] for v in ref["fingerprints"]],
           "scores": [s[g] for s in ref["scores"]], "selections": [s[g] for s in ref["selections"]],
           "margins": [m[g] for m in ref["margins"]]}
    if k_rep is not None:
        out["k_rep"] = k_rep[:, g:g + 1]
    return out


def _gpu_sets(res, n_clusters, Hkv):
    """GPU selection rows j * Hkv + g as one [Hkv, cnt] array per cluster."""
    return [np.stack([res["sel_idx"][j * Hkv + g, :res["sel_cnt"][j * Hkv + g]] for g in range(Hkv)]).astype(np.int64)
            for j in range(n_clusters)]


@pytest.mark.parametrize("w,c,sigma", [(GQA, 3, 1.0), (G7, 4, 1.0), (G8, 5, 1.0), (GQA, 3, 1.0 / math.sqrt(128))])
def test_bound_representative_keys(dev, w, c, sigma):
    gu.log(f"[variants] bounds {w.name} sigma={sigma:.3f}")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    res = gu.run_gpu(w, d, cs, dev, rep_bounds=True, score_scale=sigma)
    ref = _oracle(w, d, cs, rep_kind="minmax", score_scale=sigma)
    mn, mx = ref["bounds"]
    # channel-wise bounds of bf16 keys are exact in fp32
    assert np.array_equal(res["k_rep"][:, :, 0, :].astype(np.float64), mn)
    assert np.array_equal(res["k_rep"][:, :, 1, :].astype(np.float64), mx)
    worst = gu.check_scores(res["scores"], ref, w.name)
    n_exact = gu.check_selection(res["sel_idx"], res["sel_cnt"], ref, EPS_VALID)
    own = _oracle(w, d, cs, rep_kind="minmax", score_scale=sigma, external_sel=gu.gpu_selections(res, len(cs) - 1))
    mx_err, rel = gu.check_output(res["out"], own["output"], f"{w.name} bounds output")
    gu.log(f"[variants] bounds {w.name}: worst score error {worst:.2e}, {n_exact} of {len(cs) - 1} exact, "
           f"output {mx_err:.2e} / {rel:.2e}")


@pytest.mark.parametrize("w,c,bounds", [(GQA, 3, False), (G7, 4, False), (GQA, 2, True)])
def test_per_kv_head_sets_block_mode(dev, w, c, bounds):
    gu.log(f"[variants] per-KV-head sets {w.name} bounds={bounds}")
    Hkv, G = w.num_kv_heads, w.num_q_heads // w.num_kv_heads
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    J = len(cs) - 1
    res = gu.run_gpu(w, d, cs, dev, kv_head_sets=True, rep_bounds=bounds)
    ref = _oracle(w, d, cs, kv_head_sets=True, rep_kind="minmax" if bounds else "mean")
    n_exact = 0
    for g in range(Hkv):
        view = _group_view(ref, g, Hkv, G, ref["k_rep"])
        gu.check_scores(res["scores"][g::Hkv], view, f"{w.name} KV head {g}")
        n_exact += gu.check_selection(res["sel_idx"][g::Hkv], res["sel_cnt"][g::Hkv], view, EPS_VALID)
    sets = _gpu_sets(res, J, Hkv)
    own = _oracle(w, d, cs, kv_head_sets=True, rep_kind="minmax" if bounds else "mean", external_sel=sets)
    mx_err, rel = gu.check_output(res["out"], own["output"], f"{w.name} per-KV-head output")
    for j, geo in enumerate(ref["geometry"]):
        if np.array_equal(sets[j], ref["selections"][j]):
            gu.check_output(res["out"][geo.s:geo.e], ref["output"][geo.s:geo.e], f"{w.name} cluster {j}")
    gu.log(f"[variants] per-KV-head {w.name}: {n_exact} of {J * Hkv} sets exact, output {mx_err:.2e} / {rel:.2e}")


def test_per_kv_head_sets_with_one_kv_head_equal_shared(dev):
    w = G8
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 5)
    a = gu.run_gpu(w, d, cs, dev, kv_head_sets=True)
    b = gu.run_gpu(w, d, cs, dev)
    for key in ("sel_idx", "sel_cnt", "out", "scores"):
        assert np.array_equal(a[key], b[key]), key


@pytest.mark.parametrize("w,c,k,sigma", [(GQA, 3, 603, 1.0), (G7, 4, 333, 1.0 / math.sqrt(128))])
def test_per_kv_head_sets_token_mode(dev, w, c, k, sigma):
    gu.log(f"[variants] per-KV-head token sets {w.name} k={k}")
    Hkv, G, B = w.num_kv_heads, w.num_q_heads // w.num_kv_heads, w.block_size
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    J = len(cs) - 1
    res = gu.run_gpu(w, d, cs, dev, top_k=k, select_tokens=True, kv_head_sets=True, score_scale=sigma)
    ref = _oracle(w, d, cs, top_k=k, select_tokens=True, kv_head_sets=True, score_scale=sigma)
    cands = gu.token_candidates(d, ref["geometry"], B)
    n_exact = 0
    for g in range(Hkv):
        view = _group_view(ref, g, Hkv, G)
        bounds = gu.token_score_bounds(view, [K[:, g:g + 1] for K in cands], 1, sigma)
        gu.check_token_scores(res["scores"][g::Hkv], view, bounds, B, f"{w.name} KV head {g}")
        n_exact += gu.check_token_selection(res["sel_idx"][g::Hkv, :k], res["sel_cnt"][g::Hkv], res["scores"][g::Hkv],
                                            view, bounds, B, f"{w.name} KV head {g}")
    own = _oracle(w, d, cs, top_k=k, select_tokens=True, kv_head_sets=True, score_scale=sigma,
                  external_sel=_gpu_sets(res, J, Hkv))
    mx_err, rel = gu.check_output(res["out"], own["output"], f"{w.name} per-KV-head token output")
    gu.log(f"[variants] per-KV-head tokens {w.name}: {n_exact} of {J * Hkv} sets exact, output {mx_err:.2e} / "
           f"{rel:.2e}")


def test_token_mode_sigma(dev):
    w, k, sigma = GQA, 603, 1.0 / math.sqrt(128)
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 3)
    res = gu.run_gpu(w, d, cs, dev, top_k=k, select_tokens=True, score_scale=sigma)
    ref = _oracle(w, d, cs, top_k=k, select_tokens=True, score_scale=sigma)
    bounds = gu.token_score_bounds(ref, gu.token_candidates(d, ref["geometry"], w.block_size), w.num_kv_heads, sigma)
    gu.check_token_scores(res["scores"], ref, bounds, w.block_size, "token sigma")
    gu.check_token_selection(res["sel_idx"][:, :k], res["sel_cnt"], res["scores"], ref, bounds, w.block_size,
                             "token sigma")
    own = _oracle(w, d, cs, top_k=k, select_tokens=True, score_scale=sigma,
                  external_sel=gu.gpu_selections(res, len(cs) - 1))
    gu.check_output(res["out"], own["output"], "token sigma output")


def test_per_kv_head_sets_full_size_sampled(dev):
    """llama128k with one set per KV head: the GPU runs the whole layer; sampled clusters are
    checked per KV head (scores, selection) and on their first and last 32-row attention tiles."""
    w = gen.WORKLOADS["llama128k"]
    Hkv, G = w.num_kv_heads, w.num_q_heads // w.num_kv_heads
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    J = len(cs) - 1
    rng = np.random.default_rng(13)
    clusters = sorted({0, J - 1, *rng.choice(np.arange(1, J - 1), size=4, replace=False).tolist()})
    geo = oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, w.top_k, cs)
    rows = gu.sample_rows([geo[j] for j in clusters], rng, tiles_per_cluster=0)
    res = gu.run_gpu(w, d, cs, dev, kv_head_sets=True, out_rows=np.concatenate(rows))
    k_rep = oracle.rep_keys(d["k_pages"], d["block_table"], w.n_tokens, w.block_size)
    sets = _gpu_sets(res, J, Hkv)
    n_exact = 0
    for j in clusters:
        g_ = geo[j]
        v = oracle.anchor_fingerprint(d["q"], g_.s, g_.anchor_end)
        sc = oracle.soft_vote_groups(oracle.block_logits(v, k_rep[g_.sink_blk:g_.sink_blk + g_.n_cand], Hkv), Hkv)
        for g in range(Hkv):
            sel, margin = oracle.select_topk(sc[g], g_.sink_blk, w.top_k)
            view = {"geometry": [g_], "fingerprints": [v[g * G:(g + 1) * G]], "scores": [sc[g]], "selections": [sel],
                    "margins": [margin], "k_rep": k_rep[:, g:g + 1]}
            r = j * Hkv + g
            gu.check_scores(res["scores"][r:r + 1], view, f"cluster {j} KV head {g}")
            n_exact += gu.check_selection(res["sel_idx"][r:r + 1], res["sel_cnt"][r:r + 1], view, EPS_VALID)
    at = 0
    for i, j in enumerate(clusters):
        o_ref = oracle.attention_rows(d["q"], d["k_pages"], d["v_pages"], d["block_table"], geo[j], sets[j], rows[i],
                                      w.block_size)
        gu.check_output(res["out"][at:at + len(rows[i])], o_ref, f"llama128k cluster {j}")
        at += len(rows[i])
    gu.log(f"[variants] llama128k per-KV-head: {n_exact} of {len(clusters) * Hkv} sampled sets exact")


def test_variants_short_last_subchunk(dev):
    """A short last sub-chunk (2368 tokens: nine of 256 and one of 64) with bound representative
    keys and per-KV-head sets together, on a two-KV-head shape."""
    w = gen.Workload("tail2", 1, 8, 2, 64, 2368, 64, 256, 4, 4, 64, 256, 8, 1, 4, 35)
    Hkv, G = w.num_kv_heads, w.num_q_heads // w.num_kv_heads
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 3)
    J = len(cs) - 1
    res = gu.run_gpu(w, d, cs, dev, kv_head_sets=True, rep_bounds=True)
    ref = _oracle(w, d, cs, kv_head_sets=True, rep_kind="minmax")
    for g in range(Hkv):
        view = _group_view(ref, g, Hkv, G, ref["k_rep"])
        gu.check_scores(res["scores"][g::Hkv], view, f"tail KV head {g}")
        gu.check_selection(res["sel_idx"][g::Hkv], res["sel_cnt"][g::Hkv], view, EPS_VALID)
    own = _oracle(w, d, cs, kv_head_sets=True, rep_kind="minmax", external_sel=_gpu_sets(res, J, Hkv))
    gu.check_output(res["out"], own["output"], "variants short tail")
