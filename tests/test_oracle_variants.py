"""Pins of the oracle's selection variants: bound representative keys (channel-wise min / max per
block, the page criticality of Quest cited in Sec. 2; reading R28), one index set per KV head
(reading R29) and the selection logit scale sigma = 1/sqrt(d) (R5), against brute force, the
upper-bound property, and the special cases that reduce them to the default selection."""
import math

import numpy as np
import pytest

import gen
import oracle
from tests import brute
from tests.test_oracle_pins import _sdpa_causal

TINY = gen.Workload("var", 1, 4, 2, 8, 256, 8, 32, 2, 3, 8, 40, 4, 1, 3, 23)


def _run(d, w, cs, **over):
    kw = dict(sub_chunk=w.sub_chunk, block_size=w.block_size, top_k=w.top_k, sink_tokens=w.sink_tokens,
              local_window=w.local_window)
    kw.update(over)
    return oracle.prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, cluster_start=cs, **kw)


def _brute(d, w, cs, **kw):
    return brute.brute_prefill_variants(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens,
                                        w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, w.top_k, cs, **kw)


@pytest.mark.parametrize("c,bounds,per_kv,sigma", [
    (1, True, False, 1.0), (2, True, False, 1.0), (3, True, True, 1.0), (2, False, True, 1.0),
    (1, False, True, 1.0), (2, True, False, 1.0 / math.sqrt(8)), (3, False, False, 1.0 / math.sqrt(8)),
])
def test_variants_match_brute_force(c, bounds, per_kv, sigma):
    w = TINY
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    r = _run(d, w, cs, rep_kind="minmax" if bounds else "mean", kv_head_sets=per_kv, score_scale=sigma)
    b = _brute(d, w, cs, bounds=bounds, per_kv_head=per_kv, score_scale=sigma)
    for j, sel in enumerate(r["selections"]):
        if per_kv:
            assert sel.shape[0] == w.num_kv_heads
            for g in range(w.num_kv_heads):
                assert tuple(int(x) for x in sel[g]) == tuple(b["selections"][g][j])
        else:
            assert tuple(int(x) for x in sel) == tuple(b["selections"][None][j])
    assert np.max(np.abs(r["output"] - b["output"])) < 1e-12


def test_bound_logit_is_an_upper_bound_and_tight_on_constant_blocks():
    """sum_i max(v_i lo_i, v_i hi_i) >= v . k for every key of the block (each term bounds v_i k_i),
    with equality when every key of the block is the same."""
    w = gen.WORKLOADS["tiny"]
    d = gen.make_layer(w)
    mn, mx = oracle.rep_bounds(d["k_pages"], d["block_table"], w.n_tokens, w.block_size)
    K = oracle.logical_rows(d["k_pages"], d["block_table"], np.arange(w.n_tokens), w.block_size)
    v = oracle.anchor_fingerprint(d["q"], 512, 768)
    x = oracle.bound_logits(v, mn, mx, w.num_kv_heads)
    nb = w.n_tokens // w.block_size
    for h in range(w.num_q_heads):
        g = (h * w.num_kv_heads) // w.num_q_heads
        dots = (K[:, g, :] @ v[h]).reshape(nb, w.block_size)
        assert np.all(x[h] >= dots.max(axis=1) - 1e-12)
        assert np.all(x[h] > dots.max(axis=1) + 1e-9)        # strict on random blocks
    const = np.ascontiguousarray(np.broadcast_to(d["k_pages"][:, :, :1, :], d["k_pages"].shape))
    mn, mx = oracle.rep_bounds(const, d["block_table"], w.n_tokens, w.block_size)
    kr = oracle.rep_keys(const, d["block_table"], w.n_tokens, w.block_size)
    assert np.array_equal(mn, mx) and np.array_equal(mn, kr)
    assert np.allclose(oracle.bound_logits(v, mn, mx, w.num_kv_heads), oracle.block_logits(v, kr, w.num_kv_heads),
                       rtol=1e-14, atol=1e-14)


def test_bound_selection_equals_mean_selection_on_block_constant_keys():
    w = gen.WORKLOADS["tiny"]
    d = gen.make_layer(w)
    d["k_pages"] = np.ascontiguousarray(np.broadcast_to(d["k_pages"][:, :, :1, :], d["k_pages"].shape))
    cs = gen.cluster_starts(w.n_sub_chunks, 2)
    a = _run(d, w, cs, rep_kind="minmax")
    b = _run(d, w, cs)
    for sa, sb, xa, xb in zip(a["selections"], b["selections"], a["scores"], b["scores"]):
        assert np.array_equal(sa, sb)
        assert np.allclose(xa, xb, rtol=1e-12, atol=1e-14)
    assert np.max(np.abs(a["output"] - b["output"])) < 1e-12


def test_per_kv_head_sets_with_one_kv_head_are_the_shared_set():
    w = gen.WORKLOADS["tiny"]                  # 4 query heads, 1 KV head
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 4)
    a = _run(d, w, cs, kv_head_sets=True)
    b = _run(d, w, cs)
    for sa, sb in zip(a["selections"], b["selections"]):
        assert sa.shape == (1, len(sb)) and np.array_equal(sa[0], sb)
    assert np.array_equal(a["output"], b["output"])


def test_per_kv_head_sets_on_replicated_heads_equal_the_shared_set():
    """Every KV head holding the same keys and every group of query heads the same queries: each
    group's vote is the shared vote divided by Hkv, so every group picks the shared set."""
    w = TINY.with_(n_tokens=512, top_k=4)
    d = gen.make_layer(w)
    G = w.num_q_heads // w.num_kv_heads
    for g in range(1, w.num_kv_heads):
        d["k_pages"][:, g] = d["k_pages"][:, 0]
        d["v_pages"][:, g] = d["v_pages"][:, 0]
        d["q"][:, g * G:(g + 1) * G] = d["q"][:, :G]
    cs = gen.cluster_starts(w.n_sub_chunks, 2)
    a = _run(d, w, cs, kv_head_sets=True)
    b = _run(d, w, cs)
    for sa, sb in zip(a["selections"], b["selections"]):
        for g in range(w.num_kv_heads):
            assert np.array_equal(sa[g], sb)
    assert np.max(np.abs(a["output"] - b["output"])) < 1e-12


@pytest.mark.parametrize("over", [dict(rep_kind="minmax"), dict(kv_head_sets=True),
                                  dict(kv_head_sets=True, select_tokens=True)])
def test_variants_dense_limit(over):
    w = TINY.with_(top_k=10 ** 6)
    d = gen.make_layer(w)
    r = _run(d, w, gen.cluster_starts(w.n_sub_chunks, 2), **over)
    ref = _sdpa_causal(d["q"], d["k_pages"], d["v_pages"], w.n_tokens)
    assert np.max(np.abs(r["output"] - ref)) < 1e-12


def test_variant_arguments_are_checked():
    w = TINY
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 2)
    with pytest.raises(ValueError):
        _run(d, w, cs, rep_kind="max")
    with pytest.raises(ValueError):
        _run(d, w, cs, rep_kind="minmax", select_tokens=True)
