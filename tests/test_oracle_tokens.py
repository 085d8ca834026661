"""Pins of the oracle's token-level selection mode (TokenSelect's granularity, paper Sec. 5.1.3,
Eq. 9; reading R27): brute force on tiny inputs, the exact reduction to block-level selection on
keys that are constant inside each block, and the dense limit."""
import numpy as np
import pytest

import gen
import oracle
from tests import brute
from tests.test_oracle_pins import _sdpa_causal

TINY = gen.Workload("tok", 1, 4, 2, 16, 192, 8, 32, 2, 3, 8, 40, 4, 1, 3, 21)


def _run(d, w, cs, **over):
    kw = dict(sub_chunk=w.sub_chunk, block_size=w.block_size, top_k=w.top_k, sink_tokens=w.sink_tokens,
              local_window=w.local_window, select_tokens=True)
    kw.update(over)
    return oracle.prefill(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, cluster_start=cs, **kw)


@pytest.mark.parametrize("c,k", [(1, 3), (2, 3), (3, 2), (3, 4)])
def test_token_selection_matches_brute_force(c, k):
    w = TINY.with_(top_k=k)
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    r = _run(d, w, cs)
    b = brute.brute_prefill_tokens(d["q"], d["k_pages"], d["v_pages"], d["block_table"], w.n_tokens, w.sub_chunk,
                                   w.block_size, w.sink_tokens, w.local_window, k, cs)
    for sel_o, sel_b, sc_o, sc_b, g in zip(r["selections"], b["selections"], r["scores"], b["scores"],
                                           r["geometry"]):
        assert g.tokens and g.n_cand == len(sc_b)
        assert tuple(int(x) for x in sel_o) == tuple(sel_b)
        for i, t in enumerate(sorted(sc_b)):
            assert t == g.sink_blk * w.block_size + i
            assert abs(sc_o[i] - sc_b[t]) < 1e-12
    assert np.max(np.abs(r["output"] - b["output"])) < 1e-12


def test_block_constant_keys_reduce_token_mode_to_block_mode():
    """When every key of a block equals the block's first key, each token of block b scores
    score_b / B, so the top kb * B tokens are exactly the tokens of the top kb blocks, and the
    attention outputs coincide."""
    w = gen.WORKLOADS["tiny"].with_(top_k=3)
    d = gen.make_layer(w)
    d["k_pages"] = np.ascontiguousarray(np.broadcast_to(d["k_pages"][:, :, :1, :], d["k_pages"].shape))
    cs = gen.cluster_starts(w.n_sub_chunks, 2)
    blk = _run(d, w, cs, select_tokens=False)
    tok = _run(d, w, cs, top_k=3 * w.block_size)
    for g, sb, st, sc_b, sc_t in zip(blk["geometry"], blk["selections"], tok["selections"], blk["scores"],
                                     tok["scores"]):
        assert np.array_equal(st, oracle.selected_positions(g, sb, w.block_size))
        assert np.allclose(np.repeat(sc_b, w.block_size) / w.block_size, sc_t, rtol=1e-12, atol=1e-15)
    assert np.max(np.abs(tok["output"] - blk["output"])) < 1e-12


def test_token_mode_dense_limit():
    w = TINY.with_(top_k=10 ** 6)
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, 2)
    r = _run(d, w, cs)
    assert all(g.sel_cnt == g.n_cand for g in r["geometry"])
    ref = _sdpa_causal(d["q"], d["k_pages"], d["v_pages"], w.n_tokens)
    assert np.max(np.abs(r["output"] - ref)) < 1e-12
