"""The allocation-free selection entry point (scale_select_cluster_static) against the handle's
scale_select_cluster on the same inputs: identical selections, counts and scores (the same
kernels on the library's static scratch), on two calls in a row, the second smaller than the
first, and the capacity error for a call whose scratch exceeds the static array."""
import numpy as np
import pytest

import gen
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_31568_amd  # noqa: F401  (fails loudly if the library is missing)

    return torch.device("cuda:0")


def _handle_selection(w, d, cs, dev_data):
    """scale_rep_keys + scale_select_cluster on a handle: k_rep, sel_idx, sel_cnt, scores."""
    import torch

    import paper_2609_31568_amd as pk

    q, kp, vp, bt = dev_data
    cfg = gu.config(w, len(cs) - 1)
    with pk.Scale(cfg) as h:
        b = pk.LayerBuffers(cfg, w.n_tokens, len(cs) - 1, device=q.device, with_scores=True)
        h.rep_keys(kp, bt, w.n_tokens, b.k_rep)
        h.select_cluster(q, w.n_tokens, b.k_rep, cs, b.sel_idx, b.sel_cnt, b.scores)
        torch.cuda.synchronize()
        return b.k_rep, b.sel_idx.cpu().numpy(), b.sel_cnt.cpu().numpy(), b.scores.cpu().numpy()


def _static_selection(w, cs, q, k_rep, fill):
    import torch

    import paper_2609_31568_amd as pk

    J = len(cs) - 1
    cfg = gu.config(w, J)
    sel = torch.full((J, max(w.top_k, 1)), fill, dtype=torch.int32, device=q.device)
    cnt = torch.full((J,), fill, dtype=torch.int32, device=q.device)
    scores = torch.full((J, w.n_tokens // w.block_size), float(fill), dtype=torch.float32, device=q.device)
    pk.scale_select_cluster_static(cfg, q, w.n_tokens, k_rep, cs, sel, cnt, scores)
    torch.cuda.synchronize()
    return sel.cpu().numpy(), cnt.cpu().numpy(), scores.cpu().numpy()


def test_static_selection_equals_handle_selection(dev):
    import paper_2609_31568_amd as pk

    big = gen.WORKLOADS["llama32k"]                       # 8 clusters of 8 sub-chunks
    small = big.with_(n_tokens=12288, n_topics=16, seed=45)    # 3 clusters, fewer candidates
    for w, fill in ((big, 7), (small, -3)):
        gu.log(f"[no-alloc] {w.name} n_tokens={w.n_tokens}")
        d = gen.make_layer(w)
        cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
        dev_data = gu.upload(d, dev)
        k_rep, sel_h, cnt_h, sc_h = _handle_selection(w, d, cs, dev_data)
        sel_s, cnt_s, sc_s = _static_selection(w, cs, dev_data[0], k_rep, fill)
        assert np.array_equal(cnt_s, cnt_h)
        assert np.array_equal(sel_s, sel_h)
        assert np.array_equal(sc_s.view(np.uint32), sc_h.view(np.uint32))
    # a call whose scratch exceeds the static array: rejected on the host, outputs untouched
    w = gen.WORKLOADS["stress1m"]
    cs = gen.cluster_starts(w.n_sub_chunks, 1)
    cfg = gu.config(w, len(cs) - 1)
    fake = 256   # an aligned address that the refused call never dereferences
    with pytest.raises(pk.ScaleError) as e:
        pk.scale_select_cluster_static(cfg, fake, w.n_tokens, fake, cs, fake, fake, None)
    assert e.value.status == pk.SCALE_ERR_CAPACITY


def test_static_selection_spill_path(dev):
    """More candidates than the top-k keeps in LDS (8192): a 640K context in blocks of 64 with 4
    query heads, so the static call's scores spill into its scratch array (about 62 MB of the
    64 MiB); the result equals the handle's selection bit for bit."""
    w = gen.Workload("spill", 1, 4, 1, 64, 655360, 64, 512, 8, 16, 64, 4096, 512, 1, 8, 44)
    gu.log(f"[no-alloc] spill n_tokens={w.n_tokens}")
    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, w.cluster)
    dev_data = gu.upload(d, dev)
    k_rep, sel_h, cnt_h, sc_h = _handle_selection(w, d, cs, dev_data)
    s, e = cs[-2] * w.sub_chunk, min(cs[-1] * w.sub_chunk, w.n_tokens)    # the last cluster
    lo = max(0, min(s, e - w.local_window))
    n_cand = lo // w.block_size - (w.sink_tokens + w.block_size - 1) // w.block_size
    assert n_cand > 8192                                                   # beyond the LDS rows
    sel_s, cnt_s, sc_s = _static_selection(w, cs, dev_data[0], k_rep, 5)
    assert np.array_equal(cnt_s, cnt_h)
    assert np.array_equal(sel_s, sel_h)
    assert np.array_equal(sc_s.view(np.uint32), sc_h.view(np.uint32))
