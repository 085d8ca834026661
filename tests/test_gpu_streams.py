"""Two handles on two streams. A handle owns its scratch and enqueues on its own stream, so two
layers running at once, interleaved call by call, give the bits each gives alone."""
import numpy as np
import pytest

import gen
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

LAYERS = [
    (gen.Workload("gqa128", 1, 8, 2, 128, 8192, 128, 512, 3, 5, 128, 1024, 12, 1, 4, 31), 3),
    (gen.Workload("g7", 1, 14, 2, 128, 4096, 64, 256, 4, 6, 64, 512, 8, 1, 3, 32), 4),
]


@pytest.fixture(scope="module")
def dev():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_31568_amd  # noqa: F401  (fails loudly if the library is missing)

    return torch.device("cuda:0")


def _prepare(w, c, dev, stream):
    import paper_2609_31568_amd as pk

    d = gen.make_layer(w)
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    cfg = gu.config(w, len(cs) - 1)
    tensors = [gu.to_dev(d[k], dev) for k in ("q", "k_pages", "v_pages", "block_table")]
    h = pk.Scale(cfg, stream=stream)
    bufs = pk.LayerBuffers(cfg, w.n_tokens, len(cs) - 1, device=dev, with_scores=True)
    return h, tensors, cs, bufs


def _host(bufs):
    return bufs.out.cpu().numpy(), bufs.sel_idx.cpu().numpy(), bufs.sel_cnt.cpu().numpy(), bufs.scores.cpu().numpy()


def test_two_handles_on_two_streams(dev):
    import torch

    import paper_2609_31568_amd as pk

    alone = []
    for w, c in LAYERS:
        h, t, cs, bufs = _prepare(w, c, dev, None)
        pk.run_layer(h, *t, w.n_tokens, cs, bufs)
        torch.cuda.synchronize()
        alone.append(_host(bufs))
        h.close()
    gu.log("[streams] each layer alone: done")
    streams = [torch.cuda.Stream(device=dev) for _ in LAYERS]     # default priority
    runs = [_prepare(w, c, dev, s) for (w, c), s in zip(LAYERS, streams)]
    torch.cuda.synchronize()                 # inputs are on the device before either stream reads them
    for _ in range(2):                       # the second pass reuses every handle's scratch
        for (w, _c), (h, t, cs, bufs) in zip(LAYERS, runs):
            pk.run_layer(h, *t, w.n_tokens, cs, bufs)
    torch.cuda.synchronize()
    for (w, _c), (h, _t, _cs, bufs), ref in zip(LAYERS, runs, alone):
        for got, want, what in zip(_host(bufs), ref, ("out", "sel_idx", "sel_cnt", "scores")):
            assert np.array_equal(got, want), f"{w.name}: {what} differs from the run alone"
        h.close()
    gu.log("[streams] both layers on two streams: bit-identical")
