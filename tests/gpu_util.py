"""Helpers for the GPU parity tests: upload generator inputs, run the library through its C ABI,
and compare with the oracle under the acceptance rules."""
from __future__ import annotations

import math
import os

import numpy as np

import gen
import oracle

# Acceptance on the attention output (max-abs and relative L2 against the fp64 oracle).
O_MAX_ABS = 1e-2
O_REL_L2 = 5e-3
# Selected indices must equal the oracle's wherever the top-k margin exceeds this.
MARGIN = 1e-3


def log(msg: str):
    """Print a progress line; with SCALE_TEST_LOG set, also append it to that file (pytest captures
    stdout, so a long test stays visible there while it runs)."""
    print(msg, flush=True)
    path = os.environ.get("SCALE_TEST_LOG")
    if path:
        with open(path, "a") as f:
            f.write(msg + "\n")


def to_dev(a: np.ndarray, dev):
    import torch

    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(dev)
    return torch.from_numpy(a).to(dev)


def config(w: gen.Workload, n_clusters: int, out_bf16=False, **over):
    import paper_2609_31568_amd as pk

    kw = dict(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
              block_size=w.block_size, sub_chunk=w.sub_chunk, top_k=w.top_k, sink_tokens=w.sink_tokens,
              local_window=w.local_window, max_tokens=w.n_tokens, max_clusters=n_clusters)
    kw.update(over)
    return pk.config_for(out_bf16=out_bf16, **kw)


def upload(data: dict, dev, n_tokens=None):
    """Device copies (q, k_pages, v_pages, block_table) of a generated layer."""
    q = data["q"] if n_tokens is None else data["q"][:n_tokens]
    return to_dev(q, dev), to_dev(data["k_pages"], dev), to_dev(data["v_pages"], dev), to_dev(data["block_table"], dev)


def run_gpu(w: gen.Workload, data: dict, cs, dev, *, out_bf16=False, n_tokens=None, with_scores=True, out_rows=None,
            dev_data=None, **over):
    """Whole path on the GPU; returns host copies of every output plus the call counter.
    With `out_rows`, only those rows of the attention output are copied back (res["out"][i] is
    row out_rows[i]). `dev_data` gives inputs already on the device (as `upload` returns them)."""
    import torch

    import paper_2609_31568_amd as pk

    n = w.n_tokens if n_tokens is None else n_tokens
    cfg = config(w, len(cs) - 1, out_bf16=out_bf16, **over)
    q, kp, vp, bt = dev_data if dev_data is not None else upload(data, dev, n)
    with pk.Scale(cfg) as h:
        bufs = pk.LayerBuffers(cfg, n, len(cs) - 1, device=dev, with_scores=with_scores)
        pk.run_layer(h, q, kp, vp, bt, n, cs, bufs)
        torch.cuda.synchronize()
        calls = h.retrieval_calls()
    out = bufs.out
    if out_rows is not None:
        out = out.index_select(0, torch.as_tensor(np.asarray(out_rows, dtype=np.int64), device=dev))
    res = {
        "k_rep": bufs.k_rep.cpu().numpy(),
        "sel_idx": bufs.sel_idx.cpu().numpy(),
        "sel_cnt": bufs.sel_cnt.cpu().numpy(),
        "out": out.float().cpu().numpy() if not out_bf16 else out.view(torch.int16).cpu().numpy(),
        "calls": calls,
    }
    if with_scores:
        res["scores"] = bufs.scores.cpu().numpy()
        res["fingerprints"] = bufs.fingerprints.cpu().numpy()
    return res


def check_rounding(gpu: np.ndarray, ref: np.ndarray, what: str):
    """GPU value = fp32 rounding of the fp64 result: |gpu - ref| <= 2^-24 |ref| (+ tiny)."""
    err = np.abs(gpu.astype(np.float64) - ref)
    bound = np.abs(ref) * 2.0 ** -24 + 1e-38
    bad = err > bound
    assert not bad.any(), f"{what}: {bad.sum()} values off by more than half an fp32 ulp, max {err.max():.3e}"


U32 = 2.0 ** -24

# Block-level soft-voting scores: fp64 arithmetic on the GPU, each score rounded once to fp32 (at
# most 9.5e-7 for a score below Hq = 32, far less for the scores of about 0.01-5 seen here); the
# acceptance is a fixed absolute tolerance.
SCORE_ATOL = 1e-6


def check_scores(gpu_scores: np.ndarray, ref, what: str):
    """Candidates within SCORE_ATOL of the fp64 oracle; every other entry of the row is -1.
    Returns the largest error seen."""
    worst = 0.0
    nb = gpu_scores.shape[1]
    for j, (g, sc) in enumerate(zip(ref["geometry"], ref["scores"])):
        row = gpu_scores[j]
        cand = np.arange(g.sink_blk, g.sink_blk + g.n_cand)
        assert np.all(np.delete(row, cand) == -1.0), f"{what} cluster {j}: non-candidate entry is not -1"
        if g.n_cand:
            err = np.abs(row[cand].astype(np.float64) - sc)
            assert np.all(err <= SCORE_ATOL), f"{what} cluster {j}: score error {err.max():.2e} above {SCORE_ATOL}"
            worst = max(worst, float(err.max()))
        assert nb >= g.sink_blk + g.n_cand
    return worst


def token_candidates(d: dict, geo, block_size: int):
    """Keys of every candidate token of each cluster (token-level selection), fp64 [n, Hkv, d]."""
    n_max = max((g.sink_blk * block_size + g.n_cand for g in geo), default=0)
    K = oracle.logical_rows(d["k_pages"], d["block_table"], np.arange(n_max), block_size)
    return [K[g.sink_blk * block_size:g.sink_blk * block_size + g.n_cand] for g in geo]


def token_score_bounds(ref, cands, num_kv_heads: int, score_scale: float = 1.0):
    """First-order error bound of the GPU's token-level soft-voting scores, per candidate.

    Logits: the fp32 fingerprint (one rounding) is split into two bf16 pieces (representation
    error <= 2^-18 |v|) and multiplied with the exact bf16 keys in fp32 accumulation over 2 d
    products: |dx| <= (2^-17 + (2 d + 8) u) sum_i |v_i k_i| =: dX. A softmax weight moves by at
    most 2 p dX; the base-2 argument x log2(e) - lse carries u |x - lse| (R = logit range plus
    log n); the normaliser is a sum of positive terms kept per lane over at most 2 n_tiles terms
    with online rescaling (each step <= 4 u), merged over 5 lane levels and the chunks; the head sums
    add Hq u. Hence |d score| <= score (2 dX + 3 u R + (4 (2 n_tiles + 6) + Hq + 16) u), plus an
    absolute 1e-30 for weights that underflow.
    """
    out = []
    for g, v, sc, K in zip(ref["geometry"], ref["fingerprints"], ref["scores"], cands):
        if g.n_cand == 0:
            out.append(np.zeros(0))
            continue
        Hq, d = v.shape
        G = Hq // num_kv_heads
        amax, xmin, xmax = 0.0, np.inf, -np.inf
        rng = 0.0
        for kv in range(num_kv_heads):
            vg = v[kv * G:(kv + 1) * G]
            Kg = K[:, kv, :]
            amax = max(amax, float((np.abs(vg) @ np.abs(Kg).T).max()) * abs(score_scale))
            x = (vg @ Kg.T) * score_scale
            rng = max(rng, float((x.max(axis=1) - x.min(axis=1)).max()))
        dX = (2.0 ** -17 + (2 * d + 8) * U32) * amax
        R = rng + math.log(g.n_cand) + 1.0
        n_tiles = -(-g.n_cand // 64)
        rel = 2 * dX + 3 * U32 * R + (4 * (2 * n_tiles + 6) + Hq + 16) * U32
        out.append(sc * rel + 1e-30)
    return out


def check_token_scores(gpu_scores: np.ndarray, ref, bounds, block_size: int, what: str, atol=None):
    """Candidate entries within the bound (and within `atol` when given); every other entry of the
    row is -1. Returns the largest relative error seen."""
    worst = 0.0
    for j, (g, sc, bd) in enumerate(zip(ref["geometry"], ref["scores"], bounds)):
        row = gpu_scores[j]
        first = g.sink_blk * block_size
        assert np.all(row[:first] == -1.0) and np.all(row[first + g.n_cand:] == -1.0), \
            f"{what} cluster {j}: non-candidate entry is not -1"
        if g.n_cand:
            err = np.abs(row[first:first + g.n_cand].astype(np.float64) - sc)
            assert np.all(err <= bd), f"{what} cluster {j}: score error {err.max():.2e} above bound"
            if atol is not None:
                assert np.all(err <= atol), f"{what} cluster {j}: score error {err.max():.2e} above {atol}"
            worst = max(worst, float((err / np.maximum(sc, 1e-300)).max()))
    return worst


def check_token_selection(gpu_sel, gpu_cnt, gpu_scores, ref, bounds, block_size: int, what: str):
    """The GPU selection is exactly the top-k of its own fp32 scores (score descending, position
    ascending); against the oracle scores it is valid to twice the bound, and equal to the oracle's
    wherever the bounds cannot reorder the threshold: every oracle-selected score minus its bound
    above every unselected score plus its bound."""
    n_exact = 0
    for j, (g, s_ref, sc, bd) in enumerate(zip(ref["geometry"], ref["selections"], ref["scores"], bounds)):
        cnt = int(gpu_cnt[j])
        assert cnt == g.sel_cnt, f"{what} cluster {j}: sel_cnt {cnt} != {g.sel_cnt}"
        got = gpu_sel[j, :cnt].astype(np.int64)
        assert np.all(gpu_sel[j, cnt:] == -1), f"{what} cluster {j}: padding is not -1"
        assert np.all(np.diff(got) > 0), f"{what} cluster {j}: not strictly ascending"
        first = g.sink_blk * block_size
        if g.n_cand == 0:
            continue
        own = gpu_scores[j, first:first + g.n_cand].astype(np.float64)
        order = np.lexsort((np.arange(g.n_cand), -own))
        assert np.array_equal(np.sort(order[:cnt]) + first, got), f"{what} cluster {j}: not the top-k of its scores"
        if cnt == g.n_cand:
            assert np.array_equal(got, s_ref)
            continue
        if cnt == 0:
            continue
        eps = 2 * float(bd.max())
        kth = np.sort(sc)[::-1][cnt - 1]
        chosen = np.zeros(g.n_cand, dtype=bool)
        chosen[got - first] = True
        assert np.all(sc[chosen] >= kth - eps), f"{what} cluster {j}: a selected token is not within eps of top-k"
        assert np.all(sc[~chosen] <= kth + eps), f"{what} cluster {j}: an unselected token beats the k-th by > eps"
        in_ref = np.zeros(g.n_cand, dtype=bool)
        in_ref[np.asarray(s_ref, dtype=np.int64) - first] = True
        if (sc[in_ref] - bd[in_ref]).min() > (sc[~in_ref] + bd[~in_ref]).max():
            assert np.array_equal(got, s_ref), f"{what} cluster {j}: differs from the oracle above the margin"
            n_exact += 1
    return n_exact


# With every score within SCORE_ATOL of the oracle's, a top-k margin above twice that leaves the GPU
# no other set to select: the k-th and (k+1)-th scores cannot swap.
MARGIN_EXACT = 2 * SCORE_ATOL


def check_selection(gpu_sel, gpu_cnt, ref, eps: float, margin_exact: float = MARGIN_EXACT):
    """Exact where the oracle's margin exceeds `margin_exact` (the scores' tolerance makes the set
    unique there; it is far below the 1e-3 of the acceptance rule); eps-valid top-k everywhere.
    Returns the number of clusters whose margin exceeds MARGIN (1e-3), all of them exact."""
    n_exact = 0
    for j, (g, s_ref, m, sc) in enumerate(zip(ref["geometry"], ref["selections"], ref["margins"], ref["scores"])):
        cnt = int(gpu_cnt[j])
        assert cnt == g.sel_cnt, f"cluster {j}: sel_cnt {cnt} != {g.sel_cnt}"
        got = gpu_sel[j, :cnt].astype(np.int64)
        assert np.all(gpu_sel[j, cnt:] == -1), f"cluster {j}: padding is not -1"
        assert np.all(np.diff(got) > 0), f"cluster {j}: not strictly ascending"
        assert np.all((got >= g.sink_blk) & (got < g.sink_blk + g.n_cand)), f"cluster {j}: non-candidate selected"
        if m > min(MARGIN, margin_exact):
            assert np.array_equal(got, s_ref), f"cluster {j}: {got} != oracle {s_ref} (margin {m:.2e})"
            n_exact += m > MARGIN
        if 0 < cnt < g.n_cand:
            kth = np.sort(sc)[::-1][cnt - 1]
            chosen = np.zeros(g.n_cand, dtype=bool)
            chosen[got - g.sink_blk] = True
            assert np.all(sc[chosen] >= kth - eps), f"cluster {j}: a selected block is not within eps of top-k"
            assert np.all(sc[~chosen] <= kth + eps), f"cluster {j}: an unselected block beats the k-th by > eps"
    return n_exact


def check_output(out: np.ndarray, ref: np.ndarray, what: str):
    err = np.abs(out.astype(np.float64) - ref)
    mx = float(err.max()) if err.size else 0.0
    rel = float(np.linalg.norm(out.astype(np.float64) - ref) / max(np.linalg.norm(ref), 1e-300))
    assert mx <= O_MAX_ABS and rel <= O_REL_L2, f"{what}: max-abs {mx:.3e}, rel-L2 {rel:.3e}"
    return mx, rel


def gpu_selections(res, n_clusters):
    return [res["sel_idx"][j, :res["sel_cnt"][j]].astype(np.int64) for j in range(n_clusters)]


def sample_rows(geo, rng, tiles_per_cluster=3, tile=32):
    """A few 32-row tiles per cluster: its first and last tile plus random ones."""
    out = []
    for g in geo:
        starts = {g.s, max(g.s, g.e - tile)}
        n_t = max(1, (g.e - g.s) // tile)
        for _ in range(tiles_per_cluster):
            starts.add(g.s + int(rng.integers(0, n_t)) * tile)
        rows = sorted({r for s0 in starts for r in range(s0, min(s0 + tile, g.e))})
        out.append(np.asarray(rows, dtype=np.int64))
    return out


def bf16_rne(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest even (test-side reference of the epilogue)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return r


def nan_free(*arrays):
    return all(not np.isnan(a).any() for a in arrays)


def isfinite_margin(m):
    return m if math.isfinite(m) else float("inf")
