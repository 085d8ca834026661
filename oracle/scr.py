"""Plain fp64 CPU oracle for cluster-level sparse prefill (Similarity Chunk Rolling, SCR).

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may import or call this module. The product path (the HIP library and its
Python binding) never does, and this module never imports the product path.

It follows the paper's statement of the method, step by step, in float64, with no blocking,
fusion or reordering beyond what the definitions say. Citations name the paper's sections and
equations (equation numbers in source order):

* Sec. 3.1, two-level chunked prefill: an outer chunk's queries are split into M = ceil(l / L)
  sub-chunks, the last one possibly short.
* Sec. 3.2, Definition 1 (Eqs. 2-4): selective sparse attention restricts the softmax of scaled
  dot-product attention (Eq. 1) to a selected subset of the cache, chosen by a selection function
  over all heads.
* Sec. 4.1, Eq. 6: the sub-chunk fingerprint is the mean of the sub-chunk's multi-head queries;
  its head-h slice is the per-head mean.
* Sec. 5.1.3, Eq. 9: one selection per cluster, driven by the anchor (first sub-chunk)
  fingerprint, shared by every member.
* Sec. 5.1.3, "selection function instantiation": head soft-voting -- per-head dot scores,
  softmax per head, sum over heads, top-k.
* Sec. 5.1.3, Eq. 10: cluster attention over three key groups (the shared top-k set, the
  attention sinks, and a local window widened to span the whole cluster) under a causal mask.
* Algorithm 2: per cluster, select -> augment with sink and local -> attend -> write.
* Sec. 5.1.1: fingerprints are L2-normalised once, so a cosine is one inner product.
* Sec. 5.1.2, Algorithm 1 with the admission rule of Eq. 8: anchor-based clustering of an outer
  chunk's sub-chunks in one left-to-right pass; a sub-chunk joins the open cluster while its
  cosine with the cluster's first sub-chunk (the anchor) reaches theta and the cluster is still
  below L_max tokens, and otherwise becomes the next anchor.

Readings where the paper is silent (block-level selection, the representative key, the
candidate set, local-window geometry, tie-break), all named R-numbers below, are listed with
their reasons in the design notes:

  R1  selection unit is a KV block of B tokens (blocks, not single tokens, are scored)
  R2  a block's representative key is the arithmetic mean of its keys, per KV head
  R4  the cluster query is the anchor fingerprint: mean of the first sub-chunk's query rows
  R5  selection logits are v . k_rep times ``score_scale`` (default 1.0, the literal text)
  R6  query head h reads KV head floor(h * Hkv / Hq)
  R7  one index set per cluster, shared by all heads (scores summed over every query head)
  R8  the soft-voting softmax runs over the candidate blocks only
  R9  candidates are the blocks strictly between the sink blocks and the local window
  R10 local window starts at lo = max(0, min(s, e - W)), rounded down to a block: it spans the
      whole cluster and at least W tokens before the cluster end
  R11 the sink is the first ceil(S / B) whole blocks, clipped to the blocks before the window
  R12 top-k order is (score descending, block index ascending); fewer candidates than k selects
      them all; the selection is emitted in ascending block order
  R13 causal: a key is visible to a query iff its position is <= the query's position
  R14 attention scale 1/sqrt(d_h) (Eqs. 1, 10) unless given
  R22 clustering compares the fingerprints of all heads concatenated (Eq. 6's v_i in R^d); a
      zero fingerprint has no direction, so its cosine is undefined (NaN) and never reaches theta
  R23 the cap test |C| L < L_max counts whole sub-chunks of L rows (the last, short sub-chunk
      too), so a cluster holds at most ceil(L_max / L) sub-chunks; clusters restart at each outer
      chunk boundary when the outer chunk length is given
  R24 the threshold test is taken in fp64
  R25 incremental prefill (Sec. 3.1's outer-chunk loop): the clusters may cover only the last
      sub-chunks [cluster_start[0], M); the cache holds every earlier token, and rows before
      cluster_start[0] * L are not computed
  R26 the overlap ratio (Eq. 7) compares the cluster's set I_C (anchor fingerprint, the cluster's
      candidates) with the union of the sets each member sub-chunk selects on its own, as the
      per-sub-chunk baseline would (its own fingerprint and its own candidate range, the
      single-sub-chunk geometry); it is undefined (NaN) when I_C is empty
  R27 token-level selection (TokenSelect's granularity, Sec. 5.1.3): the candidates are the single
      tokens between the sink blocks and the local window, each scored per head with its own key;
      top_k counts tokens. Sinks and the local window keep their block rounding (R10, R11)
  R28 bound representative keys (the query-aware page criticality of Quest, cited in Sec. 2): per
      block and KV head the channel-wise minimum and maximum of the valid keys, and the logit
      sigma * sum_i max(v_i mn_i, v_i mx_i), an upper bound of v . k over the block's keys (for
      sigma > 0); it replaces R2's mean in block-level selection
  R29 per-KV-head index sets: instead of R7's one set per cluster, every KV head g gets its own
      top-k, voted by the softmax weights of its own query heads only; query head h attends over
      the set of g(h)
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = [
    "ClusterGeometry",
    "geometry",
    "bf16_to_f64",
    "logical_kv",
    "logical_rows",
    "selected_positions",
    "rep_keys",
    "rep_bounds",
    "anchor_fingerprint",
    "block_logits",
    "bound_logits",
    "soft_vote",
    "soft_vote_groups",
    "group_sets",
    "select_topk",
    "key_positions",
    "attention_rows",
    "cluster_attention",
    "prefill",
    "retrieval_calls",
    "subchunk_fingerprints",
    "normalized",
    "anchor_clustering",
    "topk_overlap",
]


def bf16_to_f64(u16) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exactly."""
    u32 = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16
    return u32.view(np.float32).astype(np.float64)


@dataclasses.dataclass(frozen=True)
class ClusterGeometry:
    """Token geometry of one cluster (all positions are token indices, half-open ranges)."""

    s: int            # first query row of the cluster
    e: int            # one past the last query row
    anchor_end: int   # the anchor sub-chunk is rows [s, anchor_end)
    lo_blk: int       # local window starts at token lo_blk * B
    sink_blk: int     # ceil(S / B): blocks reserved for the sink
    sink_eff: int     # sink blocks actually used: [0, sink_eff)
    n_cand: int       # candidate blocks are [sink_blk, sink_blk + n_cand) (tokens: see below)
    sel_cnt: int      # min(k, n_cand)
    tokens: bool = False   # token-level selection (R27): candidates are the TOKENS
                           # [sink_blk * B, lo_blk * B), n_cand and sel_cnt count tokens


def geometry(n_tokens: int, sub_chunk: int, block_size: int, sink_tokens: int, local_window: int,
             top_k: int, cluster_start, select_tokens: bool = False) -> list[ClusterGeometry]:
    """Per-cluster geometry (Sec. 3.1 sub-chunks; Sec. 5.1.3 and Eq. 10 key groups; R9-R12).

    ``cluster_start`` holds sub-chunk indices: cluster j covers sub-chunks
    [cluster_start[j], cluster_start[j+1]). It may start past 0 (R25): incremental prefill of the
    last outer chunks, whose keys follow those of the earlier, already prefilled ones in the cache.
    """
    L, B, S, W, k = sub_chunk, block_size, sink_tokens, local_window, top_k
    M = -(-n_tokens // L)
    cs = [int(x) for x in cluster_start]
    if len(cs) < 2 or cs[0] < 0 or cs[-1] != M or any(b <= a for a, b in zip(cs, cs[1:])):
        raise ValueError("cluster_start must rise strictly to ceil(n_tokens / sub_chunk) from >= 0")
    out = []
    sink_blk = -(-S // B)
    for j in range(len(cs) - 1):
        s = cs[j] * L
        e = min(cs[j + 1] * L, n_tokens)
        anchor_end = min(s + L, e)
        lo = max(0, min(s, e - W))
        lo_blk = lo // B
        sink_eff = min(sink_blk, lo_blk)
        n_cand = max(0, lo_blk - sink_blk) * (B if select_tokens else 1)
        out.append(ClusterGeometry(s, e, anchor_end, lo_blk, sink_blk, sink_eff, n_cand, min(k, n_cand),
                                   bool(select_tokens)))
    return out


def retrieval_calls(n_clusters_per_layer) -> int:
    """One selection call per cluster per layer, degenerate clusters included (Sec. 5.1.2)."""
    return int(sum(int(n) for n in n_clusters_per_layer))


def logical_kv(pages, block_table, blocks) -> np.ndarray:
    """Keys (or values) of the given logical blocks as float64 [len(blocks) * B, Hkv, d].

    ``pages`` is the paged cache [n_pages, Hkv, B, d]; ``block_table[b]`` is the page holding
    logical block b.
    """
    blocks = np.asarray(blocks, dtype=np.int64)
    if blocks.size == 0:
        return np.zeros((0, pages.shape[1], pages.shape[3]), dtype=np.float64)
    phys = np.asarray(block_table)[blocks]
    x = bf16_to_f64(pages[phys])                   # [nb, Hkv, B, d]
    return x.transpose(0, 2, 1, 3).reshape(-1, pages.shape[1], pages.shape[3])


def logical_rows(pages, block_table, positions, block_size: int) -> np.ndarray:
    """Keys (or values) at the given token positions as float64 [len(positions), Hkv, d]."""
    positions = np.asarray(positions, dtype=np.int64)
    if positions.size == 0:
        return np.zeros((0, pages.shape[1], pages.shape[3]), dtype=np.float64)
    phys = np.asarray(block_table)[positions // block_size]
    return bf16_to_f64(pages[phys, :, positions % block_size, :])


def rep_keys(k_pages, block_table, n_tokens: int, block_size: int, blocks=None) -> np.ndarray:
    """R2: k_rep[b][g] = mean of K[t][g] over the valid tokens t of block b. [n, Hkv, d] fp64."""
    n_blocks = -(-n_tokens // block_size)
    blocks = np.arange(n_blocks) if blocks is None else np.asarray(blocks)
    Hkv, d = k_pages.shape[1], k_pages.shape[3]
    out = np.empty((len(blocks), Hkv, d), dtype=np.float64)
    for i, b in enumerate(blocks):
        n_valid = min(block_size, n_tokens - int(b) * block_size)
        keys = bf16_to_f64(k_pages[int(block_table[int(b)]), :, :n_valid, :])   # [Hkv, n_valid, d]
        out[i] = keys.sum(axis=1) / n_valid
    return out


def rep_bounds(k_pages, block_table, n_tokens: int, block_size: int, blocks=None):
    """R28: channel-wise minimum and maximum of K[t][g] over the valid tokens t of block b.
    Returns (mn, mx), each [n, Hkv, d] fp64."""
    n_blocks = -(-n_tokens // block_size)
    blocks = np.arange(n_blocks) if blocks is None else np.asarray(blocks)
    Hkv, d = k_pages.shape[1], k_pages.shape[3]
    mn = np.empty((len(blocks), Hkv, d), dtype=np.float64)
    mx = np.empty((len(blocks), Hkv, d), dtype=np.float64)
    for i, b in enumerate(blocks):
        n_valid = min(block_size, n_tokens - int(b) * block_size)
        keys = bf16_to_f64(k_pages[int(block_table[int(b)]), :, :n_valid, :])   # [Hkv, n_valid, d]
        mn[i] = keys.min(axis=1)
        mx[i] = keys.max(axis=1)
    return mn, mx


def anchor_fingerprint(q, s: int, anchor_end: int) -> np.ndarray:
    """Eq. 6 on the anchor sub-chunk (Eq. 9): v[h] = mean over rows p in [s, anchor_end) of q[p][h].

    ``q`` is [N, Hq, d] bf16 bits (or any array indexable by row). Returns [Hq, d] fp64.
    """
    rows = bf16_to_f64(q[s:anchor_end])
    return rows.sum(axis=0) / (anchor_end - s)


def block_logits(v, k_rep_cand, num_kv_heads: int, score_scale: float = 1.0) -> np.ndarray:
    """Per-head dot scores of the selection function (R5, R6): x[h][b] = sigma * v[h] . k_rep[b][g(h)].

    ``v`` [Hq, d]; ``k_rep_cand`` [n_cand, Hkv, d]. Returns [Hq, n_cand].
    """
    Hq = v.shape[0]
    x = np.empty((Hq, k_rep_cand.shape[0]), dtype=np.float64)
    for h in range(Hq):
        g = (h * num_kv_heads) // Hq
        x[h] = score_scale * (k_rep_cand[:, g, :] @ v[h])
    return x


def bound_logits(v, mn_cand, mx_cand, num_kv_heads: int, score_scale: float = 1.0) -> np.ndarray:
    """R28: x[h][b] = sigma * sum_i max(v[h][i] mn[b][g(h)][i], v[h][i] mx[b][g(h)][i]).

    ``v`` [Hq, d]; ``mn_cand``, ``mx_cand`` [n_cand, Hkv, d]. Returns [Hq, n_cand].
    """
    Hq = v.shape[0]
    x = np.empty((Hq, mn_cand.shape[0]), dtype=np.float64)
    for h in range(Hq):
        g = (h * num_kv_heads) // Hq
        x[h] = score_scale * np.maximum(mn_cand[:, g, :] * v[h], mx_cand[:, g, :] * v[h]).sum(axis=1)
    return x


def soft_vote_groups(x, num_kv_heads: int) -> np.ndarray:
    """R29: the soft-voting scores of each KV head's own query heads: [Hkv, n_cand]."""
    Hq = x.shape[0]
    G = Hq // num_kv_heads
    return np.stack([soft_vote(x[g * G:(g + 1) * G]) for g in range(num_kv_heads)])


def group_sets(sel, num_kv_heads: int) -> list:
    """A selection as one index array per KV head: a 2-D [Hkv, cnt] array is one set per KV head
    (R29); a 1-D array is one set shared by every head (R7)."""
    a = np.asarray(sel, dtype=np.int64)
    if a.ndim == 2:
        if a.shape[0] != num_kv_heads:
            raise ValueError("per-KV-head selection needs one row per KV head")
        return [a[g] for g in range(num_kv_heads)]
    return [a] * num_kv_heads


def soft_vote(x) -> np.ndarray:
    """Head soft-voting (Sec. 5.1.3): softmax over candidates per head, then sum over heads (R7, R8)."""
    if x.shape[1] == 0:
        return np.zeros(0, dtype=np.float64)
    m = x.max(axis=1, keepdims=True)
    ex = np.exp(x - m)
    p = ex / ex.sum(axis=1, keepdims=True)
    return p.sum(axis=0)


def select_topk(scores, first_block: int, k: int):
    """R12: the top min(k, n) candidates by (score descending, block index ascending).

    Returns (selected block indices in ascending order, margin), where the margin is the gap
    between the k-th and (k+1)-th score in that order (+inf when every candidate is selected).
    """
    n = len(scores)
    idx = np.arange(first_block, first_block + n)
    order = np.lexsort((idx, -np.asarray(scores)))        # primary key: -score; ties: index
    cnt = min(k, n)
    sel = np.sort(idx[order[:cnt]])
    margin = math.inf if n <= k else float(scores[order[cnt - 1]] - scores[order[cnt]]) if cnt > 0 else math.inf
    return sel.astype(np.int64), margin


def selected_positions(geo: ClusterGeometry, sel, block_size: int) -> np.ndarray:
    """Token positions of the selected set: every token of each selected block, or the selected
    tokens themselves (R27)."""
    sel = np.asarray(sel, dtype=np.int64)
    if geo.tokens:
        return sel
    return (sel[:, None] * block_size + np.arange(block_size)[None, :]).reshape(-1)


def key_positions(geo: ClusterGeometry, sel, p: int, block_size: int) -> np.ndarray:
    """Eq. 10 key set of query row p: sink blocks, the shared selected set, and the local
    window [lo_blk * B, p] (causal, R13). The three groups are disjoint by construction (R9)."""
    B = block_size
    sink = np.arange(0, geo.sink_eff * B)
    local = np.arange(geo.lo_blk * B, p + 1)
    return np.concatenate([sink, selected_positions(geo, sel, B), local])


def attention_rows(q, k_pages, v_pages, block_table, geo: ClusterGeometry, sel, rows, block_size: int,
                   softmax_scale: float | None = None, heads=None) -> np.ndarray:
    """Eq. 10 for the query rows ``rows`` (all inside the cluster), fp64: [len(rows), len(heads), d].

    Every row attends to its own key set (``key_positions``); the softmax subtracts the row max.
    ``sel`` may be any index set (the oracle's own or one under test).
    """
    rows = np.asarray(rows, dtype=np.int64)
    Hq, d = q.shape[1], q.shape[2]
    Hkv = k_pages.shape[1]
    heads = np.arange(Hq) if heads is None else np.asarray(heads)
    scale = 1.0 / math.sqrt(d) if not softmax_scale else float(softmax_scale)
    B = block_size
    if len(rows) and (rows.min() < geo.s or rows.max() >= geo.e):
        raise ValueError("rows outside the cluster")
    out = np.empty((len(rows), len(heads), d), dtype=np.float64)
    if len(rows) == 0:
        return out
    # Logical keys/values of every position any requested row can see: the sink and selected
    # sets (visible to every row) then the local window up to the last requested row. With one
    # set per KV head (R29) each KV head has its own selected positions.
    p_max = int(rows.max())
    qx = bf16_to_f64(q[rows])                            # [nr, Hq, d]
    sets = group_sets(sel, Hkv)
    per_set = {}                                         # keyed by set: a shared set is read once

    def keys_of(g):
        key = id(sets[g])
        if key not in per_set:
            fixed = np.concatenate([np.arange(geo.sink_eff * B), selected_positions(geo, sets[g], B)])
            pos = np.concatenate([fixed, np.arange(geo.lo_blk * B, p_max + 1)]).astype(np.int64)
            # Mask from the key-set definition: key t is visible to row p iff t is in Kset(p).
            n_fixed = len(fixed)
            visible = np.ones((len(rows), len(pos)), dtype=bool)
            visible[:, n_fixed:] = pos[None, n_fixed:] <= rows[:, None]
            per_set[key] = (logical_rows(k_pages, block_table, pos, B), logical_rows(v_pages, block_table, pos, B),
                            visible)
        K, V, visible = per_set[key]
        return K[:, g, :], V[:, g, :], visible

    for hi, h in enumerate(heads):
        g = (int(h) * Hkv) // Hq
        Kg, Vg, visible = keys_of(g)
        s = (qx[:, h, :] @ Kg.T) * scale                    # [nr, nk]
        s = np.where(visible, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        w = np.exp(s - m)
        out[:, hi, :] = (w @ Vg) / w.sum(axis=1, keepdims=True)
    return out


def cluster_attention(q, k_pages, v_pages, block_table, geo, sel, block_size, softmax_scale=None,
                      row_chunk: int = 512) -> np.ndarray:
    """Eq. 10 over every row of the cluster: [e - s, Hq, d] fp64."""
    out = np.empty((geo.e - geo.s, q.shape[1], q.shape[2]), dtype=np.float64)
    for r0 in range(geo.s, geo.e, row_chunk):
        rows = np.arange(r0, min(r0 + row_chunk, geo.e))
        out[r0 - geo.s: r0 - geo.s + len(rows)] = attention_rows(
            q, k_pages, v_pages, block_table, geo, sel, rows, block_size, softmax_scale)
    return out


def prefill(q, k_pages, v_pages, block_table, n_tokens: int, *, sub_chunk: int, block_size: int,
            top_k: int, sink_tokens: int, local_window: int, cluster_start, score_scale: float = 1.0,
            softmax_scale: float | None = None, with_output: bool = True, external_sel=None,
            select_tokens: bool = False, rep_kind: str = "mean", kv_head_sets: bool = False) -> dict:
    """Algorithm 2 for one layer with a given cluster assignment.

    For each cluster: anchor fingerprint -> block logits -> soft-voting scores -> top-k
    (selection) -> attention of every row over sink + selected + local keys.
    ``external_sel`` (list of index arrays) replaces the oracle's own selection in the attention
    step, so attention can be checked under another selection.
    ``rep_kind`` "minmax" scores blocks by the R28 bound; ``kv_head_sets`` gives every KV head its
    own set (R29): a cluster's scores are then [Hkv, n_cand], its selection [Hkv, cnt] and its
    margins [Hkv].
    Returns a dict with geometry, k_rep, fingerprints, scores, selections, margins, output.
    """
    if rep_kind not in ("mean", "minmax"):
        raise ValueError("rep_kind is 'mean' or 'minmax'")
    if rep_kind == "minmax" and select_tokens:
        raise ValueError("bound representative keys apply to block-level selection")
    geo = geometry(n_tokens, sub_chunk, block_size, sink_tokens, local_window, top_k, cluster_start,
                   select_tokens)
    k_rep = rep_keys(k_pages, block_table, n_tokens, block_size)
    bounds = rep_bounds(k_pages, block_table, n_tokens, block_size) if rep_kind == "minmax" else None
    Hkv = k_pages.shape[1]
    B = block_size
    fps, scores, sels, margins = [], [], [], []
    for g in geo:
        v = anchor_fingerprint(q, g.s, g.anchor_end)
        if select_tokens:
            # R27: the candidates are single tokens, scored with their own keys
            cand = logical_rows(k_pages, block_table, np.arange(g.sink_blk * B, g.sink_blk * B + g.n_cand), B)
            first = g.sink_blk * B
            x = block_logits(v, cand, Hkv, score_scale)
        elif rep_kind == "minmax":
            c = slice(g.sink_blk, g.sink_blk + g.n_cand)
            first = g.sink_blk
            x = bound_logits(v, bounds[0][c], bounds[1][c], Hkv, score_scale)
        else:
            first = g.sink_blk
            x = block_logits(v, k_rep[g.sink_blk:g.sink_blk + g.n_cand], Hkv, score_scale)
        if kv_head_sets:
            sc = soft_vote_groups(x, Hkv) if x.shape[1] else np.zeros((Hkv, 0))
            picks = [select_topk(sc[kv], first, top_k) for kv in range(Hkv)]
            sel = np.stack([p[0] for p in picks]) if picks else np.zeros((Hkv, 0), dtype=np.int64)
            margin = np.array([p[1] for p in picks])
        else:
            sc = soft_vote(x)
            sel, margin = select_topk(sc, first, top_k)
        fps.append(v)
        scores.append(sc)
        sels.append(sel)
        margins.append(margin)
    out = None
    if with_output:
        out = np.full((n_tokens, q.shape[1], q.shape[2]), np.nan, dtype=np.float64)
        for j, g in enumerate(geo):
            sel = sels[j] if external_sel is None else np.asarray(external_sel[j], dtype=np.int64)
            out[g.s:g.e] = cluster_attention(q, k_pages, v_pages, block_table, g, sel, block_size,
                                             softmax_scale)
    return {
        "geometry": geo,
        "k_rep": k_rep,
        "bounds": bounds,
        "fingerprints": fps,
        "scores": scores,
        "selections": sels,
        "margins": margins,
        "output": out,
        "retrieval_calls": len(geo),
        "degenerate": sum(1 for g in geo if g.n_cand <= top_k),
    }


def subchunk_fingerprints(q, n_tokens: int, sub_chunk: int) -> np.ndarray:
    """Eq. 6 for every sub-chunk of the outer chunk: v_i is the mean over the sub-chunk's rows of the
    multi-head query, all heads concatenated (R22); the last sub-chunk may be short (Sec. 3.1).

    ``q`` is [N, Hq, d] bf16 bits. Returns [M, Hq * d] fp64, M = ceil(N / L).
    """
    m = -(-n_tokens // sub_chunk)
    out = np.empty((m, q.shape[1] * q.shape[2]), dtype=np.float64)
    for i in range(m):
        rows = bf16_to_f64(q[i * sub_chunk:min((i + 1) * sub_chunk, n_tokens)])
        out[i] = rows.reshape(rows.shape[0], -1).sum(axis=0) / rows.shape[0]
    return out


def normalized(v) -> np.ndarray:
    """Sec. 5.1.1: v / ||v||_2 per fingerprint (a zero fingerprint gives NaN, R22)."""
    v = np.asarray(v, dtype=np.float64)
    with np.errstate(invalid="ignore", divide="ignore"):
        return v / np.linalg.norm(v, axis=-1, keepdims=True)


def anchor_clustering(vt, theta: float, sub_chunk: int, l_max: int, outer_subchunks: int = 0,
                      first: int = 0) -> np.ndarray:
    """Algorithm 1 (Sec. 5.1.2): one left-to-right pass over the normalised fingerprints ``vt``.

    The open cluster starts at anchor a; sub-chunk j joins while cos(v_a, v_j) = vt[a] . vt[j]
    reaches ``theta`` and the cluster's current size |C| satisfies |C| * L < L_max (Eq. 8); the
    first j that fails either test closes the cluster and becomes the next anchor. With
    ``outer_subchunks`` > 0 the pass also closes a cluster at every outer-chunk boundary (R23).
    The pass starts at sub-chunk ``first`` (the outer chunks still to prefill, R25).
    Returns cluster_start as int32 [n_clusters + 1] in sub-chunk units (first ``first``, last M).
    """
    vt = np.asarray(vt, dtype=np.float64)
    m = vt.shape[0]
    starts = []
    a = first
    while a < m:
        starts.append(a)
        end = m if outer_subchunks <= 0 else min(m, (a // outer_subchunks + 1) * outer_subchunks)
        size = 1
        j = a + 1
        while j < end and float(vt[a] @ vt[j]) >= theta and size * sub_chunk < l_max:
            size += 1
            j += 1
        a = j
    starts.append(m)
    return np.asarray(starts, dtype=np.int32)


def topk_overlap(cluster_sets, subchunk_sets, cluster_start) -> np.ndarray:
    """Eq. 7 per cluster (R26): rho(C) = |I_C & U_j I_j| / |I_C|, with I_C the cluster's selection and
    I_j the selections of its member sub-chunks j in [cluster_start[c], cluster_start[c + 1]) made
    one sub-chunk at a time; ``subchunk_sets[j]`` is indexed by absolute sub-chunk. NaN when I_C is
    empty."""
    out = np.empty(len(cluster_sets), dtype=np.float64)
    for c, i_c in enumerate(cluster_sets):
        i_c = set(int(x) for x in i_c)
        union = set()
        for j in range(int(cluster_start[c]), int(cluster_start[c + 1])):
            union |= set(int(x) for x in subchunk_sets[j])
        out[c] = len(i_c & union) / len(i_c) if i_c else math.nan
    return out
