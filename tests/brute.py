"""Brute-force references used to pin the oracle on tiny inputs.

Written separately from the oracle and in a different style: token-level loops, explicit
position sets, an explicit N x N visibility mask, and exhaustive subset enumeration. Nothing here
imports the oracle or the HIP path.

* Selection (paper Sec. 5.1.3, Eq. 9 and head soft-voting): a block's logit for head h is the
  average over the block's tokens t and the anchor rows p of q[p][h] . k[t][g(h)] -- by bilinearity
  this equals the anchor-mean query dotted with the block-mean key. Softmax per head over the
  candidate blocks, summed over heads; the chosen set is the k-subset with the largest total score,
  ties broken toward the lexicographically smallest sorted index tuple.
* Attention (Eq. 10): dense softmax over all N keys under a boolean mask built from the three key
  groups (sink, selected blocks, cluster-spanning local window) and the causal rule.
"""
from __future__ import annotations

import itertools
import math

import numpy as np


def widen(u16):
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def unpage(pages, block_table):
    """[n_pages, Hkv, B, d] bf16 bits + table -> logical fp64 [n_blocks * B, Hkv, d]."""
    nb = len(block_table)
    Hkv, B, d = pages.shape[1], pages.shape[2], pages.shape[3]
    out = np.empty((nb * B, Hkv, d))
    for b in range(nb):
        blk = widen(pages[int(block_table[b])])        # [Hkv, B, d]
        for t in range(B):
            out[b * B + t] = blk[:, t, :]
    return out


def cluster_layout(n_tokens, L, B, S, W, cluster_start):
    """(s, e, anchor_end, lo_blk, sink_eff, cand list) per cluster, from the definitions."""
    res = []
    for j in range(len(cluster_start) - 1):
        s = int(cluster_start[j]) * L
        e = min(int(cluster_start[j + 1]) * L, n_tokens)
        anchor_end = min(s + L, e)
        # the local window covers the whole cluster and at least W tokens ending at e
        lo = s if e - s >= W else max(0, e - W)
        lo_blk = lo // B
        sink_blocks = [b for b in range(math.ceil(S / B)) if b < lo_blk]
        cand = [b for b in range(lo_blk) if b >= math.ceil(S / B)]
        res.append((s, e, anchor_end, lo_blk, len(sink_blocks), cand))
    return res


def brute_scores(q, K, anchor_rows, cand, B, Hkv, score_scale=1.0):
    """Soft-voting score of every candidate block, by explicit loops. q fp64 [N, Hq, d], K fp64
    logical [N, Hkv, d]."""
    Hq = q.shape[1]
    G = Hq // Hkv
    total = {b: 0.0 for b in cand}
    for h in range(Hq):
        g = h // G
        logits = {}
        for b in cand:
            acc = 0.0
            for p in anchor_rows:
                acc += float(np.dot(K[b * B:(b + 1) * B, g, :], q[p, h, :]).sum())
            logits[b] = score_scale * acc / (len(anchor_rows) * B)
        if not logits:
            continue
        mx = max(logits.values())
        den = sum(math.exp(x - mx) for x in logits.values())
        for b in cand:
            total[b] += math.exp(logits[b] - mx) / den
    return total


def brute_select(scores: dict, k: int, rel_tie: float = 1e-12):
    cand = sorted(scores)
    if len(cand) <= k:
        return tuple(cand)
    best, best_sum = None, -math.inf
    for combo in itertools.combinations(cand, k):     # generated in lexicographic order
        ssum = sum(scores[b] for b in combo)
        if best is None or ssum > best_sum + rel_tie * max(1.0, abs(best_sum)):
            best, best_sum = combo, ssum
    return best


def visibility_mask(n_tokens, layout, selections, B):
    """Explicit N x N mask: vis[p][t] is True iff key t is in query p's key set."""
    vis = np.zeros((n_tokens, n_tokens), dtype=bool)
    for (s, e, _a, lo_blk, sink_eff, _c), sel in zip(layout, selections):
        allowed = set(range(sink_eff * B))
        for b in sel:
            allowed.update(range(b * B, (b + 1) * B))
        for p in range(s, e):
            keys = set(allowed)
            keys.update(range(lo_blk * B, p + 1))
            for t in keys:
                if t <= p:
                    vis[p, t] = True
                else:
                    raise AssertionError("a key after its query would be visible")
    return vis


def masked_attention(q, K, V, vis, scale=None):
    """Dense softmax attention under an explicit mask, every head. fp64 [N, Hq, d]."""
    N, Hq, d = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    out = np.empty_like(q)
    for h in range(Hq):
        g = h // G
        s = (q[:, h, :] @ K[:N, g, :].T) * scale
        s = np.where(vis, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        w = np.exp(s)
        out[:, h, :] = (w @ V[:N, g, :]) / w.sum(axis=1, keepdims=True)
    return out


def brute_prefill(q_bits, k_pages, v_pages, block_table, n_tokens, L, B, S, W, k, cluster_start,
                  score_scale=1.0):
    q = widen(q_bits)
    K = unpage(k_pages, block_table)
    V = unpage(v_pages, block_table)
    Hkv = k_pages.shape[1]
    layout = cluster_layout(n_tokens, L, B, S, W, cluster_start)
    sels, scores = [], []
    for (s, e, a_end, lo_blk, sink_eff, cand) in layout:
        sc = brute_scores(q, K, range(s, a_end), cand, B, Hkv, score_scale)
        scores.append(sc)
        sels.append(brute_select(sc, k))
    vis = visibility_mask(n_tokens, layout, sels, B)
    return {"layout": layout, "scores": scores, "selections": sels, "mask": vis,
            "output": masked_attention(q, K, V, vis)}


def brute_prefill_tokens(q_bits, k_pages, v_pages, block_table, n_tokens, L, B, S, W, k, cluster_start,
                         score_scale=1.0):
    """Token-level selection by explicit loops: every single token between the sink blocks and the
    local window is a candidate scored with its own key; exhaustive best-total k-subset; explicit
    mask; dense masked softmax."""
    q = widen(q_bits)
    K = unpage(k_pages, block_table)
    V = unpage(v_pages, block_table)
    Hkv = k_pages.shape[1]
    Hq = q.shape[1]
    G = Hq // Hkv
    layout = cluster_layout(n_tokens, L, B, S, W, cluster_start)
    sels, scores = [], []
    for (s, e, a_end, lo_blk, sink_eff, cand_blocks) in layout:
        cand = [t for b in cand_blocks for t in range(b * B, (b + 1) * B)]
        total = {t: 0.0 for t in cand}
        for h in range(Hq):
            g = h // G
            logits = {}
            for t in cand:
                acc = 0.0
                for p in range(s, a_end):
                    acc += float(np.dot(K[t, g, :], q[p, h, :]))
                logits[t] = score_scale * acc / (a_end - s)
            if not logits:
                continue
            mx = max(logits.values())
            den = sum(math.exp(x - mx) for x in logits.values())
            for t in cand:
                total[t] += math.exp(logits[t] - mx) / den
        scores.append(total)
        sels.append(brute_select(total, k))
    vis = np.zeros((n_tokens, n_tokens), dtype=bool)
    for (s, e, _a, lo_blk, sink_eff, _c), sel in zip(layout, sels):
        allowed = set(range(sink_eff * B)) | set(sel)
        for p in range(s, e):
            for t in allowed | set(range(lo_blk * B, p + 1)):
                assert t <= p, "a key after its query would be visible"
                vis[p, t] = True
    return {"layout": layout, "scores": scores, "selections": sels, "mask": vis,
            "output": masked_attention(q, K, V, vis)}


def brute_prefill_variants(q_bits, k_pages, v_pages, block_table, n_tokens, L, B, S, W, k, cluster_start,
                           score_scale=1.0, bounds=False, per_kv_head=False):
    """Block-level selection with the two variants by explicit loops.

    bounds: a block's logit for head h is sigma * sum over channels i of the larger of v_i * lo_i
    and v_i * hi_i, lo_i / hi_i the smallest / largest channel-i key value among the block's tokens
    (found by scanning the tokens), v the anchor-row mean (summed row by row).
    per_kv_head: the softmax weights are summed over the query heads of each KV head separately;
    every KV head picks its own best-total k-subset and its query heads attend under its own mask.
    """
    q = widen(q_bits)
    K = unpage(k_pages, block_table)
    V = unpage(v_pages, block_table)
    Hkv = k_pages.shape[1]
    Hq, d = q.shape[1], q.shape[2]
    G = Hq // Hkv
    layout = cluster_layout(n_tokens, L, B, S, W, cluster_start)
    groups = list(range(Hkv)) if per_kv_head else [None]
    sels = {gr: [] for gr in groups}
    for (s, e, a_end, lo_blk, sink_eff, cand) in layout:
        totals = {gr: {b: 0.0 for b in cand} for gr in groups}
        for h in range(Hq):
            g = h // G
            v = [0.0] * d
            for p in range(s, a_end):
                for i in range(d):
                    v[i] += q[p, h, i]
            v = [x / (a_end - s) for x in v]
            logits = {}
            for b in cand:
                if bounds:
                    acc = 0.0
                    for i in range(d):
                        lo_i = min(K[t, g, i] for t in range(b * B, (b + 1) * B))
                        hi_i = max(K[t, g, i] for t in range(b * B, (b + 1) * B))
                        acc += max(v[i] * lo_i, v[i] * hi_i)
                    logits[b] = score_scale * acc
                else:
                    logits[b] = score_scale * sum(float(np.dot(K[t, g, :], v)) for t in range(b * B, (b + 1) * B)) / B
            if not logits:
                continue
            mx = max(logits.values())
            den = sum(math.exp(x - mx) for x in logits.values())
            gr = g if per_kv_head else None
            for b in cand:
                totals[gr][b] += math.exp(logits[b] - mx) / den
        for gr in groups:
            sels[gr].append(brute_select(totals[gr], k))
    out = np.empty_like(q)
    for gr in groups:
        vis = visibility_mask(n_tokens, layout, sels[gr], B)
        full = masked_attention(q, K, V, vis)
        heads = range(Hq) if gr is None else range(gr * G, (gr + 1) * G)
        for h in heads:
            out[:, h, :] = full[:, h, :]
    return {"layout": layout, "selections": sels, "output": out}
