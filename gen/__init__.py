"""Seeded synthetic inputs for cluster-level sparse prefill (topic-structured Q/K/V).

This module only draws inputs; it holds none of the method's arithmetic. The numbers come from
``topicgen.c`` (counter-based SplitMix64 + Box-Muller, bf16 round-to-nearest-even), so every element
is a pure function of (seed, layer, tensor, index). The workloads stand in for the long-context
benchmarks the paper prefills (InfiniteBench, RULER; paper Sec. V, experimental setup): queries
follow topic runs over sub-chunks, KV blocks carry random topics, so block selection has a
meaningful answer.

The cluster assignment ``cluster_starts(M, c)`` (runs of ``c`` consecutive sub-chunks) is an input
of the method, equal to the anchor clustering of Algorithm 1 with the threshold disabled and
``L_max = c * L``.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtopicgen.so")
_lib = None


def build(verbose: bool = False) -> str:
    """Compile ``topicgen.c`` into ``libtopicgen.so`` (gcc, OpenMP)."""
    import subprocess

    src = os.path.join(_HERE, "topicgen.c")
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", src, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        build()
    lib = ctypes.CDLL(LIB_PATH)
    u64, i32, i64 = ctypes.c_uint64, ctypes.c_int, ctypes.c_int64
    p = ctypes.c_void_p
    lib.tg_stream_key.argtypes = [u64, u64, u64]
    lib.tg_stream_key.restype = u64
    lib.tg_draw.argtypes = [u64, u64]
    lib.tg_draw.restype = u64
    lib.tg_normal.argtypes = [u64, u64]
    lib.tg_normal.restype = ctypes.c_double
    lib.tg_bf16.argtypes = [ctypes.c_double]
    lib.tg_bf16.restype = ctypes.c_uint16
    lib.tg_topics.argtypes = [u64, i32, i32, i32, p]
    lib.tg_query_topics.argtypes = [u64, i32, i32, i32, i32, i32, ctypes.c_double, ctypes.c_double, p, p]
    lib.tg_kv_topics.argtypes = [u64, i32, i32, i32, p]
    lib.tg_fill_q.argtypes = [u64, i32, p, p, p, i32, i32, i32, i64, i64, p]
    lib.tg_fill_kv.argtypes = [u64, i32, p, p, i32, i32, i32, i64, i64, p, p]
    _lib = lib
    return lib


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: attention shape, SCR geometry and generator parameters."""

    name: str
    layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    n_tokens: int
    block_size: int
    sub_chunk: int
    cluster: int
    top_k: int
    sink_tokens: int
    local_window: int
    n_topics: int
    run_lo: int
    run_hi: int
    seed: int
    q_scale_lo: float = 2.0   # topic strength of a query run, drawn uniformly in [lo, hi]
    q_scale_hi: float = 2.0

    @property
    def n_blocks(self) -> int:
        return -(-self.n_tokens // self.block_size)

    @property
    def n_sub_chunks(self) -> int:
        return -(-self.n_tokens // self.sub_chunk)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # 1 layer, 4 query heads / 1 KV head, d 64, 2K context
    "tiny": Workload("tiny", 1, 4, 1, 64, 2048, 64, 256, 4, 4, 64, 256, 8, 1, 4, 0),
    # Llama-3-8B attention shape (32q / 8kv, d 128), one layer, 32K context
    "llama32k": Workload("llama32k", 1, 32, 8, 128, 32768, 128, 512, 8, 16, 128, 4096, 64, 2, 8, 1),
    # same layer at 128K context: the headline workload
    "llama128k": Workload("llama128k", 1, 32, 8, 128, 131072, 128, 512, 8, 32, 128, 4096, 256, 2, 16, 2),
    # one GPU's share of the 128K layer split four ways by KV head (8q / 2kv): the attention shape
    # of one shard; its selection votes over its own 8 heads (the cross-shard score sum is the one
    # exchange of the split and is not run here)
    "llama128k_tp4": Workload("llama128k_tp4", 1, 8, 2, 128, 131072, 128, 512, 8, 32, 128, 4096, 256, 2, 16, 6),
    # Qwen2-7B-shaped stack (28 layers, 28q / 4kv, d 128), 256K context
    "qwen256k": Workload("qwen256k", 28, 28, 4, 128, 262144, 128, 1024, 4, 32, 128, 8192, 512, 1, 8, 3),
    # Llama-3-8B layer at 1M context; the cluster size is swept over {1, 2, 4, 8, 16}
    "stress1m": Workload("stress1m", 1, 32, 8, 128, 1048576, 128, 512, 8, 64, 128, 4096, 2048, 1, 32, 4),
    # the 128K layer with query runs of varying coherence (topic strength 2 .. 6, so same-topic
    # sub-chunk fingerprints have cosines from about 0.94 to 0.993): the similarity-threshold
    # clustering workload; its fixed cluster size (8) is the L_max / L cap of the paper's default
    "scr128k": Workload("scr128k", 1, 32, 8, 128, 131072, 128, 512, 8, 32, 128, 4096, 256, 2, 16, 5,
                        q_scale_lo=2.0, q_scale_hi=6.0),
}


def cluster_starts(n_sub_chunks: int, c: int) -> np.ndarray:
    """Cluster boundaries in sub-chunk units: runs of ``c`` consecutive sub-chunks, last one short."""
    if c <= 0:
        raise ValueError("cluster size must be positive")
    starts = list(range(0, n_sub_chunks, c)) + [n_sub_chunks]
    return np.asarray(starts, dtype=np.int32)


def bf16_bits_to_f64(u16: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float64."""
    u32 = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16
    return u32.view(np.float32).astype(np.float64)


def topics(w: Workload, layer: int = 0) -> np.ndarray:
    lib = _load()
    t = np.empty((w.n_topics, w.head_dim), dtype=np.float64)
    lib.tg_topics(w.seed, layer, w.n_topics, w.head_dim, t.ctypes.data)
    return t


def query_runs(w: Workload, layer: int = 0):
    """(topic, topic strength) of every sub-chunk: int32 [M], float64 [M]."""
    lib = _load()
    qt = np.empty(w.n_sub_chunks, dtype=np.int32)
    qs = np.empty(w.n_sub_chunks, dtype=np.float64)
    lib.tg_query_topics(w.seed, layer, w.n_topics, w.run_lo, w.run_hi, w.n_sub_chunks, float(w.q_scale_lo),
                        float(w.q_scale_hi), qt.ctypes.data, qs.ctypes.data)
    return qt, qs


def query_topics(w: Workload, layer: int = 0) -> np.ndarray:
    return query_runs(w, layer)[0]


def kv_topics(w: Workload, layer: int = 0) -> np.ndarray:
    lib = _load()
    kt = np.empty(w.n_blocks, dtype=np.int32)
    lib.tg_kv_topics(w.seed, layer, w.n_topics, w.n_blocks, kt.ctypes.data)
    return kt


def q_rows(w: Workload, row0: int, n_rows: int, layer: int = 0, *, _topics=None, _qruns=None,
           out: np.ndarray | None = None) -> np.ndarray:
    """Q rows [row0, row0 + n_rows) as bf16 bits, shape [n_rows, Hq, d]."""
    lib = _load()
    t = topics(w, layer) if _topics is None else _topics
    qt, qs = query_runs(w, layer) if _qruns is None else _qruns
    if row0 < 0 or row0 + n_rows > w.n_tokens:
        raise ValueError("row range outside the context")
    q = out if out is not None else np.empty((n_rows, w.num_q_heads, w.head_dim), dtype=np.uint16)
    assert q.shape == (n_rows, w.num_q_heads, w.head_dim) and q.dtype == np.uint16 and q.flags.c_contiguous
    lib.tg_fill_q(w.seed, layer, t.ctypes.data, qt.ctypes.data, qs.ctypes.data, w.sub_chunk, w.num_q_heads,
                  w.head_dim, row0, n_rows, q.ctypes.data)
    return q


def kv_blocks(w: Workload, blk0: int, n_blk: int, layer: int = 0, *, want_k=True, want_v=True,
              _topics=None, _kvtopic=None, out_k=None, out_v=None):
    """K and V pages for logical blocks [blk0, blk0 + n_blk), bf16 bits [n_blk, Hkv, B, d] each."""
    lib = _load()
    if w.n_tokens % w.block_size:
        raise ValueError("the generator writes whole blocks only")
    t = topics(w, layer) if _topics is None else _topics
    kt = kv_topics(w, layer) if _kvtopic is None else _kvtopic
    if blk0 < 0 or blk0 + n_blk > w.n_blocks:
        raise ValueError("block range outside the context")
    shape = (n_blk, w.num_kv_heads, w.block_size, w.head_dim)
    k = (out_k if out_k is not None else np.empty(shape, dtype=np.uint16)) if want_k else None
    v = (out_v if out_v is not None else np.empty(shape, dtype=np.uint16)) if want_v else None
    for a in (k, v):
        if a is not None:
            assert a.shape == shape and a.dtype == np.uint16 and a.flags.c_contiguous
    lib.tg_fill_kv(w.seed, layer, t.ctypes.data, kt.ctypes.data, w.block_size, w.num_kv_heads,
                   w.head_dim, blk0, n_blk, None if k is None else k.ctypes.data,
                   None if v is None else v.ctypes.data)
    return k, v


def make_layer(w: Workload, layer: int = 0) -> dict:
    """All inputs of one layer: q [N, Hq, d], k_pages / v_pages [n_blocks, Hkv, B, d] (bf16 bits),
    identity block table, and the topic labels that generated them."""
    t = topics(w, layer)
    qt, qs = query_runs(w, layer)
    kt = kv_topics(w, layer)
    q = q_rows(w, 0, w.n_tokens, layer, _topics=t, _qruns=(qt, qs))
    k, v = kv_blocks(w, 0, w.n_blocks, layer, _topics=t, _kvtopic=kt)
    return {
        "q": q,
        "k_pages": k,
        "v_pages": v,
        "block_table": np.arange(w.n_blocks, dtype=np.int32),
        "qtopic": qt,
        "qscale": qs,
        "kvtopic": kt,
        "topics": t,
    }


def stream_key(seed: int, layer: int, tensor: int) -> int:
    return int(_load().tg_stream_key(seed, layer, tensor))


def draw(key: int, n: int) -> int:
    return int(_load().tg_draw(key, n))


def normal(key: int, i: int) -> float:
    return float(_load().tg_normal(key, i))


def bf16_round(x: float) -> int:
    return int(_load().tg_bf16(x))
