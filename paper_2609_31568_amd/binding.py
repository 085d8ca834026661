"""ctypes binding of libscale.so, the C ABI in include/scale.h.

Argument marshalling only: every step of the path runs in the library's HIP kernels. Device
tensors are torch tensors (or raw integer addresses); torch supplies memory and the stream.
Importing this module loads the library and raises if it has not been built: there is no other
implementation to fall back to.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIB_PATH

SCALE_OK = 0
SCALE_ERR_INVALID_ARG = -1
SCALE_ERR_UNSUPPORTED = -2
SCALE_ERR_OUT_OF_MEMORY = -3
SCALE_ERR_CAPACITY = -4
SCALE_ERR_HIP = -5
SCALE_OUT_F32 = 0
SCALE_OUT_BF16 = 1
SCALE_REP_MEAN = 0
SCALE_REP_BOUNDS = 1

EXPORTS = (
    "scale_init", "scale_free", "scale_rep_keys", "scale_select_cluster", "scale_sparse_prefill",
    "scale_status_string", "scale_retrieval_calls", "scale_cluster_geometry", "scale_enable_timing",
    "scale_stage_times", "scale_cluster_subchunks", "scale_rep_keys_range", "scale_select_cluster_tokens",
    "scale_init_variant", "scale_fingerprints", "scale_select_cluster_static", "scale_enable_stage_timing",
)
STAGES = ("rep_keys", "fingerprint", "logits", "vote_topk", "attention", "cluster", "gather")


class ScaleError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


class scale_config(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("sub_chunk", ctypes.c_int32),
        ("top_k", ctypes.c_int32),
        ("sink_tokens", ctypes.c_int32),
        ("local_window", ctypes.c_int32),
        ("max_tokens", ctypes.c_int32),
        ("max_clusters", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("score_scale", ctypes.c_float),
        ("out_dtype", ctypes.c_int32),
    ]


class scale_variant(ctypes.Structure):
    _fields_ = [
        ("select_tokens", ctypes.c_int32),
        ("rep_kind", ctypes.c_int32),
        ("kv_head_sets", ctypes.c_int32),
    ]


class Config:
    """A scale_config and the scale_variant it is used with; fields of either read and write by name."""

    _VARIANT = {name for name, _ in scale_variant._fields_}

    def __init__(self, base: scale_config, variant: scale_variant):
        object.__setattr__(self, "base", base)
        object.__setattr__(self, "variant", variant)

    def __getattr__(self, name):
        return getattr(self.variant if name in Config._VARIANT else self.base, name)

    def __setattr__(self, name, value):
        setattr(self.variant if name in Config._VARIANT else self.base, name, value)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libscale.so is not built ({LIB_PATH}); run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.scale_init.argtypes = [ctypes.POINTER(scale_config), vp, ctypes.POINTER(vp)]
    lib.scale_init.restype = ctypes.c_int
    lib.scale_init_variant.argtypes = [ctypes.POINTER(scale_config), ctypes.POINTER(scale_variant), vp,
                                       ctypes.POINTER(vp)]
    lib.scale_init_variant.restype = ctypes.c_int
    lib.scale_free.argtypes = [vp]
    lib.scale_free.restype = None
    lib.scale_rep_keys.argtypes = [vp, vp, vp, i32, vp]
    lib.scale_rep_keys.restype = ctypes.c_int
    lib.scale_select_cluster.argtypes = [vp, vp, i32, vp, vp, i32, vp, vp, vp]
    lib.scale_select_cluster.restype = ctypes.c_int
    lib.scale_select_cluster_tokens.argtypes = [vp, vp, i32, vp, vp, vp, i32, vp, vp, vp]
    lib.scale_select_cluster_tokens.restype = ctypes.c_int
    lib.scale_fingerprints.argtypes = [vp, vp, i32]
    lib.scale_fingerprints.restype = ctypes.c_int
    lib.scale_select_cluster_static.argtypes = [ctypes.POINTER(scale_config), vp, vp, i32, vp, vp, i32, vp, vp, vp]
    lib.scale_select_cluster_static.restype = ctypes.c_int
    lib.scale_sparse_prefill.argtypes = [vp, vp, vp, vp, vp, i32, vp, i32, vp, vp, vp]
    lib.scale_sparse_prefill.restype = ctypes.c_int
    lib.scale_status_string.argtypes = [ctypes.c_int]
    lib.scale_status_string.restype = ctypes.c_char_p
    lib.scale_retrieval_calls.argtypes = [vp, ctypes.POINTER(i64)]
    lib.scale_retrieval_calls.restype = ctypes.c_int
    lib.scale_cluster_geometry.argtypes = [ctypes.POINTER(scale_config), ctypes.POINTER(scale_variant), i32, vp,
                                           i32, vp]
    lib.scale_cluster_geometry.restype = ctypes.c_int
    lib.scale_enable_timing.argtypes = [vp, ctypes.c_int]
    lib.scale_enable_timing.restype = ctypes.c_int
    lib.scale_enable_stage_timing.argtypes = [vp, ctypes.c_uint32]
    lib.scale_enable_stage_timing.restype = ctypes.c_int
    lib.scale_stage_times.argtypes = [vp, vp, vp, ctypes.c_int]
    lib.scale_stage_times.restype = ctypes.c_int
    lib.scale_cluster_subchunks.argtypes = [vp, vp, i32, i32, ctypes.c_double, i32, i32, vp, vp, vp]
    lib.scale_rep_keys_range.argtypes = [vp, vp, vp, i32, i32, vp]
    lib.scale_rep_keys_range.restype = ctypes.c_int
    lib.scale_cluster_subchunks.restype = ctypes.c_int
    return lib


lib = _load()


def status_string(status: int) -> str:
    return lib.scale_status_string(int(status)).decode()


def _ptr(x):
    """Address of a torch tensor / numpy array / int, or None for NULL."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _check(status: int, where: str):
    if status != SCALE_OK:
        raise ScaleError(status, where)


def _cluster_start(cs) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(cs, dtype=np.int32))
    return a


def make_config(*, num_q_heads, num_kv_heads, head_dim, block_size, sub_chunk, top_k, sink_tokens,
                local_window, max_tokens, max_clusters, softmax_scale=0.0, score_scale=0.0,
                out_dtype=SCALE_OUT_F32, select_tokens=False, rep_kind=SCALE_REP_MEAN,
                kv_head_sets=False) -> Config:
    return Config(scale_config(num_q_heads, num_kv_heads, head_dim, block_size, sub_chunk, top_k, sink_tokens,
                               local_window, max_tokens, max_clusters, softmax_scale, score_scale, out_dtype),
                  scale_variant(1 if select_tokens else 0, int(rep_kind), 1 if kv_head_sets else 0))


def scale_cluster_geometry(cfg: Config, n_tokens: int, cluster_start) -> np.ndarray:
    """Host-only geometry: int32 [n_clusters, 6] = (s, e, lo_blk, sink_eff, n_cand, sel_cnt)."""
    cs = _cluster_start(cluster_start)
    n = len(cs) - 1
    geo = np.zeros((max(n, 0), 6), dtype=np.int32)
    _check(lib.scale_cluster_geometry(ctypes.byref(cfg.base), ctypes.byref(cfg.variant), int(n_tokens),
                                      cs.ctypes.data, n, geo.ctypes.data), "scale_cluster_geometry")
    return geo


def _stream_handle(stream):
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Scale:
    """One library handle (scale_init ... scale_free), bound to the current device and a stream."""

    def __init__(self, cfg: Config, stream=None):
        self.cfg = cfg
        self.stream = _stream_handle(stream)
        h = ctypes.c_void_p()
        _check(lib.scale_init_variant(ctypes.byref(cfg.base), ctypes.byref(cfg.variant), self.stream,
                                      ctypes.byref(h)), "scale_init_variant")
        self._h = h

    def close(self):
        if self._h is not None and self._h.value:
            lib.scale_free(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def handle(self):
        return self._h

    def rep_keys(self, k_pages, block_table, n_tokens: int, k_rep):
        _check(lib.scale_rep_keys(self._h, _ptr(k_pages), _ptr(block_table), int(n_tokens), _ptr(k_rep)),
               "scale_rep_keys")

    def rep_keys_range(self, k_pages, block_table, first_block: int, n_tokens: int, k_rep):
        _check(lib.scale_rep_keys_range(self._h, _ptr(k_pages), _ptr(block_table), int(first_block), int(n_tokens),
                                        _ptr(k_rep)), "scale_rep_keys_range")

    def select_cluster(self, q, n_tokens: int, k_rep, cluster_start, sel_idx, sel_cnt, scores_out=None):
        cs = _cluster_start(cluster_start)
        _check(lib.scale_select_cluster(self._h, _ptr(q), int(n_tokens), _ptr(k_rep), cs.ctypes.data, len(cs) - 1,
                                        _ptr(sel_idx), _ptr(sel_cnt), _ptr(scores_out)),
               "scale_select_cluster")

    def select_cluster_tokens(self, q, n_tokens: int, k_pages, block_table, cluster_start, sel_idx, sel_cnt,
                              scores_out=None):
        cs = _cluster_start(cluster_start)
        _check(lib.scale_select_cluster_tokens(self._h, _ptr(q), int(n_tokens), _ptr(k_pages), _ptr(block_table),
                                               cs.ctypes.data, len(cs) - 1, _ptr(sel_idx), _ptr(sel_cnt),
                                               _ptr(scores_out)),
               "scale_select_cluster_tokens")

    def fingerprints(self, out, n_clusters: int):
        _check(lib.scale_fingerprints(self._h, _ptr(out), int(n_clusters)), "scale_fingerprints")

    def sparse_prefill(self, q, k_pages, v_pages, block_table, n_tokens: int, cluster_start, sel_idx, sel_cnt, out):
        cs = _cluster_start(cluster_start)
        _check(lib.scale_sparse_prefill(self._h, _ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(block_table),
                                        int(n_tokens), cs.ctypes.data, len(cs) - 1, _ptr(sel_idx), _ptr(sel_cnt),
                                        _ptr(out)),
               "scale_sparse_prefill")

    def cluster_subchunks(self, q, n_tokens: int, theta: float, l_max: int, outer_subchunks: int = 0,
                          with_band: bool = False, first_subchunk: int = 0):
        """Anchor-based clustering of the sub-chunks [first_subchunk, M); returns cluster_start
        (int32 [n + 1]) and, with ``with_band``, the cosine band [M - first][span] (include/scale.h)."""
        L = self.cfg.sub_chunk
        m = -(-int(n_tokens) // L) - int(first_subchunk)
        cs = np.zeros(max(m, 0) + 1, dtype=np.int32)
        n = ctypes.c_int32()
        band = None
        if with_band:
            band = np.full((max(m, 0), max(cluster_span(l_max, L, outer_subchunks, m), 0)), np.nan, dtype=np.float64)
        _check(lib.scale_cluster_subchunks(self._h, _ptr(q), int(n_tokens), int(first_subchunk), float(theta),
                                           int(l_max), int(outer_subchunks), cs.ctypes.data, ctypes.byref(n),
                                           None if band is None or band.size == 0 else band.ctypes.data),
               "scale_cluster_subchunks")
        cs = cs[:n.value + 1].copy()
        return (cs, band) if with_band else cs

    def enable_timing(self, enable: bool = True):
        _check(lib.scale_enable_timing(self._h, 1 if enable else 0), "scale_enable_timing")

    def enable_stage_timing(self, stages=()):
        """Time only the named stages (names of STAGES); an empty selection turns timing off."""
        mask = 0
        for name in stages:
            mask |= 1 << STAGES.index(name)
        _check(lib.scale_enable_stage_timing(self._h, mask), "scale_enable_stage_timing")

    def stage_times(self, reset: bool = False) -> dict:
        """{stage: (device ms accumulated, launches)}; synchronises the handle's stream."""
        ms = np.zeros(len(STAGES), dtype=np.float64)
        n = np.zeros(len(STAGES), dtype=np.int64)
        _check(lib.scale_stage_times(self._h, ms.ctypes.data, n.ctypes.data, 1 if reset else 0), "scale_stage_times")
        return {s: (float(ms[i]), int(n[i])) for i, s in enumerate(STAGES)}

    def retrieval_calls(self) -> int:
        n = ctypes.c_int64()
        _check(lib.scale_retrieval_calls(self._h, ctypes.byref(n)), "scale_retrieval_calls")
        return int(n.value)


# Same names as the C ABI, for callers that prefer the flat form.
def scale_init(cfg: Config, stream=None) -> Scale:
    return Scale(cfg, stream)


def scale_free(h: Scale) -> None:
    h.close()


def scale_rep_keys(h: Scale, k_pages, block_table, n_tokens, k_rep):
    h.rep_keys(k_pages, block_table, n_tokens, k_rep)


def scale_select_cluster(h: Scale, q, n_tokens, k_rep, cluster_start, sel_idx, sel_cnt, scores_out=None):
    h.select_cluster(q, n_tokens, k_rep, cluster_start, sel_idx, sel_cnt, scores_out)


def scale_select_cluster_tokens(h: Scale, q, n_tokens, k_pages, block_table, cluster_start, sel_idx, sel_cnt,
                                scores_out=None):
    h.select_cluster_tokens(q, n_tokens, k_pages, block_table, cluster_start, sel_idx, sel_cnt, scores_out)


def scale_fingerprints(h: Scale, out, n_clusters):
    h.fingerprints(out, n_clusters)


def scale_select_cluster_static(cfg: Config, q, n_tokens, k_rep, cluster_start, sel_idx, sel_cnt, scores_out=None,
                                stream=None):
    """The allocation-free selection (no handle; the library's static device scratch)."""
    cs = _cluster_start(cluster_start)
    _check(lib.scale_select_cluster_static(ctypes.byref(cfg.base), _stream_handle(stream), _ptr(q), int(n_tokens),
                                           _ptr(k_rep), cs.ctypes.data, len(cs) - 1, _ptr(sel_idx), _ptr(sel_cnt),
                                           _ptr(scores_out)), "scale_select_cluster_static")


def scale_sparse_prefill(h: Scale, q, k_pages, v_pages, block_table, n_tokens, cluster_start, sel_idx, sel_cnt, out):
    h.sparse_prefill(q, k_pages, v_pages, block_table, n_tokens, cluster_start, sel_idx, sel_cnt, out)


def scale_retrieval_calls(h: Scale) -> int:
    return h.retrieval_calls()


def scale_cluster_subchunks(h: Scale, q, n_tokens, first_subchunk, theta, l_max, outer_subchunks=0, with_band=False):
    return h.cluster_subchunks(q, n_tokens, theta, l_max, outer_subchunks, with_band, first_subchunk)


def scale_rep_keys_range(h: Scale, k_pages, block_table, first_block, n_tokens, k_rep):
    h.rep_keys_range(k_pages, block_table, first_block, n_tokens, k_rep)


def cluster_span(l_max: int, sub_chunk: int, outer_subchunks: int, m: int) -> int:
    """Width of the cosine band of scale_cluster_subchunks (include/scale.h)."""
    cap = -(-int(l_max) // int(sub_chunk))
    if outer_subchunks > 0:
        cap = min(cap, int(outer_subchunks))
    return min(cap, int(m)) - 1
