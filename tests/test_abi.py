"""C-ABI contract checks that need no GPU: exported symbols, status strings, host-side validation
and the host geometry (compared with the oracle's). No call here reaches the device: every
scale_init below carries a config the host rejects before its first HIP call."""
import ctypes
import os
import re

import numpy as np
import pytest

import gen
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _pk():
    import paper_2609_31568_amd as pk

    return pk


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "scale.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(scale_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    pk = _pk()
    declared = _declared_functions()
    assert set(declared) == set(pk.EXPORTS)
    lib = ctypes.CDLL(pk.build.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings():
    pk = _pk()
    for code in (0, -1, -2, -3, -4, -5):
        assert pk.status_string(code) and pk.status_string(code) != "unknown status"
    assert pk.status_string(7) == "unknown status"


def _cfg(**over):
    pk = _pk()
    kw = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=128, sub_chunk=512, top_k=32,
              sink_tokens=128, local_window=4096, max_tokens=131072, max_clusters=32)
    kw.update(over)
    return pk.make_config(**kw)


@pytest.mark.parametrize("over,status", [
    (dict(num_q_heads=0), -1),
    (dict(num_q_heads=30), -1),            # not a multiple of the KV heads
    (dict(num_kv_heads=0), -1),
    (dict(top_k=-1), -1),
    (dict(sink_tokens=-1), -1),
    (dict(local_window=-5), -1),
    (dict(max_tokens=0), -1),
    (dict(max_clusters=0), -1),
    (dict(softmax_scale=-1.0), -1),
    (dict(softmax_scale=float("nan")), -1),
    (dict(score_scale=float("inf")), -1),
    (dict(out_dtype=2), -1),
    (dict(head_dim=96), -2),
    (dict(block_size=32), -2),
    (dict(sub_chunk=192), -2),             # not a multiple of the block size
    (dict(num_q_heads=72, num_kv_heads=8), -2),   # group of 9 query heads
    (dict(select_tokens=2), -1),
    (dict(select_tokens=1, top_k=1 << 20, max_clusters=4096), -2),   # gathered rows past int32
    (dict(rep_kind=2), -1),
    (dict(kv_head_sets=2), -1),
    (dict(select_tokens=1, rep_kind=1), -2),          # token selection scores the keys themselves
])
def test_init_rejects_bad_config_before_any_hip_call(over, status):
    pk = _pk()
    over = dict(over)
    raw = {k: over.pop(k) for k in ("select_tokens", "rep_kind", "kv_head_sets") if k in over}
    cfg = _cfg(**over)
    for k, v in raw.items():
        setattr(cfg, k, v)                  # the raw field, past make_config's conversions
    h = ctypes.c_void_p(1234)
    st = pk.lib.scale_init_variant(ctypes.byref(cfg.base), ctypes.byref(cfg.variant), None, ctypes.byref(h))
    assert st == status
    assert h.value is None
    if not raw:                             # the default path through scale_init rejects it the same way
        h = ctypes.c_void_p(1234)
        assert pk.lib.scale_init(ctypes.byref(cfg.base), None, ctypes.byref(h)) == status
        assert h.value is None
    assert pk.lib.scale_init(None, None, ctypes.byref(h)) == -1
    assert pk.lib.scale_init(ctypes.byref(_cfg().base), None, None) == -1
    assert pk.lib.scale_init_variant(None, None, None, ctypes.byref(h)) == -1


def test_calls_reject_null_handle():
    pk = _pk()
    lib = pk.lib
    cs = np.array([0, 1], dtype=np.int32)
    assert lib.scale_rep_keys(None, 1, None, 128, 1) == -1
    assert lib.scale_select_cluster(None, 1, 128, 1, cs.ctypes.data, 1, 1, 1, None) == -1
    assert lib.scale_sparse_prefill(None, 1, 1, 1, None, 128, cs.ctypes.data, 1, 1, 1, 1) == -1
    n = ctypes.c_int64()
    assert lib.scale_retrieval_calls(None, ctypes.byref(n)) == -1
    out = np.zeros(4, dtype=np.int32)
    k = ctypes.c_int32()
    assert lib.scale_cluster_subchunks(None, 1, 128, 0, 0.95, 4096, 0, out.ctypes.data, ctypes.byref(k), None) == -1
    assert lib.scale_rep_keys_range(None, 1, None, 0, 128, 1) == -1
    assert lib.scale_select_cluster_tokens(None, 1, 128, 1, None, cs.ctypes.data, 1, 1, 1, None) == -1
    assert lib.scale_fingerprints(None, 1, 1) == -1
    lib.scale_free(None)        # no-op


def test_cluster_span_rule():
    """Band width of scale_cluster_subchunks: the cluster cap in sub-chunks, bounded by the outer
    chunk and the sub-chunk count, minus one."""
    pk = _pk()
    assert pk.cluster_span(4096, 512, 0, 256) == 7
    assert pk.cluster_span(4097, 512, 0, 256) == 8
    assert pk.cluster_span(4096, 512, 4, 256) == 3
    assert pk.cluster_span(10 ** 9, 512, 16, 256) == 15
    assert pk.cluster_span(10 ** 9, 512, 0, 5) == 4
    assert pk.cluster_span(100, 512, 0, 256) == 0


@pytest.mark.parametrize("name,c", [("tiny", 4), ("tiny", 1), ("llama32k", 8), ("llama128k", 8),
                                    ("qwen256k", 4), ("stress1m", 16), ("stress1m", 1)])
def test_host_geometry_matches_oracle(name, c):
    pk = _pk()
    w = gen.WORKLOADS[name]
    cs = gen.cluster_starts(w.n_sub_chunks, c)
    cfg = _cfg(num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
               block_size=w.block_size, sub_chunk=w.sub_chunk, top_k=w.top_k, sink_tokens=w.sink_tokens,
               local_window=w.local_window, max_tokens=w.n_tokens, max_clusters=len(cs) - 1)
    geo = pk.scale_cluster_geometry(cfg, w.n_tokens, cs)
    ref = oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, w.top_k, cs)
    assert geo.shape == (len(ref), 6)
    for row, g in zip(geo, ref):
        assert tuple(int(x) for x in row) == (g.s, g.e, g.lo_blk, g.sink_eff, g.n_cand, g.sel_cnt)
    # token-level selection: candidates and the budget count tokens
    k_tok = w.top_k * w.block_size + 37
    cfg.select_tokens, cfg.top_k = 1, k_tok
    geo = pk.scale_cluster_geometry(cfg, w.n_tokens, cs)
    ref = oracle.geometry(w.n_tokens, w.sub_chunk, w.block_size, w.sink_tokens, w.local_window, k_tok, cs,
                          select_tokens=True)
    for row, g in zip(geo, ref):
        assert g.tokens and tuple(int(x) for x in row) == (g.s, g.e, g.lo_blk, g.sink_eff, g.n_cand, g.sel_cnt)


def test_geometry_short_last_subchunk_and_odd_clusters():
    pk = _pk()
    n = 64 * 37          # 2368 tokens: 9 full sub-chunks of 256 and one of 64
    cs = np.array([0, 3, 4, 9, 10], dtype=np.int32)
    cfg = _cfg(num_q_heads=4, num_kv_heads=1, head_dim=64, block_size=64, sub_chunk=256, top_k=4,
               sink_tokens=64, local_window=300, max_tokens=n, max_clusters=4)
    geo = pk.scale_cluster_geometry(cfg, n, cs)
    ref = oracle.geometry(n, 256, 64, 64, 300, 4, cs)
    for row, g in zip(geo, ref):
        assert tuple(int(x) for x in row) == (g.s, g.e, g.lo_blk, g.sink_eff, g.n_cand, g.sel_cnt)
    assert geo[-1][1] == n and geo[-1][0] == 9 * 256


def test_geometry_of_a_suffix_of_clusters():
    """Incremental prefill: clusters covering only the last sub-chunks have the geometry those
    clusters have in the whole partition."""
    pk = _pk()
    cfg = _cfg(num_q_heads=4, num_kv_heads=1, head_dim=64, block_size=64, sub_chunk=256, top_k=4,
               sink_tokens=64, local_window=300, max_tokens=8192, max_clusters=8)
    full = np.array([0, 3, 4, 9, 12, 16, 20, 32], dtype=np.int32)
    g_full = pk.scale_cluster_geometry(cfg, 8192, full)
    for cut in (1, 3, 5):
        g = pk.scale_cluster_geometry(cfg, 8192, full[cut:])
        assert np.array_equal(g, g_full[cut:])
        ref = oracle.geometry(8192, 256, 64, 64, 300, 4, full[cut:])
        assert [tuple(int(x) for x in r) for r in g] == [(r.s, r.e, r.lo_blk, r.sink_eff, r.n_cand, r.sel_cnt)
                                                       for r in ref]


@pytest.mark.parametrize("cs,n,status", [
    ([0, 2, 2, 8], 2048, -1),        # not strictly increasing
    ([-1, 8], 2048, -1),             # starts below 0
    ([0, 7], 2048, -1),              # does not end at M
    ([0, 9], 2048, -1),
    ([0, 8], 2000, -2),              # n_tokens not a multiple of the block size
    ([0, 4, 8], 4096 + 64, -1),      # M changes with n_tokens
])
def test_geometry_rejects_malformed_clusters(cs, n, status):
    pk = _pk()
    cfg = _cfg(num_q_heads=4, num_kv_heads=1, head_dim=64, block_size=64, sub_chunk=256, top_k=4,
               sink_tokens=64, local_window=256, max_tokens=8192, max_clusters=8)
    arr = np.asarray(cs, dtype=np.int32)
    geo = np.zeros((len(cs), 6), dtype=np.int32)
    st = pk.lib.scale_cluster_geometry(ctypes.byref(cfg.base), None, n, arr.ctypes.data, len(cs) - 1,
                                       geo.ctypes.data)
    assert st == status


def test_geometry_capacity():
    pk = _pk()
    cfg = _cfg(num_q_heads=4, num_kv_heads=1, head_dim=64, block_size=64, sub_chunk=256, top_k=4,
               sink_tokens=64, local_window=256, max_tokens=2048, max_clusters=2)
    geo = np.zeros((8, 6), dtype=np.int32)
    cs = gen.cluster_starts(8, 1)
    assert pk.lib.scale_cluster_geometry(ctypes.byref(cfg.base), None, 2048, cs.ctypes.data, 8, geo.ctypes.data) == -4
    cs = gen.cluster_starts(16, 8)
    assert pk.lib.scale_cluster_geometry(ctypes.byref(cfg.base), None, 4096, cs.ctypes.data, 2, geo.ctypes.data) == -4


def test_c_client_of_the_header(tmp_path):
    """include/scale.h is plain C: a C99 program (tests/c/abi_host.c) compiles against it with
    warnings as errors, links against libscale.so and runs the host-only calls."""
    import shutil
    import subprocess

    if shutil.which("gcc") is None:
        pytest.skip("gcc is not available")
    pk = _pk()
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    lib = pk.build.LIB_PATH
    exe = tmp_path / "abi_host"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(root, "include"),
           os.path.join(root, "tests", "c", "abi_host.c"), lib, f"-Wl,-rpath,{os.path.dirname(lib)}",
           "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0, run.stdout + run.stderr
    assert run.stdout.count("ok ") == 5
