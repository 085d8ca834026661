"""Planted mistakes in the oracle must fail a pin (CPU only).

Each mutant below is one plausible slip in `oracle/scr.py` -- a dropped or shifted key group, a
wrong bound, a transposed index, a wrong softmax domain or divisor, an off-by-one margin. The
test copies the oracle, the input generator and the CPU pin files into a temporary directory,
plants the mistake in the copy, and runs the pins that cover that part of the oracle in a child
pytest: at least one of them must fail. An unmutated copy run the same way must pass, so a
failure is the mutant's and not the harness's. The planted mistakes live only in the temporary
copies; the oracle itself is never modified.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "scr.py")

PINS = "tests/test_oracle_pins.py"
VARIANTS = "tests/test_oracle_variants.py"
TOKENS = "tests/test_oracle_tokens.py"
CLUSTERING = "tests/test_oracle_clustering.py"

# (name, text in oracle/scr.py (exactly one occurrence), replacement, pin files that must catch it)
MUTANTS = [
    # block-level path: geometry, representative keys, fingerprint, logits, soft-voting, top-k, attention
    ("head_map_strided", "        g = (h * num_kv_heads) // Hq\n        x[h] = score_scale * (k_rep_cand",
     "        g = h % num_kv_heads\n        x[h] = score_scale * (k_rep_cand", [PINS]),
    ("sink_not_clipped", "sink_eff = min(sink_blk, lo_blk)", "sink_eff = sink_blk", [PINS]),
    ("window_fixed_W", "        lo = max(0, min(s, e - W))\n", "        lo = max(0, e - W)\n", [PINS]),
    ("window_rounded_up", "lo_blk = lo // B", "lo_blk = -(-lo // B)", [PINS]),
    ("candidates_into_window", "n_cand = max(0, lo_blk - sink_blk) * (B if",
     "n_cand = max(0, lo_blk - sink_blk + 1) * (B if", [PINS]),
    ("softmax_over_all_blocks", "            sc = soft_vote(x)\n",
     "            sc = soft_vote(block_logits(v, k_rep[0:g.lo_blk], Hkv, score_scale))[g.sink_blk:] "
     "if not select_tokens and rep_kind == 'mean' else soft_vote(x)\n", [PINS]),
    ("cluster_mean_query", "v = anchor_fingerprint(q, g.s, g.anchor_end)", "v = anchor_fingerprint(q, g.s, g.e)",
     [PINS]),
    ("ties_highest_index", "order = np.lexsort((idx, -np.asarray(scores)))",
     "order = np.lexsort((-idx, -np.asarray(scores)))", [PINS]),
    ("selection_unsorted", "sel = np.sort(idx[order[:cnt]])", "sel = idx[order[:cnt]]", [PINS]),
    ("margin_off_by_one", "float(scores[order[cnt - 1]] - scores[order[cnt]])",
     "float(scores[order[cnt - 2]] - scores[order[cnt - 1]])", [PINS]),
    ("causal_strict", "visible[:, n_fixed:] = pos[None, n_fixed:] <= rows[:, None]",
     "visible[:, n_fixed:] = pos[None, n_fixed:] < rows[:, None]", [PINS]),
    ("rep_key_first_token", "        out[i] = keys.sum(axis=1) / n_valid\n", "        out[i] = keys[:, 0, :]\n", [PINS]),
    ("fingerprint_sum", "    return rows.sum(axis=0) / (anchor_end - s)\n", "    return rows.sum(axis=0)\n", [PINS]),
    ("attention_values_from_keys", "logical_rows(v_pages, block_table, pos, B),",
     "logical_rows(k_pages, block_table, pos, B),", [PINS]),
    ("attention_head_map_strided", "        g = (int(h) * Hkv) // Hq\n        Kg, Vg, visible = keys_of(g)",
     "        g = int(h) % Hkv\n        Kg, Vg, visible = keys_of(g)", [PINS]),
    ("attention_drops_sink", "fixed = np.concatenate([np.arange(geo.sink_eff * B), selected_positions",
     "fixed = np.concatenate([np.arange(0), selected_positions", [PINS]),
    ("attention_unnormalised", "out[:, hi, :] = (w @ Vg) / w.sum(axis=1, keepdims=True)",
     "out[:, hi, :] = (w @ Vg) / w.shape[1]", [PINS]),
    ("softmax_not_per_head", "p = ex / ex.sum(axis=1, keepdims=True)", "p = ex / ex.sum()", [PINS]),
    ("attention_scale_1_over_d", "scale = 1.0 / math.sqrt(d) if", "scale = 1.0 / d if", [PINS]),
    ("partial_block_divisor", "        out[i] = keys.sum(axis=1) / n_valid",
     "        out[i] = keys.sum(axis=1) / block_size", [PINS]),
    ("sel_cnt_plus_one", "n_cand, min(k, n_cand),", "n_cand, min(k + 1, n_cand),", [PINS]),
    ("logit_scale_dropped", "x[h] = score_scale * (k_rep_cand[:, g, :] @ v[h])", "x[h] = (k_rep_cand[:, g, :] @ v[h])",
     [PINS]),
    # selection variants: bound representative keys, per-KV-head sets
    ("bounds_min", "np.maximum(mn_cand[:, g, :] * v[h], mx_cand[:, g, :] * v[h])",
     "np.minimum(mn_cand[:, g, :] * v[h], mx_cand[:, g, :] * v[h])", [VARIANTS]),
    ("bounds_max_only", "np.maximum(mn_cand[:, g, :] * v[h], mx_cand[:, g, :] * v[h]).sum(axis=1)",
     "(mx_cand[:, g, :] * v[h]).sum(axis=1)", [VARIANTS]),
    ("bounds_mean_as_min", "mn[i] = keys.min(axis=1)", "mn[i] = keys.mean(axis=1)", [VARIANTS]),
    ("groups_strided", "soft_vote(x[g * G:(g + 1) * G])", "soft_vote(x[g::num_kv_heads])", [VARIANTS]),
    ("every_kv_head_set_0", "return [a[g] for g in range(num_kv_heads)]", "return [a[0] for g in range(num_kv_heads)]",
     [VARIANTS]),
    ("kv_sets_from_shared_vote", "sc = soft_vote_groups(x, Hkv) if x.shape[1]",
     "sc = np.stack([soft_vote(x)] * Hkv) if x.shape[1]", [VARIANTS]),
    # token-level selection
    ("token_first_off_by_one", "            first = g.sink_blk * B\n", "            first = g.sink_blk * B + 1\n",
     [TOKENS]),
    ("token_block_keys", "np.arange(g.sink_blk * B, g.sink_blk * B + g.n_cand), B)",
     "np.arange(g.sink_blk * B, g.sink_blk * B + g.n_cand) // B * B, B)", [TOKENS]),
    ("token_count_per_block", "(B if select_tokens else 1)", "(B - 1 if select_tokens else 1)", [TOKENS]),
    ("token_positions_shifted", "if geo.tokens:\n        return sel\n", "if geo.tokens:\n        return sel + 1\n",
     [TOKENS]),
    # anchor clustering (Algorithm 1, Eq. 8) and the overlap ratio (Eq. 7)
    ("clustering_predecessor", "float(vt[a] @ vt[j]) >= theta", "float(vt[j - 1] @ vt[j]) >= theta", [CLUSTERING]),
    ("clustering_strict", "float(vt[a] @ vt[j]) >= theta and", "float(vt[a] @ vt[j]) > theta and", [CLUSTERING]),
    ("clustering_cap_off_by_one", "size * sub_chunk < l_max", "size * sub_chunk <= l_max", [CLUSTERING]),
    ("clustering_short_divisor", "sum(axis=0) / rows.shape[0]", "sum(axis=0) / sub_chunk", [CLUSTERING]),
    ("clustering_outer_off_by_one", "(a // outer_subchunks + 1) * outer_subchunks)",
     "(a // outer_subchunks + 1) * outer_subchunks + 1)", [CLUSTERING]),
    ("clustering_flatten_transposed", "rows.reshape(rows.shape[0], -1).sum(axis=0)",
     "rows.transpose(0, 2, 1).reshape(rows.shape[0], -1).sum(axis=0)", [CLUSTERING]),
    ("overlap_over_union", "len(i_c & union) / len(i_c)", "len(i_c & union) / len(union)", [CLUSTERING]),
]


def _copy_tree(dst):
    """The oracle, the generator (with its built helper) and the CPU test files, into dst."""
    ignore = shutil.ignore_patterns("__pycache__", "*.pyc", "c")
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(dst, "oracle"), ignore=ignore)
    shutil.copytree(os.path.join(ROOT, "gen"), os.path.join(dst, "gen"), ignore=ignore)
    shutil.copytree(os.path.join(ROOT, "tests"), os.path.join(dst, "tests"), ignore=ignore)
    shutil.copy(os.path.join(ROOT, "pytest.ini"), dst)


def _run_pins(dst, files):
    env = {k: v for k, v in os.environ.items() if k != "PYTHONPATH"}
    env["OMP_NUM_THREADS"] = "1"
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider", *files]
    r = subprocess.run(cmd, cwd=dst, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, (r.stdout + r.stderr).strip().splitlines()[-1:] or [""]


def test_mutants_fail_a_pin(tmp_path):
    src = open(ORACLE_SRC).read()
    for name, old, _new, _files in MUTANTS:
        assert src.count(old) == 1, f"mutant {name}: its text occurs {src.count(old)} times in the oracle"

    def one(item):
        i, (name, old, new, files) = item
        dst = os.path.join(tmp_path, f"m{i:02d}")
        _copy_tree(dst)
        if name != "control":
            with open(os.path.join(dst, "oracle", "scr.py"), "w") as f:
                f.write(src.replace(old, new))
        return name, _run_pins(dst, files)

    control = ("control", "", "", [PINS, VARIANTS, TOKENS, CLUSTERING])
    jobs = list(enumerate([control] + MUTANTS))
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as pool:
        results = dict(pool.map(one, jobs))
    rc, tail = results.pop("control")
    assert rc == 0, f"the unmutated copy fails its pins: {tail}"
    survivors = [f"{name}: {tail}" for name, (rc, tail) in results.items() if rc != 1]
    assert not survivors, "mutants that no pin catches (or that broke the harness):\n" + "\n".join(survivors)
