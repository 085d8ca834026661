"""Pins of the oracle's anchor-based clustering (paper Sec. 5.1.1-5.1.2, Algorithm 1, Eq. 8) and of
the sub-chunk fingerprints it compares (Eq. 6), checked against brute force, closed forms and
the generator's ground-truth topic runs rather than against the oracle's own formulas."""
import itertools
import math

import numpy as np
import pytest

import gen
import oracle


def _bits(x):
    """float array -> bf16 bit patterns (values chosen to be exact in bf16)."""
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def test_fingerprint_of_constant_rows_is_the_row():
    rng = np.random.default_rng(1)
    row = rng.integers(-8, 8, size=(3, 4)).astype(np.float64) / 4.0      # exact in bf16
    q = np.broadcast_to(_bits(row), (10, 3, 4)).copy()
    fp = oracle.subchunk_fingerprints(q, 10, 4)                           # sub-chunks of 4, 4, 2 rows
    assert fp.shape == (3, 12)
    assert np.array_equal(fp, np.broadcast_to(row.reshape(-1), (3, 12)))


def test_fingerprint_short_last_subchunk_divides_by_its_own_rows():
    q = np.zeros((6, 1, 2), dtype=np.float64)
    q[4:, 0, 0] = [1.0, 3.0]                                              # last sub-chunk: rows 4, 5
    fp = oracle.subchunk_fingerprints(_bits(q), 6, 4)
    assert fp[1, 0] == 2.0 and fp[0, 0] == 0.0
    # head-major flattening: the per-head slices are the per-head means of the anchor helper
    w = gen.WORKLOADS["tiny"]
    d = gen.make_layer(w)
    fp = oracle.subchunk_fingerprints(d["q"], w.n_tokens, w.sub_chunk)
    for i in (0, 3, 7):
        s = i * w.sub_chunk
        assert np.array_equal(fp[i], oracle.anchor_fingerprint(d["q"], s, s + w.sub_chunk).reshape(-1))


def _partitions(m):
    """Every split of [0, m) into consecutive non-empty ranges, as cluster_start lists."""
    for cuts in itertools.product((0, 1), repeat=m - 1):
        yield [0] + [i + 1 for i, c in enumerate(cuts) if c] + [m]


def _satisfies_definition(starts, vt, theta, L, l_max):
    """The properties that define Algorithm 1's output: every member is within theta of its
    cluster's first sub-chunk, no cluster exceeds the cap, and every cluster that is not the last
    one was closed by the next sub-chunk failing the similarity test or by the cap."""
    cap = math.ceil(l_max / L)
    for a, e in zip(starts[:-1], starts[1:]):
        if e - a > cap:
            return False
        if any(not (vt[a] @ vt[j] >= theta) for j in range(a + 1, e)):
            return False
        if e < len(vt) and (e - a) < cap and vt[a] @ vt[e] >= theta:
            return False                                                   # could have admitted e
    return True


@pytest.mark.parametrize("seed", range(12))
def test_clustering_is_the_unique_partition_of_its_definition(seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 8))
    # directions clustered around a few centres so that every theta below splits somewhere
    centres = rng.normal(size=(3, 6))
    vt = oracle.normalized(centres[rng.integers(0, 3, size=m)] + 0.3 * rng.normal(size=(m, 6)))
    theta = float(rng.uniform(0.5, 0.99))
    L, l_max = 512, int(rng.choice([512, 1000, 1536, 4096]))
    valid = [p for p in _partitions(m) if _satisfies_definition(p, vt, theta, L, l_max)]
    assert len(valid) == 1
    assert oracle.anchor_clustering(vt, theta, L, l_max).tolist() == valid[0]


def test_clustering_extremes():
    rng = np.random.default_rng(3)
    vt = oracle.normalized(rng.normal(size=(21, 5)))
    # theta above 1: nothing is ever admitted
    assert oracle.anchor_clustering(vt, 1.5, 512, 4096).tolist() == list(range(22))
    # theta -1: the cap alone decides, which is the fixed-size partition of ceil(L_max / L)
    for l_max in (512, 1024, 1000, 4096, 4097):
        c = math.ceil(l_max / 512)
        assert np.array_equal(oracle.anchor_clustering(vt, -1.0, 512, l_max), gen.cluster_starts(21, c))
    # a cap at or below one sub-chunk gives singletons whatever the similarity
    assert oracle.anchor_clustering(vt, -1.0, 512, 300).tolist() == list(range(22))


def test_clustering_follows_the_anchor_not_the_predecessor():
    """Fingerprints that turn by a fixed angle per sub-chunk: every consecutive pair passes theta,
    but the cosine to the anchor decays as cos(k alpha), so each cluster holds
    floor(arccos(theta) / alpha) + 1 sub-chunks (a predecessor rule would keep one cluster)."""
    alpha = math.acos(0.995)
    theta = 0.95
    ang = alpha * np.arange(40)
    vt = np.stack([np.cos(ang), np.sin(ang)], axis=1)
    k = int(math.floor(math.acos(theta) / alpha)) + 1
    starts = oracle.anchor_clustering(vt, theta, 512, 10 ** 9)
    sizes = np.diff(starts)
    assert np.all(sizes[:-1] == k) and sizes[-1] <= k
    assert all(vt[i] @ vt[i + 1] >= theta for i in range(39))


def test_clustering_recovers_the_generators_topic_runs():
    """At a threshold between the cross-topic and the same-topic cosines, the clusters are the
    generator's topic runs (consecutive sub-chunks of one topic), cut by the cap."""
    w = gen.WORKLOADS["tiny"].with_(n_tokens=16384, n_topics=16, run_lo=1, run_hi=6, seed=11,
                                    q_scale_lo=2.0, q_scale_hi=5.0)
    d = gen.make_layer(w)
    vt = oracle.normalized(oracle.subchunk_fingerprints(d["q"], w.n_tokens, w.sub_chunk))
    topic = d["qtopic"]
    same = np.equal.outer(topic, topic)
    cos = vt @ vt.T
    lo_same, hi_cross = cos[same].min(), cos[~same].max()
    theta = 0.5 * (lo_same + hi_cross)
    assert hi_cross < theta < lo_same                                     # the data has the gap
    l_max = 4 * w.sub_chunk
    expected = [0]
    a = 0
    for j in range(1, len(topic) + 1):
        if j == len(topic) or topic[j] != topic[a] or j - a == 4:
            expected.append(j)
            a = j
    assert oracle.anchor_clustering(vt, theta, w.sub_chunk, l_max).tolist() == expected


def test_clustering_restarts_at_outer_chunk_boundaries():
    vt = oracle.normalized(np.ones((20, 3)))                               # everything identical
    assert oracle.anchor_clustering(vt, 0.9, 512, 4096).tolist() == [0, 8, 16, 20]
    assert oracle.anchor_clustering(vt, 0.9, 512, 4096, outer_subchunks=6).tolist() == [0, 6, 12, 18, 20]
    assert oracle.anchor_clustering(vt, 0.9, 512, 2048, outer_subchunks=6).tolist() == [0, 4, 6, 10, 12, 16, 18, 20]


def test_zero_fingerprint_never_joins_nor_admits():
    v = np.ones((5, 2))
    v[2] = 0.0
    vt = oracle.normalized(v)
    assert oracle.anchor_clustering(vt, 0.5, 512, 4096).tolist() == [0, 2, 3, 5]


def test_admission_at_exact_equality():
    """Eq. 8 admits at cos = theta: unit vectors whose inner products are exact in fp64."""
    vt = np.array([[1.0, 0.0], [0.6, 0.8], [0.6, -0.8], [0.0, 1.0]])
    assert oracle.anchor_clustering(vt, 0.6, 512, 4096).tolist() == [0, 3, 4]


def test_generator_strength_draws_leave_topics_unchanged():
    """The per-run topic strength comes from a stream of its own: topics and run lengths do not
    move when the strength range changes, runs share one strength, and it lies in the range."""
    w = gen.WORKLOADS["tiny"].with_(n_tokens=16384, run_lo=1, run_hi=5)
    t0, s0 = gen.query_runs(w)
    t1, s1 = gen.query_runs(w.with_(q_scale_lo=1.0, q_scale_hi=7.0))
    assert np.array_equal(t0, t1) and np.all(s0 == 2.0)
    assert np.all((s1 >= 1.0) & (s1 <= 7.0)) and len(np.unique(s1)) > 1
    # continuous strengths differ between runs, so each constant-strength segment is one run
    cut = np.concatenate([[0], np.flatnonzero(np.diff(s1)) + 1, [len(s1)]])
    lengths = np.diff(cut)
    assert np.all((lengths[:-1] >= 1) & (lengths[:-1] <= 5)) and 1 <= lengths[-1] <= 5
    assert all(len(set(t1[a:b].tolist())) == 1 for a, b in zip(cut[:-1], cut[1:]))
    assert np.array_equal(gen.q_rows(w, 0, 300), gen.q_rows(w.with_(q_scale_lo=2.0, q_scale_hi=2.0), 0, 300))


def test_clustering_from_a_first_subchunk():
    """Incremental clustering of the outer chunks still to run equals the tail of the whole pass
    whenever the first sub-chunk starts an outer chunk."""
    rng = np.random.default_rng(5)
    vt = oracle.normalized(np.repeat(rng.normal(size=(6, 4)), 5, axis=0) + 0.05 * rng.normal(size=(30, 4)))
    full = oracle.anchor_clustering(vt, 0.9, 512, 4096, outer_subchunks=10)
    for first in (10, 20):
        tail = oracle.anchor_clustering(vt, 0.9, 512, 4096, outer_subchunks=10, first=first)
        assert tail[0] == first and tail[-1] == 30
        assert np.array_equal(tail, full[np.searchsorted(full, first):])


def test_topk_overlap_by_hand():
    cs = [0, 3, 4]
    cluster_sets = [[1, 2, 5, 9], [2]]
    sub = [[1, 2], [7, 8], [5, 6], [3]]          # sub-chunk 3 alone forms cluster 1
    rho = oracle.topk_overlap(cluster_sets, sub, cs)
    assert rho[0] == 0.75 and rho[1] == 0.0
    assert math.isnan(oracle.topk_overlap([[]], [[1]], [0, 1])[0])
