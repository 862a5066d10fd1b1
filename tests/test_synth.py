"""The seeded input generators: determinism, thread-count independence and the
shape statistics of the stand-in workloads (CPU only)."""
import hashlib
import os
import subprocess
import sys

import numpy as np
import pytest

from paper_1909_01315_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# recorded outputs of this generator (counter-based SplitMix64; independent of numpy)
C1_GRAPH_SHA = "27d193728f57282166ef080ad5da0fae7c8cbfe45b1994a7e3401c984cc2132f"
C1_X_SHA = "839b8bae612b7de580a06af65d39960b33b8cd2a77935228b3ddeb2f5848ed34"


def sha(*arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def is_sorted_by_dst_src(g):
    key = g.dst.astype(np.int64) * (g.n_src + 1) + g.src
    return bool(np.all(np.diff(key) >= 0))


def test_c1_shape_and_hash():
    g = synth.graph_c1()
    assert (g.n_src, g.n_dst, g.n_edges) == (1024, 1024, 17408)
    assert is_sorted_by_dst_src(g)
    loops = np.zeros(1024, dtype=np.int64)
    np.add.at(loops, g.src[g.src == g.dst], 1)
    assert np.all(loops >= 1), "every node carries its appended self-loop"
    pairs = g.src.astype(np.int64) * 1024 + g.dst
    assert np.unique(pairs).size < g.n_edges, "duplicate edges are kept"
    assert sha(g.src, g.dst) == C1_GRAPH_SHA
    x = synth.normal(synth.feat_seed(1), "X", (1024, 16))
    assert sha(x) == C1_X_SHA


def test_same_seed_same_arrays():
    a = synth.normal(7, "t", (1001, 3))
    b = synth.normal(7, "t", (1001, 3))
    c = synth.normal(7, "u", (1001, 3))
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    u = synth.uniform(7, "w", (5000,), 0.0, 1.0)
    assert u.min() >= 0.0 and u.max() < 1.0 and abs(u.mean() - 0.5) < 0.02
    n = synth.normal(7, "n", (200000,))
    assert abs(n.mean()) < 0.01 and abs(n.std() - 1.0) < 0.01


def test_thread_count_does_not_change_output():
    code = ("from paper_1909_01315_amd import synth; import hashlib;"
            "g=synth.rmat_graph(3, 12, 4000, 30000);"
            "x=synth.normal(3,'x',(30001,));"
            "print(hashlib.sha256(g.src.tobytes()+g.dst.tobytes()+x.tobytes()).hexdigest())")
    outs = []
    for t in ("1", "3"):
        env = dict(os.environ, OMP_NUM_THREADS=t)
        outs.append(subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, check=True,
                                   capture_output=True, text=True).stdout.strip())
    assert outs[0] == outs[1]


def test_c2_chung_lu_gcn_weights():
    g = synth.graph_c2()
    assert g.n_src == g.n_dst == 20000
    assert 100000 < g.n_edges < 110000
    assert is_sorted_by_dst_src(g)
    pairs = g.src.astype(np.int64) * 20000 + g.dst
    assert np.unique(pairs).size == g.n_edges, "no duplicates"
    assert int(np.sum(g.src == g.dst)) == 20000, "exactly the added self-loops"
    outdeg = np.bincount(g.src, minlength=20000)
    indeg = np.bincount(g.dst, minlength=20000)
    w = g.extra["gcn_w"][:, 0]
    np.testing.assert_allclose(w, 1.0 / np.sqrt(outdeg[g.src] * indeg[g.dst]), rtol=1e-7)
    assert indeg.max() > 200, "power-law hubs"


def test_c5_relational_encoding():
    g = synth.graph_c5()
    n, r = synth.C5_N, synth.C5_R
    assert (g.n_src, g.n_dst, g.n_edges) == (n * r, n, synth.C5_E)
    et = g.extra["etype"]
    assert np.array_equal(g.src, et * n + g.extra["orig_src"])
    assert np.all(np.diff(g.dst) >= 0)
    p0 = np.mean(et == 0)
    assert 0.28 < p0 < 0.32, "Zipf(1.2) over 50 relations puts about 30% on relation 0"
    # per-(dst, relation) normalisation
    key = g.dst.astype(np.int64) * r + et
    _, inv, cnt = np.unique(key, return_inverse=True, return_counts=True)
    np.testing.assert_allclose(g.extra["norm"][:, 0], 1.0 / cnt[inv], rtol=1e-7)


def test_c4_rmat_statistics():
    g = synth.graph_c4()
    assert (g.n_src, g.n_edges) == (synth.C4_N, synth.C4_E)
    assert is_sorted_by_dst_src(g)
    st = synth.degree_stats(g)
    assert 0.40 < st["empty"] / g.n_dst < 0.44, "about 42% of destinations have no in-edge"
    assert st["median"] == 1.0
    assert 60000 < st["max"] < 120000
    key = g.dst.astype(np.int64) * g.n_src + g.src
    assert np.all(np.diff(key) > 0), "deduplicated and strictly sorted"


def test_bf16_inputs_round_to_nearest_even():
    x = np.array([1.0, 1.00390625, 1.005859375, -2.5], dtype=np.float32)  # 1 + 2^-8 is a tie
    b = synth.to_bf16_bits(x)
    assert list(b) == [0x3F80, 0x3F80, 0x3F81, 0xC020]


def test_shuffle_within_rows_keeps_each_rows_edges():
    g = synth.uniform_graph(5, 300, 120, 5000)
    r = synth.shuffle_within_rows(g, 17)
    r2 = synth.shuffle_within_rows(g, 17)
    assert np.array_equal(r.src, r2.src) and np.array_equal(r.dst, r2.dst)  # seeded
    assert np.array_equal(r.dst, g.dst)  # still grouped by destination, rows in place
    assert not np.array_equal(r.src, g.src)
    ptr = np.concatenate([[0], np.cumsum(np.bincount(g.dst, minlength=g.n_dst))])
    unsorted = 0
    for v in range(g.n_dst):
        a, b = r.src[ptr[v]:ptr[v + 1]], g.src[ptr[v]:ptr[v + 1]]
        assert np.array_equal(np.sort(a), b)
        unsorted += int(not np.array_equal(a, b))
    assert unsorted > g.n_dst // 2
