"""Seeded synthetic inputs shaped like the paper's workloads.

This module is the only code shared by the CPU oracle's tests and the GPU
path's tests and benchmark.  It draws graphs and dense tensors; it holds none
of the message-passing arithmetic.  The heavy lifting is in ``synth.c``
(counter-based SplitMix64, OpenMP), so every array depends only on
(seed, stream, index) and is identical for any thread count and machine.

Edge ids: every generated graph lists its edges sorted by (destination,
source); the edge id is the position in that list.

Workloads (the paper's datasets are not available; these stand in for them):

* ``c1`` tiny uniform multigraph: N=1,024, 16,384 uniform (src, dst) pairs
  plus one self-loop per node (E=17,408).
* ``c2`` Chung-Lu power law (exponent 2.5), N=20,000, 90,000 draws, self-loops
  and duplicates dropped, one self-loop per node added; GCN edge weights
  1/sqrt(outdeg(src) * indeg(dst)) with degrees counted after the self-loops.
* ``c3`` R-MAT (0.57, 0.19, 0.19, 0.05) at scale 18 on N=232,965 nodes (the
  node count of the paper's Reddit table row), deduplicated, E=114,600,000.
* ``c4`` R-MAT at scale 22 on N=2,449,029 nodes with E=61,859,140 (the node and
  edge counts of the paper's ogbn-products table row), deduplicated.
* ``c5`` relational multigraph: N=100,000, E=2,000,000 uniform edges, edge
  types from a Zipf(1.2) law truncated to 50 relations, seen as a bipartite
  graph whose source id is ``etype * N + src`` (num_src = 50 N), with the
  per-relation normalisation 1/|{e': dst_e' = dst_e, etype_e' = etype_e}|.
"""
from __future__ import annotations

import ctypes
import os
import zlib
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

SEED_BASE = 190901315

_I64 = ctypes.c_int64
_U64 = ctypes.c_uint64
_P = ctypes.c_void_p


def build(verbose: bool = False) -> str:
    """Compile synth.c into libsynth.so next to it (gcc, OpenMP)."""
    import subprocess

    cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-Wall", "-o", _LIB_PATH,
           os.path.join(_HERE, "synth.c"), "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.synth_fill_normal_f32.argtypes = [_U64, _U64, _I64, _P]
    lib.synth_fill_uniform_f32.argtypes = [_U64, _U64, _I64, ctypes.c_float, ctypes.c_float, _P]
    lib.synth_f32_to_bf16.argtypes = [_I64, _P, _P]
    lib.synth_permutation.argtypes = [_U64, _U64, _I64, _P]
    lib.synth_sort_coo.argtypes = [_I64, _P, _P, _I64, _I64]
    lib.synth_sort_coo.restype = ctypes.c_int
    lib.synth_uniform_edges.argtypes = [_U64, _U64, _I64, _I64, _I64, _P, _P]
    lib.synth_zipf.argtypes = [_U64, _U64, _I64, ctypes.c_int32, ctypes.c_double, _P]
    lib.synth_chung_lu.argtypes = [_U64, _I64, _I64, ctypes.c_double, _P, _P]
    lib.synth_chung_lu.restype = _I64
    lib.synth_rmat.argtypes = [_U64, ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                               _I64, _I64, _P, _P]
    lib.synth_rmat.restype = _I64
    lib.synth_count_dst_type.argtypes = [_I64, _I64, ctypes.c_int32, _P, _P, _P]
    lib.synth_bincount.argtypes = [_I64, _P, _I64, _P]
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def stream_id(name: str) -> int:
    """Stable stream number for a named tensor."""
    return zlib.crc32(name.encode()) & 0xFFFFFFFF


# ---------------------------------------------------------------------------
# dense tensors


def normal(seed: int, name: str, shape) -> np.ndarray:
    """float32 array of i.i.d. N(0, 1) draws for tensor ``name``."""
    out = np.empty(shape, dtype=np.float32)
    _load().synth_fill_normal_f32(seed, stream_id(name), out.size, _ptr(out))
    return out


def uniform(seed: int, name: str, shape, lo: float = 0.0, hi: float = 1.0) -> np.ndarray:
    """float32 array of i.i.d. U[lo, hi) draws on a 2^-24 grid."""
    out = np.empty(shape, dtype=np.float32)
    _load().synth_fill_uniform_f32(seed, stream_id(name), out.size, lo, hi, _ptr(out))
    return out


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even bf16 bit patterns (uint16) of a float32 array."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().synth_f32_to_bf16(x.size, _ptr(x), _ptr(out))
    return out


def permutation(seed: int, name: str, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    _load().synth_permutation(seed, stream_id(name), n, _ptr(out))
    return out


def bincount(idx: np.ndarray, n: int) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    out = np.empty(n, dtype=np.int64)
    _load().synth_bincount(idx.size, _ptr(idx), n, _ptr(out))
    return out


# ---------------------------------------------------------------------------
# graphs


@dataclass
class Graph:
    """A directed multigraph as an edge list; edge id = position."""

    name: str
    n_src: int
    n_dst: int
    src: np.ndarray  # int32 (E,)
    dst: np.ndarray  # int32 (E,)
    extra: dict = field(default_factory=dict)

    @property
    def n_edges(self) -> int:
        return int(self.src.shape[0])


def sort_coo(src: np.ndarray, dst: np.ndarray, n_src: int, n_dst: int):
    """Return (src, dst) sorted by (dst, src)."""
    src = np.ascontiguousarray(src, dtype=np.int32).copy()
    dst = np.ascontiguousarray(dst, dtype=np.int32).copy()
    rc = _load().synth_sort_coo(src.size, _ptr(src), _ptr(dst), max(n_src, 1), max(n_dst, 1))
    if rc != 0:
        raise RuntimeError(f"synth_sort_coo failed ({rc})")
    return src, dst


def uniform_graph(seed: int, n_src: int, n_dst: int, n_edges: int, self_loops: bool = False,
                  name: str = "uniform") -> Graph:
    """Uniform random multigraph (duplicates and self-loops kept), optionally plus one self-loop per node."""
    lib = _load()
    src = np.empty(n_edges, dtype=np.int32)
    dst = np.empty(n_edges, dtype=np.int32)
    if n_edges:
        lib.synth_uniform_edges(seed, stream_id("edges"), n_edges, n_src, n_dst, _ptr(src), _ptr(dst))
    if self_loops:
        assert n_src == n_dst
        loop = np.arange(n_src, dtype=np.int32)
        src = np.concatenate([src, loop])
        dst = np.concatenate([dst, loop])
    src, dst = sort_coo(src, dst, n_src, n_dst)
    return Graph(name, n_src, n_dst, src, dst)


def knn_graph(seed: int, n: int, k: int, name: str = "knn") -> Graph:
    """Constant in-degree graph (a k-nearest-neighbour graph's shape): every
    node receives k edges from uniform random sources (Appendix E's
    sensitivity study contrasts such graphs with power-law ones)."""
    lib = _load()
    src = np.empty(n * k, dtype=np.int32)
    dummy = np.empty(n * k, dtype=np.int32)
    if n * k:
        lib.synth_uniform_edges(seed, stream_id("knn"), n * k, n, n, _ptr(src), _ptr(dummy))
    dst = np.repeat(np.arange(n, dtype=np.int32), k)
    src, dst = sort_coo(src, dst, n, n)
    return Graph(name, n, n, src, dst)


def graph_c1() -> Graph:
    g = uniform_graph(SEED_BASE + 1, 1024, 1024, 16384, self_loops=True, name="c1")
    return g


def graph_c2() -> Graph:
    n, draws = 20000, 90000
    src = np.empty(draws + n, dtype=np.int32)
    dst = np.empty(draws + n, dtype=np.int32)
    e = _load().synth_chung_lu(SEED_BASE + 2, n, draws, 2.5, _ptr(src), _ptr(dst))
    g = Graph("c2", n, n, src[:e].copy(), dst[:e].copy())
    outdeg = bincount(g.src, n).astype(np.float64)
    indeg = bincount(g.dst, n).astype(np.float64)
    g.extra["gcn_w"] = (1.0 / np.sqrt(outdeg[g.src] * indeg[g.dst])).astype(np.float32).reshape(-1, 1)
    return g


def rmat_graph(seed: int, scale: int, n: int, n_edges: int, name: str = "rmat",
               abc=(0.57, 0.19, 0.19)) -> Graph:
    src = np.empty(n_edges, dtype=np.int32)
    dst = np.empty(n_edges, dtype=np.int32)
    rc = _load().synth_rmat(seed, scale, abc[0], abc[1], abc[2], n, n_edges, _ptr(src), _ptr(dst))
    if rc != n_edges:
        raise RuntimeError(f"synth_rmat failed ({rc})")
    return Graph(name, n, n, src, dst)


C3_N, C3_E = 232965, 114600000
C4_N, C4_E = 2449029, 61859140


def shuffle_within_rows(g: Graph, seed: int, name: str = "row order") -> Graph:
    """The same edges with each destination's in-edges in a seeded random
    order instead of ascending source: edges sorted by (destination, random
    key), edge ids renumbered to the new positions.  Rows then list their
    sources in no particular order, as an edge list in arrival order does."""
    key = permutation(seed, name, g.n_edges).astype(np.int64)
    order = np.argsort((g.dst.astype(np.int64) << 32) | key, kind="stable")
    return Graph(g.name + " (rows shuffled)", g.n_src, g.n_dst, np.ascontiguousarray(g.src[order]),
                 np.ascontiguousarray(g.dst[order]), dict(g.extra))


def graph_c3() -> Graph:
    return rmat_graph(SEED_BASE + 3, 18, C3_N, C3_E, name="c3")


def graph_c4() -> Graph:
    return rmat_graph(SEED_BASE + 4, 22, C4_N, C4_E, name="c4")


C5_N, C5_E, C5_R = 100000, 2000000, 50


def graph_c5() -> Graph:
    """Relational multigraph seen as a bipartite graph over (etype * N + src) -> dst."""
    lib = _load()
    seed = SEED_BASE + 5
    n, e, r = C5_N, C5_E, C5_R
    src = np.empty(e, dtype=np.int32)
    dst = np.empty(e, dtype=np.int32)
    lib.synth_uniform_edges(seed, stream_id("edges"), e, n, n, _ptr(src), _ptr(dst))
    et = np.empty(e, dtype=np.int32)
    lib.synth_zipf(seed, stream_id("etype"), e, r, 1.2, _ptr(et))
    comp = (et.astype(np.int64) * n + src).astype(np.int32)
    comp, dst = sort_coo(comp, dst, n * r, n)
    etype = (comp // n).astype(np.int32)
    cnt = np.empty(e, dtype=np.int32)
    lib.synth_count_dst_type(e, n, r, _ptr(dst), _ptr(etype), _ptr(cnt))
    g = Graph("c5", n * r, n, comp, dst)
    g.extra["etype"] = etype
    g.extra["orig_src"] = (comp % n).astype(np.int32)
    g.extra["n_nodes"] = n
    g.extra["n_rel"] = r
    g.extra["norm"] = (1.0 / cnt.astype(np.float64)).astype(np.float32).reshape(-1, 1)
    return g


GRAPHS = {"c1": graph_c1, "c2": graph_c2, "c3": graph_c3, "c4": graph_c4, "c5": graph_c5}


def config_graph(name: str) -> Graph:
    return GRAPHS[name]()


def feat_seed(k: int) -> int:
    """Seed for the input features of workload k (1..5)."""
    return SEED_BASE + 100 + k


def grad_seed(k: int) -> int:
    """Seed for the upstream gradients of workload k (1..5)."""
    return SEED_BASE + 200 + k


def degree_stats(g: Graph) -> dict:
    """Summary of the in-degree distribution (used by tests and the design notes)."""
    indeg = bincount(g.dst, g.n_dst)
    nz = indeg[indeg > 0]
    s = np.sort(indeg)
    share = {}
    for t in (64, 1024, 16384):
        share[t] = float(indeg[indeg > t].sum()) / max(g.n_edges, 1)
    return {
        "max": int(s[-1]) if s.size else 0,
        "median": float(np.median(indeg)) if s.size else 0.0,
        "p99": float(np.percentile(indeg, 99)) if s.size else 0.0,
        "empty": int((indeg == 0).sum()),
        "nonempty": int(nz.size),
        "edge_share_above": share,
        "self_loops": int((g.src == g.dst).sum()) if g.n_src == g.n_dst else 0,
    }
