"""Python access to the CPU oracle (``oracle.c``).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The GPU library and
its binding never import it, and it imports nothing from them.

Arrays are numpy arrays shaped (rows, heads, feat) -- a 2-D (rows, d) array is
read as (rows, 1, d) -- with dtype float32, float64, or uint16 holding bf16 bit
patterns.  The last two dimensions must be contiguous; the row stride may be
larger than heads * feat.

Operator names follow the paper's message functions: ``copy_lhs`` (copy_u),
``copy_rhs`` (copy_e), ``add``, ``sub``, ``mul``, ``div``, ``dot``; reducers
``sum``, ``mean``, ``max``, ``min``; targets ``u`` (source), ``e`` (edge),
``v`` (destination).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

OPS = {"copy_lhs": 0, "copy_rhs": 1, "add": 2, "sub": 3, "mul": 4, "div": 5, "dot": 6}
REDUCES = {"sum": 0, "mean": 1, "max": 2, "min": 3}
TARGETS = {"u": 0, "e": 1, "v": 2}
_DT = {np.dtype(np.float32): 0, np.dtype(np.uint16): 1, np.dtype(np.float64): 2}

BUILD_CMD = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-std=c99", "-Wall", "-Wextra", "-shared",
             "-fPIC", "-o", _LIB_PATH, os.path.join(_HERE, "oracle.c"), "-lm"]


def build(verbose: bool = False) -> str:
    if verbose:
        print(" ".join(BUILD_CMD))
    subprocess.run(BUILD_CMD, check=True)
    return _LIB_PATH


class _Tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("rows", ctypes.c_int64), ("heads", ctypes.c_int64), ("feat", ctypes.c_int64),
                ("stride", ctypes.c_int64)]


class _Graph(ctypes.Structure):
    _fields_ = [("n_src", ctypes.c_int64), ("n_dst", ctypes.c_int64), ("n_edges", ctypes.c_int64),
                ("src", ctypes.c_void_p), ("dst", ctypes.c_void_p)]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        P, I, I64, F = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
        sig = {
            "oracle_degrees": [P, P, P],
            "oracle_csr": [P, I, P, P, P],
            "oracle_gspmm": [P, I, I, P, P, P, P, P, P, I64],
            "oracle_gsddmm": [P, I, P, I, P, I, P, P, I64],
            "oracle_gspmm_backward": [P, I, I, P, P, P, P, P, P, P, I64],
            "oracle_gsddmm_backward": [P, I, P, I, P, I, P, P, P, P, I64],
            "oracle_edge_softmax": [P, P, P, P, I64, P],
            "oracle_edge_softmax_backward": [P, P, P, P, P, I64, P],
            "oracle_leaky_relu": [P, P, F],
            "oracle_leaky_relu_backward": [P, P, P, F],
        }
        for name, args in sig.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        lib.oracle_round_bf16.argtypes = [I64, P, P]
        lib.oracle_round_bf16.restype = None
        _lib = lib
    return _lib


class OGraph:
    """Edge list (edge e: src[e] -> dst[e]) held for the oracle."""

    def __init__(self, src, dst, n_src: int, n_dst: int):
        self.src = np.ascontiguousarray(src, dtype=np.int32)
        self.dst = np.ascontiguousarray(dst, dtype=np.int32)
        assert self.src.shape == self.dst.shape
        self.n_src, self.n_dst = int(n_src), int(n_dst)
        self._g = _Graph(self.n_src, self.n_dst, self.src.size, self.src.ctypes.data, self.dst.ctypes.data)

    @classmethod
    def of(cls, g) -> "OGraph":
        """From any object with src, dst, n_src, n_dst attributes."""
        return cls(g.src, g.dst, g.n_src, g.n_dst)

    @property
    def n_edges(self) -> int:
        return int(self.src.size)

    @property
    def ref(self):
        return ctypes.byref(self._g)


def _as3(a):
    if a is None:
        return None
    a = np.asarray(a)
    if a.ndim == 2:
        a = a.reshape(a.shape[0], 1, a.shape[1])
    assert a.ndim == 3, "tensors are (rows, heads, feat)"
    return a


def _desc(a):
    """ctypes descriptor of a (rows, heads, feat) array; keeps a reference."""
    if a is None:
        return None
    a = _as3(a)
    if a.dtype not in _DT:
        raise TypeError(f"unsupported dtype {a.dtype}")
    it = a.itemsize
    h, f = a.shape[1], a.shape[2]
    if a.shape[0] > 1:
        if a.strides[2] != it or a.strides[1] != f * it or a.strides[0] % it:
            raise ValueError("last two dims must be contiguous")
        stride = a.strides[0] // it
    else:
        stride = h * f
    return _Tensor(a.ctypes.data, _DT[a.dtype], 0, a.shape[0], h, f, stride)


def _ref(d):
    return ctypes.byref(d) if d is not None else None


def _sel(sel):
    if sel is None:
        return None, None, 0
    s = np.ascontiguousarray(sel, dtype=np.int64)
    return s, s.ctypes.data, s.size


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments ({rc})")


def _rows_of(g: OGraph, target: str) -> int:
    return {"u": g.n_src, "e": g.n_edges, "v": g.n_dst}[target]


def msg_shape(op: str, lhs, rhs):
    if op == "copy_lhs":
        return lhs.shape[1], lhs.shape[2]
    if op == "copy_rhs":
        return rhs.shape[1], rhs.shape[2]
    return max(lhs.shape[1], rhs.shape[1]), max(lhs.shape[2], rhs.shape[2])


def degrees(g: OGraph):
    ind = np.empty(g.n_dst, dtype=np.int64)
    outd = np.empty(g.n_src, dtype=np.int64)
    _check(_load().oracle_degrees(g.ref, ind.ctypes.data, outd.ctypes.data), "degrees")
    return ind, outd


def csr(g: OGraph, reverse: bool = False):
    """(indptr int64, indices int32, eids int32): in-CSR, or the reverse graph's CSR."""
    n = g.n_src if reverse else g.n_dst
    indptr = np.empty(n + 1, dtype=np.int64)
    indices = np.empty(max(g.n_edges, 1), dtype=np.int32)
    eids = np.empty(max(g.n_edges, 1), dtype=np.int32)
    _check(_load().oracle_csr(g.ref, int(reverse), indptr.ctypes.data, indices.ctypes.data, eids.ctypes.data),
           "csr")
    return indptr, indices[:g.n_edges], eids[:g.n_edges]


def gspmm(g: OGraph, op: str, reduce: str, lhs=None, rhs=None, out_dtype=None, rows=None):
    """z_v = reduce over in-edges (u, e, v) of op(lhs[u], rhs[e]).

    Returns out, or (out, arg_u, arg_e) for max/min.  With ``rows``, output row
    k is node rows[k]."""
    lhs, rhs = _as3(lhs), _as3(rhs)
    h, f = msg_shape(op, lhs, rhs)
    dt = out_dtype or (lhs if lhs is not None else rhs).dtype
    sel, sp, ns = _sel(rows)
    nrow = ns if rows is not None else g.n_dst
    out = np.zeros((nrow, h, f), dtype=dt)
    cmp = reduce in ("max", "min")
    au = np.empty((nrow, h, f), dtype=np.int32) if cmp else None
    ae = np.empty((nrow, h, f), dtype=np.int32) if cmp else None
    dl, dr, do = _desc(lhs), _desc(rhs), _desc(out)
    rc = _load().oracle_gspmm(g.ref, OPS[op], REDUCES[reduce], _ref(dl), _ref(dr), _ref(do),
                              au.ctypes.data if cmp else None, ae.ctypes.data if cmp else None, sp,
                              ctypes.c_int64(ns))
    _check(rc, "gspmm")
    return (out, au, ae) if cmp else out


def gsddmm(g: OGraph, op: str, lhs, lhs_target: str, rhs, rhs_target: str, out_dtype=None, edges=None):
    """m_e = op(lhs at its target, rhs at its target); dot reduces the feature dim."""
    lhs, rhs = _as3(lhs), _as3(rhs)
    if op == "dot":
        h, f = max(lhs.shape[1], rhs.shape[1]), 1
    else:
        h, f = msg_shape(op, lhs, rhs)
    dt = out_dtype or (lhs if lhs is not None else rhs).dtype
    sel, sp, ns = _sel(edges)
    nrow = ns if edges is not None else g.n_edges
    out = np.zeros((nrow, h, f), dtype=dt)
    dl, dr, do = _desc(lhs), _desc(rhs), _desc(out)
    rc = _load().oracle_gsddmm(g.ref, OPS[op], _ref(dl), TARGETS[lhs_target], _ref(dr), TARGETS[rhs_target],
                               _ref(do), sp, ctypes.c_int64(ns))
    _check(rc, "gsddmm")
    return out


def gspmm_backward(g: OGraph, op: str, reduce: str, lhs, rhs, grad_out, arg_e=None, want_lhs=True,
                   want_rhs=True, sel=None):
    """(grad_lhs, grad_rhs) of gspmm; with ``sel`` exactly one gradient is computed on the listed rows."""
    lhs, rhs, grad_out = _as3(lhs), _as3(rhs), _as3(grad_out)
    want_lhs = want_lhs and op != "copy_rhs"
    want_rhs = want_rhs and op != "copy_lhs"
    s, sp, ns = _sel(sel)
    gl = gr = None
    dt = grad_out.dtype
    if want_lhs:
        gl = np.zeros((ns if sel is not None else g.n_src, lhs.shape[1], lhs.shape[2]), dtype=dt)
    if want_rhs:
        gr = np.zeros((ns if sel is not None else g.n_edges, rhs.shape[1], rhs.shape[2]), dtype=dt)
    ae = None if arg_e is None else np.ascontiguousarray(arg_e, dtype=np.int32)
    dl, dr, dg, dgl, dgr = _desc(lhs), _desc(rhs), _desc(grad_out), _desc(gl), _desc(gr)
    rc = _load().oracle_gspmm_backward(g.ref, OPS[op], REDUCES[reduce], _ref(dl), _ref(dr),
                                       ae.ctypes.data if ae is not None else None, _ref(dg), _ref(dgl), _ref(dgr),
                                       sp, ctypes.c_int64(ns))
    _check(rc, "gspmm_backward")
    return gl, gr


def gsddmm_backward(g: OGraph, op: str, lhs, lhs_target: str, rhs, rhs_target: str, grad_out, want_lhs=True,
                    want_rhs=True, sel=None):
    lhs, rhs, grad_out = _as3(lhs), _as3(rhs), _as3(grad_out)
    want_lhs = want_lhs and op != "copy_rhs"
    want_rhs = want_rhs and op != "copy_lhs"
    s, sp, ns = _sel(sel)
    gl = gr = None
    dt = grad_out.dtype
    if want_lhs:
        gl = np.zeros((ns if sel is not None else _rows_of(g, lhs_target), lhs.shape[1], lhs.shape[2]), dtype=dt)
    if want_rhs:
        gr = np.zeros((ns if sel is not None else _rows_of(g, rhs_target), rhs.shape[1], rhs.shape[2]), dtype=dt)
    dl, dr, dg, dgl, dgr = _desc(lhs), _desc(rhs), _desc(grad_out), _desc(gl), _desc(gr)
    rc = _load().oracle_gsddmm_backward(g.ref, OPS[op], _ref(dl), TARGETS[lhs_target], _ref(dr),
                                        TARGETS[rhs_target], _ref(dg), _ref(dgl), _ref(dgr), sp, ctypes.c_int64(ns))
    _check(rc, "gsddmm_backward")
    return gl, gr


def _sel_count(g: OGraph, rows):
    ind, _ = degrees(g)
    return int(ind[np.asarray(rows, dtype=np.int64)].sum())


def edge_softmax(g: OGraph, score, rows=None):
    """Softmax over each destination's in-edges.  With ``rows``: (values, edge ids) for their in-edges."""
    score = _as3(score)
    s, sp, ns = _sel(rows)
    nrow = _sel_count(g, rows) if rows is not None else g.n_edges
    out = np.zeros((nrow,) + score.shape[1:], dtype=score.dtype)
    eids = np.empty(max(nrow, 1), dtype=np.int64)
    ds, do = _desc(score), _desc(out)
    rc = _load().oracle_edge_softmax(g.ref, _ref(ds), _ref(do), sp, ctypes.c_int64(ns), eids.ctypes.data)
    _check(rc, "edge_softmax")
    return (out, eids[:nrow]) if rows is not None else out


def edge_softmax_backward(g: OGraph, out, grad_out, rows=None):
    out, grad_out = _as3(out), _as3(grad_out)
    s, sp, ns = _sel(rows)
    nrow = _sel_count(g, rows) if rows is not None else g.n_edges
    gs = np.zeros((nrow,) + out.shape[1:], dtype=grad_out.dtype)
    eids = np.empty(max(nrow, 1), dtype=np.int64)
    d1, d2, d3 = _desc(out), _desc(grad_out), _desc(gs)
    rc = _load().oracle_edge_softmax_backward(g.ref, _ref(d1), _ref(d2), _ref(d3), sp, ctypes.c_int64(ns),
                                              eids.ctypes.data)
    _check(rc, "edge_softmax_backward")
    return (gs, eids[:nrow]) if rows is not None else gs


def leaky_relu(x, slope: float = 0.2):
    x = _as3(x)
    y = np.zeros(x.shape, dtype=x.dtype)
    dx, dy = _desc(x), _desc(y)
    _check(_load().oracle_leaky_relu(_ref(dx), _ref(dy), ctypes.c_float(slope)), "leaky_relu")
    return y


def leaky_relu_backward(x, dy, slope: float = 0.2):
    x, dy = _as3(x), _as3(dy)
    dx = np.zeros(x.shape, dtype=dy.dtype)
    a, b, c = _desc(x), _desc(dy), _desc(dx)
    _check(_load().oracle_leaky_relu_backward(_ref(a), _ref(b), _ref(c), ctypes.c_float(slope)),
           "leaky_relu_backward")
    return dx


def round_bf16(x) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (the oracle's own rounding)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().oracle_round_bf16(ctypes.c_int64(x.size), x.ctypes.data, out.ctypes.data)
    return out


def bf16_to_f32(bits) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)
