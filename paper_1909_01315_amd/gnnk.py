"""Python binding of libgnnk.so (the C ABI declared in include/gnnk.h).

Argument marshalling only: every operation runs in the HIP library.  PyTorch
provides device memory (outputs are allocated here with torch.empty and
handed to the library, which computes their sizes' contents) and the current
HIP stream.  There is no CPU fallback: if the library is missing or cannot be
loaded, every call raises.

Tensors are torch tensors on the GPU, float32 or bfloat16, shaped (rows, heads,
feat) -- a 2-D (rows, d) tensor is read as (rows, 1, d) -- with the last two
dimensions contiguous (the row stride may be larger).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgnnk.so")

OK, EINVAL, EUNSUPPORTED, EHIP, ERANGE, ENOMEM = range(6)
I32, I64 = 0, 1
F32, BF16 = 0, 1
OPS = {"copy_lhs": 0, "copy_rhs": 1, "add": 2, "sub": 3, "mul": 4, "div": 5, "dot": 6}
REDUCES = {"sum": 0, "mean": 1, "max": 2, "min": 3}
TARGETS = {"u": 0, "e": 1, "v": 2}

_lib = None


class GnnkError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"gnnk status {status}: {msg}")
        self.status = status


class _Tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("rows", ctypes.c_int64), ("heads", ctypes.c_int32),
                ("feat", ctypes.c_int32), ("row_stride", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class _Info(ctypes.Structure):
    _fields_ = [("num_src", ctypes.c_int64), ("num_dst", ctypes.c_int64), ("num_edges", ctypes.c_int64),
                ("ptr_type", ctypes.c_int32), ("identity_eids", ctypes.c_int32),
                ("max_in_degree", ctypes.c_int64), ("max_out_degree", ctypes.c_int64),
                ("empty_dst_rows", ctypes.c_int64), ("empty_src_rows", ctypes.c_int64),
                ("seg_edges", ctypes.c_int64), ("hub_dst_rows", ctypes.c_int64), ("hub_src_rows", ctypes.c_int64),
                ("segments_in", ctypes.c_int64), ("segments_out", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_size_t), ("seg_edges_out", ctypes.c_int64),
                ("seg_edges_gather", ctypes.c_int64), ("segments_gather", ctypes.c_int64),
                ("seg_edges_in_gather", ctypes.c_int64), ("segments_in_gather", ctypes.c_int64)]


SYMBOLS = {
    "graph_workspace_bytes": [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p],
    "graph_create_coo": [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                         ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p],
    "graph_create_csr": [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int,
                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                         ctypes.c_void_p],
    "graph_info": [ctypes.c_void_p, ctypes.c_void_p],
    "graph_in_degrees": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "graph_out_degrees": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "graph_csr_export": [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                         ctypes.c_void_p],
    "graph_validate": [ctypes.c_void_p, ctypes.c_void_p],
    "graph_destroy": [ctypes.c_void_p],
    "gspmm": [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "gspmm_noalloc": [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "gsddmm": [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
               ctypes.c_void_p, ctypes.c_void_p],
    "gspmm_backward": [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                       ctypes.c_void_p],
    "gsddmm_backward": [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "edge_softmax": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "edge_softmax_backward": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "edge_leaky_relu": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float, ctypes.c_void_p],
    "edge_leaky_relu_backward": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float,
                                 ctypes.c_void_p],
    "gat_aggregate": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float,
                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "gat_aggregate_backward": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float,
                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                               ctypes.c_void_p],
    "graph_scratch_bytes": [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p],
    "graph_attach_scratch": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t],
    "gnnk_scratch_needed": [ctypes.c_void_p],
    "gnnk_set_option": [ctypes.c_char_p, ctypes.c_int64],
    "gnnk_last_error": [],
}


def load():
    """Load libgnnk.so (raises if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built (run __graft_entry__.build() or "
                              "python -m paper_1909_01315_amd.build)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, args in SYMBOLS.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        lib.gnnk_last_error.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def _check(status: int):
    if status != OK:
        raise GnnkError(status, load().gnnk_last_error().decode())


def _stream(stream=None) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


SCRATCH_ARGMAX, SCRATCH_WIDE_SUMS = 1, 2


def _run(g, call, stream=None):
    """Run call() (a C entry point on g); when it ran short of scratch, lend g
    a buffer of the size it asked for on the call's stream and run it again
    (outputs are overwritten, never accumulated, so a repeated call gives the
    same result).  A call that needs several parts asks for them in turn."""
    st = call()
    for _ in range(4):
        if st != ENOMEM:
            break
        need = ctypes.c_size_t(0)
        load().gnnk_scratch_needed(ctypes.byref(need))
        if need.value == 0:  # short of something else (a workspace)
            break
        g.lend_scratch(need.value, stream)
        st = call()
    _check(st)


def _as3(t: torch.Tensor) -> torch.Tensor:
    if t.dim() == 2:
        t = t.unsqueeze(1)
    if t.dim() != 3:
        raise ValueError("tensors are (rows, heads, feat)")
    return t


def _desc(t):
    """ctypes descriptor of a (rows, heads, feat) GPU tensor."""
    if t is None:
        return None
    t = _as3(t)
    if not t.is_cuda:
        raise ValueError("tensors must be on the GPU")
    if t.dtype == torch.float32:
        dt = F32
    elif t.dtype == torch.bfloat16:
        dt = BF16
    else:
        raise TypeError(f"unsupported dtype {t.dtype}")
    rows, h, f = t.shape
    if t.numel() == 0:  # no element is addressed: any strides will do
        return _Tensor(t.data_ptr(), rows, h, f, h * f, dt, 0)
    if (f > 1 and t.stride(2) != 1) or (h > 1 and t.stride(1) != f):
        raise ValueError("the last two dimensions must be contiguous")
    stride = t.stride(0) if rows > 1 else h * f
    if stride < h * f:
        raise ValueError("row stride smaller than heads * feat")
    return _Tensor(t.data_ptr(), rows, h, f, stride, dt, 0)


def _ref(d):
    return ctypes.byref(d) if d is not None else None


def _ptr(t):
    return t.data_ptr() if t is not None else None


def set_option(key: str, value: int):
    _check(load().gnnk_set_option(key.encode(), int(value)))


class Graph:
    """A gnnk graph handle with its device workspace (and any borrowed arrays)."""

    def __init__(self, handle, keep, num_src, num_dst, num_edges):
        self._h = handle
        self._keep = keep  # tensors the handle points into
        self._lent = {}    # stream handle -> scratch buffer lent for that stream
        self.num_src, self.num_dst, self.num_edges = num_src, num_dst, num_edges

    @property
    def device(self):
        return self._keep[0].device

    def scratch_bytes(self, max_cols: int, argmax: bool = False, wide_sums: bool = False) -> int:
        """Bytes of scratch any call with messages of at most max_cols columns needs."""
        n = ctypes.c_size_t(0)
        flags = (SCRATCH_ARGMAX if argmax else 0) | (SCRATCH_WIDE_SUMS if wide_sums else 0)
        _check(load().graph_scratch_bytes(self.handle, int(max_cols), flags, ctypes.byref(n)))
        return n.value

    def lend_scratch(self, nbytes: int, stream=None):
        """Lend the handle a scratch buffer of at least nbytes for the calls on
        `stream` (default: the current stream), allocated on that stream; the
        buffer it replaces goes back to torch's allocator, which reuses it only
        for work ordered after the calls already queued on that stream."""
        s = stream if stream is not None else torch.cuda.current_stream()
        old = self._lent.get(s.cuda_stream)
        size = max(int(nbytes), int(old.numel() * 5 // 4) if old is not None else 0, 256)
        with torch.cuda.stream(s):
            buf = torch.empty(size, dtype=torch.uint8, device=self.device)
        _check(load().graph_attach_scratch(self.handle, s.cuda_stream, buf.data_ptr(), size))
        self._lent[s.cuda_stream] = buf

    @staticmethod
    def _workspace(num_src, num_dst, num_edges, ptr_t, device):
        nbytes = ctypes.c_size_t(0)
        _check(load().graph_workspace_bytes(num_src, num_dst, num_edges, ptr_t, ctypes.byref(nbytes)))
        return torch.empty(max(nbytes.value, 1), dtype=torch.uint8, device=device)

    @classmethod
    def from_coo(cls, src: torch.Tensor, dst: torch.Tensor, num_src: int, num_dst: int, ptr64: bool = False,
                 stream=None) -> "Graph":
        assert src.dtype == torch.int32 and dst.dtype == torch.int32 and src.is_cuda and dst.is_cuda
        src, dst = src.contiguous(), dst.contiguous()
        E = src.numel()
        ptr_t = I64 if ptr64 else I32
        ws = cls._workspace(num_src, num_dst, E, ptr_t, src.device)
        h = ctypes.c_void_p()
        _check(load().graph_create_coo(num_src, num_dst, E, src.data_ptr(), dst.data_ptr(), ptr_t, ws.data_ptr(),
                                       ws.numel(), _stream(stream), ctypes.byref(h)))
        return cls(h, [ws], num_src, num_dst, E)

    @classmethod
    def from_csr(cls, indptr: torch.Tensor, indices: torch.Tensor, eids, num_src: int, stream=None) -> "Graph":
        assert indptr.dtype in (torch.int32, torch.int64) and indices.dtype == torch.int32
        indptr, indices = indptr.contiguous(), indices.contiguous()
        if eids is not None:
            assert eids.dtype == torch.int32
            eids = eids.contiguous()
        num_dst = indptr.numel() - 1
        E = indices.numel()
        ptr_t = I64 if indptr.dtype == torch.int64 else I32
        ws = cls._workspace(num_src, num_dst, E, ptr_t, indices.device)
        h = ctypes.c_void_p()
        _check(load().graph_create_csr(num_src, num_dst, E, indptr.data_ptr(), ptr_t, indices.data_ptr(),
                                       _ptr(eids), ws.data_ptr(), ws.numel(), _stream(stream), ctypes.byref(h)))
        return cls(h, [ws, indptr, indices, eids], num_src, num_dst, E)

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("graph destroyed")
        return self._h

    def info(self) -> dict:
        inf = _Info()
        _check(load().graph_info(self.handle, ctypes.byref(inf)))
        return {name: getattr(inf, name) for name, _ in _Info._fields_}

    def in_degrees(self, stream=None) -> torch.Tensor:
        out = torch.empty(self.num_dst, dtype=torch.int32, device=self._keep[0].device)
        _check(load().graph_in_degrees(self.handle, out.data_ptr(), _stream(stream)))
        return out

    def out_degrees(self, stream=None) -> torch.Tensor:
        out = torch.empty(self.num_src, dtype=torch.int32, device=self._keep[0].device)
        _check(load().graph_out_degrees(self.handle, out.data_ptr(), _stream(stream)))
        return out

    def csr_export(self, reverse: bool = False, stream=None):
        inf = self.info()
        dev = self._keep[0].device
        rows = self.num_src if reverse else self.num_dst
        pdt = torch.int64 if inf["ptr_type"] == I64 else torch.int32
        indptr = torch.empty(rows + 1, dtype=pdt, device=dev)
        indices = torch.empty(max(self.num_edges, 1), dtype=torch.int32, device=dev)
        eids = torch.empty(max(self.num_edges, 1), dtype=torch.int32, device=dev)
        _check(load().graph_csr_export(self.handle, int(reverse), indptr.data_ptr(), indices.data_ptr(),
                                       eids.data_ptr(), _stream(stream)))
        return indptr, indices[:self.num_edges], eids[:self.num_edges]

    def validate(self, stream=None):
        _check(load().graph_validate(self.handle, _stream(stream)))

    def destroy(self):
        if self._h is not None:
            _check(load().graph_destroy(self._h))
            self._h = None
            self._keep = None
            self._lent = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def rows_of(self, target: str) -> int:
        return {"u": self.num_src, "e": self.num_edges, "v": self.num_dst}[target]


def _msg_shape(op, lhs, rhs):
    if op == "copy_lhs":
        return lhs.shape[1], lhs.shape[2]
    if op == "copy_rhs":
        return rhs.shape[1], rhs.shape[2]
    return max(lhs.shape[1], rhs.shape[1]), max(lhs.shape[2], rhs.shape[2])


def _dev_dtype(*ts):
    for t in ts:
        if t is not None:
            return t.device, t.dtype
    raise ValueError("no tensor given")


def gspmm(g: Graph, op: str, reduce: str, lhs=None, rhs=None, out=None, want_args: bool = False, arg_lhs=None,
          arg_rhs=None, stream=None):
    """out[v] = reduce over in-edges (u, e, v) of op(lhs[u], rhs[e]).

    Returns out, or (out, arg_lhs, arg_rhs) for max/min with want_args (the
    arg arrays may be passed in preallocated)."""
    lhs = _as3(lhs) if lhs is not None else None
    rhs = _as3(rhs) if rhs is not None else None
    h, f = _msg_shape(op, lhs, rhs)
    dev, dt = _dev_dtype(lhs, rhs)
    if out is None:
        out = torch.empty((g.num_dst, h, f), dtype=dt, device=dev)
    arg_l, arg_r = arg_lhs, arg_rhs
    if want_args:
        if arg_l is None:
            arg_l = torch.empty((g.num_dst, h, f), dtype=torch.int32, device=dev)
        if arg_r is None:
            arg_r = torch.empty((g.num_dst, h, f), dtype=torch.int32, device=dev)
    dl, dr, do = _desc(lhs), _desc(rhs), _desc(out)
    _run(g, lambda: load().gspmm(g.handle, OPS[op], REDUCES[reduce], _ref(dl), _ref(dr), _ref(do), _ptr(arg_l),
                                 _ptr(arg_r), _stream(stream)), stream)
    return (out, arg_l, arg_r) if want_args else out


def gspmm_noalloc(g: Graph, op: str, reduce: str, lhs=None, rhs=None, out=None, arg_lhs=None, arg_rhs=None,
                  stream=None):
    """gspmm with the library's fixed per-GPU scratch buffer (no buffer is
    lent or allocated by the call; outputs and arg arrays are the caller's,
    allocated here only when not given).  Returns out, or (out, arg_lhs,
    arg_rhs) when arg arrays are given."""
    lhs = _as3(lhs) if lhs is not None else None
    rhs = _as3(rhs) if rhs is not None else None
    if out is None:
        h, f = _msg_shape(op, lhs, rhs)
        dev, dt = _dev_dtype(lhs, rhs)
        out = torch.empty((g.num_dst, h, f), dtype=dt, device=dev)
    dl, dr, do = _desc(lhs), _desc(rhs), _desc(out)
    _check(load().gspmm_noalloc(g.handle, OPS[op], REDUCES[reduce], _ref(dl), _ref(dr), _ref(do), _ptr(arg_lhs),
                                _ptr(arg_rhs), _stream(stream)))
    return (out, arg_lhs, arg_rhs) if (arg_lhs is not None or arg_rhs is not None) else out


def gsddmm(g: Graph, op: str, lhs, lhs_target: str, rhs, rhs_target: str, out=None, stream=None):
    """out[e] = op(lhs at its target, rhs at its target); targets 'u', 'e', 'v'."""
    lhs = _as3(lhs) if lhs is not None else None
    rhs = _as3(rhs) if rhs is not None else None
    if op == "dot":
        h, f = max(lhs.shape[1], rhs.shape[1]), 1
    else:
        h, f = _msg_shape(op, lhs, rhs)
    dev, dt = _dev_dtype(lhs, rhs)
    if out is None:
        out = torch.empty((g.num_edges, h, f), dtype=dt, device=dev)
    dl, dr, do = _desc(lhs), _desc(rhs), _desc(out)
    _run(g, lambda: load().gsddmm(g.handle, OPS[op], _ref(dl), TARGETS[lhs_target], _ref(dr), TARGETS[rhs_target],
                                  _ref(do), _stream(stream)), stream)
    return out


def gspmm_backward(g: Graph, op: str, reduce: str, lhs, rhs, grad_out, arg_rhs=None, want_lhs: bool = True,
                   want_rhs: bool = True, grad_lhs=None, grad_rhs=None, stream=None):
    """(grad_lhs, grad_rhs) of gspmm (either may be None)."""
    lhs = _as3(lhs) if lhs is not None else None
    rhs = _as3(rhs) if rhs is not None else None
    grad_out = _as3(grad_out)
    if want_lhs and lhs is not None and grad_lhs is None:
        grad_lhs = torch.empty(lhs.shape, dtype=grad_out.dtype, device=grad_out.device)
    if want_rhs and rhs is not None and grad_rhs is None:
        grad_rhs = torch.empty(rhs.shape, dtype=grad_out.dtype, device=grad_out.device)
    if not want_lhs:
        grad_lhs = None
    if not want_rhs:
        grad_rhs = None
    d = [_desc(x) for x in (lhs, rhs, grad_out, grad_lhs, grad_rhs)]
    _run(g, lambda: load().gspmm_backward(g.handle, OPS[op], REDUCES[reduce], _ref(d[0]), _ref(d[1]), None,
                                          _ptr(arg_rhs), _ref(d[2]), _ref(d[3]), _ref(d[4]), _stream(stream)), stream)
    return grad_lhs, grad_rhs


def gsddmm_backward(g: Graph, op: str, lhs, lhs_target: str, rhs, rhs_target: str, grad_out, want_lhs=True,
                    want_rhs=True, grad_lhs=None, grad_rhs=None, stream=None):
    lhs = _as3(lhs) if lhs is not None else None
    rhs = _as3(rhs) if rhs is not None else None
    grad_out = _as3(grad_out)
    if want_lhs and lhs is not None and grad_lhs is None:
        grad_lhs = torch.empty(lhs.shape, dtype=grad_out.dtype, device=grad_out.device)
    if want_rhs and rhs is not None and grad_rhs is None:
        grad_rhs = torch.empty(rhs.shape, dtype=grad_out.dtype, device=grad_out.device)
    if not want_lhs:
        grad_lhs = None
    if not want_rhs:
        grad_rhs = None
    d = [_desc(x) for x in (lhs, rhs, grad_out, grad_lhs, grad_rhs)]
    _run(g, lambda: load().gsddmm_backward(g.handle, OPS[op], _ref(d[0]), TARGETS[lhs_target], _ref(d[1]),
                                           TARGETS[rhs_target], _ref(d[2]), _ref(d[3]), _ref(d[4]), _stream(stream)),
         stream)
    return grad_lhs, grad_rhs


def edge_softmax(g: Graph, score, out=None, stream=None):
    score = _as3(score)
    if out is None:
        out = torch.empty(score.shape, dtype=score.dtype, device=score.device)
    d1, d2 = _desc(score), _desc(out)
    _run(g, lambda: load().edge_softmax(g.handle, _ref(d1), _ref(d2), _stream(stream)), stream)
    return out


def edge_softmax_backward(g: Graph, out, grad_out, grad_score=None, stream=None):
    out, grad_out = _as3(out), _as3(grad_out)
    if grad_score is None:
        grad_score = torch.empty(out.shape, dtype=grad_out.dtype, device=grad_out.device)
    d1, d2, d3 = _desc(out), _desc(grad_out), _desc(grad_score)
    _run(g, lambda: load().edge_softmax_backward(g.handle, _ref(d1), _ref(d2), _ref(d3), _stream(stream)), stream)
    return grad_score


def gat_aggregate(g: Graph, feat, el, er, slope: float = 0.2, out=None, attn=None, want_attn: bool = False,
                  stats=None, want_stats: bool = False, stream=None):
    """Fused attention: out[v, h] = sum over in-edges of softmax_v(leaky(el[u, h] + er[v, h])) * feat[u, h, :].
    Returns out, followed by attn (with want_attn or attn given) and by the per-row statistics
    (num_dst, H, 2) fp32 (with want_stats or stats given) that gat_aggregate_backward takes."""
    feat, el, er = _as3(feat), _as3(el), _as3(er)
    if out is None:
        out = torch.empty((g.num_dst, feat.shape[1], feat.shape[2]), dtype=feat.dtype, device=feat.device)
    if want_attn and attn is None:
        attn = torch.empty((g.num_edges, feat.shape[1], 1), dtype=feat.dtype, device=feat.device)
    if want_stats and stats is None:
        stats = torch.empty((g.num_dst, feat.shape[1], 2), dtype=torch.float32, device=feat.device)
    d = [_desc(x) for x in (feat, el, er, out, attn, stats)]
    _run(g, lambda: load().gat_aggregate(g.handle, _ref(d[0]), _ref(d[1]), _ref(d[2]), ctypes.c_float(slope),
                                         _ref(d[3]), _ref(d[4]), _ref(d[5]), _stream(stream)), stream)
    res = (out,) + ((attn,) if attn is not None else ()) + ((stats,) if stats is not None else ())
    return res if len(res) > 1 else out


def gat_aggregate_backward(g: Graph, feat, el, er, slope: float, stats, grad_out, want_feat: bool = True,
                           want_el: bool = True, want_er: bool = True, stream=None):
    """(grad_feat, grad_el, grad_er) of gat_aggregate from its per-row statistics (any may be None)."""
    feat, el, er, grad_out = _as3(feat), _as3(el), _as3(er), _as3(grad_out)
    gf = torch.empty(feat.shape, dtype=feat.dtype, device=feat.device) if want_feat else None
    gl = torch.empty(el.shape, dtype=feat.dtype, device=feat.device) if want_el else None
    gr = torch.empty(er.shape, dtype=feat.dtype, device=feat.device) if want_er else None
    d = [_desc(x) for x in (feat, el, er, stats, grad_out, gf, gl, gr)]
    _run(g, lambda: load().gat_aggregate_backward(g.handle, _ref(d[0]), _ref(d[1]), _ref(d[2]),
                                                  ctypes.c_float(slope), _ref(d[3]), _ref(d[4]), _ref(d[5]),
                                                  _ref(d[6]), _ref(d[7]), _stream(stream)), stream)
    return gf, gl, gr


def edge_leaky_relu(x, slope: float = 0.2, y=None, stream=None):
    x = _as3(x)
    if y is None:
        y = torch.empty(x.shape, dtype=x.dtype, device=x.device)
    d1, d2 = _desc(x), _desc(y)
    _check(load().edge_leaky_relu(_ref(d1), _ref(d2), ctypes.c_float(slope), _stream(stream)))
    return y


def edge_leaky_relu_backward(x, dy, slope: float = 0.2, dx=None, stream=None):
    x, dy = _as3(x), _as3(dy)
    if dx is None:
        dx = torch.empty(x.shape, dtype=dy.dtype, device=dy.device)
    d1, d2, d3 = _desc(x), _desc(dy), _desc(dx)
    _check(load().edge_leaky_relu_backward(_ref(d1), _ref(d2), _ref(d3), ctypes.c_float(slope), _stream(stream)))
    return dx
