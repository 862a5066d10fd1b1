"""Autograd functions and layers (paper_1909_01315_amd.nn) against plain
PyTorch references of the same computations in float64 (index_add /
scatter_reduce over the edge list), forward and backward, and the memory
property of fused message passing: no tensor of E x D elements is formed.

Tolerances: single primitives as everywhere (1e-5 relative + 1e-6 absolute);
chains of primitives (GAT), whose fp32 intermediates are rounded between
steps, 1e-4 relative + 1e-5 absolute; gradients of dense layer weights, which
torch forms with fp32 matrix products over every node, 1e-4 relative + 1e-5
of the largest entry."""
import numpy as np
import pytest
import torch

from paper_1909_01315_amd import gnnk, nn, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


class G:
    """a graph on the GPU (gnnk handle) and its edge list in torch"""

    def __init__(self, src, dst, n_src, n_dst):
        self.src = torch.from_numpy(np.ascontiguousarray(src)).long()
        self.dst = torch.from_numpy(np.ascontiguousarray(dst)).long()
        self.n_src, self.n_dst = n_src, n_dst
        self.h = gnnk.Graph.from_coo(self.src.int().to(DEV), self.dst.int().to(DEV), n_src, n_dst)


@pytest.fixture(scope="module")
def c1():
    sg = synth.graph_c1()
    return G(sg.src, sg.dst, sg.n_src, sg.n_dst)


@pytest.fixture(scope="module")
def c2():
    sg = synth.graph_c2()
    return G(sg.src, sg.dst, sg.n_src, sg.n_dst)


def close(a, b, rel=1e-5, ab=1e-6, name=""):
    a = a.detach().double().cpu()
    b = b.detach().double().cpu()
    assert a.shape == b.shape, (a.shape, b.shape)
    bad = (a - b).abs() > ab + rel * b.abs()
    assert not bad.any(), f"{name}: {int(bad.sum())} of {bad.numel()} out of tolerance, max err {(a - b).abs().max()}"


# ---- plain references (float64, CPU) --------------------------------------


def bcast(t):
    return t if t.dim() == 3 else t.view(t.shape[0], 1, -1)


def phi(op, x, w):
    return {"copy_lhs": lambda: x, "copy_rhs": lambda: w, "add": lambda: x + w, "sub": lambda: x - w,
            "mul": lambda: x * w, "div": lambda: x / w}[op]()


def ref_gspmm(g, op, reduce, X, W):
    x = X[g.src] if X is not None else None
    m = phi(op, x, W)
    out = torch.zeros((g.n_dst,) + m.shape[1:], dtype=m.dtype)
    if reduce in ("sum", "mean"):
        out = out.index_add(0, g.dst, m)
        if reduce == "mean":
            deg = torch.bincount(g.dst, minlength=g.n_dst).clamp(min=1).to(m.dtype)
            out = out / deg.view(-1, *([1] * (m.dim() - 1)))
        return out
    idx = g.dst.view(-1, *([1] * (m.dim() - 1))).expand_as(m)
    red = out.scatter_reduce(0, idx, m, "amax" if reduce == "max" else "amin", include_self=False)
    has = torch.bincount(g.dst, minlength=g.n_dst) > 0
    return torch.where(has.view(-1, *([1] * (m.dim() - 1))), red, torch.zeros_like(red))


def at(g, t, target):
    return {"u": lambda: t[g.src], "v": lambda: t[g.dst], "e": lambda: t}[target]()


def ref_gsddmm(g, op, L, lt, R, rt):
    l = at(g, L, lt) if L is not None else None
    r = at(g, R, rt) if R is not None else None
    if op == "dot":
        return (l * r).sum(-1, keepdim=True)
    return phi(op, l, r)


def ref_softmax(g, s):
    idx = g.dst.view(-1, 1, 1).expand_as(s)
    mx = torch.full((g.n_dst,) + s.shape[1:], -torch.inf, dtype=s.dtype).scatter_reduce(0, idx, s, "amax")
    ex = torch.exp(s - mx[g.dst])
    den = torch.zeros((g.n_dst,) + s.shape[1:], dtype=s.dtype).index_add(0, g.dst, ex)
    return ex / den[g.dst]


def leaf(t, dev):
    return t.detach().to(dev).requires_grad_(True)


# ---- functions -------------------------------------------------------------


@pytest.mark.parametrize("op", ["copy_lhs", "copy_rhs", "add", "sub", "mul", "div"])
@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_gspmm_autograd(c1, c2, op, reduce):
    # max/min on c2 (no multi-edges): torch splits the gradient of tied
    # maxima, the library gives it to the smallest edge id
    if reduce == "max":
        c1 = c2
    torch.manual_seed(0)
    X = torch.randn(c1.n_src, 2, 8, dtype=torch.float32)
    W = torch.rand(len(c1.src), 2, 1, dtype=torch.float32) + 0.5
    Gout = torch.randn(c1.n_dst, 2, 8, dtype=torch.float64)
    Xg, Wg = leaf(X, DEV), leaf(W, DEV)
    out = nn.gspmm(c1.h, op, reduce, Xg if op != "copy_rhs" else None, Wg if op != "copy_lhs" else None)
    if op == "copy_rhs":
        Gout = torch.randn(c1.n_dst, 2, 1, dtype=torch.float64)
    (out.double() * Gout.to(DEV)).sum().backward()
    Xr, Wr = leaf(X.double(), "cpu"), leaf(W.double(), "cpu")
    ref = ref_gspmm(c1, op, reduce, Xr if op != "copy_rhs" else None, Wr if op != "copy_lhs" else None)
    (ref * Gout).sum().backward()
    close(out, ref, name="forward")
    if op != "copy_rhs":
        close(Xg.grad, Xr.grad, name="dX")
    if op != "copy_lhs":
        close(Wg.grad, Wr.grad, name="dW")


@pytest.mark.parametrize("op", ["add", "sub", "mul", "div", "dot"])
@pytest.mark.parametrize("lt,rt", [("u", "v"), ("u", "e"), ("v", "u")])
def test_gsddmm_autograd(c1, op, lt, rt):
    torch.manual_seed(1)
    rows = {"u": c1.n_src, "v": c1.n_dst, "e": len(c1.src)}
    L = torch.randn(rows[lt], 2, 8)
    R = torch.rand(rows[rt], 2, 8) + 0.5
    Lg, Rg = leaf(L, DEV), leaf(R, DEV)
    out = nn.gsddmm(c1.h, op, Lg, lt, Rg, rt)
    Gout = torch.randn(out.shape, dtype=torch.float64)
    (out.double() * Gout.to(DEV)).sum().backward()
    Lr, Rr = leaf(L.double(), "cpu"), leaf(R.double(), "cpu")
    ref = ref_gsddmm(c1, op, Lr, lt, Rr, rt)
    (ref * Gout).sum().backward()
    close(out, ref, name="forward")
    close(Lg.grad, Lr.grad, name="dL")
    close(Rg.grad, Rr.grad, name="dR")


def test_edge_softmax_and_leaky_autograd(c1):
    torch.manual_seed(2)
    s = torch.randn(len(c1.src), 4, 1)
    sg = leaf(s, DEV)
    a = nn.edge_softmax(c1.h, nn.leaky_relu(sg, 0.2))
    Gout = torch.randn(a.shape, dtype=torch.float64)
    (a.double() * Gout.to(DEV)).sum().backward()
    sr = leaf(s.double(), "cpu")
    ar = ref_softmax(c1, torch.nn.functional.leaky_relu(sr, 0.2))
    (ar * Gout).sum().backward()
    close(a, ar, name="softmax")
    close(sg.grad, sr.grad, rel=1e-4, ab=1e-5, name="d score")


# ---- layers ----------------------------------------------------------------


def copy_params(dst_mod, src_mod):
    with torch.no_grad():
        for (n1, p1), (n2, p2) in zip(dst_mod.named_parameters(), src_mod.named_parameters()):
            assert n1 == n2
            p1.copy_(p2.double().cpu())


def test_graphconv_and_sage(c2):
    torch.manual_seed(3)
    X = torch.randn(c2.n_src, 32)
    w = nn.gcn_norm(c2.h, c2.src.int().to(DEV), c2.dst.int().to(DEV))
    for kind in ("gcn", "sage"):
        layer = (nn.GraphConv(32, 16) if kind == "gcn" else nn.SAGEConv(32, 16)).to(DEV)
        ref_layer = (nn.GraphConv(32, 16) if kind == "gcn" else nn.SAGEConv(32, 16)).double()
        copy_params(ref_layer, layer)
        Xg = leaf(X, DEV)
        out = layer(c2.h, Xg, w) if kind == "gcn" else layer(c2.h, Xg)
        Gout = torch.randn(out.shape, dtype=torch.float64)
        (out.double() * Gout.to(DEV)).sum().backward()
        Xr = leaf(X.double(), "cpu")
        if kind == "gcn":
            h = ref_layer.linear(Xr).view(c2.n_src, 1, -1)
            ref = ref_gspmm(c2, "mul", "sum", h, w.double().cpu()).view(c2.n_dst, -1) + ref_layer.bias
        else:
            hn = ref_gspmm(c2, "copy_lhs", "mean", Xr.view(c2.n_src, 1, -1), None).view(c2.n_dst, -1)
            ref = ref_layer.fc_self(Xr) + ref_layer.fc_neigh(hn)
        (ref * Gout).sum().backward()
        close(out, ref, rel=1e-4, ab=1e-5, name=f"{kind} forward")
        close(Xg.grad, Xr.grad, rel=1e-4, ab=1e-5, name=f"{kind} dX")
        for (n, p), (_, pr) in zip(layer.named_parameters(), ref_layer.named_parameters()):
            close(p.grad, pr.grad, rel=1e-4, ab=1e-5 * float(pr.grad.abs().max()), name=f"{kind} d{n}")


def test_gatconv(c2):
    torch.manual_seed(4)
    X = torch.randn(c2.n_src, 24)
    layer = nn.GATConv(24, 16, 8).to(DEV)
    ref_layer = nn.GATConv(24, 16, 8).double()
    copy_params(ref_layer, layer)
    Xg = leaf(X, DEV)
    out, a = layer(c2.h, Xg, return_attention=True)
    Gout = torch.randn(out.shape, dtype=torch.float64)
    (out.double() * Gout.to(DEV)).sum().backward()
    Xr = leaf(X.double(), "cpu")
    feat = ref_layer.fc(Xr).view(-1, 8, 16)
    el = (feat * ref_layer.attn_l).sum(-1, keepdim=True)
    er = (feat * ref_layer.attn_r).sum(-1, keepdim=True)
    s = torch.nn.functional.leaky_relu(el[c2.src] + er[c2.dst], 0.2)
    ar = ref_softmax(c2, s)
    ref = torch.zeros(c2.n_dst, 8, 16, dtype=torch.float64).index_add(0, c2.dst, feat[c2.src] * ar)
    (ref * Gout).sum().backward()
    close(a, ar, rel=1e-4, ab=1e-5, name="attention")
    close(out, ref, rel=1e-4, ab=1e-5, name="gat forward")
    close(Xg.grad, Xr.grad, rel=1e-4, ab=1e-5, name="gat dX")
    for (n, p), (_, pr) in zip(layer.named_parameters(), ref_layer.named_parameters()):
        close(p.grad, pr.grad, rel=1e-4, ab=1e-5 * float(pr.grad.abs().max()), name=f"gat d{n}")


def test_relgraphconv_bipartite():
    rng = np.random.default_rng(5)
    N, E, R = 300, 4000, 6
    src = rng.integers(0, N, E).astype(np.int32)
    dst = np.sort(rng.integers(0, N, E)).astype(np.int32)
    et = rng.integers(0, R, E).astype(np.int32)
    bsrc = (et.astype(np.int64) * N + src).astype(np.int32)
    g = G(bsrc, dst, R * N, N)
    norm = nn.rel_norm(torch.from_numpy(et).to(DEV), torch.from_numpy(dst).to(DEV), R, N)
    torch.manual_seed(5)
    X = torch.randn(N, 12)
    layer = nn.RelGraphConv(12, 10, R).to(DEV)
    ref_layer = nn.RelGraphConv(12, 10, R).double()
    copy_params(ref_layer, layer)
    Xg = leaf(X, DEV)
    out = layer(g.h, Xg, norm)
    Gout = torch.randn(out.shape, dtype=torch.float64)
    (out.double() * Gout.to(DEV)).sum().backward()
    Xr = leaf(X.double(), "cpu")
    # the formula itself: sum_r D_r^-1 A_r X W_r + X W_0 + b
    ref = ref_layer.loop(Xr)
    etl = torch.from_numpy(et).long()
    srcl, dstl = torch.from_numpy(src).long(), torch.from_numpy(dst).long()
    for r in range(R):
        m = etl == r
        cnt = torch.bincount(dstl[m], minlength=N).clamp(min=1).double()
        agg = torch.zeros(N, 12, dtype=torch.float64).index_add(0, dstl[m], Xr[srcl[m]])
        ref = ref + (agg / cnt.view(-1, 1)) @ ref_layer.weight[r]
    (ref * Gout).sum().backward()
    close(out, ref, rel=1e-4, ab=1e-5, name="rgcn forward")
    close(Xg.grad, Xr.grad, rel=1e-4, ab=1e-5, name="rgcn dX")
    close(layer.weight.grad, ref_layer.weight.grad, rel=1e-4, ab=1e-5 * float(ref_layer.weight.grad.abs().max()),
          name="rgcn dW")


def test_fused_message_passing_never_materialises_edge_messages():
    """GAT forward + backward with E x D = 2M x 128: the peak of allocated
    device memory above the inputs stays far below one E x D fp32 tensor."""
    rng = np.random.default_rng(6)
    N, E, H, F = 20000, 2_000_000, 8, 16
    src = rng.integers(0, N, E).astype(np.int32)
    dst = np.sort(rng.integers(0, N, E)).astype(np.int32)
    g = G(src, dst, N, N)
    layer = nn.GATConv(H * F, F, H).to(DEV)
    X = torch.randn(N, H * F, device=DEV, requires_grad=True)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    out = layer(g.h, X)
    out.sum().backward()
    torch.cuda.synchronize()
    peak = torch.cuda.max_memory_allocated() - base
    ed_bytes = E * H * F * 4
    assert peak < 0.5 * ed_bytes, f"peak {peak / 1e6:.0f} MB vs E x D x 4 = {ed_bytes / 1e6:.0f} MB"
