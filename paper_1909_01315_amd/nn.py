"""Autograd functions and message-passing layers on the gnnk primitives.

Section 3 of the paper reduces every message-passing layer to g-SDDMM and
g-SpMM, and Theorem 1 makes their gradients operators of the same two kinds;
Section 4.2 lets the framework own the tensors.  This module is that
framework side: torch.autograd.Function wrappers whose forward and backward
both call the HIP library (no message tensor of E x D elements is ever formed,
which is the memory saving of fused message passing the paper reports), and
the aggregation layers of the paper's experiments built from them:

  GraphConv     GCN, symmetric normalisation, u_mul_e/sum
  SAGEConv      GraphSAGE with mean aggregation, copy_u/mean
  GATConv       multi-head attention: u_add_v -> leaky ReLU -> edge softmax ->
                u_mul_e/sum (the chain of Appendix E)
  RelGraphConv  R-GCN aggregation: per-relation transformed source rows
                gathered by (relation, source) on a bipartite encoding and
                summed with 1/in-degree-per-relation weights

Dense projections (the node-wise update) are ordinary torch layers.  Graph
handles come from gnnk.Graph; the caller keeps them alive while tensors that
depend on them are in use.
"""
from __future__ import annotations

import math

import torch

from . import gnnk


def _c(t):
    return t.contiguous() if t is not None else None


class _GSpMM(torch.autograd.Function):
    @staticmethod
    def forward(ctx, g, op, reduce, lhs, rhs):
        cmp = reduce in ("max", "min")
        if cmp:
            out, _, arg_e = gnnk.gspmm(g, op, reduce, lhs, rhs, want_args=True)
        else:
            out, arg_e = gnnk.gspmm(g, op, reduce, lhs, rhs), None
        ctx.g, ctx.op, ctx.reduce = g, op, reduce
        ctx.save_for_backward(lhs, rhs, arg_e)
        if arg_e is not None:
            ctx.mark_non_differentiable(arg_e)
        return out

    @staticmethod
    def backward(ctx, dz):
        lhs, rhs, arg_e = ctx.saved_tensors
        want_l = lhs is not None and ctx.needs_input_grad[3]
        want_r = rhs is not None and ctx.needs_input_grad[4]
        if not (want_l or want_r):
            return None, None, None, None, None
        dl, dr = gnnk.gspmm_backward(ctx.g, ctx.op, ctx.reduce, lhs, rhs, _c(dz), arg_rhs=arg_e, want_lhs=want_l,
                                     want_rhs=want_r)
        if dl is not None and lhs.dim() != dl.dim():
            dl = dl.view(lhs.shape)
        if dr is not None and rhs.dim() != dr.dim():
            dr = dr.view(rhs.shape)
        return None, None, None, dl, dr


class _GSDDMM(torch.autograd.Function):
    @staticmethod
    def forward(ctx, g, op, lhs, lhs_target, rhs, rhs_target):
        out = gnnk.gsddmm(g, op, lhs, lhs_target, rhs, rhs_target)
        ctx.g, ctx.op, ctx.lt, ctx.rt = g, op, lhs_target, rhs_target
        ctx.save_for_backward(lhs, rhs)
        return out

    @staticmethod
    def backward(ctx, dm):
        lhs, rhs = ctx.saved_tensors
        want_l = lhs is not None and ctx.needs_input_grad[2]
        want_r = rhs is not None and ctx.needs_input_grad[4]
        if not (want_l or want_r):
            return None, None, None, None, None, None
        dl, dr = gnnk.gsddmm_backward(ctx.g, ctx.op, lhs, ctx.lt, rhs, ctx.rt, _c(dm), want_lhs=want_l,
                                      want_rhs=want_r)
        if dl is not None and lhs.dim() != dl.dim():
            dl = dl.view(lhs.shape)
        if dr is not None and rhs.dim() != dr.dim():
            dr = dr.view(rhs.shape)
        return None, None, dl, None, dr, None


class _EdgeSoftmax(torch.autograd.Function):
    @staticmethod
    def forward(ctx, g, score):
        a = gnnk.edge_softmax(g, score)
        ctx.g = g
        ctx.save_for_backward(a)
        return a

    @staticmethod
    def backward(ctx, da):
        (a,) = ctx.saved_tensors
        return None, gnnk.edge_softmax_backward(ctx.g, a, _c(da)).view(a.shape)


class _LeakyReLU(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, slope):
        ctx.slope = slope
        ctx.save_for_backward(x)
        return gnnk.edge_leaky_relu(x, slope).view(x.shape)

    @staticmethod
    def backward(ctx, dy):
        (x,) = ctx.saved_tensors
        return gnnk.edge_leaky_relu_backward(x, _c(dy).view(x.shape), ctx.slope).view(x.shape), None


class _FusedGAT(torch.autograd.Function):
    """gat_aggregate forward (one pass per destination) keeping only the
    per-row statistics (max score, 1 / sum); backward by
    gat_aggregate_backward, which recomputes the attention from them, so no
    tensor of E x H elements is formed in either direction.  Both this
    backward and the unfused one need H * F / vector width <= 64 (the
    attention gradient is a per-head reduction across one lane group)."""

    @staticmethod
    def forward(ctx, g, feat, el, er, slope):
        out, stats = gnnk.gat_aggregate(g, feat, el, er, slope, want_stats=True)
        ctx.g, ctx.slope = g, slope
        ctx.save_for_backward(feat, el, er, stats)
        return out

    @staticmethod
    def backward(ctx, dout):
        feat, el, er, stats = ctx.saved_tensors
        g = ctx.g
        nf = ctx.needs_input_grad
        dfeat, d_el, d_er = gnnk.gat_aggregate_backward(g, feat, el, er, ctx.slope, stats, _c(dout),
                                                        want_feat=nf[1], want_el=nf[2], want_er=nf[3])
        view = lambda t, like: t.view(like.shape) if t is not None else None
        return None, view(dfeat, feat), view(d_el, el), view(d_er, er), None


# ---------------------------------------------------------------------------
# functional API (same names and argument order as the C ABI)


def gspmm(g, op: str, reduce: str, lhs=None, rhs=None):
    """Differentiable g-SpMM: out[v] = reduce over in-edges of op(lhs[u], rhs[e])."""
    return _GSpMM.apply(g, op, reduce, _c(lhs), _c(rhs))


def gsddmm(g, op: str, lhs, lhs_target: str, rhs, rhs_target: str):
    """Differentiable g-SDDMM: out[e] = op(lhs at its target, rhs at its target)."""
    return _GSDDMM.apply(g, op, _c(lhs), lhs_target, _c(rhs), rhs_target)


def edge_softmax(g, score):
    """Differentiable softmax over the in-edges of each destination."""
    return _EdgeSoftmax.apply(g, _c(score))


def leaky_relu(x, slope: float = 0.2):
    """Differentiable leaky ReLU computed by the library's edge kernel."""
    return _LeakyReLU.apply(_c(x), float(slope))


def gat_aggregate(g, feat, el, er, slope: float = 0.2):
    """Differentiable fused attention aggregation (gat_aggregate)."""
    return _FusedGAT.apply(g, _c(feat), _c(el), _c(er), float(slope))


def degrees(g):
    """(in_degree, out_degree) int32 device tensors."""
    return g.in_degrees(), g.out_degrees()


def gcn_norm(g, src, dst):
    """Edge weights 1/sqrt(outdeg(src) * indeg(dst)) (GCN's symmetric
    normalisation, degrees with multi-edges counted), shape (E, 1, 1)."""
    indeg, outdeg = degrees(g)
    w = torch.rsqrt(outdeg[src.long()].double().clamp(min=1) * indeg[dst.long()].double().clamp(min=1))
    return w.float().view(-1, 1, 1)


# ---------------------------------------------------------------------------
# layers


class GraphConv(torch.nn.Module):
    """GCN layer: H' = A_norm (H W) + b, with A_norm's weights given per edge
    (gcn_norm) and the aggregation a u_mul_e/sum g-SpMM."""

    def __init__(self, in_feats: int, out_feats: int, bias: bool = True):
        super().__init__()
        self.linear = torch.nn.Linear(in_feats, out_feats, bias=False)
        self.bias = torch.nn.Parameter(torch.zeros(out_feats)) if bias else None

    def forward(self, g, x, edge_weight):
        h = self.linear(x).view(x.shape[0], 1, -1)
        out = gspmm(g, "mul", "sum", h, edge_weight).view(g.num_dst, -1)
        return out + self.bias if self.bias is not None else out


class SAGEConv(torch.nn.Module):
    """GraphSAGE with mean aggregation: H' = H W_self + mean_{u in N(v)} H_u W_neigh."""

    def __init__(self, in_feats: int, out_feats: int, bias: bool = True):
        super().__init__()
        self.fc_self = torch.nn.Linear(in_feats, out_feats, bias=bias)
        self.fc_neigh = torch.nn.Linear(in_feats, out_feats, bias=False)

    def forward(self, g, x):
        h_neigh = gspmm(g, "copy_lhs", "mean", x.view(x.shape[0], 1, -1)).view(g.num_dst, -1)
        return self.fc_self(x[: g.num_dst]) + self.fc_neigh(h_neigh)


class GATConv(torch.nn.Module):
    """Multi-head graph attention: per-head scores el[u] + er[v] (u_add_v),
    leaky ReLU, softmax over in-edges, and the attention-weighted sum of the
    projected source features (u_mul_e/sum) -- the chain of Appendix E."""

    def __init__(self, in_feats: int, out_feats: int, num_heads: int, negative_slope: float = 0.2,
                 fused: bool = False):
        super().__init__()
        self.H, self.F = num_heads, out_feats
        self.fused = fused  # one-pass gat_aggregate in forward
        self.fc = torch.nn.Linear(in_feats, out_feats * num_heads, bias=False)
        self.attn_l = torch.nn.Parameter(torch.empty(1, num_heads, out_feats))
        self.attn_r = torch.nn.Parameter(torch.empty(1, num_heads, out_feats))
        self.slope = negative_slope
        gain = math.sqrt(2.0)
        torch.nn.init.xavier_normal_(self.fc.weight, gain=gain)
        torch.nn.init.xavier_normal_(self.attn_l, gain=gain)
        torch.nn.init.xavier_normal_(self.attn_r, gain=gain)

    def forward(self, g, x, return_attention: bool = False):
        feat = self.fc(x).view(-1, self.H, self.F)
        el = (feat * self.attn_l).sum(-1, keepdim=True)  # (N, H, 1)
        er = (feat[: g.num_dst] * self.attn_r).sum(-1, keepdim=True)
        if self.fused and not return_attention:
            return gat_aggregate(g, feat, el, er, self.slope)
        s = leaky_relu(gsddmm(g, "add", el, "u", er, "v"), self.slope)  # (E, H, 1)
        a = edge_softmax(g, s)
        out = gspmm(g, "mul", "sum", feat, a)  # (N_dst, H, F)
        return (out, a) if return_attention else out


class RelGraphConv(torch.nn.Module):
    """R-GCN aggregation (the formula of Appendix D, experiment configurations): for each
    relation r, sum over r-edges into v of W_r h_u / |N_r(v)|, plus a self
    term.  The per-relation products W_r h_u are computed densely for all
    (r, u) and gathered by the g-SpMM on the bipartite graph whose source id
    is r * N + u; the 1 / |N_r(v)| weights are the edge operand."""

    def __init__(self, in_feats: int, out_feats: int, num_rels: int, self_loop: bool = True):
        super().__init__()
        self.R = num_rels
        self.weight = torch.nn.Parameter(torch.empty(num_rels, in_feats, out_feats))
        torch.nn.init.xavier_uniform_(self.weight, gain=math.sqrt(2.0))
        self.loop = torch.nn.Linear(in_feats, out_feats, bias=True) if self_loop else None

    def forward(self, g_rel, x, norm):
        # g_rel: bipartite handle with num_src = R * N; norm: (E, 1, 1)
        xr = torch.matmul(x.unsqueeze(0), self.weight).reshape(self.R * x.shape[0], 1, -1)  # (R, N, out)
        out = gspmm(g_rel, "mul", "sum", xr, norm).view(g_rel.num_dst, -1)
        return out + self.loop(x[: g_rel.num_dst]) if self.loop is not None else out


def rel_norm(etype, dst, num_rels: int, num_dst: int):
    """1 / |{e': dst_e' = dst_e, etype_e' = etype_e}| per edge, (E, 1, 1) fp32."""
    key = dst.long() * num_rels + etype.long()
    cnt = torch.bincount(key, minlength=num_rels * num_dst)
    return (1.0 / cnt[key].double()).float().view(-1, 1, 1)
