"""GPU parity: every entry point of the C ABI against the oracle, element by
element, on the small workloads (c1 uniform multigraph, c2 Chung-Lu GCN graph)
and on edge cases.  Tolerances are in tests/_gpu.py."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_1909_01315_amd import gnnk, synth
from _gpu import Pair, assert_close, assert_exact, check_formats, dev, host

pytestmark = pytest.mark.gpu

S1 = synth.feat_seed(1)
G1 = synth.grad_seed(1)


@pytest.fixture(scope="module")
def c1():
    return Pair.of(synth.graph_c1())


@pytest.fixture(scope="module")
def c2():
    sg = synth.graph_c2()
    p = Pair.of(sg)
    p.w = sg.extra["gcn_w"]
    return p


@pytest.fixture(autouse=True)
def reset_options():
    yield
    gnnk.set_option("seg_edges", 0)
    gnnk.set_option("no_split", 0)
    gnnk.set_option("small_deg", -1)
    gnnk.set_option("fused_dw", -1)
    gnnk.set_option("sddmm_split", 0)


def feats(seed, name, shape, lo=None, hi=None):
    if lo is None:
        return synth.normal(seed, name, shape)
    return synth.uniform(seed, name, shape, lo, hi)


# ---------------------------------------------------------------------------
# A0: graph formats


def test_graph_formats_c1_c2(c1, c2):
    check_formats(c1)
    check_formats(c2)


def test_graph_formats_bipartite_int64():
    sg = synth.uniform_graph(5, 300, 120, 4000)
    p = Pair.of(sg, ptr64=True)
    assert p.g.info()["ptr_type"] == gnnk.I64
    check_formats(p)


def test_graph_create_csr_with_edge_ids():
    """An in-CSR whose edge ids are a permutation: formats and a g-SpMM follow the ids."""
    rng = np.random.default_rng(3)
    n, E = 200, 3000
    src = rng.integers(0, n, E).astype(np.int32)
    dst = rng.integers(0, n, E).astype(np.int32)
    o = orc.OGraph(src, dst, n, n)
    indptr, indices, eids = orc.csr(o)
    # shuffle positions within each row so edge ids are not ascending
    for v in range(n):
        b, e = indptr[v], indptr[v + 1]
        perm = rng.permutation(e - b) + b
        indices[b:e] = indices[perm]
        eids[b:e] = eids[perm]
    g = gnnk.Graph.from_csr(dev(indptr), dev(indices), dev(eids), n)
    assert g.info()["identity_eids"] == 0
    gp, gi, ge = g.csr_export()
    assert_exact(gi, indices)
    assert_exact(ge, eids)
    rp, ri, re_ = orc.csr(o, reverse=True)
    hp, hi, he = g.csr_export(reverse=True)
    assert_exact(hi, ri)
    assert_exact(he, re_)
    X = feats(S1, "csrX", (n, 8))
    W = feats(S1, "csrW", (E, 1), 0.0, 1.0)
    out = gnnk.gspmm(g, "mul", "sum", dev(X), dev(W))
    assert_close(out, orc.gspmm(o, "mul", "sum", X, W))
    o2, au, ae = gnnk.gspmm(g, "copy_lhs", "max", dev(X), None, want_args=True)
    r2, rau, rae = orc.gspmm(o, "copy_lhs", "max", X)
    assert_exact(o2, r2)
    assert_exact(au, rau)
    assert_exact(ae, rae)
    M = gnnk.gsddmm(g, "dot", dev(X), "u", dev(X), "v")
    assert_close(M, orc.gsddmm(o, "dot", X, "u", X, "v"))


# ---------------------------------------------------------------------------
# A1 / A2: g-SpMM forward

OPS = ["copy_lhs", "copy_rhs", "add", "sub", "mul", "div"]


@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("reduce", ["sum", "mean"])
@pytest.mark.parametrize("wshape", [(1, 1), (1, 16), (4, 1), (4, 4)])
def test_gspmm_sum_mean_c1(c1, op, reduce, wshape):
    E, N = c1.o.n_edges, c1.o.n_src
    xh, xf = (1, 16) if wshape[0] == 1 else (4, 4)
    X = feats(S1, "X", (N, xh, xf))
    W = feats(S1, f"W{wshape}", (E,) + wshape, 0.5, 1.5)
    L = X if op != "copy_rhs" else None
    R = W if op != "copy_lhs" else None
    ref = orc.gspmm(c1.o, op, reduce, L, R)
    out = gnnk.gspmm(c1.g, op, reduce, dev(L) if L is not None else None, dev(R) if R is not None else None)
    assert_close(out, ref, name=f"{op}/{reduce}")


def test_copy_u_sum_of_ones_is_in_degree_bit_exact(c1, c2):
    for p in (c1, c2):
        ones = torch.ones((p.o.n_src, 1, 4), dtype=torch.float32, device="cuda")
        out = gnnk.gspmm(p.g, "copy_lhs", "sum", ones)
        ind, _ = orc.degrees(p.o)
        assert_exact(out[:, 0, 0], ind.astype(np.float32))


@pytest.mark.parametrize("D", [16, 64, 256, 512])
def test_gspmm_gcn_c2(c2, D):
    X = feats(synth.feat_seed(2), f"X{D}", (c2.o.n_src, D))
    ref = orc.gspmm(c2.o, "mul", "sum", X, c2.w)
    out = gnnk.gspmm(c2.g, "mul", "sum", dev(X), dev(c2.w))
    assert_close(out, ref, name=f"c2 D={D}")


@pytest.fixture(scope="module")
def hot():
    """300 nodes, 4,000 edges, a third of them into destination 7 and a
    quarter out of source 3 (rows of a thousand edges: hub segments)"""
    rng = np.random.default_rng(44)
    E = 4000
    src = rng.integers(0, 300, E).astype(np.int32)
    dst = rng.integers(0, 300, E).astype(np.int32)
    dst[rng.random(E) < 0.33] = 7
    src[rng.random(E) < 0.25] = 3
    return Pair(src, dst, 300, 300)


@pytest.mark.parametrize("H,F", [(1, 512), (1, 300), (2, 256), (8, 40), (3, 129), (4, 100)])
@pytest.mark.parametrize("seg", [0, 64])
def test_sums_over_rows_wider_than_a_wavefront(hot, H, F, seg):
    """Sums over the features of rows wider than one pass of 64 lanes: the
    u_dot_v score, the edge-weight gradient of u_mul_e/sum with a weight per
    edge and per head (also for max, through the winner masks), the node
    gradient of a per-head node operand, and the g-SDDMM backward of a dot;
    with the automatic segment size and with 64-edge hub segments (fp32 and a
    bf16 case)."""
    gnnk.set_option("seg_edges", seg)
    p = Pair(hot.o.src, hot.o.dst, 300, 300) if seg else hot
    o, g = p.o, p.g
    S = synth.feat_seed(40)
    X = feats(S, f"wX{H}{F}", (o.n_src, H, F))
    Y = feats(S, f"wY{H}{F}", (o.n_dst, H, F))
    dM = feats(G1, f"wdM{H}", (o.n_edges, H, 1))
    M = orc.gsddmm(o, "dot", X, "u", Y, "v")
    assert_close(gnnk.gsddmm(g, "dot", dev(X), "u", dev(Y), "v"), M, name="dot")
    gl, gr = orc.gsddmm_backward(o, "dot", X, "u", Y, "v", dM)
    dl, dr = gnnk.gsddmm_backward(g, "dot", dev(X), "u", dev(Y), "v", dev(dM))
    assert_close(dl, gl, name="dot grad lhs")
    assert_close(dr, gr, name="dot grad rhs")
    dZ = feats(G1, f"wdZ{H}{F}", (o.n_dst, H, F))
    for wshape in ((H, 1), (1, 1)):
        W = feats(S, f"wW{wshape}", (o.n_edges,) + wshape, 0.5, 1.5)
        for red in ("sum", "mean", "max"):
            ae = None
            if red == "max":
                _, _, ae = orc.gspmm(o, "mul", red, X, W)
            rl, rr = orc.gspmm_backward(o, "mul", red, X, W, dZ, arg_e=ae)
            ql, qr = gnnk.gspmm_backward(g, "mul", red, dev(X), dev(W), dev(dZ),
                                         arg_rhs=dev(ae) if ae is not None else None)
            assert_close(ql, rl, name=f"grad x {wshape} {red}")
            assert_close(qr, rr, name=f"grad w {wshape} {red}")
    # a per-head node operand times a full edge operand: its gradient sums
    # each head's F columns on the reverse graph
    Ln = feats(S, f"wL{H}", (o.n_src, H, 1))
    We = feats(S, f"wWe{H}{F}", (o.n_edges, H, F), 0.5, 1.5)
    rl, rr = orc.gspmm_backward(o, "div", "sum", Ln, We, dZ)
    ql, qr = gnnk.gspmm_backward(g, "div", "sum", dev(Ln), dev(We), dev(dZ))
    assert_close(ql, rl, name="grad per-head node operand")
    assert_close(qr, rr, name="grad full edge operand")
    if H == 2 and seg == 0:
        Xb, Yb = synth.to_bf16_bits(X), synth.to_bf16_bits(Y)
        assert_close(gnnk.gsddmm(g, "dot", dev(Xb), "u", dev(Yb), "v"), orc.gsddmm(o, "dot", Xb, "u", Yb, "v"),
                     kind="bf16", name="bf16 dot")


@pytest.mark.parametrize("op,reduce", [("copy_lhs", "max"), ("copy_lhs", "min"), ("mul", "max"), ("add", "min"),
                                       ("sub", "max"), ("div", "min"), ("copy_rhs", "max")])
@pytest.mark.parametrize("wshape", [(1, 1), (1, 16)])
def test_gspmm_max_min_c1(c1, op, reduce, wshape):
    E, N = c1.o.n_edges, c1.o.n_src
    X = feats(S1, "Xm", (N, 1, 16))
    W = feats(S1, f"Wm{wshape}", (E,) + wshape, 0.5, 1.5)
    L = X if op != "copy_rhs" else None
    R = W if op != "copy_lhs" else None
    ref, rau, rae = orc.gspmm(c1.o, op, reduce, L, R)
    out, au, ae = gnnk.gspmm(c1.g, op, reduce, dev(L) if L is not None else None,
                             dev(R) if R is not None else None, want_args=True)
    assert_exact(out, ref, "value")
    assert_exact(ae, rae, "arg edge")
    assert_exact(au, rau, "arg node")


def test_max_ties_from_multi_edges(c1):
    """Duplicated edges give exactly equal messages: the smaller edge id must win."""
    X = np.round(feats(S1, "Xt", (c1.o.n_src, 1, 16)) * 2).astype(np.float32)  # many exact ties
    ref, rau, rae = orc.gspmm(c1.o, "copy_lhs", "max", X)
    out, au, ae = gnnk.gspmm(c1.g, "copy_lhs", "max", dev(X), want_args=True)
    assert_exact(out, ref)
    assert_exact(ae, rae)


@pytest.mark.parametrize("ident", [True, False])
@pytest.mark.parametrize("seg", [0, 64])
@pytest.mark.parametrize("D", [16, 100, 300, 512])
def test_argmax_scatter_masks(hot, ident, seg, D):
    """The max/min backward's winner masks, built row by row when edge ids are
    the in-CSR positions (the hot graph's edges sorted by destination) and by
    winning column otherwise: hub rows cut into 64-edge segments (seg 64) or
    whole, and mask widths of one to sixteen words (partial blocks of four):
    the gradient against the oracle."""
    gnnk.set_option("seg_edges", seg)
    src, dst = hot.o.src, hot.o.dst
    if ident:
        order = np.argsort(dst, kind="stable")
        src, dst = src[order], dst[order]
    p = Pair(src, dst, 300, 300)
    assert p.g.info()["identity_eids"] == int(ident)
    X = feats(S1, f"amX{D}", (300, 1, D))
    dZ = feats(G1, f"amdZ{D}", (300, 1, D))
    for red in ("max", "min"):
        _, _, ae = orc.gspmm(p.o, "copy_lhs", red, X)
        ref, _ = orc.gspmm_backward(p.o, "copy_lhs", red, X, None, dZ, arg_e=ae, want_rhs=False)
        dX, _ = gnnk.gspmm_backward(p.g, "copy_lhs", red, dev(X), None, dev(dZ), arg_rhs=dev(ae))
        assert_close(dX, ref, name=f"{red} D={D}")


# ---------------------------------------------------------------------------
# A3: g-SDDMM forward

TARGET_PAIRS = [("u", "v"), ("u", "e"), ("e", "v"), ("v", "u"), ("u", "u"), ("e", "e"), ("v", "e")]


@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("lt,rt", TARGET_PAIRS)
def test_gsddmm_elementwise_bit_exact(c1, op, lt, rt):
    rows = {"u": c1.o.n_src, "e": c1.o.n_edges, "v": c1.o.n_dst}
    L = feats(S1, f"L{lt}", (rows[lt], 4, 4))
    R = feats(S1, f"R{rt}", (rows[rt], 4, 1), 0.5, 1.5)
    Lx = L if op != "copy_rhs" else None
    Rx = R if op != "copy_lhs" else None
    ref = orc.gsddmm(c1.o, op, Lx, lt, Rx, rt)
    out = gnnk.gsddmm(c1.g, op, dev(Lx) if Lx is not None else None, lt, dev(Rx) if Rx is not None else None, rt)
    assert_exact(out, ref, f"{lt}_{op}_{rt}")


# F / 4 lanes per head: 4, 2, 1, (13 columns: one per lane), 8, 16, 32
@pytest.mark.parametrize("shape", [(1, 16), (2, 8), (4, 4), (1, 13), (2, 32), (1, 64), (1, 128)])
@pytest.mark.parametrize("lt,rt", [("u", "v"), ("u", "e"), ("v", "u")])
def test_gsddmm_dot(c1, shape, lt, rt):
    rows = {"u": c1.o.n_src, "e": c1.o.n_edges, "v": c1.o.n_dst}
    L = feats(S1, f"dL{lt}", (rows[lt],) + shape)
    R = feats(S1, f"dR{rt}", (rows[rt],) + shape)
    ref = orc.gsddmm(c1.o, "dot", L, lt, R, rt)
    out = gnnk.gsddmm(c1.g, "dot", dev(L), lt, dev(R), rt)
    assert_close(out, ref, name="dot")


@pytest.mark.parametrize("shapes", [((2, 32), (2, 1)), ((1, 64), (1, 1)), ((8, 16), (8, 1)), ((8, 16), (1, 1))])
@pytest.mark.parametrize("seg", [2048, 64])
@pytest.mark.parametrize("fused", [1, 0, -1])
def test_edge_gradient_in_the_reverse_pass_is_bit_identical(shapes, seg, fused):
    """u_mul_e/sum backward with both gradients: with the option fused_dw = 1
    the edge-weight gradient is computed inside the reverse pass (64+
    columns), with 0 (and alone) it is a g-SDDMM, with -1 (the default) the
    first for one weight per edge and the second for per-head weights.  Both sum the same fp64 products
    in the same lane order: bit-identical."""
    gnnk.set_option("seg_edges", seg)
    gnnk.set_option("fused_dw", fused)
    sg = synth.graph_c2()
    p = Pair.of(sg)
    (xh, xf), (wh, wf) = shapes
    X = feats(S1, f"fX{xh}{xf}", (p.o.n_src, xh, xf))
    W = feats(S1, f"fW{wh}", (p.o.n_edges, wh, wf), 0.5, 1.5)
    dZ = feats(G1, f"fdZ{xh}{xf}", (p.o.n_dst, xh, xf))
    dX, dW = gnnk.gspmm_backward(p.g, "mul", "sum", dev(X), dev(W), dev(dZ))
    _, dW1 = gnnk.gspmm_backward(p.g, "mul", "sum", dev(X), dev(W), dev(dZ), want_lhs=False)
    assert torch.equal(dW, dW1)
    _, ref = orc.gspmm_backward(p.o, "mul", "sum", X, W, dZ, want_lhs=False)
    assert_close(dW, ref, name="edge gradient")
    gl, _ = orc.gspmm_backward(p.o, "mul", "sum", X, W, dZ, want_rhs=False)
    assert_close(dX, gl, name="dX")


@pytest.mark.parametrize("split", [1, 2, 3, 4, 8])
@pytest.mark.parametrize("seg", [512, 64])
def test_gsddmm_hub_segments_split_across_wavefronts(hot, split, seg):
    """A hub segment of a g-SDDMM shared by several wavefronts, each taking
    whole batches of it (the parts past the segment's end are empty): the
    same results as one wavefront per segment, bit for bit where the oracle's
    result is one rounding"""
    gnnk.set_option("seg_edges", seg)
    p = Pair(hot.o.src, hot.o.dst, 300, 300)
    gnnk.set_option("sddmm_split", split)
    el = feats(S1, "el", (300, 8, 1))
    er = feats(S1, "er", (300, 8, 1))
    assert_exact(gnnk.gsddmm(p.g, "add", dev(el), "u", dev(er), "v"), orc.gsddmm(p.o, "add", el, "u", er, "v"),
                 "u_add_v")
    X = feats(S1, "X", (300, 2, 32))
    Y = feats(S1, "Y", (300, 2, 32))
    assert_exact(gnnk.gsddmm(p.g, "mul", dev(X), "u", dev(Y), "v"), orc.gsddmm(p.o, "mul", X, "u", Y, "v"), "u_mul_v")
    assert_close(gnnk.gsddmm(p.g, "dot", dev(X), "u", dev(Y), "v"), orc.gsddmm(p.o, "dot", X, "u", Y, "v"),
                 name="u_dot_v")


@pytest.mark.parametrize("H,F", [(4, 3), (1, 12), (2, 6), (3, 4), (1, 3), (2, 8), (1, 20)])
@pytest.mark.parametrize("fused", [0, -1])
def test_whole_row_sums_of_a_partial_run(hot, H, F, fused):
    """The gradient of a one-value edge weight sums dZ[v] . X[u] over the whole
    row.  Rows of three vectors (12 fp32 columns, 3 columns) fill three lanes
    of a run of four: the fourth lane must add nothing and still store its
    slot's edge (a case found by the random cases)"""
    gnnk.set_option("fused_dw", fused)
    X = feats(S1, "X", (300, H, F))
    W = feats(S1, "W", (hot.o.n_edges, 1, 1), 0.5, 1.5)
    dZ = feats(S1, "dZ", (300, H, F))
    _, gr = orc.gspmm_backward(hot.o, "mul", "sum", X, W, dZ, want_lhs=False)
    _, dr = gnnk.gspmm_backward(hot.g, "mul", "sum", dev(X), dev(W), dev(dZ), want_lhs=False)
    assert_close(dr, gr, name=f"dW ({H}, {F})")


def test_gsddmm_u_add_v_scores(c1):
    el = feats(S1, "el", (c1.o.n_src, 4, 1))
    er = feats(S1, "er", (c1.o.n_dst, 4, 1))
    assert_exact(gnnk.gsddmm(c1.g, "add", dev(el), "u", dev(er), "v"), orc.gsddmm(c1.o, "add", el, "u", er, "v"))


# ---------------------------------------------------------------------------
# A4 / A5 / A9: edge softmax and leaky ReLU


@pytest.mark.parametrize("H", [1, 4, 8])
def test_edge_softmax_c1(c1, H):
    s = feats(S1, f"s{H}", (c1.o.n_edges, H, 1))
    assert_close(gnnk.edge_softmax(c1.g, dev(s)), orc.edge_softmax(c1.o, s), name="softmax")
    a = orc.edge_softmax(c1.o, s)
    gout = feats(G1, f"gs{H}", (c1.o.n_edges, H, 1))
    ds = gnnk.edge_softmax_backward(c1.g, dev(a), dev(gout))
    assert_close(ds, orc.edge_softmax_backward(c1.o, a, gout), name="softmax backward")


def assert_close_nan(gpu, ref, name):
    """NaN exactly where the oracle has NaN (a destination whose scores are
    all -inf: 0 / 0), the fp32 tolerance elsewhere"""
    g = host(gpu).reshape(np.shape(ref)) if isinstance(gpu, torch.Tensor) else gpu
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(g), nan), f"{name}: NaN positions differ"
    assert_close(np.where(nan, 0.0, g).astype(np.float32), np.where(nan, 0.0, ref).astype(np.float32), name=name)


@pytest.mark.parametrize("seg", [0, 64])
@pytest.mark.parametrize("H", [1, 4])
def test_edge_softmax_masked_scores(c2, seg, H):
    """Scores of -inf (masked edges) get attention 0; a destination with
    every score masked gets NaN (0 / 0) as the definition gives.  seg 64
    sends the rows of more than 64 in-edges to the hub-row blocks."""
    gnnk.set_option("seg_edges", seg)
    p = Pair(c2.o.src, c2.o.dst, c2.o.n_src, c2.o.n_dst)
    E = c2.o.n_edges
    rng = np.random.default_rng(4400 + H)
    s = feats(synth.feat_seed(2), f"ms{H}", (E, H, 1))
    s[rng.random((E, H, 1)) < 0.4] = -np.inf
    ind = np.bincount(c2.o.dst, minlength=c2.o.n_dst)
    ptr = np.concatenate([[0], np.cumsum(ind)])
    big = np.argsort(-ind, kind="stable")[:3]
    for v in big[:2]:                    # whole rows masked, one a hub row
        s[ptr[v]:ptr[v + 1]] = -np.inf
    v = big[2]                           # a hub row with one finite score in its middle
    s[ptr[v]:ptr[v + 1]] = -np.inf
    s[(ptr[v] + ptr[v + 1]) // 2] = 0.5
    ref = orc.edge_softmax(c2.o, s)
    assert np.isnan(ref).any() and (ref == 0.0).any()
    assert_close_nan(gnnk.edge_softmax(p.g, dev(s)), ref, name="masked softmax")
    assert_close(gnnk.edge_softmax(p.g, dev(s))[ptr[v]:ptr[v + 1]], ref[ptr[v]:ptr[v + 1]], name="one finite score")
    # the backward of the masked attention (zeros, and no NaN rows)
    a = np.where(np.isnan(ref), 0.0, ref).astype(np.float32)
    gout = feats(synth.grad_seed(2), f"mg{H}", (E, H, 1))
    assert_close(gnnk.edge_softmax_backward(p.g, dev(a), dev(gout)), orc.edge_softmax_backward(c2.o, a, gout),
                 name="masked softmax backward")


@pytest.mark.parametrize("seg", [0, 64])
def test_gat_aggregate_masked_sources(c2, seg):
    """Fused attention with el = -inf for some (source, head) pairs: every
    out-edge of such a source scores -inf in that head (attention 0); a
    destination whose in-edges are all masked in a head gets NaN there, as
    the oracle's chain gives."""
    gnnk.set_option("seg_edges", seg)
    p = Pair(c2.o.src, c2.o.dst, c2.o.n_src, c2.o.n_dst)
    N, H, F = c2.o.n_src, 4, 8
    fs = synth.feat_seed(2)
    feat = feats(fs, "mfeat", (N, H, F))
    el = feats(fs, "mel", (N, H, 1))
    er = feats(fs, "mer", (c2.o.n_dst, H, 1))
    el[np.random.default_rng(4500).random((N, H, 1)) < 0.5] = -np.inf
    sc = orc.leaky_relu(orc.gsddmm(c2.o, "add", el, "u", er, "v"), 0.2)
    a = orc.edge_softmax(c2.o, sc)
    ref = orc.gspmm(c2.o, "mul", "sum", feat, a)
    assert np.isnan(ref).any()
    out, attn = gnnk.gat_aggregate(p.g, dev(feat), dev(el), dev(er), 0.2, want_attn=True)
    assert_close_nan(attn, a, name="masked fused attention")
    assert_close_nan(out, ref, name="masked fused output")


def test_leaky_relu_bit_exact(c1):
    x = feats(S1, "lx", (c1.o.n_edges, 4, 1))
    x[:7] = 0.0
    dy = feats(G1, "ldy", (c1.o.n_edges, 4, 1))
    assert_exact(gnnk.edge_leaky_relu(dev(x), 0.2), orc.leaky_relu(x, 0.2))
    assert_exact(gnnk.edge_leaky_relu_backward(dev(x), dev(dy), 0.2), orc.leaky_relu_backward(x, dy, 0.2))


# ---------------------------------------------------------------------------
# A6 / A7: g-SpMM backward


@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("reduce", ["sum", "mean", "max", "min"])
# ((2, 32), (2, 1)) and ((1, 64), (1, 1)): the edge gradient sums 8 and 16
# lanes per head (the DPP steps of the lane reductions)
@pytest.mark.parametrize("shapes", [((1, 16), (1, 1)), ((1, 16), (1, 16)), ((4, 4), (4, 1)), ((4, 1), (4, 4)),
                                    ((2, 32), (2, 1)), ((1, 64), (1, 1))])
def test_gspmm_backward_c1(c1, op, reduce, shapes):
    (xh, xf), (wh, wf) = shapes
    if op == "copy_lhs":
        wh, wf = xh, xf
    if op == "copy_rhs":
        xh, xf = wh, wf
    E, N = c1.o.n_edges, c1.o.n_src
    X = feats(S1, f"bX{xh}{xf}", (N, xh, xf))
    W = feats(S1, f"bW{wh}{wf}", (E, wh, wf), 0.5, 1.5)
    L = X if op != "copy_rhs" else None
    R = W if op != "copy_lhs" else None
    Ld = dev(L) if L is not None else None
    Rd = dev(R) if R is not None else None
    H, F = max(xh, wh), max(xf, wf)
    dZ = feats(G1, f"dZ{H}{F}", (c1.o.n_dst, H, F))
    ae = None
    if reduce in ("max", "min"):
        _, _, rae = orc.gspmm(c1.o, op, reduce, L, R)
        ae = rae
        _, _, gae = gnnk.gspmm(c1.g, op, reduce, Ld, Rd, want_args=True)
        assert_exact(gae, rae)
    gl, gr = orc.gspmm_backward(c1.o, op, reduce, L, R, dZ, arg_e=ae)
    dl, dr = gnnk.gspmm_backward(c1.g, op, reduce, Ld, Rd, dev(dZ), arg_rhs=dev(ae) if ae is not None else None)
    if gl is not None:
        assert_close(dl, gl, name="grad_lhs")
    if gr is not None:
        assert_close(dr, gr, name="grad_rhs")


# ---------------------------------------------------------------------------
# A8: g-SDDMM backward


@pytest.mark.parametrize("op", OPS + ["dot"])
@pytest.mark.parametrize("lt,rt", TARGET_PAIRS)
def test_gsddmm_backward_c1(c1, op, lt, rt):
    rows = {"u": c1.o.n_src, "e": c1.o.n_edges, "v": c1.o.n_dst}
    L = feats(S1, f"gL{lt}", (rows[lt], 2, 8))
    R = feats(S1, f"gR{rt}", (rows[rt], 2, 1 if op != "dot" else 8), 0.5, 1.5)
    Lx = L if op != "copy_rhs" else None
    Rx = R if op != "copy_lhs" else None
    H, F = 2, 8
    gshape = (c1.o.n_edges, H, 1 if op == "dot" else F)
    if op == "copy_rhs":
        gshape = (c1.o.n_edges,) + R.shape[1:]
    dM = feats(G1, f"dM{gshape}", gshape)
    gl, gr = orc.gsddmm_backward(c1.o, op, Lx, lt, Rx, rt, dM)
    dl, dr = gnnk.gsddmm_backward(c1.g, op, dev(Lx) if Lx is not None else None, lt,
                                  dev(Rx) if Rx is not None else None, rt, dev(dM))
    if gl is not None:
        assert_close(dl, gl, name="grad_lhs")
    if gr is not None:
        assert_close(dr, gr, name="grad_rhs")


# ---------------------------------------------------------------------------
# A10: schedules (node- vs edge-balanced) agree; hub segments; determinism


@pytest.mark.parametrize("setting", [("seg_edges", 64), ("seg_edges", 32), ("seg_edges", 2048), ("no_split", 1),
                                     ("small_deg", 0), ("small_deg", 64)])
def test_schedules_agree_c2(c2, setting):
    key, val = setting
    gnnk.set_option(key, val)
    p = Pair(c2.o.src, c2.o.dst, c2.o.n_src, c2.o.n_dst)
    info = p.g.info()
    if key == "seg_edges" and val < 2048:
        assert info["hub_dst_rows"] > 0 and info["segments_in"] > info["hub_dst_rows"]
    if key == "seg_edges" and val == 2048:
        assert info["hub_dst_rows"] == 0  # c2's largest in-degree is 985
    X = feats(synth.feat_seed(2), "sX", (c2.o.n_src, 1, 64))
    ref = orc.gspmm(c2.o, "mul", "sum", X, c2.w)
    assert_close(gnnk.gspmm(p.g, "mul", "sum", dev(X), dev(c2.w)), ref, name=f"{setting} sum")
    rm, rau, rae = orc.gspmm(c2.o, "copy_lhs", "max", X)
    m, au, ae = gnnk.gspmm(p.g, "copy_lhs", "max", dev(X), want_args=True)
    assert_exact(m, rm)
    assert_exact(ae, rae)
    mean = gnnk.gspmm(p.g, "copy_lhs", "mean", dev(X))
    assert_close(mean, orc.gspmm(c2.o, "copy_lhs", "mean", X), name="mean")
    s = feats(synth.feat_seed(2), "ss", (c2.o.n_edges, 2, 1))
    a = orc.edge_softmax(c2.o, s)
    assert_close(gnnk.edge_softmax(p.g, dev(s)), a, name="softmax")
    gs = feats(synth.grad_seed(2), "gss", (c2.o.n_edges, 2, 1))
    assert_close(gnnk.edge_softmax_backward(p.g, dev(a), dev(gs)), orc.edge_softmax_backward(c2.o, a, gs),
                 name="softmax bwd")
    dZ = feats(synth.grad_seed(2), "sdZ", (c2.o.n_dst, 1, 64))
    gl, gr = orc.gspmm_backward(c2.o, "mul", "sum", X, c2.w, dZ)
    dl, dr = gnnk.gspmm_backward(p.g, "mul", "sum", dev(X), dev(c2.w), dev(dZ))
    assert_close(dl, gl, name="dX")
    assert_close(dr, gr, name="dW")
    M = gnnk.gsddmm(p.g, "dot", dev(X), "u", dev(X), "v")
    assert_close(M, orc.gsddmm(c2.o, "dot", X, "u", X, "v"), name="dot")


def test_determinism_with_hub_segments(c2):
    gnnk.set_option("seg_edges", 32)
    p = Pair(c2.o.src, c2.o.dst, c2.o.n_src, c2.o.n_dst)
    X = dev(feats(synth.feat_seed(2), "detX", (c2.o.n_src, 1, 64)))
    W = dev(c2.w)
    a = gnnk.gspmm(p.g, "mul", "sum", X, W).clone()
    b = gnnk.gspmm(p.g, "mul", "sum", X, W).clone()
    assert torch.equal(a, b)
    dZ = dev(feats(synth.grad_seed(2), "detdZ", (c2.o.n_dst, 1, 64)))
    d1 = gnnk.gspmm_backward(p.g, "mul", "sum", X, W, dZ)[0].clone()
    d2 = gnnk.gspmm_backward(p.g, "mul", "sum", X, W, dZ)[0].clone()
    assert torch.equal(d1, d2)


# ---------------------------------------------------------------------------
# bf16, row strides, edge cases, errors


def test_bf16_c1(c1):
    N, E = c1.o.n_src, c1.o.n_edges
    X = synth.to_bf16_bits(feats(S1, "bfX", (N, 1, 16)))
    W = synth.to_bf16_bits(feats(S1, "bfW", (E, 1, 1), 0.5, 1.5))
    for op, L, R in (("copy_lhs", X, None), ("mul", X, W)):
        for red in ("sum", "mean"):
            ref = orc.gspmm(c1.o, op, red, L, R)
            out = gnnk.gspmm(c1.g, op, red, dev(L), dev(R) if R is not None else None)
            assert out.dtype == torch.bfloat16
            assert_close(out, ref, kind="bf16", name=f"bf16 {op}/{red}")
    ref, rau, rae = orc.gspmm(c1.o, "copy_lhs", "max", X)
    out, au, ae = gnnk.gspmm(c1.g, "copy_lhs", "max", dev(X), want_args=True)
    assert_exact(out, ref)
    assert_exact(ae, rae)
    M = gnnk.gsddmm(c1.g, "dot", dev(X), "u", dev(X), "v")
    assert_close(M, orc.gsddmm(c1.o, "dot", X, "u", X, "v"), kind="bf16")
    dZ = synth.to_bf16_bits(feats(G1, "bfdZ", (N, 1, 16)))
    gl, _ = orc.gspmm_backward(c1.o, "copy_lhs", "sum", X, None, dZ)
    dl, _ = gnnk.gspmm_backward(c1.g, "copy_lhs", "sum", dev(X), None, dev(dZ))
    assert_close(dl, gl, kind="bf16")
    gl, _ = orc.gspmm_backward(c1.o, "copy_lhs", "max", X, None, dZ, arg_e=rae)
    dl, _ = gnnk.gspmm_backward(c1.g, "copy_lhs", "max", dev(X), None, dev(dZ), arg_rhs=ae)
    assert_close(dl, gl, kind="bf16")
    s = synth.to_bf16_bits(feats(S1, "bfs", (E, 8, 1)))
    assert_close(gnnk.edge_softmax(c1.g, dev(s)), orc.edge_softmax(c1.o, s), kind="bf16")


@pytest.mark.parametrize("pad", [4, 2, 1])
def test_padded_row_stride(c1, pad):
    N = c1.o.n_src
    full = feats(S1, f"pad{pad}", (N, 16 + pad))
    X = full[:, :16]
    W = feats(S1, "padW", (c1.o.n_edges, 1), 0.5, 1.5)
    Xd = dev(full)[:, :16]
    ref = orc.gspmm(c1.o, "mul", "sum", np.ascontiguousarray(X), W)
    assert_close(gnnk.gspmm(c1.g, "mul", "sum", Xd, dev(W)), ref)
    out_full = torch.zeros((N, 16 + pad), device="cuda")
    gnnk.gspmm(c1.g, "mul", "sum", Xd, dev(W), out=out_full[:, :16].unsqueeze(1))
    assert_close(out_full[:, :16], ref[:, 0, :])
    assert torch.all(out_full[:, 16:] == 0)


def test_empty_graph():
    p = Pair(np.zeros(0, np.int32), np.zeros(0, np.int32), 5, 7)
    X = torch.ones((5, 1, 8), device="cuda")
    assert torch.all(gnnk.gspmm(p.g, "copy_lhs", "sum", X) == 0)
    assert torch.all(gnnk.gspmm(p.g, "copy_lhs", "mean", X) == 0)
    m, au, ae = gnnk.gspmm(p.g, "copy_lhs", "max", X, want_args=True)
    assert torch.all(m == 0) and torch.all(au == -1) and torch.all(ae == -1)
    assert gnnk.gsddmm(p.g, "dot", X, "u", torch.ones((7, 1, 8), device="cuda"), "v").shape == (0, 1, 1)
    dl, _ = gnnk.gspmm_backward(p.g, "copy_lhs", "sum", X, None, torch.ones((7, 1, 8), device="cuda"))
    assert torch.all(dl == 0)
    p.g.validate()


def test_single_node_self_loops_and_isolated():
    src = np.array([0, 0, 0, 2], np.int32)
    dst = np.array([0, 0, 2, 2], np.int32)
    p = Pair(src, dst, 4, 4)
    X = feats(S1, "tinyX", (4, 1, 3))
    assert_close(gnnk.gspmm(p.g, "copy_lhs", "mean", dev(X)), orc.gspmm(p.o, "copy_lhs", "mean", X))
    s = feats(S1, "tinys", (4, 1, 1))
    a = host(gnnk.edge_softmax(p.g, dev(s)))
    assert_close(a, orc.edge_softmax(p.o, s))


def test_bipartite_relational_small():
    """The relational encoding: num_src = R * N, source id etype * N + src."""
    rng = np.random.default_rng(9)
    n, r, E = 50, 5, 600
    src = rng.integers(0, n, E)
    et = rng.integers(0, r, E)
    dst = rng.integers(0, n, E).astype(np.int32)
    comp = (et * n + src).astype(np.int32)
    p = Pair(comp, dst, n * r, n)
    X = feats(S1, "relX", (n * r, 1, 64))
    W = feats(S1, "relW", (E, 1, 1), 0.1, 1.0)
    assert_close(gnnk.gspmm(p.g, "mul", "sum", dev(X), dev(W)), orc.gspmm(p.o, "mul", "sum", X, W))
    dZ = feats(G1, "reldZ", (n, 1, 64))
    M = gnnk.gsddmm(p.g, "dot", dev(X), "u", dev(dZ), "v")
    assert_close(M, orc.gsddmm(p.o, "dot", X, "u", dZ, "v"))
    check_formats(p)


def test_invalid_arguments(c1):
    X = torch.ones((c1.o.n_src, 1, 16), device="cuda")
    with pytest.raises(gnnk.GnnkError) as e:
        gnnk.gspmm(c1.g, "dot", "sum", X, X)
    assert e.value.status == gnnk.EINVAL
    with pytest.raises(gnnk.GnnkError):
        gnnk.gspmm(c1.g, "mul", "sum", X, torch.ones((c1.o.n_edges, 3, 1), device="cuda"))
    with pytest.raises(gnnk.GnnkError):
        gnnk.gspmm(c1.g, "copy_lhs", "sum", X[:-1])
    with pytest.raises(gnnk.GnnkError) as e:
        gnnk.gspmm(c1.g, "copy_lhs", "sum", X, want_args=True)
    assert e.value.status == gnnk.EUNSUPPORTED
    with pytest.raises(gnnk.GnnkError):
        gnnk.gspmm_backward(c1.g, "copy_lhs", "max", X, None, torch.ones((c1.o.n_dst, 1, 16), device="cuda"))
    with pytest.raises(gnnk.GnnkError):
        gnnk.gsddmm(c1.g, "add", X, "u", X.to(torch.bfloat16), "v")
