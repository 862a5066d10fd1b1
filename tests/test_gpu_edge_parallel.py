"""GPU parity of the forced schedules against the oracle: the row engine
(schedule 1) and the edge-parallel (COO) walks, deterministic (2) and with
fp64 atomics for split rows (3), for g-SpMM sum and mean, g-SDDMM and the
backward passes built on them, with sub-chunks small enough that many rows
cross sub-chunk boundaries.  Every schedule must match the oracle (the
paper's Table 1: both parallelisations are valid for these reducers); the
automatic choice (schedule 0) is covered by every other parity test."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_1909_01315_amd import gnnk, synth
from _gpu import Pair, assert_close, assert_exact, dev

pytestmark = pytest.mark.gpu

S = synth.feat_seed(11)
GS = synth.grad_seed(11)
OPS = ["copy_lhs", "copy_rhs", "add", "sub", "mul", "div"]
SCHEDULES = [1, 2, 3]


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
    gnnk.set_option("schedule", 0)
    gnnk.set_option("edge_chunk", 0)


def feats(seed, name, shape, lo=None, hi=None):
    return synth.normal(seed, name, shape) if lo is None else synth.uniform(seed, name, shape, lo, hi)


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("chunk", [0, 8, 36])
@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("reduce", ["sum", "mean"])
def test_gspmm_edge_parallel_c1(c1, schedule, chunk, op, reduce):
    gnnk.set_option("schedule", schedule)
    gnnk.set_option("edge_chunk", chunk)
    E, N = c1.o.n_edges, c1.o.n_src
    X = feats(S, "X", (N, 4, 4))
    W = feats(S, "W", (E, 4, 1), 0.5, 1.5)
    L = X if op != "copy_rhs" else None
    R = W if op != "copy_lhs" else None
    ref = orc.gspmm(c1.o, op, reduce, L, R)
    out = gnnk.gspmm(c1.g, op, reduce, dev(L) if L is not None else None, dev(R) if R is not None else None)
    assert_close(out, ref, name=f"{op}/{reduce} schedule {schedule} chunk {chunk}")


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("D", [16, 64, 100, 256, 512])
@pytest.mark.parametrize("chunk", [0, 64])
def test_gspmm_gcn_edge_parallel_c2(c2, schedule, D, chunk):
    gnnk.set_option("schedule", schedule)
    gnnk.set_option("edge_chunk", chunk)
    X = feats(synth.feat_seed(2), f"X{D}", (c2.o.n_src, D))
    ref = orc.gspmm(c2.o, "mul", "sum", X, c2.w)
    out = gnnk.gspmm(c2.g, "mul", "sum", dev(X), dev(c2.w))
    assert_close(out, ref, name=f"c2 D={D} schedule {schedule}")
    ones = torch.ones((c2.o.n_src, 1, 4), dtype=torch.float32, device="cuda")
    deg = gnnk.gspmm(c2.g, "copy_lhs", "sum", ones)
    ind, _ = orc.degrees(c2.o)
    assert_exact(deg[:, 0, 0], ind.astype(np.float32), "in-degree")


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("op", ["copy_lhs", "mul", "div", "sub"])
@pytest.mark.parametrize("reduce", ["sum", "mean"])
def test_gspmm_backward_edge_parallel_c1(c1, schedule, op, reduce):
    gnnk.set_option("schedule", schedule)
    gnnk.set_option("edge_chunk", 16)
    E, N = c1.o.n_edges, c1.o.n_src
    X = feats(S, "bX", (N, 1, 16))
    W = feats(S, "bW", (E, 1, 16 if op == "copy_lhs" else 1), 0.5, 1.5)
    L, R = X, (W if op != "copy_lhs" else None)
    dZ = feats(GS, "bdZ", (c1.o.n_dst, 1, 16))
    gl, gr = orc.gspmm_backward(c1.o, op, reduce, L, R, dZ)
    dl, dr = gnnk.gspmm_backward(c1.g, op, reduce, dev(L), dev(R) if R is not None else None, dev(dZ))
    assert_close(dl, gl, name="grad_lhs")
    if gr is not None:
        assert_close(dr, gr, name="grad_rhs")


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("shape", [(2, 32), (1, 64), (1, 128)])
def test_gsddmm_dot_wide_heads_c1(c1, schedule, shape):
    """dot products reduced over 8, 16 and 32 lanes per head"""
    gnnk.set_option("schedule", schedule)
    L = feats(S, f"wL{shape}", (c1.o.n_src,) + shape)
    R = feats(S, f"wR{shape}", (c1.o.n_dst,) + shape)
    assert_close(gnnk.gsddmm(c1.g, "dot", dev(L), "u", dev(R), "v"), orc.gsddmm(c1.o, "dot", L, "u", R, "v"),
                 name=f"dot {shape}")


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("op", ["add", "sub", "mul", "div", "dot", "copy_lhs"])
@pytest.mark.parametrize("lt,rt", [("u", "v"), ("v", "u"), ("u", "e"), ("e", "v")])
def test_gsddmm_edge_parallel_c1(c1, schedule, op, lt, rt):
    gnnk.set_option("schedule", schedule)
    gnnk.set_option("edge_chunk", 12)
    rows = {"u": c1.o.n_src, "e": c1.o.n_edges, "v": c1.o.n_dst}
    L = feats(S, f"sL{lt}", (rows[lt], 2, 8))
    R = feats(S, f"sR{rt}", (rows[rt], 2, 8), 0.5, 1.5)
    Rx = R if op != "copy_lhs" else None
    ref = orc.gsddmm(c1.o, op, L, lt, Rx, rt)
    out = gnnk.gsddmm(c1.g, op, dev(L), lt, dev(Rx) if Rx is not None else None, rt)
    if op in ("dot",):
        assert_close(out, ref, name=f"{op} {lt}{rt}")
    else:
        assert_exact(out, ref, name=f"{op} {lt}{rt}")


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_gsddmm_backward_and_gat_chain_edge_parallel_c2(c2, schedule):
    gnnk.set_option("schedule", schedule)
    X = feats(synth.feat_seed(2), "gX", (c2.o.n_src, 8, 16))
    dM = feats(synth.grad_seed(2), "gdM", (c2.o.n_edges, 8, 1))
    gl, gr = orc.gsddmm_backward(c2.o, "dot", X, "u", X, "v", dM)
    dl, dr = gnnk.gsddmm_backward(c2.g, "dot", dev(X), "u", dev(X), "v", dev(dM))
    assert_close(dl, gl, name="d lhs")
    assert_close(dr, gr, name="d rhs")
    a = orc.edge_softmax(c2.o, feats(synth.feat_seed(2), "gs", (c2.o.n_edges, 8, 1)))
    Z = gnnk.gspmm(c2.g, "mul", "sum", dev(X), dev(a))
    assert_close(Z, orc.gspmm(c2.o, "mul", "sum", X, a), name="attention aggregation")


def test_edge_parallel_deterministic_c2(c2):
    gnnk.set_option("schedule", 2)
    gnnk.set_option("edge_chunk", 32)
    X = dev(feats(synth.feat_seed(2), "dX", (c2.o.n_src, 1, 64)))
    W = dev(c2.w)
    a = gnnk.gspmm(c2.g, "mul", "sum", X, W).clone()
    b = gnnk.gspmm(c2.g, "mul", "sum", X, W).clone()
    assert torch.equal(a, b)


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_edge_parallel_edge_cases(schedule):
    gnnk.set_option("schedule", schedule)
    # isolated nodes, a single hub row, self-loops, bipartite, int64 offsets
    src = np.array([0, 0, 1, 2, 2, 2, 2, 5, 5, 3], dtype=np.int32)
    dst = np.array([4, 4, 4, 4, 1, 0, 4, 4, 2, 4], dtype=np.int32)
    for n_src, n_dst, ptr64 in ((6, 7, False), (6, 7, True)):
        p = Pair(src, dst, n_src, n_dst, ptr64=ptr64)
        X = feats(S, "ecX", (n_src, 1, 8))
        for reduce in ("sum", "mean"):
            for chunk in (4, 8, 0):
                gnnk.set_option("edge_chunk", chunk)
                assert_close(gnnk.gspmm(p.g, "copy_lhs", reduce, dev(X)), orc.gspmm(p.o, "copy_lhs", reduce, X))
        assert_close(gnnk.gsddmm(p.g, "dot", dev(X), "u", dev(feats(S, "ecY", (n_dst, 1, 8))), "v"),
                     orc.gsddmm(p.o, "dot", X, "u", feats(S, "ecY", (n_dst, 1, 8)), "v"))
    empty = Pair(np.zeros(0, np.int32), np.zeros(0, np.int32), 3, 4)
    z = gnnk.gspmm(empty.g, "copy_lhs", "sum", dev(feats(S, "ezX", (3, 1, 8))))
    assert_exact(z, np.zeros((4, 1, 8), np.float32))


def test_edge_parallel_bf16_c1(c1):
    gnnk.set_option("schedule", 2)
    gnnk.set_option("edge_chunk", 20)
    N, E = c1.o.n_src, c1.o.n_edges
    X = synth.to_bf16_bits(feats(S, "bfX", (N, 1, 16)))
    W = synth.to_bf16_bits(feats(S, "bfW", (E, 1, 1), 0.5, 1.5))
    ref = orc.gspmm(c1.o, "mul", "sum", X, W)
    out = gnnk.gspmm(c1.g, "mul", "sum", dev(X), dev(W))
    assert_close(out, ref, kind="bf16")
