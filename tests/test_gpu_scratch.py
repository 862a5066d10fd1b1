"""Scratch memory lent by the caller (the boundary allocates nothing): a
compute call on a stream without a lent buffer returns GNNK_ENOMEM before
launching anything and reports what it needs; the bound of
graph_scratch_bytes covers every call kind; one handle serves two streams at
once, each with its own buffer, with every result equal to the oracle's."""
import ctypes

import numpy as np
import pytest
import torch

import oracle as orc
from paper_1909_01315_amd import gnnk, synth
from _gpu import Pair, assert_close, assert_exact, dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def reset_options():
    yield
    gnnk.set_option("seg_edges", 0)


@pytest.fixture(scope="module")
def sg2():
    return synth.graph_c2()


def hub_pair(sg):
    """c2 with 64-edge segments: its long rows need fp64 partials"""
    gnnk.set_option("seg_edges", 64)
    p = Pair.of(sg)
    info = p.g.info()
    assert info["segments_in"] > 0 and info["segments_out"] > 0
    return p


def test_call_without_scratch_fails_before_launching(sg2):
    p = hub_pair(sg2)
    lib = gnnk.load()
    X = synth.normal(synth.feat_seed(31), "X", (p.o.n_src, 1, 64))
    Xd = dev(X)
    out = torch.full((p.o.n_dst, 1, 64), 7.0, device="cuda")
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    call = lambda: lib.gspmm(p.g.handle, gnnk.OPS["copy_lhs"], gnnk.REDUCES["sum"], gnnk._ref(gnnk._desc(Xd)), None,
                             gnnk._ref(gnnk._desc(out)), None, None, s.cuda_stream)
    assert call() == gnnk.ENOMEM
    assert b"scratch" in lib.gnnk_last_error()
    need = ctypes.c_size_t(0)
    assert lib.gnnk_scratch_needed(ctypes.byref(need)) == gnnk.OK
    assert need.value >= p.g.info()["segments_in"] * 64 * 8
    torch.cuda.synchronize()
    assert bool((out == 7.0).all()), "nothing may run when the call is short of scratch"
    # a buffer one byte short of the need is still short
    buf = torch.empty(need.value, dtype=torch.uint8, device="cuda")
    assert lib.graph_attach_scratch(p.g.handle, s.cuda_stream, buf.data_ptr(), need.value - 1) == gnnk.OK
    assert call() == gnnk.ENOMEM
    assert lib.graph_attach_scratch(p.g.handle, s.cuda_stream, buf.data_ptr(), need.value) == gnnk.OK
    assert call() == gnnk.OK
    s.synchronize()
    assert_close(out, orc.gspmm(p.o, "copy_lhs", "sum", X), name="sum with the lent buffer")
    # the buffer is taken back; misaligned and oversubscribed attachments are refused
    assert lib.graph_attach_scratch(p.g.handle, s.cuda_stream, None, 0) == gnnk.OK
    assert call() == gnnk.ENOMEM
    assert lib.graph_attach_scratch(p.g.handle, s.cuda_stream, buf.data_ptr() + 8, 1024) == gnnk.EINVAL
    streams = [torch.cuda.Stream() for _ in range(17)]
    sts = [lib.graph_attach_scratch(p.g.handle, t.cuda_stream, buf.data_ptr(), 1024) for t in streams]
    assert sts[:16] == [gnnk.OK] * 16 and sts[16] == gnnk.EINVAL
    p.g.destroy()


@pytest.mark.parametrize("kind", ["max", "mul_sum", "dot"])
def test_multi_pass_call_short_of_scratch_runs_nothing(sg2, kind):
    """Calls made of several passes (the max backward's winner masks and the
    walk that reads them; dX and the edge gradient of u_mul_e/sum; the two
    node gradients of a dot) with a lent buffer too small for a later pass:
    GNNK_ENOMEM, the buffer untouched (no pass ran), and gnnk_scratch_needed()
    the whole call's need, with which the same call then succeeds."""
    p = hub_pair(sg2)
    lib = gnnk.load()
    s = torch.cuda.Stream()
    S = synth.feat_seed(32)
    X = synth.normal(S, "mX", (p.o.n_src, 1, 64))
    Y = synth.normal(S, "mY", (p.o.n_dst, 1, 64))
    W = synth.uniform(S, "mW", (p.o.n_edges, 1, 1), 0.5, 1.5)
    dZ = synth.normal(synth.grad_seed(32), "mdZ", (p.o.n_dst, 1, 64))
    dM = synth.normal(synth.grad_seed(32), "mdM", (p.o.n_edges, 1, 1))
    if kind == "max":
        _, _, ae = orc.gspmm(p.o, "copy_lhs", "max", X)
        ref, _ = orc.gspmm_backward(p.o, "copy_lhs", "max", X, None, dZ, arg_e=ae, want_rhs=False)
    elif kind == "mul_sum":
        ref = orc.gspmm_backward(p.o, "mul", "sum", X, W, dZ)
    else:
        ref = orc.gsddmm_backward(p.o, "dot", X, "u", Y, "v", dM)
    # the need of the whole call, from a call without any buffer
    lib.graph_attach_scratch(p.g.handle, s.cuda_stream, None, 0)
    g_handle = p.g.handle
    need = ctypes.c_size_t(0)
    if kind == "dot":
        Xd, Yd, dMd = dev(X), dev(Y), dev(dM)
        gl, gr = torch.empty_like(Xd), torch.empty_like(Yd)
        d = [gnnk._desc(t) for t in (Xd, Yd, dMd, gl, gr)]
        call = lambda: lib.gsddmm_backward(g_handle, gnnk.OPS["dot"], gnnk._ref(d[0]), gnnk.TARGETS["u"],
                                           gnnk._ref(d[1]), gnnk.TARGETS["v"], gnnk._ref(d[2]), gnnk._ref(d[3]),
                                           gnnk._ref(d[4]), s.cuda_stream)
    else:
        Xd, dZd = dev(X), dev(dZ)
        gl = torch.empty_like(Xd)
        if kind == "max":
            aed = dev(ae)
            d = [gnnk._desc(t) for t in (Xd, dZd, gl)]
            call = lambda: lib.gspmm_backward(g_handle, gnnk.OPS["copy_lhs"], gnnk.REDUCES["max"], gnnk._ref(d[0]),
                                              None, None, aed.data_ptr(), gnnk._ref(d[1]), gnnk._ref(d[2]), None,
                                              s.cuda_stream)
        else:
            Wd = dev(W)
            gw = torch.empty_like(Wd)
            d = [gnnk._desc(t) for t in (Xd, Wd, dZd, gl, gw)]
            call = lambda: lib.gspmm_backward(g_handle, gnnk.OPS["mul"], gnnk.REDUCES["sum"], gnnk._ref(d[0]),
                                              gnnk._ref(d[1]), None, None, gnnk._ref(d[2]), gnnk._ref(d[3]),
                                              gnnk._ref(d[4]), s.cuda_stream)
    torch.cuda.synchronize()
    assert call() == gnnk.ENOMEM
    assert lib.gnnk_scratch_needed(ctypes.byref(need)) == gnnk.OK
    assert need.value > 0
    # a buffer short by 4 KiB, filled with a pattern that no pass may touch
    short = need.value - 4096 if need.value > 4096 else 0
    if short > 0:
        buf = torch.full((short,), 0x5A, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        assert lib.graph_attach_scratch(g_handle, s.cuda_stream, buf.data_ptr(), short) == gnnk.OK
        assert call() == gnnk.ENOMEM
        n2 = ctypes.c_size_t(0)
        assert lib.gnnk_scratch_needed(ctypes.byref(n2)) == gnnk.OK and n2.value == need.value
        s.synchronize()
        assert bool((buf == 0x5A).all()), "no pass may run when the call is short of scratch"
    # exactly the reported need suffices, in one go
    full = torch.empty(need.value, dtype=torch.uint8, device="cuda")
    assert lib.graph_attach_scratch(g_handle, s.cuda_stream, full.data_ptr(), need.value) == gnnk.OK
    assert call() == gnnk.OK
    s.synchronize()
    if kind == "max":
        assert_close(gl, ref, name="max backward")
    elif kind == "mul_sum":
        assert_close(gl, ref[0], name="dX")
        assert_close(gw, ref[1], name="dW")
    else:
        assert_close(gl, ref[0], name="dX")
        assert_close(gr, ref[1], name="dY")
    lib.graph_attach_scratch(g_handle, s.cuda_stream, None, 0)
    p.g.destroy()


def test_one_handle_on_two_streams_at_once(sg2):
    """Calls of every scratch-using kind queued on two streams without any
    synchronisation between them (so their kernels overlap), each stream
    with a buffer of graph_scratch_bytes; no call asks for more, and every
    result equals the oracle's."""
    p = hub_pair(sg2)
    o, g = p.o, p.g
    N, H, F = o.n_src, 4, 16
    fs, gs = synth.feat_seed(32), synth.grad_seed(32)
    X1 = synth.normal(fs, "X1", (N, H, F))
    X2 = synth.normal(fs, "X2", (N, 1, H * F))
    a = synth.uniform(fs, "a", (o.n_edges, H, 1), 0.1, 1.0)
    el = synth.normal(fs, "el", (N, H, 1))
    er = synth.normal(fs, "er", (o.n_dst, H, 1))
    dz = synth.normal(gs, "dz", (o.n_dst, H, F))
    dm = synth.normal(gs, "dm", (o.n_dst, 1, H * F))
    d = {k: dev(v) for k, v in dict(X1=X1, X2=X2, a=a, el=el, er=er, dz=dz, dm=dm).items()}
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for s in (s1, s2):
        g.lend_scratch(g.scratch_bytes(H * F, argmax=True), s)
    lent = {k: v.data_ptr() for k, v in g._lent.items()}
    torch.cuda.synchronize()
    res1, res2 = [], []
    for _ in range(3):
        with torch.cuda.stream(s1):
            z = gnnk.gspmm(g, "mul", "sum", d["X1"], d["a"], stream=s1)
            dx, da = gnnk.gspmm_backward(g, "mul", "sum", d["X1"], d["a"], d["dz"], stream=s1)
            fo, st = gnnk.gat_aggregate(g, d["X1"], d["el"], d["er"], 0.2, want_stats=True, stream=s1)
            gf, gl, gr = gnnk.gat_aggregate_backward(g, d["X1"], d["el"], d["er"], 0.2, st, d["dz"], stream=s1)
            res1.append((z, dx, da, fo, gf, gl, gr))
        with torch.cuda.stream(s2):
            m, au, ae = gnnk.gspmm(g, "copy_lhs", "max", d["X2"], want_args=True, stream=s2)
            dxm, _ = gnnk.gspmm_backward(g, "copy_lhs", "max", d["X2"], None, d["dm"], arg_rhs=ae, stream=s2)
            mean = gnnk.gspmm(g, "copy_lhs", "mean", d["X2"], stream=s2)
            res2.append((m, ae, dxm, mean))
    torch.cuda.synchronize()
    assert {k: v.data_ptr() for k, v in g._lent.items()} == lent, "the bound covered every call"
    rz = orc.gspmm(o, "mul", "sum", X1, a)
    rdx, rda = orc.gspmm_backward(o, "mul", "sum", X1, a, dz)
    sc = orc.leaky_relu(orc.gsddmm(o, "add", el, "u", er, "v"), 0.2)
    att = orc.edge_softmax(o, sc)
    rfo = orc.gspmm(o, "mul", "sum", X1, att)
    s64 = orc.gsddmm(o, "add", el.astype(np.float64), "u", er.astype(np.float64), "v")
    att64 = orc.edge_softmax(o, orc.leaky_relu(s64, 0.2))
    rgf, _ = orc.gspmm_backward(o, "mul", "sum", X1.astype(np.float64), att64, dz.astype(np.float64),
                                want_rhs=False)
    rm, _, rae = orc.gspmm(o, "copy_lhs", "max", X2)
    rdxm, _ = orc.gspmm_backward(o, "copy_lhs", "max", X2, None, dm, arg_e=rae)
    rmean = orc.gspmm(o, "copy_lhs", "mean", X2)
    for z, dx, da, fo, gf, gl, gr in res1:
        assert_close(z, rz, name="s1 u_mul_e/sum")
        assert_close(dx, rdx, name="s1 dX")
        assert_close(da, rda, name="s1 d attention")
        assert_close(fo, rfo, name="s1 fused attention")
        assert_close(gf, rgf, name="s1 fused d feat")
        assert torch.equal(gl, res1[0][5]) and torch.equal(gr, res1[0][6])
    for m, ae, dxm, mean in res2:
        assert_exact(m, rm, "s2 max")
        assert_exact(ae, rae, "s2 arg edge")
        assert_close(dxm, rdxm, name="s2 argmax scatter")
        assert_close(mean, rmean, name="s2 mean")
    g.destroy()
