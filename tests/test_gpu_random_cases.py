"""Seeded random cases: every entry point against the oracle on graphs and
settings drawn together, so that combinations no hand-written case lists
are still covered.  Each case draws

  - a graph: 1-200 sources and destinations, 0-3000 edges, sometimes a hot
    source and a hot destination (hub rows), sometimes sorted by destination
    (identity edge ids), int32 or int64 offsets, built from the edge list or
    from the in-CSR (with or without explicit edge ids);
  - library options: hub segment size, small-row threshold, schedule
    (row engine, edge-parallel ordered, edge-parallel with atomics), the
    edge-parallel chunk, the runtime-layout kernels and the wavefronts per
    hub segment of a g-SDDMM;
  - shapes: H in {1, 2, 4, 8}, F from 1 to 40 (now and then a row wider than
    one pass of the wavefront: F of 100-300), each operand full (H, F), per
    head (H, 1) or one value (1, 1); fp32 or bf16; node tables with a padded
    row stride;
  - the stream: the current one or a second stream;

then runs g-SpMM (op and reducer drawn), its backward, g-SDDMM (op and
targets drawn), its backward, edge softmax and its backward, leaky ReLU and
its backward, and the fused attention layer with its backward.  Tolerances are those of tests/_gpu.py;
max/min values and their arg edges compare bit for bit.  The case number,
seed and draws are printed before the GPU work of a case."""
import contextlib
import os
import sys

import numpy as np
import pytest
import torch

import oracle as orc
from paper_1909_01315_amd import gnnk
from _gpu import Pair, assert_close, assert_exact, dev, host
from test_gpu_gat import oracle_gat, oracle_gat_backward

pytestmark = pytest.mark.gpu

# other seed ranges and counts: GNNK_RANDOM_SEED0, GNNK_RANDOM_CASES
SEED0 = int(os.environ.get("GNNK_RANDOM_SEED0", "90000"))
N_CASES = int(os.environ.get("GNNK_RANDOM_CASES", "400"))
OPS = ["copy_lhs", "copy_rhs", "add", "sub", "mul", "div"]
TARGETS = ["u", "e", "v"]


@pytest.fixture(autouse=True)
def reset_options():
    yield
    for k, v in (("seg_edges", 0), ("small_deg", -1), ("schedule", 0), ("no_fast", 0), ("no_split", 0),
                 ("edge_chunk", 0), ("sddmm_split", 0)):
        gnnk.set_option(k, v)


def draw_graph(rng):
    n_src = int(rng.integers(1, 200))
    n_dst = int(rng.integers(1, 200))
    E = int(rng.integers(0, 3000)) if rng.random() < 0.95 else 0
    src = rng.integers(0, n_src, E).astype(np.int32)
    dst = rng.integers(0, n_dst, E).astype(np.int32)
    if E and rng.random() < 0.35:
        dst[rng.random(E) < 0.4] = int(rng.integers(0, n_dst))
        src[rng.random(E) < 0.3] = int(rng.integers(0, n_src))
    if rng.random() < 0.3:
        order = np.argsort(dst, kind="stable")
        src, dst = src[order], dst[order]
    return src, dst, n_src, n_dst, bool(rng.random() < 0.3)


def draw_options(rng):
    return {"seg_edges": int(rng.choice([0, 32, 64, 256])), "small_deg": int(rng.choice([-1, -1, 0, 4, 64])),
            "schedule": int(rng.choice([0, 0, 0, 2, 3])), "no_fast": int(rng.choice([0, 0, 0, 1])),
            "edge_chunk": int(rng.choice([0, 0, 8, 36]))}


class CsrPair:
    """The graph built from the oracle's in-CSR (graph_create_csr), with the
    edge ids of its positions or, when they are the identity, none."""

    def __init__(self, src, dst, n_src, n_dst, ptr64, with_eids):
        self.o = orc.OGraph(src, dst, n_src, n_dst)
        ip, ii, ie = orc.csr(self.o)
        ident = np.array_equal(ie, np.arange(len(ie), dtype=ie.dtype))
        eids = None if (ident and not with_eids) else dev(ie.astype(np.int32))
        self.g = gnnk.Graph.from_csr(dev(ip.astype(np.int64 if ptr64 else np.int32)), dev(ii.astype(np.int32)),
                                     eids, n_src)
        torch.cuda.synchronize()


def kind_shape(rng, H, F):
    return [(H, F), (H, 1), (1, 1)][int(rng.choice(3, p=[0.6, 0.25, 0.15]))]


def table(rng, rows, shape, bf16, positive=False, pad=0):
    """(oracle array, device tensor): normal values, or uniform in [0.5, 1.5]
    for divisors; bf16 as bit patterns on the oracle side; a padded row
    stride on the device when pad > 0."""
    h, f = shape
    a = rng.uniform(0.5, 1.5, (rows, h, f)) if positive else rng.standard_normal((rows, h, f))
    a = a.astype(np.float32)
    if bf16:
        a = orc.round_bf16(a)
    t = dev(a)
    if pad and rows > 1:
        buf = torch.zeros((rows, h * f + pad), dtype=t.dtype, device=t.device)
        buf[:, :h * f] = t.reshape(rows, h * f)
        t = buf[:, :h * f].unflatten(1, (h, f))
    return a, t


def check(kind, gpu, ref, name):
    assert_close(gpu, ref, kind=kind, name=name)


def gat_grad_bounds(o, feat, el, er, dz, slope):
    """Error bounds of the attention gradients from the magnitudes of the
    terms they sum.  Both sides round the attention a to fp32 (the oracle
    between its steps, the fused kernel from exp2 and 1/l), so the sum of a
    row's attention is 1 only to within fp32 rounding, and d_er = P - S Q
    (exactly 0 when the slope is the same over the row) keeps |S| times that
    error.  A sum of terms t_e computed from fp32-rounded factors is within a
    small multiple of 2^-24 sum |t_e| of the exact one: 2^-20 sum |t_e| is
    used (16 units of fp32 rounding), per output, on top of the usual
    tolerance."""
    s = (el[o.src, :, 0].astype(np.float64) + er[o.dst, :, 0].astype(np.float64))
    lk = np.where(s > 0, 1.0, slope)
    a = orc.edge_softmax(o, orc.leaky_relu(orc.gsddmm(o, "add", el, "u", er, "v"), slope))[:, :, 0]
    a = a.astype(np.float64)
    dabs = np.einsum("ehf,ehf->eh", np.abs(feat[o.src]).astype(np.float64), np.abs(dz[o.dst]).astype(np.float64))
    s_abs = np.zeros((o.n_dst, feat.shape[1]))
    np.add.at(s_abs, o.dst, a * dabs)
    t = a * (dabs + s_abs[o.dst]) * lk
    b_er = np.zeros((o.n_dst, feat.shape[1]))
    np.add.at(b_er, o.dst, t)
    b_el = np.zeros((o.n_src, feat.shape[1]))
    np.add.at(b_el, o.src, t)
    b_feat = np.zeros(feat.shape)
    np.add.at(b_feat, o.src, a[:, :, None] * np.abs(dz[o.dst]))
    u = 2.0 ** -20
    return u * b_feat, u * b_el[:, :, None], u * b_er[:, :, None]


def check_bound(gpu, ref, bound, name, rel=1e-5):
    """|gpu - ref| <= max(1e-6 + rel |ref|, bound) per element (bf16 results
    as their values)"""
    g = host(gpu)
    g = (orc.bf16_to_f32(g) if g.dtype == np.uint16 else g).astype(np.float64).reshape(ref.shape)
    r = np.asarray(ref, np.float64)
    tol = np.maximum(1e-6 + rel * np.abs(r), bound)
    bad = ~(np.abs(g - r) <= tol)
    assert not bad.any(), f"{name}: {int(bad.sum())} of {bad.size} out of bound; first at " \
                          f"{np.argwhere(bad)[0]}: gpu {g[bad][0]} ref {r[bad][0]} tol {tol[bad][0]}"


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_case(case):
    rng = np.random.default_rng(SEED0 + case)
    src, dst, n_src, n_dst, ptr64 = draw_graph(rng)
    opts = draw_options(rng)
    # drawn from a stream of its own, so that the other draws of a case stay
    # those of the seed
    opts["sddmm_split"] = int(np.random.default_rng([SEED0 + case, 1]).choice([0, 0, 1, 2, 3]))
    build = ["coo", "coo", "csr", "csr_eids"][int(rng.integers(4))]
    side = bool(rng.random() < 0.3)
    if rng.random() < 0.1:
        H = int(rng.choice([1, 2, 3]))
        F = int(rng.choice([100, 129, 300]))
    else:
        H = int(rng.choice([1, 2, 4, 8]))
        F = int(rng.choice([1, 2, 3, 4, 5, 8, 13, 16, 32, 40]))
    bf16 = bool(rng.random() < 0.2)
    kind = "bf16" if bf16 else "f32"
    pad = int(rng.choice([0, 0, 1, 4]))
    op = OPS[int(rng.integers(len(OPS)))]
    red = ["sum", "mean", "max", "min"][int(rng.integers(4))]
    lt, rt = (TARGETS[int(i)] for i in rng.integers(0, 3, 2))
    sop = (OPS + ["dot"])[int(rng.integers(len(OPS) + 1))]
    print(f"case {case}: n_src {n_src} n_dst {n_dst} E {len(src)} ptr64 {ptr64} {build} side stream {side} "
          f"{opts} H {H} F {F} {kind} pad {pad} gspmm {op}/{red} gsddmm {sop} {lt},{rt}", flush=True)
    sys.stdout.flush()
    for k, v in opts.items():
        gnnk.set_option(k, v)
    stream = torch.cuda.Stream() if side else None
    if stream is not None:
        stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext():
        run_case(rng, src, dst, n_src, n_dst, ptr64, build, opts, H, F, bf16, kind, pad, op, red, lt, rt, sop)
    torch.cuda.synchronize()


def run_case(rng, src, dst, n_src, n_dst, ptr64, build, opts, H, F, bf16, kind, pad, op, red, lt, rt, sop):
    if build == "coo":
        p = Pair(src, dst, n_src, n_dst, ptr64=ptr64)
    else:
        p = CsrPair(src, dst, n_src, n_dst, ptr64, build == "csr_eids")
    E = p.o.n_edges
    rows = {"u": n_src, "e": E, "v": n_dst}

    # g-SpMM forward and backward
    ls = kind_shape(rng, H, F) if op != "copy_rhs" else None
    rs = kind_shape(rng, H, F) if op != "copy_lhs" else None
    if ls and rs and ls != (H, F) and rs != (H, F):
        ls = (H, F)
    L, Ld = table(rng, n_src, ls, bf16, pad=pad) if ls else (None, None)
    R, Rd = table(rng, E, rs, bf16, positive=True) if rs else (None, None)
    if red in ("max", "min"):
        ref, rau, rae = orc.gspmm(p.o, op, red, L, R)
        out, au, ae = gnnk.gspmm(p.g, op, red, Ld, Rd, want_args=True)
        assert_exact(out, ref, "gspmm value")
        assert_exact(ae, rae, "gspmm arg edge")
        assert_exact(au, rau, "gspmm arg node")
    else:
        ref, rae, ae = orc.gspmm(p.o, op, red, L, R), None, None
        check(kind, gnnk.gspmm(p.g, op, red, Ld, Rd), ref, "gspmm")
    dZ, dZd = table(rng, n_dst, ref.shape[1:], bf16)
    gl, gr = orc.gspmm_backward(p.o, op, red, L, R, dZ, arg_e=rae)
    dl, dr = gnnk.gspmm_backward(p.g, op, red, Ld, Rd, dZd, arg_rhs=ae)
    if gl is not None:
        check(kind, dl, gl, "gspmm grad lhs")
    if gr is not None:
        check(kind, dr, gr, "gspmm grad rhs")

    # g-SDDMM forward and backward
    if sop == "dot":
        # a dot of a full operand with a full, per-head or single value
        ls2, rs2 = (H, F), kind_shape(rng, H, F)
        if rng.random() < 0.5:
            ls2, rs2 = rs2, ls2
    else:
        ls2 = kind_shape(rng, H, F) if sop != "copy_rhs" else None
        rs2 = kind_shape(rng, H, F) if sop != "copy_lhs" else None
    L2, L2d = table(rng, rows[lt], ls2, bf16, pad=pad if lt != "e" else 0) if ls2 else (None, None)
    R2, R2d = table(rng, rows[rt], rs2, bf16, positive=True) if rs2 else (None, None)
    M = orc.gsddmm(p.o, sop, L2, lt, R2, rt)
    check(kind, gnnk.gsddmm(p.g, sop, L2d, lt, R2d, rt), M, "gsddmm")
    dM, dMd = table(rng, E, M.shape[1:], bf16)
    gl, gr = orc.gsddmm_backward(p.o, sop, L2, lt, R2, rt, dM)
    dl, dr = gnnk.gsddmm_backward(p.g, sop, L2d, lt, R2d, rt, dMd)
    if gl is not None:
        check(kind, dl, gl, "gsddmm grad lhs")
    if gr is not None:
        check(kind, dr, gr, "gsddmm grad rhs")

    # edge softmax forward and backward (one score per head, or F per head)
    ssh = (H, 1) if rng.random() < 0.6 else (H, F)
    s, sd = table(rng, E, ssh, bf16)
    a = orc.edge_softmax(p.o, s)
    ad = gnnk.edge_softmax(p.g, sd)
    check(kind, ad, a, "edge softmax")
    g_, gd = table(rng, E, ssh, bf16)
    check(kind, gnnk.edge_softmax_backward(p.g, dev(a), gd), orc.edge_softmax_backward(p.o, a, g_),
          "edge softmax backward")

    # leaky ReLU on an edge tensor (one fp32 operation: bit for bit), with a
    # padded row stride sometimes
    x, xd = table(rng, E, (H, F), bf16, pad=pad)
    dy, dyd = table(rng, E, (H, F), bf16)
    assert_exact(gnnk.edge_leaky_relu(xd, 0.2), orc.leaky_relu(x, 0.2), "leaky relu")
    assert_exact(gnnk.edge_leaky_relu_backward(xd, dyd, 0.2), orc.leaky_relu_backward(x, dy, 0.2),
                 "leaky relu backward")

    # fused attention layer: a head of feat must fit one wavefront of vectors
    # (8 bf16 or 4 fp32 values per lane, fewer as F and the row stride
    # allow).  It rounds nothing between its steps, so for bf16 the reference
    # is the oracle chain on the exactly widened inputs, at the bf16 tolerance.
    vec = next(v for v in ((8, 4, 2, 1) if bf16 else (4, 2, 1))
               if F % v == 0 and (pad == 0 or n_src < 2 or (H * F + pad) % v == 0))
    if F // vec <= 64 and opts["schedule"] == 0:
        wide = orc.bf16_to_f32 if bf16 else (lambda x: x)
        feat, featd = table(rng, n_src, (H, F), bf16, pad=pad)
        el, eld = table(rng, n_src, (H, 1), bf16)
        er, erd = table(rng, n_dst, (H, 1), bf16)
        feat, el, er = wide(feat), wide(el), wide(er)
        ref, ref_a = oracle_gat(p.o, feat, el, er, 0.2)
        out, attn, st = gnnk.gat_aggregate(p.g, featd, eld, erd, 0.2, want_attn=True, want_stats=True)
        check(kind, out, ref, "gat out")
        check(kind, attn, ref_a, "gat attention")
        dz, dzd = table(rng, n_dst, (H, F), bf16)
        dz = wide(dz)
        rf, rl, rr = oracle_gat_backward(p.o, feat, el, er, 0.2, dz)
        gf, gl_, gr_ = gnnk.gat_aggregate_backward(p.g, featd, eld, erd, 0.2, st, dzd)
        bf, bl, br = gat_grad_bounds(p.o, feat, el, er, dz, 0.2)
        rel = 1e-2 if bf16 else 1e-5
        check_bound(gf, rf, bf, "gat d feat", rel)
        check_bound(gl_, rl, bl, "gat d el", rel)
        check_bound(gr_, rr, br, "gat d er", rel)
    p.g.destroy()
