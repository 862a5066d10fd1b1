"""Seeded random cases: every entry point against the oracle on graphs and
settings drawn together, so that combinations no hand-written case lists
are still covered.  Each case draws

  - a graph: 1-200 sources and destinations, 0-3000 edges, sometimes a hot
    source and a hot destination (hub rows), sometimes sorted by destination
    (identity edge ids), int32 or int64 offsets;
  - library options: hub segment size, small-row threshold, schedule
    (row engine, edge-parallel ordered, edge-parallel with atomics) and the
    runtime-layout kernels;
  - shapes: H in {1, 2, 4, 8}, F from 1 to 40, each operand full (H, F),
    per head (H, 1) or one value (1, 1); fp32 or bf16; node tables with a
    padded row stride;

then runs g-SpMM (op and reducer drawn), its backward, g-SDDMM (op and
targets drawn), its backward, edge softmax and its backward, and the fused
attention layer with its backward.  Tolerances are those of tests/_gpu.py;
max/min values and their arg edges compare bit for bit.  The case number,
seed and draws are printed before the GPU work of a case."""
import sys

import numpy as np
import pytest
import torch

import oracle as orc
from paper_1909_01315_amd import gnnk
from _gpu import Pair, assert_close, assert_exact, dev, host
from test_gpu_gat import oracle_gat, oracle_gat_backward

pytestmark = pytest.mark.gpu

N_CASES = 160
OPS = ["copy_lhs", "copy_rhs", "add", "sub", "mul", "div"]
TARGETS = ["u", "e", "v"]


@pytest.fixture(autouse=True)
def reset_options():
    yield
    for k, v in (("seg_edges", 0), ("small_deg", -1), ("schedule", 0), ("no_fast", 0), ("no_split", 0)):
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
            "schedule": int(rng.choice([0, 0, 0, 2, 3])), "no_fast": int(rng.choice([0, 0, 0, 1]))}


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


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_case(case):
    rng = np.random.default_rng(90_000 + case)
    src, dst, n_src, n_dst, ptr64 = draw_graph(rng)
    opts = draw_options(rng)
    H = int(rng.choice([1, 2, 4, 8]))
    F = int(rng.choice([1, 2, 3, 4, 5, 8, 13, 16, 32, 40]))
    bf16 = bool(rng.random() < 0.2)
    kind = "bf16" if bf16 else "f32"
    pad = int(rng.choice([0, 0, 1, 4]))
    op = OPS[int(rng.integers(len(OPS)))]
    red = ["sum", "mean", "max", "min"][int(rng.integers(4))]
    lt, rt = (TARGETS[int(i)] for i in rng.integers(0, 3, 2))
    sop = (OPS + ["dot"])[int(rng.integers(len(OPS) + 1))]
    print(f"case {case}: n_src {n_src} n_dst {n_dst} E {len(src)} ptr64 {ptr64} {opts} H {H} F {F} {kind} "
          f"pad {pad} gspmm {op}/{red} gsddmm {sop} {lt},{rt}", flush=True)
    sys.stdout.flush()
    for k, v in opts.items():
        gnnk.set_option(k, v)
    p = Pair(src, dst, n_src, n_dst, ptr64=ptr64)
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
        ls2 = rs2 = (H, F)
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

    # edge softmax forward and backward
    s, sd = table(rng, E, (H, 1), bf16)
    a = orc.edge_softmax(p.o, s)
    ad = gnnk.edge_softmax(p.g, sd)
    check(kind, ad, a, "edge softmax")
    g_, gd = table(rng, E, (H, 1), bf16)
    check(kind, gnnk.edge_softmax_backward(p.g, dev(a), gd), orc.edge_softmax_backward(p.o, a, g_),
          "edge softmax backward")

    # fused attention layer (fp32; a row of feat must fit one wavefront of
    # vectors: 4, 2 or 1 floats per lane as F and the row stride allow)
    vec = next(v for v in (4, 2, 1) if F % v == 0 and (pad == 0 or n_src < 2 or (H * F + pad) % v == 0))
    if not bf16 and H * F // vec <= 64 and opts["schedule"] == 0:
        feat, featd = table(rng, n_src, (H, F), False, pad=pad)
        el, eld = table(rng, n_src, (H, 1), False)
        er, erd = table(rng, n_dst, (H, 1), False)
        ref, ref_a = oracle_gat(p.o, feat, el, er, 0.2)
        out, attn, st = gnnk.gat_aggregate(p.g, featd, eld, erd, 0.2, want_attn=True, want_stats=True)
        check(kind, out, ref, "gat out")
        check(kind, attn, ref_a, "gat attention")
        dz, dzd = table(rng, n_dst, (H, F), False)
        rf, rl, rr = oracle_gat_backward(p.o, feat, el, er, 0.2, dz)
        gf, gl_, gr_ = gnnk.gat_aggregate_backward(p.g, featd, eld, erd, 0.2, st, dzd)
        check(kind, gf, rf, "gat d feat")
        check(kind, gl_, rl, "gat d el")
        check(kind, gr_, rr, "gat d er")
    torch.cuda.synchronize()
    p.g.destroy()
