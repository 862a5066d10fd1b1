"""Per-operator timing against the HBM roofline on the synthetic workloads.

For every (workload, operator, dtype, direction) the call is timed with HIP
events on the stream it runs on: 3 untimed calls, then 20 timed ones; the
median and the minimum are reported.  B_alg is the operator's algorithmic
byte count (gather model):

* every edge gathers its neighbour's row (E x D x s) and reads its index
  (4 B) and its edge operand (E x W x s);
* operands on the row itself are read once per row and outputs are written
  once (N x D x s);
* row offsets once ((N + 1) x 4 or 8 B);
* reverse-graph passes read edge operands through the reverse edge ids
  (+4 B per edge);
* max/min backward passes each (row, column) gradient to its one winner:
  the arg edges, dZ and dX are touched once each (N x D x (4 + 2 s)), plus
  8 B per edge for the walk.

B_alg GB/s = B_alg / median time, and "B_alg / 8 TB/s" is that rate over the
MI355X HBM peak; "of copy" is the same rate over what a plain 1 GiB device
copy reaches on the same box (bytes read + written over the median of 5
copies, measured first), the achievable stream bandwidth.  Both are
gather-model rates: where the gathered table fits the 256 MB Infinity Cache
they exceed 1, and only where it cannot (the 61.9M-edge graph's tables) are
they fractions of a bound.  bench.py prices the operators of its step against
the bytes that must cross HBM and the counted bytes past L2.
edge.feat/s = E x (message columns) / time.

Usage: python -m paper_1909_01315_amd.opbench [--configs c2,c3,c3r,c4,c5] [--out FILE.md]
       [--warm W] [--reps K] [--mark]
Every graph and input is seeded and synthetic.  Needs a GPU and the built
library.
"""
from __future__ import annotations

import argparse
import sys
import time

import numpy as np
import torch

from . import gnnk, synth

PEAK_GBS = 8000.0


def _time(fn, warm: int = 3, reps: int = 20):
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        fn()
        e1.record(st)
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts)), float(np.min(ts))


def _log(msg):
    print(f"[opbench] {msg}", file=sys.stderr, flush=True)


class Rows:
    """warm, reps: untimed and timed calls per operator.  mark: before and
    after each operator, a one-element int32 fill on the device, so that a
    hardware counter run (rocprofv3 --pmc, one call per operator) can tell
    which dispatches belong to which operator."""

    def __init__(self, warm: int = 3, reps: int = 20, mark: bool = False):
        self.rows = []
        self.warm, self.reps = warm, reps
        self.mark = torch.zeros(1, dtype=torch.int32, device="cuda") if mark else None

    def add(self, cfg, op, dtype, direction, b_alg, feat_cols, E, fn):
        if self.mark is not None:
            self.mark.fill_(len(self.rows) + 1)
            torch.cuda.synchronize()
        med, mn = _time(fn, self.warm, self.reps)
        if self.mark is not None:
            self.mark.fill_(-len(self.rows) - 1)
            torch.cuda.synchronize()
        gbs = b_alg / med / 1e6
        self.rows.append(dict(config=cfg, op=op, dtype=dtype, dir=direction, b_alg=b_alg, ms=med, ms_min=mn,
                              gbs=gbs, frac=gbs / PEAK_GBS, ef=E * feat_cols / (med * 1e-3) if feat_cols else None))
        _log(f"{cfg} {op} {dtype} {direction}: {med:.3f} ms (min {mn:.3f}), {gbs:.0f} GB/s, B_alg / 8 TB/s {gbs / PEAK_GBS:.2f}")


def _graph(sg, ptr64=False):
    dev = torch.device("cuda:0")
    s, d = torch.from_numpy(sg.src).to(dev), torch.from_numpy(sg.dst).to(dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    g = gnnk.Graph.from_coo(s, d, sg.n_src, sg.n_dst, ptr64=ptr64)
    torch.cuda.synchronize()
    _log(f"{sg.name}: device graph build {1e3 * (time.perf_counter() - t0):.1f} ms")
    return g


def c2(R: Rows):
    sg = synth.graph_c2()
    g = _graph(sg)
    N, E = sg.n_dst, sg.n_edges
    w = torch.from_numpy(sg.extra["gcn_w"]).cuda().view(E, 1, 1)
    for D in (16, 64, 256, 512):
        X = torch.randn((N, 1, D), device="cuda")
        Z = torch.empty((N, 1, D), device="cuda")
        b = E * (D * 4 + 4 + 4) + N * D * 4 + (N + 1) * 4
        R.add("c2", f"u_mul_e/sum D={D} (GCN weights)", "f32", "fwd", b, D, E,
              lambda: gnnk.gspmm(g, "mul", "sum", X, w, out=Z))
    g.destroy()


def c3(R: Rows):
    sg = synth.graph_c3()
    g = _graph(sg)
    N, E = sg.n_dst, sg.n_edges
    H, F, D = 8, 16, 128
    off = (N + 1) * 4
    cu = dict(device="cuda")
    X = torch.randn((N, H, F), **cu)
    X1 = X.view(N, 1, D)
    dZ = torch.randn((N, H, F), **cu)
    dZ1 = dZ.view(N, 1, D)
    a = torch.rand((E, H, 1), **cu)
    w = torch.rand((E, 1, 1), **cu)
    el, er = torch.randn((N, H, 1), **cu), torch.randn((N, H, 1), **cu)
    Z, Z1, dX = torch.empty((N, H, F), **cu), torch.empty((N, 1, D), **cu), torch.empty((N, H, F), **cu)
    M8, M1 = torch.empty((E, H, 1), **cu), torch.empty((E, 1, 1), **cu)
    S2, S3 = torch.empty((E, H, 1), **cu), torch.empty((E, H, 1), **cu)
    au = torch.empty((N, 1, D), dtype=torch.int32, **cu)
    ae = torch.empty((N, 1, D), dtype=torch.int32, **cu)
    dl, dr = torch.empty((N, H, 1), **cu), torch.empty((N, H, 1), **cu)
    gl = torch.randn((E, H, 1), **cu)

    R.add("c3", "u_mul_e/sum H=8 F=16, attention (E,8)", "f32", "fwd",
          E * (512 + 32 + 4) + N * 512 + off, D, E, lambda: gnnk.gspmm(g, "mul", "sum", X, a, out=Z))
    R.add("c3", "u_mul_e/sum H=1 D=128, w (E,1)", "f32", "fwd",
          E * (512 + 4 + 4) + N * 512 + off, D, E, lambda: gnnk.gspmm(g, "mul", "sum", X1, w, out=Z1))
    R.add("c3", "u_dot_v H=8 F=16 -> (E,8)", "f32", "fwd",
          E * (512 + 4 + 32) + N * 512 + off, D, E, lambda: gnnk.gsddmm(g, "dot", X, "u", X, "v", out=M8))
    R.add("c3", "u_dot_v H=1 D=128 -> (E,1)", "f32", "fwd",
          E * (512 + 4 + 4) + N * 512 + off, D, E, lambda: gnnk.gsddmm(g, "dot", X1, "u", X1, "v", out=M1))
    R.add("c3", "copy_u/mean D=128", "f32", "fwd",
          E * (512 + 4) + N * 512 + off, D, E, lambda: gnnk.gspmm(g, "copy_lhs", "mean", X1, out=Z1))
    R.add("c3", "copy_u/max D=128 + arg edge", "f32", "fwd",
          E * (512 + 4) + N * 512 * 2 + off, D, E,
          lambda: gnnk.gspmm(g, "copy_lhs", "max", X1, out=Z1, want_args=True, arg_lhs=au, arg_rhs=ae))
    R.add("c3", "u_add_v H=8 -> (E,8)", "f32", "fwd",
          E * (32 + 4 + 32) + N * 32 + off, H, E, lambda: gnnk.gsddmm(g, "add", el, "u", er, "v", out=M8))
    R.add("c3", "leaky ReLU (E,8)", "f32", "fwd", 2 * E * 32, H, E,
          lambda: gnnk.edge_leaky_relu(M8, 0.2, y=S2))
    R.add("c3", "edge softmax (E,8)", "f32", "fwd", 2 * E * 32 + off, H, E,
          lambda: gnnk.edge_softmax(g, S2, out=S3))
    R.add("c3", "fused attention (u_add_v, leaky, softmax, u_mul_e/sum) H=8 F=16", "f32", "fwd",
          E * (512 + 32 + 4) + N * (512 + 32) + off, D, E, lambda: gnnk.gat_aggregate(g, X, el, er, 0.2, out=Z))
    _, stats = gnnk.gat_aggregate(g, X, el, er, 0.2, want_stats=True)
    # pass A gathers feat and el per edge (dZ, er, stats per row); pass B
    # gathers dZ and a 16-byte record per edge (feat, el per row)
    R.add("c3", "fused attention backward (two passes, no E-sized tensor)", "f32", "bwd",
          E * (512 + 32 + 4) + N * (512 + 32 + 64 + 32 + 128) + off +
          E * (512 + 128 + 4) + N * (512 + 32 + 512 + 32) + off, D, E,
          lambda: gnnk.gat_aggregate_backward(g, X, el, er, 0.2, stats, dZ))
    # backward passes
    R.add("c3", "u_mul_e/sum H=8: d feat (reverse graph)", "f32", "bwd",
          E * (512 + 32 + 4 + 4) + N * 512 + off, D, E,
          lambda: gnnk.gspmm_backward(g, "mul", "sum", X, a, dZ, grad_lhs=dX, want_rhs=False))
    R.add("c3", "u_mul_e/sum H=8: d attention (per-head u_dot_v)", "f32", "bwd",
          E * (512 + 4 + 32) + N * 512 + off, D, E,
          lambda: gnnk.gspmm_backward(g, "mul", "sum", X, a, dZ, want_lhs=False, grad_rhs=M8))
    R.add("c3", "u_mul_e/sum H=8: d feat and d attention in one reverse pass", "f32", "bwd",
          E * (512 + 32 + 4 + 4 + 32) + N * (512 + 512) + off, D, E,
          lambda: gnnk.gspmm_backward(g, "mul", "sum", X, a, dZ, grad_lhs=dX, grad_rhs=M8))
    R.add("c3", "copy_u/mean D=128: dX (reverse graph)", "f32", "bwd",
          E * (512 + 4) + N * (512 + 4) + off, D, E,
          lambda: gnnk.gspmm_backward(g, "copy_lhs", "mean", X1, None, dZ1, grad_lhs=Z1))
    gnnk.gspmm(g, "copy_lhs", "max", X1, out=Z1, want_args=True, arg_lhs=au, arg_rhs=ae)
    R.add("c3", "copy_u/max D=128: dX (argmax scatter)", "f32", "bwd",
          E * (4 + 4) + N * 512 * 3 + off, D, E,
          lambda: gnnk.gspmm_backward(g, "copy_lhs", "max", X1, None, dZ1, arg_rhs=ae, grad_lhs=Z1))
    R.add("c3", "edge softmax (E,8)", "f32", "bwd", 3 * E * 32 + off, H, E,
          lambda: gnnk.edge_softmax_backward(g, S3, gl, grad_score=S2))
    R.add("c3", "leaky ReLU (E,8)", "f32", "bwd", 3 * E * 32, H, E,
          lambda: gnnk.edge_leaky_relu_backward(M8, gl, 0.2, dx=S2))
    R.add("c3", "u_add_v H=8: d el, d er", "f32", "bwd",
          E * (32 + 4) + E * 32 + 2 * N * 32 + 2 * off, H, E,
          lambda: gnnk.gsddmm_backward(g, "add", el, "u", er, "v", gl, grad_lhs=dl, grad_rhs=dr))
    g.destroy()


def c3r(R: Rows):
    """The gated c3 operators on the same graph with each destination's
    in-edges in random source order (synth.shuffle_within_rows): what the
    row order contributes (the generated graphs list sources in ascending
    order, which the segment order turns into L2 locality)."""
    sg = synth.shuffle_within_rows(synth.graph_c3(), synth.SEED_BASE + 300)
    g = _graph(sg)
    N, E = sg.n_dst, sg.n_edges
    H, F, D = 8, 16, 128
    off = (N + 1) * 4
    cu = dict(device="cuda")
    X = torch.randn((N, H, F), **cu)
    X1 = X.view(N, 1, D)
    dZ = torch.randn((N, H, F), **cu)
    a = torch.rand((E, H, 1), **cu)
    Z, Z1, dX = torch.empty((N, H, F), **cu), torch.empty((N, 1, D), **cu), torch.empty((N, H, F), **cu)
    M8 = torch.empty((E, H, 1), **cu)
    tag = "c3 rows shuffled"
    R.add(tag, "u_mul_e/sum H=8 F=16, attention (E,8)", "f32", "fwd",
          E * (512 + 32 + 4) + N * 512 + off, D, E, lambda: gnnk.gspmm(g, "mul", "sum", X, a, out=Z))
    R.add(tag, "u_dot_v H=8 F=16 -> (E,8)", "f32", "fwd",
          E * (512 + 4 + 32) + N * 512 + off, D, E, lambda: gnnk.gsddmm(g, "dot", X, "u", X, "v", out=M8))
    R.add(tag, "copy_u/mean D=128", "f32", "fwd",
          E * (512 + 4) + N * 512 + off, D, E, lambda: gnnk.gspmm(g, "copy_lhs", "mean", X1, out=Z1))
    R.add(tag, "u_mul_e/sum H=8: d feat and d attention in one reverse pass", "f32", "bwd",
          E * (512 + 32 + 4 + 4 + 32) + N * (512 + 512) + off, D, E,
          lambda: gnnk.gspmm_backward(g, "mul", "sum", X, a, dZ, grad_lhs=dX, grad_rhs=M8))
    g.destroy()


def c4(R: Rows):
    sg = synth.graph_c4()
    g = _graph(sg, ptr64=True)
    N, E = sg.n_dst, sg.n_edges
    D = 100
    off = (N + 1) * 8
    cu = dict(device="cuda")
    for dt, s, name in ((torch.float32, 4, "f32"), (torch.bfloat16, 2, "bf16")):
        X = torch.randn((N, 1, D), **cu).to(dt)
        Y = torch.randn((N, 1, D), **cu).to(dt)
        dZ = torch.randn((N, 1, D), **cu).to(dt)
        Z = torch.empty((N, 1, D), dtype=dt, **cu)
        dX = torch.empty((N, 1, D), dtype=dt, **cu)
        M = torch.empty((E, 1, 1), dtype=dt, **cu)
        au = torch.empty((N, 1, D), dtype=torch.int32, **cu)
        ae = torch.empty((N, 1, D), dtype=torch.int32, **cu)
        R.add("c4", "copy_u/sum D=100 (int64 offsets)", name, "fwd",
              E * (D * s + 4) + N * D * s + off, D, E, lambda: gnnk.gspmm(g, "copy_lhs", "sum", X, out=Z))
        R.add("c4", "copy_u/max D=100 + arg edge", name, "fwd",
              E * (D * s + 4) + N * D * (s + 4) + off, D, E,
              lambda: gnnk.gspmm(g, "copy_lhs", "max", X, out=Z, want_args=True, arg_lhs=au, arg_rhs=ae))
        R.add("c4", "u_dot_v D=100 -> (E,1)", name, "fwd",
              E * (D * s + 4 + s) + N * D * s + off, D, E, lambda: gnnk.gsddmm(g, "dot", X, "u", Y, "v", out=M))
        R.add("c4", "copy_u/sum D=100: dX (reverse graph)", name, "bwd",
              E * (D * s + 4) + N * D * s + off, D, E,
              lambda: gnnk.gspmm_backward(g, "copy_lhs", "sum", X, None, dZ, grad_lhs=dX))
        R.add("c4", "copy_u/max D=100: dX (argmax scatter)", name, "bwd",
              E * (4 + 4) + N * D * (4 + 2 * s) + off, D, E,
              lambda: gnnk.gspmm_backward(g, "copy_lhs", "max", X, None, dZ, arg_rhs=ae, grad_lhs=dX))
        gM = torch.randn((E, 1, 1), **cu).to(dt)
        R.add("c4", "u_dot_v D=100: dX (reverse graph) and dY", name, "bwd",
              2 * (E * (D * s + 4 + s) + N * D * s + off) + E * 4, D, E,
              lambda: gnnk.gsddmm_backward(g, "dot", X, "u", Y, "v", gM, grad_lhs=dX, grad_rhs=Z))
        del X, Y, dZ, Z, dX, M, au, ae, gM
    g.destroy()


def c5(R: Rows):
    sg = synth.graph_c5()
    g = _graph(sg)
    Ns, N, E = sg.n_src, sg.n_dst, sg.n_edges
    D = 64
    off = (N + 1) * 4
    cu = dict(device="cuda")
    X = torch.randn((Ns, 1, D), **cu)
    dZ = torch.randn((N, 1, D), **cu)
    c = torch.from_numpy(sg.extra["norm"]).cuda().view(E, 1, 1)
    Z = torch.empty((N, 1, D), **cu)
    M = torch.empty((E, 1, 1), **cu)
    R.add("c5", "u_mul_e/sum D=64 (relational, 5M sources)", "f32", "fwd",
          E * (D * 4 + 4 + 4) + N * D * 4 + off, D, E, lambda: gnnk.gspmm(g, "mul", "sum", X, c, out=Z))
    R.add("c5", "u_dot_v D=64 (X_rel at u, dZ at v) -> (E,1)", "f32", "fwd",
          E * (D * 4 + 4 + 4) + N * D * 4 + off, D, E, lambda: gnnk.gsddmm(g, "dot", X, "u", dZ, "v", out=M))
    g.destroy()


CONFIGS = {"c2": c2, "c3": c3, "c3r": c3r, "c4": c4, "c5": c5}


def copy_bandwidth() -> float:
    """GB/s of a plain 1 GiB device copy, bytes read + written over the median
    of 5 copies"""
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    med, _ = _time(lambda: dst.copy_(src), warm=1, reps=5)
    return 2 * src.numel() * 4 / med / 1e6


def to_markdown(rows, copy_gbs) -> str:
    out = [f"Plain 1 GiB device copy on this box: {copy_gbs:.0f} GB/s (read + write).", "",
           "| workload | operator | dtype | dir | B_alg GB | median ms | min ms | B_alg GB/s | B_alg / 8 TB/s | of copy | "
           "edge.feat/s |",
           "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        ef = f"{r['ef']:.3g}" if r["ef"] else "-"
        out.append(f"| {r['config']} | {r['op']} | {r['dtype']} | {r['dir']} | {r['b_alg'] / 1e9:.3f} | {r['ms']:.3f} | "
                   f"{r['ms_min']:.3f} | {r['gbs']:.0f} | {r['frac']:.2f} | {r['gbs'] / copy_gbs:.2f} | {ef} |")
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--configs", default="c2,c3,c4,c5")
    ap.add_argument("--out", default=None)
    ap.add_argument("--warm", type=int, default=3, help="untimed calls per operator")
    ap.add_argument("--reps", type=int, default=20, help="timed calls per operator")
    ap.add_argument("--mark", action="store_true",
                    help="a one-element int32 fill before each operator (for counter runs)")
    args = ap.parse_args()
    gnnk.load()
    assert torch.cuda.is_available(), "the operator benchmark needs a GPU"
    copy_gbs = copy_bandwidth()
    _log(f"plain device copy: {copy_gbs:.0f} GB/s")
    R = Rows(args.warm, args.reps, args.mark)
    for name in args.configs.split(","):
        CONFIGS[name](R)
        torch.cuda.empty_cache()
    md = to_markdown(R.rows, copy_gbs)
    print(md)
    if args.out:
        with open(args.out, "w") as f:
            f.write(md + "\n")


if __name__ == "__main__":
    main()
