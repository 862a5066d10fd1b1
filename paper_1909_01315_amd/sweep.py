"""Sensitivity of the two primitives to graph shape, feature width and
parallelisation (the kernel study of Appendix E, on MI355X).

Appendix E of the paper compares node-parallel and edge-parallel g-SpMM and
g-SDDMM over CSR and COO while the per-head feature width F varies, on a
constant-degree (k-NN-like) graph and on power-law graphs; its figure values
are not printed in the text, so this is a characterisation, not a
comparison.  Here the row engine (node-parallel, degree-sorted roles: the
CSR kernels) is set against the edge-parallel walk over the COO form
(deterministic split-row partials, and fp64 atomics for split rows).

Usage: python -m paper_1909_01315_amd.sweep [--out FILE.md] [--graphs knn,rmat]
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

SCHEDULES = {1: "row engine", 2: "edge (ordered)", 3: "edge (atomics)"}


def _time(fn, reps: int = 5) -> float:
    for _ in range(2):
        fn()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def _graphs(names):
    for n in names:
        t0 = time.perf_counter()
        if n == "knn":
            g = synth.knn_graph(synth.SEED_BASE + 50, 1 << 20, 32, name="knn k=32, N=1,048,576")
        elif n == "rmat":
            g = synth.graph_c4()
            g.name = "R-MAT N=2,449,029 E=61.9M"
        elif n == "rmat_dense":
            g = synth.graph_c3()
            g.name = "R-MAT N=232,965 E=114.6M"
        else:
            raise ValueError(n)
        print(f"[sweep] {g.name}: built in {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)
        yield g


def run(graph_names, feats=(1, 2, 4, 8, 16, 32, 64, 128)):
    dev = torch.device("cuda:0")
    rows = []
    for sg in _graphs(graph_names):
        g = gnnk.Graph.from_coo(torch.from_numpy(sg.src).to(dev), torch.from_numpy(sg.dst).to(dev), sg.n_src,
                                sg.n_dst)
        E = sg.n_edges
        w = torch.rand((E, 1, 1), device=dev)
        for F in feats:
            X = torch.randn((sg.n_src, 1, F), device=dev)
            Y = torch.randn((sg.n_dst, 1, F), device=dev)
            Z = torch.empty((sg.n_dst, 1, F), device=dev)
            M = torch.empty((E, 1, 1), device=dev)
            for sch in SCHEDULES:
                gnnk.set_option("schedule", sch)
                t_spmm = _time(lambda: gnnk.gspmm(g, "mul", "sum", X, w, out=Z))
                t_sddmm = _time(lambda: gnnk.gsddmm(g, "dot", X, "u", Y, "v", out=M)) if sch != 3 else float("nan")
                b_spmm = E * (F * 4 + 4 + 4) + sg.n_dst * F * 4
                b_sddmm = E * (F * 4 + 4 + 4) + sg.n_dst * F * 4
                rows.append((sg.name, F, SCHEDULES[sch], t_spmm, b_spmm / t_spmm / 1e6, t_sddmm,
                             b_sddmm / t_sddmm / 1e6 if t_sddmm == t_sddmm else float("nan")))
                print(f"[sweep] {sg.name} F={F:3d} {SCHEDULES[sch]:15s} spmm {t_spmm:8.3f} ms  sddmm "
                      f"{t_sddmm:8.3f} ms", file=sys.stderr, flush=True)
            del X, Y, Z, M
        gnnk.set_option("schedule", 0)
        g.destroy()
        torch.cuda.empty_cache()
    return rows


def to_markdown(rows) -> str:
    out = ["| graph | F | walk | g-SpMM u_mul_e/sum ms | GB/s | g-SDDMM u_dot_v ms | GB/s |",
           "|---|---|---|---|---|---|---|"]
    for name, F, sch, ts, bs, td, bd in rows:
        td_s = f"{td:.3f}" if td == td else "-"
        bd_s = f"{bd:.0f}" if bd == bd else "-"
        out.append(f"| {name} | {F} | {sch} | {ts:.3f} | {bs:.0f} | {td_s} | {bd_s} |")
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--graphs", default="knn,rmat")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    gnnk.load()
    assert torch.cuda.is_available(), "the sweep needs a GPU"
    md = to_markdown(run(args.graphs.split(",")))
    print(md)
    if args.out:
        with open(args.out, "w") as f:
            f.write(md + "\n")


if __name__ == "__main__":
    main()
