#!/usr/bin/env python3
"""Throughput of the g-SpMM / g-SDDMM hot path on one MI355X.

Workload: the 114.6M-edge R-MAT graph (a=0.57, b=0.19, c=0.19, d=0.05,
N=232,965 nodes, deduplicated), D=128 fp32 features seen as 8 heads x 16.  The
graph and every input are seeded synthetic stand-ins (the paper's datasets are
not available); they are built on the host and copied to HBM before timing.

One step is one pass over the whole hot path:
  GAT layer forward   gsddmm u_add_v -> leaky ReLU -> edge_softmax ->
                      gspmm u_mul_e/sum (X (N,8,16), attention (E,8,1))
  GAT layer backward  gspmm_backward (dX on the reverse graph, d attention as
                      a per-head u_dot_v) -> edge_softmax_backward -> leaky
                      ReLU backward -> gsddmm_backward of u_add_v
  GraphSAGE           gspmm copy_u/mean on (N,128) and its backward
  max aggregation     gspmm copy_u/max with argmax and its argmax scatter
  attention score     gsddmm u_dot_v (N,8,16).(N,8,16) -> (E,8,1)

The metric is edge-feature throughput: the sum over the step's g-SpMM /
g-SDDMM / edge-softmax passes of E x (feature columns of that pass's message),
divided by the step time.

Every operator is timed with HIP events recorded on the stream it runs on and
reported against two ceilings (the "rooflines" list; "roofline" is the
operator that takes the longest):
  * achieved / peak: the bytes that must cross HBM at least once (every input
    element read once, every output element written once, the index arrays
    the operator walks), over its time, against the 8 TB/s HBM peak: at most
    1 by construction.  "effective_gbs" is the gather model instead (every
    edge gathers its neighbour's row), which counts re-reads that the L2 and
    the 256 MB Infinity Cache serve and can exceed the peak.
  * past_l2: the L2-to-fabric bytes of the operator from two rocprofv3
    counter runs of this script (FETCH_SIZE, then WRITE_SIZE, each scaled by
    what the counter reads for the 1 GiB device copy issued after the timed
    region), over its time, against the rate random-row gathers reach when
    the Infinity Cache serves every L2 miss, measured in the same run (the
    same kernel over a uniformly random graph from a table of the same size);
    for the 61.9M-edge rows, whose table the cache cannot hold, against the
    HBM peak.  Reported while the library sources hash to the digest recorded
    with the counters, else null.
Two rows of the 61.9M-edge R-MAT graph (2,449,029 nodes, D=100 fp32: a 980 MB
table, four times the Infinity Cache), timed after the step, are the
HBM-bound reference: copy_u/sum and u_dot_v.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
       [--no-c4] [--mark]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "g-SpMM/g-SDDMM edge·feat/s and HBM GB/s vs peak, 114.6M-edge R-MAT, D=128"
HBM_PEAK_GBS = 8000.0
CSRC = os.path.join(ROOT, "paper_1909_01315_amd", "csrc")

# L2-to-fabric bytes per operator (fetched, written) from two rocprofv3
# counter runs of this script (FETCH_SIZE, then WRITE_SIZE, per dispatch,
# summed over the dispatches of each operator, each counter scaled by what it
# reads for the 1 GiB device copy after the timed region), for the library
# sources with this digest; any other source state reports null.
MEASURED_TRAFFIC = {
    "sources_sha256": "7f7701f6fc9b713ff8f3b24049a6ba68ebc0e87e1322d39ee4146982e95e644c",
    "ops": {
        "gsddmm u_add_v": (975519108, 3770025728),
        "leaky_relu": (3667139078, 3667379328),
        "edge_softmax": (6693548516, 3711487648),
        "gspmm u_mul_e/sum": (15841954416, 578011776),
        "gspmm_backward u_mul_e/sum (dX, d_attention)": (42347297902, 4399529344),
        "edge_softmax_backward": (10913796995, 3733532992),
        "leaky_relu_backward": (7334258701, 3667254272),
        "gsddmm_backward u_add_v": (19963675419, 31044640),
        "gspmm copy_u/mean": (10630264301, 578010240),
        "gspmm_backward copy_u/mean": (11704602589, 577952128),
        "gspmm copy_u/max": (11250424239, 1045948672),
        "gspmm_backward copy_u/max": (5065323504, 2435773984),
        "gsddmm u_dot_v": (11754932283, 3821094848),
        "c4 gspmm copy_u/sum": (21624294348, 1144795882),
        "c4 gsddmm u_dot_v": (22160211589, 386185669),
    },
}


def sources_digest():
    """sha256 over the library's kernel and host sources (name + content)."""
    import hashlib

    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def op_bytes(N, E, D, H, s=4, idx=4, ptr=4):
    """Per operator of the step: (bytes that must cross HBM at least once,
    gather-model bytes).  s: bytes per feature element; idx: per index; ptr:
    per row offset.  Node tables are N x D (or N x H) elements, edge tensors
    E x H; the reverse-graph passes also walk the reverse edge ids."""
    off = (N + 1) * ptr
    nD, nH, eH = N * D * s, N * H * s, E * H * s
    ix = E * idx
    return {
        # el, er read, scores written; the in-CSR's neighbour ids
        "gsddmm u_add_v": (2 * nH + ix + off + eH, E * H * s + ix + nH + eH + off),
        "leaky_relu": (2 * eH, 2 * eH),
        "edge_softmax": (2 * eH + off, 2 * eH + off),
        # X and the attention read, Z written
        "gspmm u_mul_e/sum": (nD + eH + ix + off + nD, E * D * s + eH + ix + nD + off),
        # dZ, X, attention read; dX, d attention written; reverse ids and edge ids
        "gspmm_backward u_mul_e/sum (dX, d_attention)": (2 * nD + eH + 2 * ix + off + nD + eH,
                                                         E * D * s + eH + 2 * ix + nD + nD + eH + off),
        "edge_softmax_backward": (3 * eH + off, 3 * eH + off),
        "leaky_relu_backward": (3 * eH, 3 * eH),
        # ds read; d_el over the reverse graph (edge ids), d_er over the in-CSR
        "gsddmm_backward u_add_v": (eH + ix + 2 * off + 2 * nH, 2 * eH + ix + 2 * off + 2 * nH),
        "gspmm copy_u/mean": (nD + ix + off + nD, E * D * s + ix + off + nD),
        # dh and in-degrees read, dX written, the reverse CSR's neighbour ids
        "gspmm_backward copy_u/mean": (nD + N * 4 + ix + off + nD, E * D * s + ix + off + N * 4 + nD),
        # X read; value, arg node and arg edge written
        "gspmm copy_u/max": (nD + ix + off + 3 * nD, E * D * s + ix + off + 3 * nD),
        # dm and arg edges read, dX written; reverse ids and the position of every edge
        "gspmm_backward copy_u/max": (3 * nD + 2 * ix + off, E * D * s + 2 * ix + off + 3 * nD),
        # X read once (both operands), scores written
        "gsddmm u_dot_v": (nD + ix + off + eH, E * D * s + ix + nD + eH + off),
    }


def timed_events(fn, stream, reps=10, warm=2):
    import torch
    for _ in range(warm):
        fn()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        e1.synchronize()
        ts.append(e0.elapsed_time(e1) / 1e3)
    ts.sort()
    return ts[len(ts) // 2]


def gather_ceiling(gnnk, synth, n_rows, D, stream, dev):
    """The rate at which random-row gathers can leave L2 when every miss is
    served by the Infinity Cache: this library's copy_u/sum over a graph of
    2^24 edges with uniformly random sources and destinations (in-degree 64
    on average, no locality beyond chance) from an (n_rows, D) fp32 table that
    the 256 MB Infinity Cache holds, in GB/s of rows gathered (the L2 of an
    XCD holds 4 MB of the table, so nearly every gathered row leaves L2)."""
    import torch

    sg = synth.uniform_graph(synth.SEED_BASE + 900, n_rows, 1 << 18, 1 << 24, name="gather ceiling")
    g = gnnk.Graph.from_coo(torch.from_numpy(sg.src).to(dev), torch.from_numpy(sg.dst).to(dev), n_rows, 1 << 18)
    table = torch.from_numpy(synth.normal(synth.SEED_BASE + 901, "table", (n_rows, 1, D))).to(dev)
    out = torch.empty((1 << 18, 1, D), dtype=torch.float32, device=dev)
    g.lend_scratch(g.scratch_bytes(D), stream)
    t = timed_events(lambda: gnnk.gspmm(g, "copy_lhs", "sum", table, out=out), stream, reps=10)
    g.destroy()
    return (sg.n_edges * D * 4) / t / 1e9, (
        f"gnnk copy_u/sum over {sg.n_edges} uniformly random edges (2^18 destinations) from a {n_rows} x {D} "
        f"fp32 table held by the Infinity Cache: rows gathered per second")


def cpu_baseline(sg, X_host, a_gpu, target_seconds=20.0):
    """The oracle, single-threaded, on a bounded sample of destination rows."""
    import numpy as np

    import oracle as orc

    og = orc.OGraph(sg.src, sg.dst, sg.n_src, sg.n_dst)
    ind = np.bincount(sg.dst, minlength=sg.n_dst)
    a = a_gpu.cpu().numpy()
    rng = np.random.default_rng(0)
    order = rng.permutation(sg.n_dst)

    # two calibration samples separate the oracle's fixed cost (its in-list
    # build over all edges) from the per-edge cost; then size the sample
    def timed(budget):
        rows = order[np.cumsum(ind[order]) <= budget]
        t0 = time.perf_counter()
        orc.gspmm(og, "mul", "sum", X_host, a, rows=rows)
        return rows, time.perf_counter() - t0

    r1, t1 = timed(100_000)
    r2, t2 = timed(1_000_000)
    e1, e2 = int(ind[r1].sum()), int(ind[r2].sum())
    per_edge = max((t2 - t1) / max(e2 - e1, 1), 1e-12)
    fixed = max(t1 - per_edge * e1, 0.0)
    budget = int(min(sg.n_edges, max(e2, (target_seconds - fixed) / per_edge)))
    rows, t = timed(budget)
    e = int(ind[rows].sum())
    D = X_host.shape[1] * X_host.shape[2]
    return {
        "value": e * D / t,
        "unit": "edge·feat/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"oracle gspmm u_mul_e/sum (X (N,8,16) fp32, attention (E,8,1)) on {rows.size} random "
                   f"destination rows of the same graph holding {e} edges; {t:.1f} s wall, including the "
                   f"oracle's own in-list build; host has {os.cpu_count()} logical CPUs, 1 used"),
    }


def roofline_row(name, ms, b_hbm, b_gather, traffic, ceiling_gbs, ceiling_what):
    t = ms / 1e3
    ach = b_hbm / t / 1e9
    row = {
        "kernel": name,
        "bound": "hbm",
        "achieved": ach,
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": ach / HBM_PEAK_GBS,
        "traffic": None,
        "ms": ms,
        "bytes_hbm_min": b_hbm,
        "bytes_gather_model": b_gather,
        "effective_gbs": b_gather / t / 1e9,
        "past_l2": None,
    }
    if traffic is not None:
        tb = traffic[0] + traffic[1]
        row["traffic"] = tb
        row["past_l2"] = {"bound": "l2-fabric", "achieved": tb / t / 1e9, "peak": ceiling_gbs, "unit": "GB/s",
                          "frac": tb / t / 1e9 / ceiling_gbs, "fetch": traffic[0], "write": traffic[1],
                          "peak_what": ceiling_what}
    return row


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle's CPU timing")
    ap.add_argument("--no-c4", action="store_true", help="skip the 61.9M-edge HBM-bound reference rows")
    ap.add_argument("--mark", action="store_true",
                    help="a one-element fill kernel before every operator of the first timed step and after its "
                         "last one, and around the 12 calls of each 61.9M-edge row, so that a counter run can tell "
                         "which dispatches belong to which operator")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus}); "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1909_01315_amd import gnnk, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    gnnk.load()  # fails loudly when the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t0 = time.perf_counter()
    sg = synth.graph_c3()
    N, E = sg.n_dst, sg.n_edges
    log(f"graph: R-MAT N={N} E={E} generated in {time.perf_counter() - t0:.1f} s")
    fs, gs = synth.feat_seed(3), synth.grad_seed(3)
    H, F = 8, 16
    D = H * F
    X_host = synth.normal(fs, "X", (N, H, F))
    el = torch.from_numpy(synth.normal(fs, "el", (N, H, 1))).to(dev)
    er = torch.from_numpy(synth.normal(fs, "er", (N, H, 1))).to(dev)
    X = torch.from_numpy(X_host).to(dev)
    X128 = X.view(N, 1, D)
    dZ = torch.from_numpy(synth.normal(gs, "dZ", (N, H, F))).to(dev)
    dh = torch.from_numpy(synth.normal(gs, "dh", (N, 1, D))).to(dev)
    dm = torch.from_numpy(synth.normal(gs, "dm", (N, 1, D))).to(dev)
    t0 = time.perf_counter()
    g = gnnk.Graph.from_coo(torch.from_numpy(sg.src).to(dev), torch.from_numpy(sg.dst).to(dev), N, N)
    torch.cuda.synchronize()
    info = g.info()
    log(f"graph formats built in {time.perf_counter() - t0:.1f} s: {info['hub_dst_rows']} hub rows in "
        f"{info['segments_in']} segments, {info['empty_dst_rows']} empty rows, max in-degree {info['max_in_degree']}")
    stream = torch.cuda.current_stream()
    # the scratch the step needs, lent before timing (messages of D columns,
    # with the max/min backward's winner masks)
    g.lend_scratch(g.scratch_bytes(D, argmax=True), stream)

    f32 = torch.float32
    e8 = lambda: torch.empty((E, H, 1), dtype=f32, device=dev)
    n8 = lambda: torch.empty((N, H, 1), dtype=f32, device=dev)
    nD = lambda: torch.empty((N, H, F), dtype=f32, device=dev)
    b = dict(s=e8(), s2=e8(), a=e8(), da=e8(), ds2=e8(), ds=e8(), M=e8(), Z=nD(), dX=nD(), del_=n8(), der=n8(),
             h=nD(), dXs=nD(), m=nD(), dXm=nD(),
             au=torch.empty((N, 1, D), dtype=torch.int32, device=dev),
             ae=torch.empty((N, 1, D), dtype=torch.int32, device=dev))

    # (name, message columns counted per edge, function)
    ops = [
        ("gsddmm u_add_v", H, lambda: gnnk.gsddmm(g, "add", el, "u", er, "v", out=b["s"])),
        ("leaky_relu", 0, lambda: gnnk.edge_leaky_relu(b["s"], 0.2, y=b["s2"])),
        ("edge_softmax", H, lambda: gnnk.edge_softmax(g, b["s2"], out=b["a"])),
        ("gspmm u_mul_e/sum", D, lambda: gnnk.gspmm(g, "mul", "sum", X, b["a"], out=b["Z"])),
        ("gspmm_backward u_mul_e/sum (dX, d_attention)", 2 * D,
         lambda: gnnk.gspmm_backward(g, "mul", "sum", X, b["a"], dZ, grad_lhs=b["dX"], grad_rhs=b["da"])),
        ("edge_softmax_backward", H, lambda: gnnk.edge_softmax_backward(g, b["a"], b["da"], grad_score=b["ds2"])),
        ("leaky_relu_backward", 0, lambda: gnnk.edge_leaky_relu_backward(b["s"], b["ds2"], 0.2, dx=b["ds"])),
        ("gsddmm_backward u_add_v", 2 * H,
         lambda: gnnk.gsddmm_backward(g, "add", el, "u", er, "v", b["ds"], grad_lhs=b["del_"], grad_rhs=b["der"])),
        ("gspmm copy_u/mean", D, lambda: gnnk.gspmm(g, "copy_lhs", "mean", X128, out=b["h"].view(N, 1, D))),
        ("gspmm_backward copy_u/mean", D,
         lambda: gnnk.gspmm_backward(g, "copy_lhs", "mean", X128, None, dh, grad_lhs=b["dXs"].view(N, 1, D))),
        ("gspmm copy_u/max", D,
         lambda: gnnk.gspmm(g, "copy_lhs", "max", X128, out=b["m"].view(N, 1, D), want_args=True, arg_lhs=b["au"],
                            arg_rhs=b["ae"])),
        ("gspmm_backward copy_u/max", D,
         lambda: gnnk.gspmm_backward(g, "copy_lhs", "max", X128, None, dm, arg_rhs=b["ae"],
                                     grad_lhs=b["dXm"].view(N, 1, D))),
        ("gsddmm u_dot_v", D, lambda: gnnk.gsddmm(g, "dot", X, "u", X, "v", out=b["M"])),
    ]
    edge_feat_per_step = float(E) * sum(c for _, c, _ in ops)
    mark = torch.zeros(1, dtype=torch.int32, device=dev) if args.mark else None

    evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(ops) + 1)]

    def step(record, marked=False):
        if record:
            evs[0].record(stream)
        for i, (_, _, fn) in enumerate(ops):
            if marked:
                mark.fill_(i + 1)
            fn()
            if record:
                evs[i + 1].record(stream)
        if marked:
            mark.fill_(len(ops) + 1)

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step(False)
    lent = {k: v.data_ptr() for k, v in g._lent.items()}
    torch.cuda.synchronize()
    per_op = np.zeros(len(ops))
    # timed region: exactly K steps between two device synchronisations
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(True, marked=mark is not None and k == 0)
        # events are read after the step is queued; reading waits for them
        evs[-1].synchronize()
        for i in range(len(ops)):
            per_op[i] += evs[i].elapsed_time(evs[i + 1])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = wall * 1e3 / args.steps
    per_op /= args.steps
    value = edge_feat_per_step / (ms_per_step / 1e3)
    assert {k: v.data_ptr() for k, v in g._lent.items()} == lent, "no scratch was lent inside the timed region"
    log(f"{ms_per_step:.2f} ms/step, {value:.4g} edge-feat/s")
    for (name, _, _), t in zip(ops, per_op):
        log(f"  {name:48s} {t:9.3f} ms")

    # after the timed region: plain 1 GiB device copies (rocprofv3 counter
    # runs scale FETCH_SIZE / WRITE_SIZE by what a copy of known size reads,
    # and their median time gives the stream bandwidth of this machine), then
    # the random-row gather ceilings of both tables
    cal_src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    cal_dst = torch.empty_like(cal_src)
    cal_bytes = cal_src.numel() * 4
    copy_gbs = 2 * cal_bytes / timed_events(lambda: cal_dst.copy_(cal_src), stream, reps=5, warm=0) / 1e9
    torch.cuda.synchronize()
    del cal_src, cal_dst
    log(f"stream bandwidth on this box: copy {copy_gbs:.0f} GB/s (read + write)")
    ceil3, ceil3_what = gather_ceiling(gnnk, synth, N, D, stream, dev)
    log(f"past-L2 gather ceiling ({N} x {D} table in the Infinity Cache): {ceil3:.0f} GB/s")

    digest_ok = MEASURED_TRAFFIC["sources_sha256"] == sources_digest()
    traffic = MEASURED_TRAFFIC["ops"] if digest_ok else {}
    nbytes = op_bytes(N, E, D, H)
    rows = []
    for (name, _, _), t in zip(ops, per_op):
        bh, bg = nbytes[name]
        rows.append(roofline_row(name, float(t), bh, bg, traffic.get(name), ceil3, ceil3_what))

    # the HBM-bound reference: the 61.9M-edge graph, whose 980 MB table is
    # four times the Infinity Cache
    if not args.no_c4:
        del b
        torch.cuda.empty_cache()
        t0 = time.perf_counter()
        s4 = synth.graph_c4()
        N4, E4, D4 = s4.n_dst, s4.n_edges, 100
        g4 = gnnk.Graph.from_coo(torch.from_numpy(s4.src).to(dev), torch.from_numpy(s4.dst).to(dev), N4, N4,
                                 ptr64=True)
        X4 = torch.from_numpy(synth.normal(synth.feat_seed(4), "X", (N4, 1, D4))).to(dev)
        Y4 = torch.from_numpy(synth.normal(synth.feat_seed(4), "Y", (N4, 1, D4))).to(dev)
        o4 = torch.empty((N4, 1, D4), dtype=f32, device=dev)
        m4 = torch.empty((E4, 1, 1), dtype=f32, device=dev)
        g4.lend_scratch(g4.scratch_bytes(D4), stream)
        log(f"c4 graph N={N4} E={E4} ready in {time.perf_counter() - t0:.1f} s")
        # the table is four times the Infinity Cache: bytes past L2 are HBM
        # traffic, against the HBM peak
        ceil4, ceil4_what = HBM_PEAK_GBS, "HBM peak (the 980 MB table is four times the Infinity Cache)"
        off4 = (N4 + 1) * 8
        for name, fn, bh, bg in (
                ("c4 gspmm copy_u/sum", lambda: gnnk.gspmm(g4, "copy_lhs", "sum", X4, out=o4),
                 2 * N4 * D4 * 4 + E4 * 4 + off4, E4 * D4 * 4 + E4 * 4 + off4 + N4 * D4 * 4),
                ("c4 gsddmm u_dot_v", lambda: gnnk.gsddmm(g4, "dot", X4, "u", Y4, "v", out=m4),
                 2 * N4 * D4 * 4 + E4 * 4 + off4 + E4 * 4, E4 * D4 * 4 + E4 * 4 + N4 * D4 * 4 + E4 * 4 + off4)):
            if mark is not None:
                mark.fill_(len(rows) + 1)
            t = timed_events(fn, stream, reps=10, warm=2)
            if mark is not None:
                mark.fill_(len(rows) + 1)
            rows.append(roofline_row(name, t * 1e3, bh, bg, traffic.get(name), ceil4, ceil4_what))
            log(f"  {name:48s} {t * 1e3:9.3f} ms")
        g4.destroy()

    dominant = max(rows[:len(ops)], key=lambda r: r["ms"])
    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle, one core)")
        cpu = cpu_baseline(sg, X_host, torch.from_numpy(synth.uniform(fs, "a_cpu", (E, H, 1), 0.0, 1.0)))
    step_hbm = sum(r["bytes_hbm_min"] for r in rows[:len(ops)])

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "edge·feat/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": ("R-MAT (0.57,0.19,0.19,0.05) N=232,965 E=114,600,000 dedup, D=128 fp32 as 8 heads x 16; "
                         "GAT fwd+bwd, SAGE mean fwd+bwd, max+argmax fwd+bwd, u_dot_v"),
            "num_nodes": N,
            "num_edges": E,
            "feat": D,
            "heads": H,
            "edge_feat_per_step": edge_feat_per_step,
            "accumulate": "f64",
        },
        "roofline": dominant,
        "rooflines": rows,
        "step_hbm_min_gbs": step_hbm / (ms_per_step / 1e3) / 1e9,
        "stream": {"copy_gbs": copy_gbs, "bytes": cal_bytes,
                   "what": "median of 5 device copies of 1 GiB, bytes read + written over time"},
        "traffic_digest_match": digest_ok,
        "ops_ms": {name: round(float(t), 4) for (name, _, _), t in zip(ops, per_op)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    g.destroy()


if __name__ == "__main__":
    main()
