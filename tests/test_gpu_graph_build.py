"""Device construction of the graph formats against the oracle's CSR (a stable
counting sort by row written from the definition): offsets, indices, edge
ids, degrees and the schedule counts compare bit for bit.  The shapes cover
every number of radix passes of the row sorts (one row: none; up to 2^8,
2^16, 2^24 and more rows: one to four), ragged last tiles, a single hot row,
unsorted edge lists (non-identity edge ids), int64 offsets, and the error
paths of both constructors."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_1909_01315_amd import gnnk
from _gpu import Pair, assert_close, assert_exact, check_formats, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def reset_options():
    yield
    gnnk.set_option("seg_edges", 0)


def random_edges(seed, n_src, n_dst, E, sort_by_dst=False):
    rng = np.random.default_rng(seed)
    src = rng.integers(0, n_src, E).astype(np.int32)
    dst = rng.integers(0, n_dst, E).astype(np.int32)
    if sort_by_dst:
        order = np.argsort(dst, kind="stable")
        src, dst = src[order], dst[order]
    return src, dst


@pytest.mark.parametrize("n_src,n_dst,E", [
    (1, 1, 5000),            # one row each way: no radix pass
    (7, 250, 10000),         # one pass
    (300, 70000, 12289),     # two and three passes, ragged last tile
    (2 ** 24 + 5, 1000, 20000),   # four passes for the reverse graph
    (1000, 2 ** 24 + 3, 9000),    # four passes for the in-CSR, mostly empty rows
    (50, 60, 1),
    (4096, 4096, 4096 * 3),  # whole tiles
])
def test_formats_every_pass_count(n_src, n_dst, E):
    src, dst = random_edges(n_src + n_dst + E, n_src, n_dst, E)
    p = Pair(src, dst, n_src, n_dst)
    check_formats(p)


@pytest.mark.parametrize("ptr64", [False, True])
def test_hot_row_and_hub_segments(ptr64):
    """Every edge but a few into destination 0 and out of source 3: one
    digit takes almost every key of a pass, and with 64-edge segments the
    hub tables have hundreds of entries; a g-SpMM over them must match."""
    gnnk.set_option("seg_edges", 64)
    E = 4096 * 3 + 17
    rng = np.random.default_rng(5)
    src = np.full(E, 3, np.int32)
    dst = np.zeros(E, np.int32)
    k = rng.choice(E, 40, replace=False)
    src[k] = rng.integers(0, 500, 40)
    dst[k] = rng.integers(0, 500, 40)
    p = Pair(src, dst, 500, 500, ptr64=ptr64)
    check_formats(p, seg_edges=64)
    X = rng.standard_normal((500, 1, 8)).astype(np.float32)
    assert_close(gnnk.gspmm(p.g, "copy_lhs", "sum", dev(X)), orc.gspmm(p.o, "copy_lhs", "sum", X))
    dZ = rng.standard_normal((500, 1, 8)).astype(np.float32)
    dX, _ = gnnk.gspmm_backward(p.g, "copy_lhs", "sum", dev(X), None, dev(dZ))
    ref, _ = orc.gspmm_backward(p.o, "copy_lhs", "sum", X, None, dZ)
    assert_close(dX, ref)


def test_identity_edge_ids_detected():
    src, dst = random_edges(8, 900, 800, 30000, sort_by_dst=True)
    p = Pair(src, dst, 900, 800)
    assert p.g.info()["identity_eids"] == 1
    check_formats(p)
    src2, dst2 = random_edges(8, 900, 800, 30000)
    q = Pair(src2, dst2, 900, 800)
    assert q.g.info()["identity_eids"] == 0
    check_formats(q)


def test_csr_constructor_matches_coo():
    """from_csr on the oracle's in-CSR (identity and shuffled edge ids, int32
    and int64 offsets) builds the same reverse graph as from_coo."""
    src, dst = random_edges(12, 3000, 2500, 70000)
    o = orc.OGraph(src, dst, 3000, 2500)
    ip, ii, ie = orc.csr(o)
    rp, ri, re_ = orc.csr(o, reverse=True)
    for ptr_dtype in (np.int32, np.int64):
        g = gnnk.Graph.from_csr(dev(ip.astype(ptr_dtype)), dev(ii), dev(ie), 3000)
        hp, hi, he = g.csr_export(reverse=True)
        assert_exact(hp.cpu().numpy().astype(np.int64), rp, "reverse indptr")
        assert_exact(hi, ri, "reverse indices")
        assert_exact(he, re_, "reverse eids")
        assert g.info()["identity_eids"] == 0
        g.destroy()
    # identity ids: the in-CSR positions are the edge ids
    order = np.argsort(dst, kind="stable")
    o2 = orc.OGraph(src[order], dst[order], 3000, 2500)
    ip2, ii2, _ = orc.csr(o2)
    g = gnnk.Graph.from_csr(dev(ip2), dev(ii2), None, 3000)
    assert g.info()["identity_eids"] == 1
    rp2, ri2, re2 = orc.csr(o2, reverse=True)
    hp, hi, he = g.csr_export(reverse=True)
    assert_exact(hi, ri2)
    assert_exact(he, re2)
    g.destroy()


def expect_einval(fn):
    with pytest.raises(gnnk.GnnkError) as e:
        fn()
    assert e.value.status == gnnk.EINVAL


def test_invalid_edge_lists_are_rejected():
    src = torch.tensor([0, 1, 2], dtype=torch.int32, device="cuda")
    dst = torch.tensor([0, 1, 1], dtype=torch.int32, device="cuda")
    expect_einval(lambda: gnnk.Graph.from_coo(src, dst, 2, 2))          # src 2 >= num_src
    expect_einval(lambda: gnnk.Graph.from_coo(src, dst - 1, 3, 2))      # dst -1
    ind = torch.tensor([0, 2, 1, 3], dtype=torch.int32, device="cuda")  # decreasing
    idx = torch.tensor([0, 1, 2], dtype=torch.int32, device="cuda")
    expect_einval(lambda: gnnk.Graph.from_csr(ind, idx, None, 3))
    ind = torch.tensor([0, 1, 2, 4], dtype=torch.int32, device="cuda")  # does not end at E
    expect_einval(lambda: gnnk.Graph.from_csr(ind, idx, None, 3))
    ind = torch.tensor([0, 1, 2, 3], dtype=torch.int32, device="cuda")
    expect_einval(lambda: gnnk.Graph.from_csr(ind, idx, None, 2))       # index 2 >= num_src
    dup = torch.tensor([0, 2, 2], dtype=torch.int32, device="cuda")
    expect_einval(lambda: gnnk.Graph.from_csr(ind, idx, dup, 3))        # not a permutation
    big = torch.tensor([0, 1, 3], dtype=torch.int32, device="cuda")
    expect_einval(lambda: gnnk.Graph.from_csr(ind, idx, big, 3))        # id out of range
    # a valid handle afterwards
    g = gnnk.Graph.from_csr(ind, idx, torch.tensor([2, 0, 1], dtype=torch.int32, device="cuda"), 3)
    # position p holds edge eids[p] from source p to destination p, so source
    # u's only out-edge is eids[u]
    hp, hi, he = g.csr_export(reverse=True)
    assert hi.cpu().tolist() == [0, 1, 2] and he.cpu().tolist() == [2, 0, 1]
    g.destroy()


def test_build_is_deterministic_and_timed():
    """Two builds of the same 2M-edge list give identical structures; the
    build time is printed for the record."""
    src, dst = random_edges(21, 200000, 200000, 2000000)
    s, d = dev(src), dev(dst)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    g1 = gnnk.Graph.from_coo(s, d, 200000, 200000)
    e1.record()
    e1.synchronize()
    g2 = gnnk.Graph.from_coo(s, d, 200000, 200000)
    print(f"device build, 2M edges, 200k nodes: {e0.elapsed_time(e1):.2f} ms")
    for rev in (False, True):
        a, b = g1.csr_export(reverse=rev), g2.csr_export(reverse=rev)
        for x, y in zip(a, b):
            assert torch.equal(x, y)
    g1.destroy()
    g2.destroy()


def test_graphs_without_nodes_or_edges():
    """zero sources, zero destinations, or both: the build and every pass
    accept empty operands and write nothing out of range"""
    z = torch.zeros(0, dtype=torch.int32, device="cuda")
    for ns, nd in ((0, 0), (0, 7), (5, 0)):
        g = gnnk.Graph.from_coo(z, z, ns, nd)
        info = g.info()
        assert info["num_edges"] == 0 and info["max_in_degree"] == 0 and info["max_out_degree"] == 0
        X = torch.randn(ns, 1, 8, device="cuda")
        out = gnnk.gspmm(g, "copy_lhs", "sum", X)
        assert out.shape == (nd, 1, 8) and torch.all(out == 0)
        m, au, ae = gnnk.gspmm(g, "copy_lhs", "max", X, want_args=True)
        assert torch.all(ae == -1)
        dz = torch.randn(nd, 1, 8, device="cuda")
        dx, _ = gnnk.gspmm_backward(g, "copy_lhs", "sum", X, None, dz)
        assert dx.shape == (ns, 1, 8) and torch.all(dx == 0)
        hp, hi, he = g.csr_export(reverse=True)
        assert hp.numel() == ns + 1 and torch.all(hp == 0)
        g.destroy()


def test_maximum_edge_count():
    """2^31 - 2^16 - 1 edges, the largest count int32 edge ids and positions
    allow (4,096 nodes, every row a hub row of about 2^19 edges): the device
    build and g-SpMM copy_u/sum of ones give the exact in- and out-degrees
    (torch.bincount; degrees stay below 2^24, exact in fp32)."""
    E = (1 << 31) - (1 << 16) - 1
    n = 4096
    gen = torch.Generator(device="cuda").manual_seed(7)
    src = torch.randint(0, n, (E,), dtype=torch.int32, device="cuda", generator=gen)
    dst = torch.randint(0, n, (E,), dtype=torch.int32, device="cuda", generator=gen)
    g = gnnk.Graph.from_coo(src, dst, n, n, ptr64=True)
    assert g.info()["num_edges"] == E
    ones = torch.ones(n, 1, 1, device="cuda")
    indeg = torch.bincount(dst.long(), minlength=n).float()
    assert torch.equal(gnnk.gspmm(g, "copy_lhs", "sum", ones).view(-1), indeg)
    outdeg = torch.bincount(src.long(), minlength=n).float()
    dx, _ = gnnk.gspmm_backward(g, "copy_lhs", "sum", ones, None, ones)
    assert torch.equal(dx.view(-1), outdeg)
    g.destroy()


def test_segment_size_follows_the_edge_count():
    """seg_edges 0 (the default): for the in-CSR the next power of two of
    E / 8192 within [64, 512], for the reverse graph's CSR the next power of
    two of E / 2048 within [64, 2048] and, for the passes of either CSR that
    gather node rows, of E / 16384 within [64, 256]; a fixed option sets all
    four"""
    for E, Si, So, Sg in ((1000, 64, 64, 64), (200_000, 64, 128, 64), (1_000_000, 128, 512, 64),
                          (3_000_000, 512, 2048, 256), (9_000_000, 512, 2048, 256)):
        src, dst = random_edges(E, 5000, 5000, E)
        p = Pair(src, dst, 5000, 5000)
        info = p.g.info()
        assert (info["seg_edges"], info["seg_edges_out"], info["seg_edges_gather"],
                info["seg_edges_in_gather"]) == (Si, So, Sg, Sg), E
        check_formats(p)
    gnnk.set_option("seg_edges", 300)
    src, dst = random_edges(1, 50, 50, 1000)
    info = Pair(src, dst, 50, 50).g.info()
    assert info["seg_edges"] == 300 and info["seg_edges_out"] == 300 and info["seg_edges_gather"] == 300
    assert info["seg_edges_in_gather"] == 300
