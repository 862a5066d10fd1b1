"""Edge softmax and its backward on hub rows: one destination with 40,000
in-edges, destinations whose degree sits just below, at and above the
segment sizes (64, 256, 2048), empty destinations, rows wider than one
pass of 64 lanes, edges in destination order and shuffled (edge ids through
the map), fp32 and bf16, against the oracle at the tolerances of
tests/_gpu.py.  A row of 40,000 edges has values near 2.5e-5, below the
absolute part of the fp32 tolerance, so the forward is also held to 1e-5
relative to each value alone."""
import functools

import numpy as np
import pytest

import oracle as orc
from paper_1909_01315_amd import gnnk
from _gpu import Pair, as_f64, assert_close, dev, host

pytestmark = pytest.mark.gpu

N = 600
SPECIAL = [63, 64, 65, 127, 128, 129, 255, 256, 257, 1000, 2047, 2048, 2049, 4097]


@pytest.fixture(autouse=True)
def reset_options():
    yield
    gnnk.set_option("seg_edges", 0)


def hub_edges(shuffled):
    rng = np.random.default_rng(7100 + shuffled)
    dst = [np.full(40_000, 5)]
    for k, d in enumerate(SPECIAL):
        dst.append(np.full(d, 10 + k))
    dst.append(rng.integers(100, N, 20_000))  # background rows of degree about 40
    dst = np.concatenate(dst).astype(np.int32)
    src = rng.integers(0, N, dst.size).astype(np.int32)
    if shuffled:
        p = rng.permutation(dst.size)
        src, dst = src[p], dst[p]
    return src, dst


def values(seed, shape, bf16):
    a = np.random.default_rng(seed).standard_normal(shape).astype(np.float32)
    return orc.round_bf16(a) if bf16 else a


@functools.lru_cache(maxsize=2)  # the two edge orders of one shape alternate
def case(shuffled, H, F, bf16):
    """edges, inputs and the oracle's results (independent of the segment size)"""
    src, dst = hub_edges(shuffled)
    o = orc.OGraph(src, dst, N, N)
    s = values(11 + H * F, (src.size, H, F), bf16)
    g = values(12 + H * F, (src.size, H, F), bf16)
    a = orc.edge_softmax(o, s)
    return src, dst, s, g, a, orc.edge_softmax_backward(o, a, g)


@pytest.mark.parametrize("shuffled", [0, 1])
@pytest.mark.parametrize("seg", [0, 256, 2048])
@pytest.mark.parametrize("H,F", [(8, 1), (4, 16), (1, 300), (3, 129)])
@pytest.mark.parametrize("bf16", [False, True])
def test_softmax_hub_rows(shuffled, seg, H, F, bf16):
    gnnk.set_option("seg_edges", seg)
    src, dst, s, g, a, ref_ds = case(shuffled, H, F, bf16)
    p = Pair(src, dst, N, N)
    a_gpu = gnnk.edge_softmax(p.g, dev(s))
    ds_gpu = gnnk.edge_softmax_backward(p.g, dev(a), dev(g))
    if bf16:
        assert_close(a_gpu, a, kind="bf16", name="softmax bf16")
        assert_close(ds_gpu, ref_ds, kind="bf16", name="softmax backward bf16")
        return
    assert_close(a_gpu, a, name="softmax")
    assert_close(ds_gpu, ref_ds, name="softmax backward")
    # forward, relative to each value alone: the exponential is within a few
    # units of 2^-24 times (1 + |s - max|) of exp (|s - max| < 10 here)
    ga, ra = as_f64(host(a_gpu)).reshape(a.shape), as_f64(a)
    err = np.abs(ga - ra)
    assert np.all(err <= 1e-5 * np.abs(ra)), f"softmax: max rel err {np.max(err / np.maximum(np.abs(ra), 1e-300)):.3g}"
    # every non-empty row sums to 1
    sums = np.zeros((N, H, F))
    np.add.at(sums, dst, ga)
    rows = np.unique(dst)
    assert np.allclose(sums[rows], 1.0, rtol=0, atol=1e-4)
