"""Pins of the CPU oracle to routes other than itself (CPU only).

Each test checks an oracle function against something the paper or the
mathematics fixes: the dense special cases of Section 3 (SpMM Y = A X and
SDDMM W = A .* (X X^T)), the incidence-matrix form of the definitions
(gather = one-hot matrix product, reduce = transposed one-hot product),
brute force on tiny graphs, central finite differences of the fp64 oracle
(Theorem 1's gradients), the reverse-graph identity of Theorem 1, invariants
(degree counts, softmax normalisation and shift invariance), permutation
invariance, the R-GCN aggregation formula of Appendix D (experiment configurations), and
library routines (numpy/scipy/torch) for CSR construction, softmax and bf16
rounding.
"""
import itertools

import numpy as np
import pytest

import oracle as orc

OPS_BIN = ["add", "sub", "mul", "div"]
OPS_SPMM = ["copy_lhs", "copy_rhs"] + OPS_BIN


def tiny_graph(seed=0, n_src=9, n_dst=7, n_edges=40, iso=True):
    """Random multigraph with duplicates and (when square) self-loops; node n_dst-1 isolated when iso."""
    rng = np.random.default_rng(seed)
    src = rng.integers(0, n_src, n_edges).astype(np.int32)
    hi = n_dst - 1 if iso else n_dst
    dst = rng.integers(0, hi, n_edges).astype(np.int32)
    # force a duplicated edge and (if square) a self-loop
    src[1], dst[1] = src[0], dst[0]
    if n_src == n_dst:
        src[2] = dst[2]
    return orc.OGraph(src, dst, n_src, n_dst)


def onehots(g):
    S = np.zeros((g.n_edges, g.n_src))
    T = np.zeros((g.n_edges, g.n_dst))
    S[np.arange(g.n_edges), g.src] = 1.0
    T[np.arange(g.n_edges), g.dst] = 1.0
    return S, T


def elem(op, a, b):
    return {"add": a + b, "sub": a - b, "mul": a * b, "div": a / b, "copy_lhs": a + 0 * b, "copy_rhs": b + 0 * a}[op]


def positive(rng, shape):
    return rng.uniform(0.5, 2.0, shape)


# ---------------------------------------------------------------------------
# P1: dense and incidence-matrix forms of the definitions


def test_spmm_special_case_dense_AX():
    """Section 3: g-SpMM with u_mul_e and scalar edge weights is SpMM Y = A X."""
    g = tiny_graph(1)
    rng = np.random.default_rng(1)
    X = rng.standard_normal((g.n_src, 1, 5))
    w = rng.uniform(0, 1, (g.n_edges, 1, 1))
    A = np.zeros((g.n_dst, g.n_src))
    for e in range(g.n_edges):  # A[v, u] = sum of weights of edges u -> v
        A[g.dst[e], g.src[e]] += w[e, 0, 0]
    Z = orc.gspmm(g, "mul", "sum", X, w)
    np.testing.assert_allclose(Z[:, 0, :], A @ X[:, 0, :], rtol=1e-13, atol=1e-13)
    # copy_u with all-one weights is A with unit entries
    Z1 = orc.gspmm(g, "copy_lhs", "sum", X)
    A1 = (A != 0).astype(float) * 0
    for e in range(g.n_edges):
        A1[g.dst[e], g.src[e]] += 1
    np.testing.assert_allclose(Z1[:, 0, :], A1 @ X[:, 0, :], rtol=1e-13, atol=1e-13)


def test_sddmm_special_case_dense_XXt():
    """Section 3: SDDMM W = A .* (X Y^T): the dot score of edge e is (X Y^T)[src_e, dst_e]."""
    g = tiny_graph(2, n_src=8, n_dst=8)
    rng = np.random.default_rng(2)
    X = rng.standard_normal((8, 1, 6))
    Y = rng.standard_normal((8, 1, 6))
    M = orc.gsddmm(g, "dot", X, "u", Y, "v")
    full = X[:, 0, :] @ Y[:, 0, :].T
    np.testing.assert_allclose(M[:, 0, 0], full[g.src, g.dst], rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("op", OPS_SPMM)
@pytest.mark.parametrize("reduce", ["sum", "mean"])
@pytest.mark.parametrize("shapes", [((3, 4), (3, 4)), ((3, 4), (3, 1)), ((3, 4), (1, 1)), ((3, 1), (3, 4))])
def test_spmm_incidence_form(op, reduce, shapes):
    """z = T^T phi(S X, W) (sum) and D^-1 of that (mean): gather and reduce as one-hot products."""
    g = tiny_graph(3)
    rng = np.random.default_rng(3)
    (hl, fl), (hr, fr) = shapes
    X = rng.standard_normal((g.n_src, hl, fl))
    W = positive(rng, (g.n_edges, hr, fr))
    S, T = onehots(g)
    H, F = max(hl, hr), max(fl, fr)
    if op == "copy_lhs":
        H, F = hl, fl
    if op == "copy_rhs":
        H, F = hr, fr
    gx = (S @ X.reshape(g.n_src, -1)).reshape(g.n_edges, hl, fl)
    if op == "copy_lhs":
        msg = gx
    elif op == "copy_rhs":
        msg = W
    else:
        msg = elem(op, np.broadcast_to(gx, (g.n_edges, H, F)), np.broadcast_to(W, (g.n_edges, H, F)))
    msg = msg.reshape(g.n_edges, -1)
    ref = (T.T @ msg).reshape(g.n_dst, H, F)
    if reduce == "mean":
        deg = T.sum(0)
        ref = ref / np.maximum(deg, 1)[:, None, None]
    Z = orc.gspmm(g, op, reduce, X if op != "copy_rhs" else None, W if op != "copy_lhs" else None)
    np.testing.assert_allclose(Z, ref, rtol=1e-12, atol=1e-12)
    assert np.all(Z[g.n_dst - 1] == 0), "isolated destination gives 0"


@pytest.mark.parametrize("op", OPS_SPMM + ["dot"])
@pytest.mark.parametrize("lt,rt", list(itertools.product("uev", "uev")))
def test_sddmm_incidence_form(op, lt, rt):
    """m = phi(gather_lt(L), gather_rt(R)) with gathers as one-hot products (identity for edges)."""
    g = tiny_graph(4, n_src=6, n_dst=6)
    rng = np.random.default_rng(4)
    S, T = onehots(g)
    G = {"u": S, "v": T, "e": np.eye(g.n_edges)}
    rows = {"u": g.n_src, "v": g.n_dst, "e": g.n_edges}
    L = rng.standard_normal((rows[lt], 2, 3))
    R = positive(rng, (rows[rt], 2, 3))
    gl = (G[lt] @ L.reshape(rows[lt], -1)).reshape(g.n_edges, 2, 3)
    gr = (G[rt] @ R.reshape(rows[rt], -1)).reshape(g.n_edges, 2, 3)
    if op == "dot":
        ref = (gl * gr).sum(-1, keepdims=True)
    else:
        ref = elem(op, gl, gr)
    M = orc.gsddmm(g, op, L, lt, R, rt)
    np.testing.assert_allclose(M, ref, rtol=1e-12, atol=1e-12)


def test_sddmm_broadcast_heads_feat():
    g = tiny_graph(5)
    rng = np.random.default_rng(5)
    X = rng.standard_normal((g.n_src, 4, 3))
    Y = rng.standard_normal((g.n_dst, 4, 1))
    M = orc.gsddmm(g, "mul", X, "u", Y, "v")
    np.testing.assert_allclose(M, X[g.src] * Y[g.dst], rtol=0, atol=0)
    D = orc.gsddmm(g, "dot", X, "u", Y, "v")
    np.testing.assert_allclose(D[:, :, 0], (X[g.src] * Y[g.dst]).sum(-1), rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------------------
# P2: invariants


def test_copy_u_sum_of_ones_is_in_degree():
    g = tiny_graph(6)
    ones = np.ones((g.n_src, 1, 3), dtype=np.float32)
    Z = orc.gspmm(g, "copy_lhs", "sum", ones)
    indeg = np.bincount(g.dst, minlength=g.n_dst)
    assert np.array_equal(Z[:, 0, 0], indeg.astype(np.float32))
    ind, outd = orc.degrees(g)
    assert np.array_equal(ind, indeg)
    assert np.array_equal(outd, np.bincount(g.src, minlength=g.n_src))


def test_mean_times_degree_is_sum():
    g = tiny_graph(7)
    X = np.random.default_rng(7).standard_normal((g.n_src, 1, 4))
    s = orc.gspmm(g, "copy_lhs", "sum", X)
    m = orc.gspmm(g, "copy_lhs", "mean", X)
    deg = np.bincount(g.dst, minlength=g.n_dst)
    np.testing.assert_allclose(m[:, 0, :] * deg[:, None], s[:, 0, :], rtol=1e-14, atol=1e-14)


def test_softmax_normalises_and_is_shift_invariant():
    g = tiny_graph(8, n_src=10, n_dst=10, n_edges=60)
    rng = np.random.default_rng(8)
    s = rng.standard_normal((g.n_edges, 3, 1)).astype(np.float32)
    a = orc.edge_softmax(g, s)
    S, T = onehots(g)
    colsum = T.T @ a.reshape(g.n_edges, -1).astype(np.float64)
    deg = T.sum(0)
    for v in range(g.n_dst):
        if deg[v] > 0:
            np.testing.assert_allclose(colsum[v], 1.0, atol=deg[v] * 2.0**-24)
    # a destination with exactly one in-edge gets exactly 1
    for v in np.nonzero(deg == 1)[0]:
        e = int(np.nonzero(g.dst == v)[0][0])
        assert np.all(a[e] == np.float32(1.0))
    # shift of every score by a per-destination constant
    c = rng.standard_normal((g.n_dst, 3, 1)).astype(np.float64)
    s64 = s.astype(np.float64)
    a1 = orc.edge_softmax(g, s64)
    a2 = orc.edge_softmax(g, s64 + c[g.dst])
    np.testing.assert_allclose(a1, a2, rtol=1e-12, atol=1e-15)


def test_softmax_single_edge_rows_exact():
    src = np.array([0, 1, 2], dtype=np.int32)
    dst = np.array([0, 1, 1], dtype=np.int32)
    g = orc.OGraph(src, dst, 3, 3)
    s = np.array([[5.0], [1.0], [1.0]], dtype=np.float32).reshape(3, 1, 1)
    a = orc.edge_softmax(g, s)
    assert a[0, 0, 0] == np.float32(1.0)
    assert a[1, 0, 0] == np.float32(0.5) and a[2, 0, 0] == np.float32(0.5)


# ---------------------------------------------------------------------------
# library routines: softmax per group, CSR by stable sort, bf16 rounding


def test_softmax_matches_scipy_per_group():
    from scipy.special import softmax

    g = tiny_graph(9, n_src=12, n_dst=12, n_edges=80)
    s = np.random.default_rng(9).standard_normal((g.n_edges, 2, 2))
    a = orc.edge_softmax(g, s)
    for v in range(g.n_dst):
        idx = np.nonzero(g.dst == v)[0]
        if idx.size:
            np.testing.assert_allclose(a[idx], softmax(s[idx], axis=0), rtol=1e-13, atol=1e-15)


def test_softmax_backward_dense_jacobian():
    g = tiny_graph(10, n_src=12, n_dst=12, n_edges=80)
    rng = np.random.default_rng(10)
    s = rng.standard_normal((g.n_edges, 2, 1))
    gout = rng.standard_normal((g.n_edges, 2, 1))
    a = orc.edge_softmax(g, s)
    ds = orc.edge_softmax_backward(g, a, gout)
    for v in range(g.n_dst):
        idx = np.nonzero(g.dst == v)[0]
        for h in range(2):
            av = a[idx, h, 0]
            J = np.diag(av) - np.outer(av, av)
            np.testing.assert_allclose(ds[idx, h, 0], J @ gout[idx, h, 0], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("reverse", [False, True])
def test_csr_matches_stable_argsort(reverse):
    g = tiny_graph(11, n_src=9, n_dst=7, n_edges=50)
    indptr, indices, eids = orc.csr(g, reverse)
    key = g.src if reverse else g.dst
    n = g.n_src if reverse else g.n_dst
    order = np.argsort(key, kind="stable")
    assert np.array_equal(eids, order)
    assert np.array_equal(indices, (g.dst if reverse else g.src)[order])
    assert np.array_equal(indptr, np.concatenate([[0], np.cumsum(np.bincount(key, minlength=n))]))


def test_bf16_rounding_matches_torch():
    import torch

    rng = np.random.default_rng(12)
    x = rng.standard_normal(20000).astype(np.float32) * np.float32(3.0)
    # exact ties: values whose low 16 bits are 0x8000, with even and odd kept LSB
    mant = rng.integers(0, 2**7, 2000).astype(np.uint32) << 16  # the 7 kept mantissa bits
    expo = rng.integers(100, 150, 2000).astype(np.uint32) << 23
    ties = (expo | mant | 0x8000).view(np.float32)
    ties2 = (expo | mant | 0x8001).view(np.float32)
    x = np.concatenate([x, ties, ties2, -ties, np.float32([0.0, -0.0, 1e-40, 3.4e38])])
    ours = orc.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_bf16_io_rounds_once_from_fp32():
    """bf16 outputs: fp64 sum -> fp32 -> bf16 (round to nearest even)."""
    g = tiny_graph(13)
    rng = np.random.default_rng(13)
    X = rng.standard_normal((g.n_src, 1, 8)).astype(np.float32)
    Xb = orc.round_bf16(X)
    Xw = orc.bf16_to_f32(Xb).astype(np.float64)
    out = orc.gspmm(g, "copy_lhs", "sum", Xb)
    ref = orc.gspmm(g, "copy_lhs", "sum", Xw)
    assert out.dtype == np.uint16
    assert np.array_equal(out, orc.round_bf16(ref.astype(np.float32)))


# ---------------------------------------------------------------------------
# P3: brute force max / min with argmax


@pytest.mark.parametrize("reduce", ["max", "min"])
@pytest.mark.parametrize("op", ["copy_lhs", "copy_rhs", "add", "mul"])
def test_max_min_brute_force(reduce, op):
    g = tiny_graph(14)
    rng = np.random.default_rng(14)
    # small integers make exact ties likely; duplicated edges give ties under copy_lhs
    X = rng.integers(-3, 4, (g.n_src, 2, 3)).astype(np.float32)
    W = rng.integers(-3, 4, (g.n_edges, 2, 1)).astype(np.float32)
    out, au, ae = orc.gspmm(g, op, reduce, X if op != "copy_rhs" else None, W if op != "copy_lhs" else None)
    H, F = out.shape[1:]
    for v in range(g.n_dst):
        for h in range(H):
            for f in range(F):
                best, be = None, -1
                for e in range(g.n_edges):  # ascending edge id
                    if g.dst[e] != v:
                        continue
                    x = X[g.src[e], h, f] if op != "copy_rhs" else None
                    w = W[e, h, 0] if op != "copy_lhs" else None
                    m = {"copy_lhs": x, "copy_rhs": w, "add": np.float32(x) + np.float32(w) if x is not None else None,
                         "mul": np.float32(x) * np.float32(w) if x is not None else None}[op]
                    if be < 0 or (m > best if reduce == "max" else m < best):
                        best, be = m, e
                if be < 0:
                    assert out[v, h, f] == 0 and ae[v, h, f] == -1 and au[v, h, f] == -1
                else:
                    assert out[v, h, f] == best and ae[v, h, f] == be and au[v, h, f] == g.src[be]


def test_max_tie_goes_to_smallest_edge():
    src = np.array([3, 1, 3, 2], dtype=np.int32)
    dst = np.array([0, 0, 0, 0], dtype=np.int32)
    g = orc.OGraph(src, dst, 4, 1)
    X = np.array([0, 7, 5, 7], dtype=np.float32).reshape(4, 1, 1)
    out, au, ae = orc.gspmm(g, "copy_lhs", "max", X)
    assert out[0, 0, 0] == 7 and ae[0, 0, 0] == 0 and au[0, 0, 0] == 3


# ---------------------------------------------------------------------------
# P4: central finite differences of the fp64 oracle (Theorem 1's gradients)


def fd_grad(fun, x, h=1e-6):
    g = np.zeros_like(x)
    flat = x.reshape(-1)
    gf = g.reshape(-1)
    for i in range(flat.size):
        old = flat[i]
        flat[i] = old + h
        fp = fun()
        flat[i] = old - h
        fm = fun()
        flat[i] = old
        gf[i] = (fp - fm) / (2 * h)
    return g


def spaced(rng, shape, lo=-2.0, gap=1e-2):
    """distinct values at least `gap` apart (max/min finite differences stay valid)"""
    n = int(np.prod(shape))
    vals = lo + gap * (rng.permutation(n) + rng.uniform(0.2, 0.8, n))
    return vals.reshape(shape)


@pytest.mark.parametrize("op", OPS_SPMM)
@pytest.mark.parametrize("reduce", ["sum", "mean", "max", "min"])
@pytest.mark.parametrize("shapes", [((2, 3), (2, 3)), ((2, 3), (2, 1)), ((2, 1), (2, 3))])
def test_gspmm_backward_finite_differences(op, reduce, shapes):
    g = tiny_graph(15, n_src=6, n_dst=5, n_edges=18)
    rng = np.random.default_rng(15)
    (hl, fl), (hr, fr) = shapes
    if op == "copy_lhs":
        hr, fr = hl, fl
    if op == "copy_rhs":
        hl, fl = hr, fr
    X = spaced(rng, (g.n_src, hl, fl)) if reduce in ("max", "min") else rng.standard_normal((g.n_src, hl, fl))
    W = 1.0 + spaced(rng, (g.n_edges, hr, fr), lo=0.0, gap=3e-2)
    L = X if op != "copy_rhs" else None
    R = W if op != "copy_lhs" else None
    res = orc.gspmm(g, op, reduce, L, R)
    out, ae = (res[0], res[2]) if reduce in ("max", "min") else (res, None)
    G = rng.standard_normal(out.shape)

    def loss():
        r = orc.gspmm(g, op, reduce, L, R)
        return float(np.sum(G * (r[0] if isinstance(r, tuple) else r)))

    gl, gr = orc.gspmm_backward(g, op, reduce, L, R, G, arg_e=ae)
    if L is not None:
        np.testing.assert_allclose(gl, fd_grad(loss, X), rtol=1e-6, atol=1e-7)
    if R is not None:
        np.testing.assert_allclose(gr, fd_grad(loss, W), rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("op", OPS_SPMM + ["dot"])
@pytest.mark.parametrize("lt,rt", [("u", "v"), ("u", "e"), ("e", "v"), ("v", "u"), ("u", "u")])
def test_gsddmm_backward_finite_differences(op, lt, rt):
    g = tiny_graph(16, n_src=6, n_dst=6, n_edges=16)
    rng = np.random.default_rng(16)
    rows = {"u": g.n_src, "v": g.n_dst, "e": g.n_edges}
    L = rng.standard_normal((rows[lt], 2, 3))
    R = 1.0 + rng.uniform(0, 1, (rows[rt], 2, 1))
    Lx = L if op != "copy_rhs" else None
    Rx = R if op != "copy_lhs" else None
    out = orc.gsddmm(g, op, Lx, lt, Rx, rt)
    G = rng.standard_normal(out.shape)

    def loss():
        return float(np.sum(G * orc.gsddmm(g, op, Lx, lt, Rx, rt)))

    gl, gr = orc.gsddmm_backward(g, op, Lx, lt, Rx, rt, G)
    if Lx is not None:
        np.testing.assert_allclose(gl, fd_grad(loss, L), rtol=1e-6, atol=1e-7)
    if Rx is not None:
        np.testing.assert_allclose(gr, fd_grad(loss, R), rtol=1e-6, atol=1e-7)


def test_edge_softmax_backward_finite_differences():
    g = tiny_graph(17, n_src=6, n_dst=6, n_edges=20)
    rng = np.random.default_rng(17)
    s = rng.standard_normal((g.n_edges, 2, 1))
    G = rng.standard_normal(s.shape)
    a = orc.edge_softmax(g, s)
    ds = orc.edge_softmax_backward(g, a, G)

    def loss():
        return float(np.sum(G * orc.edge_softmax(g, s)))

    np.testing.assert_allclose(ds, fd_grad(loss, s), rtol=1e-6, atol=1e-8)


def test_leaky_relu_against_torch_and_fd():
    import torch

    rng = np.random.default_rng(18)
    x = rng.standard_normal((50, 4, 1)).astype(np.float32)
    x[0, 0, 0] = 0.0
    y = orc.leaky_relu(x, 0.2)
    ref = torch.nn.functional.leaky_relu(torch.from_numpy(x), 0.2).numpy()
    assert np.array_equal(y, ref)
    x64 = x.astype(np.float64) + 0.05 * np.sign(x + 1e-3)  # keep away from the kink
    G = rng.standard_normal(x64.shape)
    dx = orc.leaky_relu_backward(x64, G, 0.2)
    np.testing.assert_allclose(dx, fd_grad(lambda: float(np.sum(G * orc.leaky_relu(x64, 0.2))), x64),
                               rtol=1e-6, atol=1e-8)
    # derivative at exactly 0 is the slope
    z = np.zeros((1, 1, 1), dtype=np.float32)
    assert orc.leaky_relu_backward(z, np.ones_like(z), 0.2)[0, 0, 0] == np.float32(0.2)


# ---------------------------------------------------------------------------
# P5: Theorem 1 -- the node gradient is a g-SpMM on the reverse graph


@pytest.mark.parametrize("op", ["copy_lhs", "mul", "div"])
def test_gspmm_dx_is_spmm_on_reverse_graph(op):
    g = tiny_graph(19)
    rev = orc.OGraph(g.dst, g.src, g.n_dst, g.n_src)  # (u,e,v) -> (v,e,u), ids kept
    rng = np.random.default_rng(19)
    X = rng.standard_normal((g.n_src, 2, 3))
    W = 1.0 + rng.uniform(0, 1, (g.n_edges, 2, 1))
    R = W if op != "copy_lhs" else None
    dZ = rng.standard_normal((g.n_dst, 2, 3))
    dx, _ = orc.gspmm_backward(g, op, "sum", X, R, dZ, want_rhs=False)
    # the lemma's message on the reverse graph: copy -> dZ, mul -> dZ * w, div -> dZ / w
    via = orc.gspmm(rev, op if op != "copy_lhs" else "copy_lhs", "sum", dZ, R)
    np.testing.assert_allclose(dx, via, rtol=1e-13, atol=1e-13)


def test_gsddmm_dot_grads_are_spmms():
    """u_dot_v: dX = sum over out-edges dM * Y[v] (reverse graph), dY = sum over in-edges dM * X[u]."""
    g = tiny_graph(20, n_src=7, n_dst=7)
    rev = orc.OGraph(g.dst, g.src, g.n_dst, g.n_src)
    rng = np.random.default_rng(20)
    X = rng.standard_normal((7, 2, 4))
    Y = rng.standard_normal((7, 2, 4))
    dM = rng.standard_normal((g.n_edges, 2, 1))
    dx, dy = orc.gsddmm_backward(g, "dot", X, "u", Y, "v", dM)
    np.testing.assert_allclose(dx, orc.gspmm(rev, "mul", "sum", Y, dM), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(dy, orc.gspmm(g, "mul", "sum", X, dM), rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------------------
# P6: permutation invariance


def test_relabelling_permutes_outputs():
    g = tiny_graph(21, n_src=8, n_dst=8, n_edges=50)
    rng = np.random.default_rng(21)
    X = rng.standard_normal((8, 1, 3))
    W = rng.uniform(0.5, 1.5, (g.n_edges, 1, 1))
    pn = rng.permutation(8)  # new id of node i is pn[i]
    pe = rng.permutation(g.n_edges)  # new edge id of edge e is pe[e]
    src2 = np.empty_like(g.src)
    dst2 = np.empty_like(g.dst)
    src2[pe] = pn[g.src]
    dst2[pe] = pn[g.dst]
    g2 = orc.OGraph(src2, dst2, 8, 8)
    X2 = np.empty_like(X)
    X2[pn] = X
    W2 = np.empty_like(W)
    W2[pe] = W
    Z = orc.gspmm(g, "mul", "sum", X, W)
    Z2 = orc.gspmm(g2, "mul", "sum", X2, W2)
    np.testing.assert_allclose(Z2[pn], Z, rtol=1e-13, atol=1e-13)
    M = orc.gsddmm(g, "dot", X, "u", X, "v")
    M2 = orc.gsddmm(g2, "dot", X2, "u", X2, "v")
    np.testing.assert_allclose(M2[pe], M, rtol=1e-13, atol=1e-13)
    # max on tie-free data agrees exactly, arg edges map through pe
    Xs = spaced(rng, (8, 1, 3))
    Xs2 = np.empty_like(Xs)
    Xs2[pn] = Xs
    o, au, ae = orc.gspmm(g, "copy_lhs", "max", Xs)
    o2, au2, ae2 = orc.gspmm(g2, "copy_lhs", "max", Xs2)
    assert np.array_equal(o2[pn], o)
    m = au >= 0
    # duplicated edges tie exactly, so the winning source (not edge) is what relabels
    assert np.array_equal(au2[pn][m], pn[au[m]])
    assert np.array_equal(g2.src[ae2[pn][m]], pn[g.src[ae[m]]])


# ---------------------------------------------------------------------------
# P7: R-GCN aggregation (Appendix D, experiment configurations): sum_r D_r^-1 A_r X_r


def test_rgcn_encoding_matches_dense_formula():
    rng = np.random.default_rng(22)
    n, r, E = 6, 3, 40
    src = rng.integers(0, n, E)
    dst = rng.integers(0, n, E)
    et = rng.integers(0, r, E)
    Xr = rng.standard_normal((r, n, 4))  # per-relation transformed features H W_r
    ref = np.zeros((n, 4))
    for rel in range(r):
        A = np.zeros((n, n))
        for e in np.nonzero(et == rel)[0]:
            A[dst[e], src[e]] += 1.0
        deg = A.sum(1)
        Dinv = np.diag(np.where(deg > 0, 1.0 / np.maximum(deg, 1), 0.0))
        ref += Dinv @ A @ Xr[rel]
    cnt = np.array([np.sum((dst == dst[e]) & (et == et[e])) for e in range(E)])
    g = orc.OGraph((et * n + src).astype(np.int32), dst.astype(np.int32), r * n, n)
    Z = orc.gspmm(g, "mul", "sum", Xr.reshape(r * n, 1, 4), (1.0 / cnt).reshape(E, 1, 1))
    np.testing.assert_allclose(Z[:, 0, :], ref, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------------------
# edge cases and sampled mode


def test_empty_graph_and_isolated_nodes():
    g = orc.OGraph(np.zeros(0, np.int32), np.zeros(0, np.int32), 3, 4)
    X = np.ones((3, 1, 2), dtype=np.float32)
    assert np.all(orc.gspmm(g, "copy_lhs", "sum", X) == 0)
    assert np.all(orc.gspmm(g, "copy_lhs", "mean", X) == 0)
    o, au, ae = orc.gspmm(g, "copy_lhs", "max", X)
    assert np.all(o == 0) and np.all(au == -1) and np.all(ae == -1)
    assert orc.gsddmm(g, "dot", X, "u", np.ones((4, 1, 2), np.float32), "v").shape == (0, 1, 1)
    dx, _ = orc.gspmm_backward(g, "copy_lhs", "sum", X, None, np.ones((4, 1, 2), np.float32))
    assert np.all(dx == 0)


def test_sampled_rows_match_full():
    g = tiny_graph(23, n_src=10, n_dst=10, n_edges=70)
    rng = np.random.default_rng(23)
    X = rng.standard_normal((10, 2, 3)).astype(np.float32)
    W = rng.uniform(0, 1, (g.n_edges, 2, 1)).astype(np.float32)
    rows = np.array([7, 0, 3, 3])
    full = orc.gspmm(g, "mul", "sum", X, W)
    assert np.array_equal(orc.gspmm(g, "mul", "sum", X, W, rows=rows), full[rows])
    edges = np.array([5, 1, 60])
    fm = orc.gsddmm(g, "dot", X, "u", X, "v")
    assert np.array_equal(orc.gsddmm(g, "dot", X, "u", X, "v", edges=edges), fm[edges])
    s = rng.standard_normal((g.n_edges, 2, 1)).astype(np.float32)
    fa = orc.edge_softmax(g, s)
    sa, eids = orc.edge_softmax(g, s, rows=rows)
    assert np.array_equal(sa, fa[eids])
    assert np.array_equal(np.sort(eids[:np.sum(g.dst == 7)]), np.nonzero(g.dst == 7)[0])
    dZ = rng.standard_normal((10, 2, 3)).astype(np.float32)
    fdx, fdw = orc.gspmm_backward(g, "mul", "sum", X, W, dZ)
    sdx, _ = orc.gspmm_backward(g, "mul", "sum", X, W, dZ, want_rhs=False, sel=rows)
    assert np.array_equal(sdx, fdx[rows])
    _, sdw = orc.gspmm_backward(g, "mul", "sum", X, W, dZ, want_lhs=False, sel=edges)
    assert np.array_equal(sdw, fdw[edges])


def test_rejects_bad_shapes():
    g = tiny_graph(24)
    X = np.ones((g.n_src, 2, 3))
    W = np.ones((g.n_edges, 3, 1))  # heads do not broadcast
    with pytest.raises(ValueError):
        orc.gspmm(g, "mul", "sum", X, W)
    with pytest.raises(ValueError):
        orc.gspmm(g, "mul", "sum", X[:-1], np.ones((g.n_edges, 2, 1)))
