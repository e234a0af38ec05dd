"""Pins for the oracle's backward pass: the transposed (source-major) CSR of
Sec. 2.2 (the CSC cache used by the backward pass) and the gradients of the
sum / mean / max aggregation of Eq. (1) with respect to x and to the edge
weights.

Pins used: numpy's stable argsort for the transpose, transposing twice,
reverse-mode differentiation by torch autograd in float64 on the CPU (a
library routine independent of the oracle), the adjoint identity
<A x, g> = <x, A^T g> against the already pinned forward oracle, closed-form
counts for max routing, and the first-edge rule on duplicate edges.
"""
import numpy as np
import pytest
import torch

import graphgen
import oracle

DYADIC = np.array([-2.0, -1.0, -0.5, 0.5, 1.0, 2.0], np.float32)


def simple_graph(seed, n_dst, n_src, e, f):
    """Random graph without repeated (src, dst) pairs, so that the messages of
    a row are distinct and max has no ties; weights are powers of two, so
    every message w * x is exact in fp32."""
    rng = np.random.default_rng(seed)
    src = rng.integers(0, n_src, e).astype(np.int32)
    dst = rng.integers(0, n_dst, e).astype(np.int32)
    _, keep = np.unique(dst.astype(np.int64) * n_src + src, return_index=True)
    keep = np.sort(keep)
    src, dst = src[keep], dst[keep]
    x = rng.standard_normal((n_src, f)).astype(np.float32)
    g = rng.standard_normal((n_dst, f)).astype(np.float32)
    w = DYADIC[rng.integers(0, DYADIC.size, src.size)]
    return src, dst, x, g, w


def row_of(rowptr):
    return np.repeat(np.arange(rowptr.size - 1), np.diff(rowptr))


# ---- transpose -------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("n_dst,n_src,e", [(1, 1, 0), (50, 70, 400), (300, 20, 3000),
                                           (20, 300, 3000)])
def test_transpose_is_stable_sort_by_source(seed, n_dst, n_src, e):
    src = graphgen.uniform_ints(seed, 1, e, n_src)
    dst = graphgen.uniform_ints(seed, 2, e, n_dst)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, n_dst, n_src=n_src)
    rpt, colt, post = oracle.csr_transpose(rp, col, n_src)
    order = np.argsort(col, kind="stable")
    assert np.array_equal(post, order)
    assert np.array_equal(colt, row_of(rp)[order])
    assert np.array_equal(rpt, np.concatenate([[0], np.cumsum(np.bincount(col, minlength=n_src))]))


@pytest.mark.parametrize("seed", range(3))
def test_transpose_twice_gives_back_the_csr(seed):
    src = graphgen.uniform_ints(seed, 1, 5000, 300)
    dst = graphgen.uniform_ints(seed, 2, 5000, 200)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 200, n_src=300)
    rpt, colt, post = oracle.csr_transpose(rp, col, 300)
    rp2, col2, post2 = oracle.csr_transpose(rpt, colt, 200)
    # back to destination-major: same rows, each row's edges now by source id
    assert np.array_equal(rp2, rp)
    q = post[post2]  # forward position of each edge of the double transpose
    assert np.array_equal(np.sort(q), np.arange(col.size))
    assert np.array_equal(row_of(rp)[q], row_of(rp)) and np.array_equal(col[q], col2)
    for r in range(200):
        seg = slice(rp[r], rp[r + 1])
        assert np.array_equal(col2[seg], np.sort(col[seg], kind="stable"))
    # a CSR whose rows are sorted by source comes back unchanged
    rp3, col3, _ = oracle.csr_transpose(*oracle.csr_transpose(rp2, col2, 300)[:2], 200)
    assert np.array_equal(rp3, rp2) and np.array_equal(col3, col2)


# ---- gradients against torch autograd -------------------------------------------

def autograd_reference(rp, col, x, g, w, reduce):
    """Forward aggregation in float64 torch ops (index_add / scatter_reduce)
    and its gradients by autograd."""
    rows = torch.from_numpy(row_of(rp))
    colt = torch.from_numpy(col.astype(np.int64))
    xt = torch.from_numpy(x.astype(np.float64)).requires_grad_(True)
    wt = torch.from_numpy(w.astype(np.float64)).requires_grad_(True)
    n_dst, f = rp.size - 1, x.shape[1]
    msg = wt[:, None] * xt[colt]
    if reduce == "max":
        out = torch.zeros(n_dst, f, dtype=torch.float64).scatter_reduce(
            0, rows[:, None].expand(-1, f), msg, "amax", include_self=False)
    else:
        out = torch.zeros(n_dst, f, dtype=torch.float64).index_add(0, rows, msg)
        if reduce == "mean":
            deg = torch.from_numpy(np.diff(rp)).clamp(min=1).to(torch.float64)
            out = out / deg[:, None]
    (out * torch.from_numpy(g.astype(np.float64))).sum().backward()
    return xt.grad.numpy(), wt.grad.numpy()


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
@pytest.mark.parametrize("weighted", [False, True])
def test_gradients_match_autograd(seed, reduce, weighted):
    n_dst, n_src = 40, 55
    src, dst, x, g, w = simple_graph(seed, n_dst, n_src, 150, 6)
    rp, col, _, wc = oracle.coo_to_csr(src, dst, n_dst, n_src=n_src, val=w)
    assert (np.diff(rp) == 0).any()  # empty rows are covered
    if not weighted:
        wc = np.ones_like(wc)
    fwd = oracle.spmm(rp, col, x=x, w=wc if weighted else None)
    am = fwd["argmax"] if reduce == "max" else None
    gx, _ = oracle.spmm_backward_x(rp, col, n_src, reduce, g=g, w=wc if weighted else None,
                                   argout=am)
    gw, _ = oracle.spmm_backward_w(rp, col, reduce, x=x, g=g, argout=am)
    ref_x, ref_w = autograd_reference(rp, col, x, g, wc, reduce)
    np.testing.assert_allclose(gx, ref_x, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(gw, ref_w, rtol=1e-12, atol=1e-12)


def test_bf16_gradient_input_widens_exactly():
    src, dst, x, g, w = simple_graph(7, 30, 30, 300, 8)
    rp, col, _, wc = oracle.coo_to_csr(src, dst, 30, val=w)
    gb = graphgen.f32_to_bf16(g)
    gwide = graphgen.bf16_to_f32(gb)
    for reduce in ("sum", "mean"):
        a, _ = oracle.spmm_backward_x(rp, col, 30, reduce, g_bf16=gb, w=wc)
        b, _ = oracle.spmm_backward_x(rp, col, 30, reduce, g=gwide, w=wc)
        assert np.array_equal(a, b)
        a, _ = oracle.spmm_backward_w(rp, col, reduce, x=x, g_bf16=gb)
        b, _ = oracle.spmm_backward_w(rp, col, reduce, x=x, g=gwide)
        assert np.array_equal(a, b)


# ---- adjoint identity and closed forms ---------------------------------------------

@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("reduce", ["sum", "mean"])
def test_adjoint_identity(seed, reduce):
    # sum and mean are linear in x and in w: <A(x, w), g> = <x, grad_x> = <w, grad_w>
    g_ = graphgen.mixed_graph(seed, n=2000, e=30_000, f=16)
    rng = np.random.default_rng(seed)
    w = DYADIC[rng.integers(0, DYADIC.size, g_.E)]
    rp, col, _, wc = oracle.coo_to_csr(g_.src, g_.dst, g_.n_dst, n_src=g_.n_src, val=w)
    G = rng.standard_normal((g_.n_dst, 16)).astype(np.float32)
    fwd = oracle.spmm(rp, col, x=g_.x, w=wc)[reduce]
    lhs = float(np.sum(fwd * G))
    gx, _ = oracle.spmm_backward_x(rp, col, g_.n_src, reduce, g=G, w=wc)
    gw, _ = oracle.spmm_backward_w(rp, col, reduce, x=g_.x, g=G)
    assert abs(lhs - float(np.sum(gx * g_.x))) <= 1e-10 * np.sum(np.abs(gx * g_.x))
    assert abs(lhs - float(np.sum(gw * wc))) <= 1e-10 * np.sum(np.abs(gw * wc))


@pytest.mark.parametrize("seed", range(3))
def test_max_backward_routes_one_unit_per_output(seed):
    # w = 1, g = 1: grad_x[u, f] counts the rows whose max for f comes from u
    g_ = graphgen.mixed_graph(seed, n=1500, e=20_000, f=8)
    rp, col, _, _ = oracle.coo_to_csr(g_.src, g_.dst, g_.n_dst, n_src=g_.n_src)
    am = oracle.spmm(rp, col, x=g_.x)["argmax"]
    ones = np.ones((g_.n_dst, 8), np.float32)
    gx, sc = oracle.spmm_backward_x(rp, col, g_.n_src, "max", g=ones, argout=am)
    for f in range(8):
        hit = am[:, f] >= 0
        cnt = np.bincount(col[am[hit, f]], minlength=g_.n_src)
        assert np.array_equal(gx[:, f], cnt)
    assert np.array_equal(gx, sc)
    # grad_w with x = 1: each edge gets the number of features it wins
    gw, _ = oracle.spmm_backward_w(rp, col, "max", x=np.ones((g_.n_src, 8), np.float32), g=ones,
                                   argout=am)
    wins = np.zeros(col.size)
    np.add.at(wins, am[am >= 0], 1)
    assert np.array_equal(gw, wins)


def test_max_backward_duplicate_edges_first_wins():
    # two copies of the same edge into row 0: the first CSR position takes it all
    src = np.array([1, 1, 0], np.int32)
    dst = np.array([0, 0, 1], np.int32)
    x = np.array([[1.0, -3.0], [2.0, 5.0]], np.float32)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 2)
    am = oracle.spmm(rp, col, x=x)["argmax"]
    assert am.tolist() == [[0, 0], [2, 2]]
    g = np.array([[10.0, 20.0], [1.0, 2.0]], np.float32)
    gx, _ = oracle.spmm_backward_x(rp, col, 2, "max", g=g, argout=am)
    assert gx.tolist() == [[1.0, 2.0], [10.0, 20.0]]
    gw, _ = oracle.spmm_backward_w(rp, col, "max", x=x, g=g, argout=am)
    assert gw.tolist() == [10.0 * 2.0 + 20.0 * 5.0, 0.0, 1.0 * 1.0 + 2.0 * -3.0]


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_listed_rows_equal_full_computation(reduce):
    g_ = graphgen.mixed_graph(3, n=1200, e=15_000, f=8)
    rp, col, _, wc = oracle.coo_to_csr(g_.src, g_.dst, g_.n_dst, n_src=g_.n_src, val=g_.w)
    am = oracle.spmm(rp, col, x=g_.x, w=wc)["argmax"]
    G = np.random.default_rng(0).standard_normal((g_.n_dst, 8)).astype(np.float32)
    full, fsc = oracle.spmm_backward_x(rp, col, g_.n_src, reduce, g=G, w=wc, argout=am)
    rows = np.array([5, 0, g_.n_src - 1, 77], np.int64)
    part, psc = oracle.spmm_backward_x(rp, col, g_.n_src, reduce, g=G, w=wc, argout=am, rows=rows)
    assert np.array_equal(part, full[rows]) and np.array_equal(psc, fsc[rows])
    fw, _ = oracle.spmm_backward_w(rp, col, reduce, x=g_.x, g=G, argout=am)
    drows = np.array([3, 900, 11], np.int64)
    pw, _ = oracle.spmm_backward_w(rp, col, reduce, x=g_.x, g=G, argout=am, rows=drows)
    sel = np.concatenate([np.arange(rp[r], rp[r + 1]) for r in drows])
    assert np.array_equal(pw[sel], fw[sel])
    assert np.isnan(np.delete(pw, sel)).all()
