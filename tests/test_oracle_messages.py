"""Pins for the oracle's edge-materialized path (explanation mode, Sec. 2.4,
with the PyG 1 materialization recalled in Sec. 2.2): messages gathered into
an E x F table in CSR order, edited by a callback c, aggregated per
destination; and the gradients of that pipeline.

Pins used: closed forms (features that encode their own row index, dyadic
weights and masks whose products are exact), equality with the already
pinned fused aggregation (identity callback; an edge mask equals a weighted
aggregation when every product is exact), brute-force Python loops with a
nonlinear callback, scipy.sparse for the segment sums, reverse-mode
differentiation by torch autograd in float64 (a library routine independent of
the oracle) for every gradient and for the whole explainer chain, the adjoint
identity, and numpy einsum for the per-edge dot products.
"""
import numpy as np
import pytest
import scipy.sparse as sp
import torch

import graphgen
import oracle

DYADIC = np.array([-2.0, -1.0, -0.5, 0.25, 0.5, 1.0, 2.0], np.float32)


def graph(seed, n_dst, n_src, e, f, distinct=False):
    """Random COO graph (duplicates kept unless distinct), N(0,1) features,
    dyadic weights and a dyadic edge mask."""
    rng = np.random.default_rng(seed)
    src = rng.integers(0, n_src, e).astype(np.int32)
    dst = rng.integers(0, n_dst, e).astype(np.int32)
    if distinct:
        _, keep = np.unique(dst.astype(np.int64) * n_src + src, return_index=True)
        keep = np.sort(keep)
        src, dst = src[keep], dst[keep]
    x = rng.standard_normal((n_src, f)).astype(np.float32)
    w = DYADIC[rng.integers(0, DYADIC.size, src.size)]
    mask = DYADIC[rng.integers(0, DYADIC.size, src.size)]
    g = rng.standard_normal((n_dst, f)).astype(np.float32)
    return src, dst, x, w, mask, g


def row_of(rowptr):
    return np.repeat(np.arange(rowptr.size - 1), np.diff(rowptr))


# ---- the gather (MESSAGE step, materialized) -----------------------------------------

@pytest.mark.parametrize("seed", range(3))
def test_gather_decodes_the_source_index(seed):
    n_src, F = 3000, 16
    x = (np.arange(n_src, dtype=np.float32)[:, None] * 1024
         + np.arange(F, dtype=np.float32)[None, :])  # exact: < 2^24
    idx = graphgen.uniform_ints(seed, 1, 5000, n_src)
    msg = oracle.message_gather(idx, x=x)
    s = msg[:, 0].astype(np.int64) // 1024
    assert np.array_equal(s, idx)
    assert np.array_equal(msg - msg[:, :1], np.broadcast_to(np.arange(F, dtype=np.float32), msg.shape))
    w = DYADIC[np.random.default_rng(seed).integers(0, DYADIC.size, idx.size)]
    msgw = oracle.message_gather(idx, x=x, w=w)
    assert np.array_equal(msgw, msg * w[:, None])  # dyadic: every product exact


def test_gather_bf16_widens_exactly():
    rng = np.random.default_rng(1)
    xb = graphgen.f32_to_bf16(rng.standard_normal((50, 24)).astype(np.float32))
    idx = rng.integers(0, 50, 700).astype(np.int32)
    msg = oracle.message_gather(idx, x_bf16=xb)
    assert np.array_equal(msg.view(np.uint32), graphgen.bf16_to_f32(xb)[idx].view(np.uint32))


def test_gather_rejects_bad_index():
    with pytest.raises(ValueError):
        oracle.message_gather(np.array([0, 5], np.int32), x=np.zeros((5, 2), np.float32))


def test_gather_weighted_rounds_once():
    # 1/3 is not dyadic: the message is the fp32 rounding of the exact product
    x = np.array([[1.0, 3.0, 0.1]], np.float32)
    w = np.array([np.float32(1.0) / np.float32(3.0)], np.float32)
    msg = oracle.message_gather(np.zeros(1, np.int32), x=x, w=w)
    exact = x[0].astype(np.float64) * np.float64(w[0])
    assert np.array_equal(msg[0], exact.astype(np.float32))


# ---- aggregation of materialized messages ----------------------------------------------

@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("bf16", [False, True])
def test_identity_callback_equals_fused_aggregation(seed, weighted, bf16):
    src, dst, x, w, _, _ = graph(seed, 40, 30, 600, 8)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 40, n_src=30)
    w_csr = w[np.argsort(dst, kind="stable")] if weighted else None
    kw = {"x_bf16": graphgen.f32_to_bf16(x)} if bf16 else {"x": x}
    agg, msg = oracle.spmm_materialized(rp, col, w=w_csr, **kw)
    ref = oracle.spmm(rp, col, w=w_csr, **kw)
    for k in ("sum", "mean", "scale", "argmax"):
        assert np.array_equal(agg[k], ref[k]), k
    assert np.array_equal(agg["max"].view(np.uint32), ref["max"].view(np.uint32))
    assert msg.shape == (col.size, 8)


@pytest.mark.parametrize("seed", range(4))
def test_edge_mask_callback_equals_weighted_aggregation(seed):
    """c(m)_p = mask[perm[p]] * m_p with dyadic mask and weights: every product
    is exact, so it is the fused aggregation with weights w * mask."""
    src, dst, x, w, mask, _ = graph(seed, 50, 40, 900, 6)
    rp, col, perm, _ = oracle.coo_to_csr(src, dst, 50, n_src=40)
    w_csr = w[perm]
    agg, _ = oracle.spmm_materialized(
        rp, col, x=x, w=w_csr, callback=lambda m: oracle.message_scale(m, mask, perm.astype(np.int32)))
    ref = oracle.spmm(rp, col, x=x, w=(w_csr * mask[perm]).astype(np.float32))
    for k in ("sum", "mean", "argmax"):
        assert np.array_equal(agg[k], ref[k]), k
    assert np.array_equal(agg["max"].view(np.uint32), ref["max"].view(np.uint32))


def test_callback_brute_force_tiny():
    """A nonlinear callback (tanh plus a per-edge shift), aggregated by
    Python loops over the COO edges in stable destination order."""
    src, dst, x, w, _, _ = graph(7, 6, 5, 25, 3)
    rp, col, perm, _ = oracle.coo_to_csr(src, dst, 6, n_src=5)

    def c(m):
        return (np.tanh(m.astype(np.float64)) + 0.125 * np.arange(m.shape[0])[:, None]).astype(np.float32)

    agg, _ = oracle.spmm_materialized(rp, col, x=x, callback=c)
    for v in range(6):
        edges = [e for e in range(src.size) if dst[e] == v]  # COO order = CSR order in the row
        for f in range(3):
            ms = []
            for e in edges:
                p = int(np.nonzero(perm == e)[0][0])
                ms.append(np.float32(np.tanh(np.float64(x[src[e], f])) + 0.125 * p))
            s = sum(float(m) for m in ms)
            assert agg["sum"][v, f] == pytest.approx(s, rel=1e-14, abs=1e-14)
            if ms:
                best = int(np.argmax(ms))  # first maximum
                assert agg["argmax"][v, f] == rp[v] + best
                assert agg["max"][v, f] == ms[best]
                assert agg["mean"][v, f] == pytest.approx(s / len(ms), rel=1e-14, abs=1e-14)
            else:
                assert agg["argmax"][v, f] == -1 and agg["max"][v, f] == 0.0


@pytest.mark.parametrize("seed", range(3))
def test_aggregate_matches_scipy_segment_sums(seed):
    rng = np.random.default_rng(seed)
    n, E, F = 200, 3000, 5
    deg = rng.multinomial(E, rng.dirichlet(np.ones(n) * 0.3))
    rp = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
    msg = rng.standard_normal((E, F)).astype(np.float32)
    agg = oracle.aggregate_messages(rp, msg)
    A = sp.csr_matrix((np.ones(E), np.arange(E), rp), shape=(n, E))
    ref = A @ msg.astype(np.float64)
    np.testing.assert_allclose(agg["sum"], ref, rtol=1e-13, atol=1e-12)
    empty = deg == 0
    assert np.all(agg["argmax"][empty] == -1) and np.all(agg["sum"][empty] == 0)


def test_aggregate_empty_graph():
    rp = np.zeros(4, np.int64)
    agg = oracle.aggregate_messages(rp, np.zeros((0, 3), np.float32))
    assert np.all(agg["sum"] == 0) and np.all(agg["argmax"] == -1) and np.all(agg["max"] == 0)


# ---- gradients ------------------------------------------------------------------------

def torch_aggregate(m, row, n, reduce, deg):
    F = m.shape[1]
    if reduce == "max":
        out = torch.zeros(n, F, dtype=m.dtype).scatter_reduce(
            0, torch.from_numpy(row)[:, None].expand(-1, F), m, reduce="amax", include_self=False)
        return out
    s = torch.zeros(n, F, dtype=m.dtype).index_add(0, torch.from_numpy(row), m)
    if reduce == "mean":
        s = s / torch.from_numpy(np.maximum(deg, 1).astype(np.float64))[:, None]
    return s


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
@pytest.mark.parametrize("gbf16", [False, True])
def test_message_backward_matches_autograd(seed, reduce, gbf16):
    src, dst, x, _, _, g = graph(seed, 200, 40, 700, 5, distinct=True)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 200, n_src=40)
    msg = oracle.message_gather(col, x=x)
    agg = oracle.aggregate_messages(rp, msg)
    gk = {"g_bf16": graphgen.f32_to_bf16(g)} if gbf16 else {"g": g}
    gw = graphgen.bf16_to_f32(graphgen.f32_to_bf16(g)) if gbf16 else g
    dmsg = oracle.message_backward(rp, reduce, argout=agg["argmax"], **gk)
    deg = np.diff(rp)
    m = torch.from_numpy(msg.astype(np.float64)).requires_grad_(True)
    out = torch_aggregate(m, row_of(rp), 200, reduce, deg)
    (out * torch.from_numpy(gw.astype(np.float64))).sum().backward()
    ref = m.grad.numpy()
    # the oracle rounds each gradient once to fp32 (exact for sum and max)
    assert np.array_equal(dmsg, ref.astype(np.float32))
    assert np.any(deg == 0)


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
def test_message_backward_adjoint(reduce):
    src, dst, x, w, _, g = graph(11, 80, 50, 2000, 7)
    rp, col, perm, _ = oracle.coo_to_csr(src, dst, 80, n_src=50)
    msg = oracle.message_gather(col, x=x, w=w[perm])
    agg = oracle.aggregate_messages(rp, msg)
    dmsg = oracle.message_backward(rp, reduce, g=g, argout=agg["argmax"])
    out = {"sum": agg["sum"], "mean": agg["mean"], "max": agg["max"].astype(np.float64)}[reduce]
    lhs = float(np.sum(out * g.astype(np.float64)))
    rhs = float(np.sum(msg.astype(np.float64) * dmsg.astype(np.float64)))
    assert rhs == pytest.approx(lhs, rel=1e-6)


def test_message_backward_max_routes_each_feature_once():
    src, dst, x, _, _, _ = graph(3, 30, 30, 500, 9)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 30, n_src=30)
    agg = oracle.aggregate_messages(rp, oracle.message_gather(col, x=x))
    ones = np.ones((30, 9), np.float32)
    dmsg = oracle.message_backward(rp, "max", g=ones, argout=agg["argmax"])
    nonempty = np.diff(rp) > 0
    assert dmsg.sum() == 9 * nonempty.sum()  # one edge per (non-empty row, feature)
    counts = np.zeros((30, 9))
    np.add.at(counts, row_of(rp), dmsg)
    assert np.array_equal(counts, np.where(nonempty[:, None], 1.0, 0.0) * ones)


@pytest.mark.parametrize("seed", range(3))
def test_edge_dot_matches_einsum(seed):
    rng = np.random.default_rng(seed)
    E, n_b, F = 500, 70, 11
    a = rng.standard_normal((E, F)).astype(np.float32)
    b = rng.standard_normal((n_b, F)).astype(np.float32)
    bidx = rng.integers(0, n_b, E).astype(np.int32)
    oidx = rng.permutation(E).astype(np.int32)
    out, sc = oracle.edge_dot(a=a, b=b, bidx=bidx, oidx=oidx)
    ref = np.einsum("pf,pf->p", a.astype(np.float64), b[bidx].astype(np.float64))
    np.testing.assert_allclose(out[oidx], ref, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(sc[oidx], np.abs(a.astype(np.float64) * b[bidx]).sum(1), rtol=1e-13)
    ab = graphgen.f32_to_bf16(np.ones((E, F), np.float32))
    out1, _ = oracle.edge_dot(a_bf16=ab, b=np.ones((E, F), np.float32))
    assert np.all(out1 == F)


@pytest.mark.parametrize("seed", range(3))
def test_message_backward_x_matches_pinned_backward(seed):
    """For the sum, dL/dmsg is G[row(p)], so the gradient through the messages
    equals the (pinned) gradient of the fused aggregation w.r.t. x."""
    src, dst, x, w, _, g = graph(seed, 45, 35, 800, 6)
    rp, col, perm, _ = oracle.coo_to_csr(src, dst, 45, n_src=35)
    dmsg = oracle.message_backward(rp, "sum", g=g)
    gx, _ = oracle.message_backward_x(col, 35, dmsg, w=w[perm])
    ref, _ = oracle.spmm_backward_x(rp, col, 35, "sum", g=g, w=w[perm])
    assert np.array_equal(gx, ref)


@pytest.mark.parametrize("reduce", ["sum", "mean", "max"])
@pytest.mark.parametrize("seed", range(2))
def test_explainer_chain_matches_autograd(reduce, seed):
    """L = <AGG(mask[perm] * (w * x[col])), G>: the oracle's pieces composed
    as an explainer would compose them give torch's float64 gradients with
    respect to the edge mask (COO order), x and the edge weights."""
    src, dst, x, w, mask, g = graph(seed, 40, 30, 500, 4, distinct=True)
    mask = np.random.default_rng(seed).uniform(0.1, 1.0, src.size).astype(np.float32)
    rp, col, perm, _ = oracle.coo_to_csr(src, dst, 40, n_src=30)
    perm32 = perm.astype(np.int32)
    w_csr = w[perm]
    m_pre = oracle.message_gather(col, x=x, w=w_csr)
    m = oracle.message_scale(m_pre, mask, perm32)
    agg = oracle.aggregate_messages(rp, m)
    dm = oracle.message_backward(rp, reduce, g=g, argout=agg["argmax"])
    dmask, _ = oracle.edge_dot(a=dm, b=m_pre, oidx=perm32)
    dpre = oracle.message_scale(dm, mask, perm32)
    gx, _ = oracle.message_backward_x(col, 30, dpre, w=w_csr)
    gw, _ = oracle.edge_dot(a=dpre, b=x, bidx=col)

    X = torch.from_numpy(x.astype(np.float64)).requires_grad_(True)
    Wt = torch.from_numpy(w_csr.astype(np.float64)).requires_grad_(True)
    M = torch.from_numpy(mask.astype(np.float64)).requires_grad_(True)
    msg = M[torch.from_numpy(perm)][:, None] * (Wt[:, None] * X[torch.from_numpy(col.astype(np.int64))])
    out = torch_aggregate(msg, row_of(rp), 40, reduce, np.diff(rp))
    (out * torch.from_numpy(g.astype(np.float64))).sum().backward()
    np.testing.assert_allclose(dmask, M.grad.numpy(), rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(gx, X.grad.numpy(), rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(gw, Wt.grad.numpy(), rtol=1e-5, atol=1e-6)
