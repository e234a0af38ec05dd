"""Pins for the oracle's aggregation (Eq. (1) with message w * h_w and the
sum / mean / max aggregators; Sec. 2.2 segmented aggregation over the
destination-sorted CSR).

Pins used: a hand-worked example (tests/golden), closed forms (x = 1 gives
in-degree; a constant feature has that constant as mean; w = 1/deg gives the
mean), a dense adjacency matmul on graphs of at most 64 nodes, scipy.sparse on
the workload graphs, the unique characterization of max/argmax, brute force on
tiny graphs, linearity and invariance under reordering the COO edges.
"""
import json
import os

import numpy as np
import pytest
import scipy.sparse as sp

import graphgen
import oracle
from checks import check_max_characterization, scaled_error

HERE = os.path.dirname(os.path.abspath(__file__))


def tiny(seed, n, e, f, weighted=False):
    rng = np.random.default_rng(seed)
    src = rng.integers(0, n, e).astype(np.int32)
    dst = rng.integers(0, n, e).astype(np.int32)
    x = rng.standard_normal((n, f)).astype(np.float32)
    w = rng.standard_normal(e).astype(np.float32) if weighted else None
    return src, dst, x, w


def csr_with_w(src, dst, n, w):
    rp, col, perm, wc = oracle.coo_to_csr(src, dst, n, val=w)
    return rp, col, perm, wc


def test_golden_worked_example():
    g = json.load(open(os.path.join(HERE, "golden", "worked_example.json")))
    src = np.array(g["src"], np.int32)
    dst = np.array(g["dst"], np.int32)
    x = np.array(g["x"], np.float32)
    w = np.array(g["w"], np.float32)
    rp, col, perm, wc = csr_with_w(src, dst, g["N"], w)
    r = oracle.spmm(rp, col, x=x)
    assert r["sum"].tolist() == g["sum"]
    assert r["mean"].tolist() == g["mean"]
    assert r["max"].tolist() == g["max"]
    assert r["argmax"].tolist() == g["argmax"]
    r = oracle.spmm(rp, col, x=x, w=wc)
    assert r["sum"].tolist() == g["weighted_sum"]
    assert r["max"].tolist() == g["weighted_max"]
    assert r["argmax"].tolist() == g["weighted_argmax"]


@pytest.mark.parametrize("seed", range(6))
def test_all_ones_gives_in_degree(seed):
    src, dst, _, _ = tiny(seed, 200, 3000, 3)
    x = np.ones((200, 3), np.float32)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 200)
    r = oracle.spmm(rp, col, x=x)
    deg = np.bincount(dst, minlength=200).astype(np.float64)
    assert np.array_equal(r["sum"], np.repeat(deg[:, None], 3, 1))
    assert np.array_equal(r["scale"], r["sum"])


def test_constant_feature_mean_is_constant():
    src, dst, _, _ = tiny(1, 300, 4000, 2)
    x = np.full((300, 2), 0.75, np.float32)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 300)
    r = oracle.spmm(rp, col, x=x)
    deg = np.bincount(dst, minlength=300)
    assert np.all(r["mean"][deg > 0] == 0.75)
    assert np.all(r["mean"][deg == 0] == 0.0)
    # max of a constant: the value itself, first edge of the row
    assert np.all(r["max"][deg > 0] == 0.75)
    assert np.array_equal(r["argmax"][deg > 0][:, 0], rp[:-1][deg > 0])


def test_inverse_degree_weights_give_mean():
    src, dst, x, _ = tiny(2, 150, 2500, 4)
    deg = np.bincount(dst, minlength=150)
    w = (1.0 / deg[dst]).astype(np.float32)
    rp, col, _, wc = csr_with_w(src, dst, 150, w)
    rw = oracle.spmm(rp, col, x=x, w=wc)
    r = oracle.spmm(rp, col, x=x)
    # fl32(1/deg) and fl32(w*x) each add at most one fp32 rounding per term
    assert scaled_error(rw["sum"], r["mean"], r["scale"] / np.maximum(deg, 1)[:, None]) < 3e-7


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("weighted", [False, True])
def test_dense_adjacency_matmul(seed, weighted):
    n = 64 if seed % 2 == 0 else 17
    src, dst, x, w = tiny(seed, n, 5 * n, 6, weighted)
    A = np.zeros((n, n), np.float64)  # A[v, u]: summed weight of edges u -> v
    np.add.at(A, (dst, src), 1.0 if w is None else w.astype(np.float64))
    ref = A @ x.astype(np.float64)
    rp, col, _, wc = csr_with_w(src, dst, n, w)
    r = oracle.spmm(rp, col, x=x, w=wc)
    if w is None:
        assert np.allclose(r["sum"], ref, rtol=0, atol=1e-12)
        deg = A.sum(1)
        assert np.allclose(r["mean"], np.where(deg[:, None] > 0, ref / np.maximum(deg, 1)[:, None], 0),
                           rtol=0, atol=1e-12)
    else:
        # messages are fl32(w * x): each term within one fp32 rounding
        assert scaled_error(r["sum"], ref, r["scale"]) < 1.2e-7


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("weighted", [False, True])
def test_brute_force_tiny(seed, weighted):
    n, e, f = 9, 40, 3
    src, dst, x, w = tiny(seed, n, e, f, weighted)
    # plain python over COO edges, in COO order; CSR position from the order
    seen = {v: [] for v in range(n)}
    for ei in range(e):
        seen[int(dst[ei])].append(ei)
    rowstart = np.concatenate([[0], np.cumsum([len(seen[v]) for v in range(n)])])
    rp, col, _, wc = csr_with_w(src, dst, n, w)
    r = oracle.spmm(rp, col, x=x, w=wc)
    for v in range(n):
        for ff in range(f):
            msgs = []
            for ei in seen[v]:
                xv = float(x[src[ei], ff])
                msgs.append(xv if w is None else float(np.float32(float(w[ei]) * xv)))
            s = sum(msgs)
            assert abs(r["sum"][v, ff] - s) <= 1e-12 * (1 + sum(abs(m) for m in msgs))
            if msgs:
                best = max(msgs)
                k = msgs.index(best)
                assert r["max"][v, ff] == np.float32(best)
                assert r["argmax"][v, ff] == rowstart[v] + k
                assert abs(r["mean"][v, ff] - s / len(msgs)) <= 1e-12 * (1 + abs(s))
            else:
                assert r["argmax"][v, ff] == -1 and r["sum"][v, ff] == 0.0


@pytest.mark.parametrize("name", ["uniform-10k", "powerlaw-1.2M"])
def test_scipy_sparse_on_workloads(name):
    g = graphgen.workload(name, seed=0)
    rp, col, _, wc = csr_with_w(g.src, g.dst, g.n_dst, g.w)
    A = sp.csr_matrix((np.ones(g.E), (g.dst, g.src)), shape=(g.n_dst, g.n_src))
    ref = A @ g.x.astype(np.float64)
    r = oracle.spmm(rp, col, x=g.x, want=("sum", "mean", "scale"))
    assert scaled_error(r["sum"], ref, r["scale"]) < 1e-14
    deg = np.diff(rp)
    assert scaled_error(r["mean"] * np.maximum(deg, 1)[:, None], ref, r["scale"]) < 1e-14
    if g.w is not None:
        Aw = sp.csr_matrix((g.w.astype(np.float64), (g.dst, g.src)), shape=(g.n_dst, g.n_src))
        refw = Aw @ g.x.astype(np.float64)
        rw = oracle.spmm(rp, col, x=g.x, w=wc, want=("sum", "scale"))
        assert scaled_error(rw["sum"], refw, rw["scale"]) < 1.2e-7


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("weighted", [False, True])
def test_max_characterization(seed, weighted):
    src, dst, x, w = tiny(seed, 120, 2000, 5, weighted)
    # coarse values force many ties
    x = np.round(x * 2) / 2
    rp, col, _, wc = csr_with_w(src, dst, 120, w)
    r = oracle.spmm(rp, col, x=x, w=wc)
    check_max_characterization(rp, col, x, wc, r["max"], r["argmax"])


def test_signed_zero_ties_keep_first_edge():
    # one row, messages -0.0, +0.0, -0.0: all equal, the first edge wins
    x = np.array([[-0.0], [0.0], [-0.0]], np.float32)
    src = np.array([0, 1, 2], np.int32)
    dst = np.zeros(3, np.int32)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 1, n_src=3)
    r = oracle.spmm(rp, col, x=x)
    assert r["argmax"][0, 0] == 0
    assert r["max"].view(np.uint32)[0, 0] == 0x80000000
    x2 = np.array([[0.0], [-0.0]], np.float32)
    rp, col, _, _ = oracle.coo_to_csr(src[:2], dst[:2], 1, n_src=2)
    r = oracle.spmm(rp, col, x=x2)
    assert r["argmax"][0, 0] == 0 and r["max"].view(np.uint32)[0, 0] == 0


def test_shuffle_invariance():
    src, dst, x, _ = tiny(4, 80, 1500, 4)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 80)
    r = oracle.spmm(rp, col, x=x)
    order = np.random.default_rng(9).permutation(src.shape[0])
    rp2, col2, _, _ = oracle.coo_to_csr(src[order], dst[order], 80)
    r2 = oracle.spmm(rp2, col2, x=x)
    assert np.array_equal(rp, rp2)
    assert scaled_error(r2["sum"], r["sum"], r["scale"]) < 1e-14
    assert np.array_equal(r2["max"], r["max"])


def test_linearity():
    src, dst, x1, _ = tiny(5, 70, 900, 3)
    x2 = np.random.default_rng(6).standard_normal((70, 3)).astype(np.float32)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 70)
    a, b = 0.5, -2.0  # exact in fp32 together with the sums below
    r1 = oracle.spmm(rp, col, x=x1)
    r2 = oracle.spmm(rp, col, x=x2)
    r12 = oracle.spmm(rp, col, x=(a * x1 + b * x2).astype(np.float32))
    assert np.allclose(r12["sum"], a * r1["sum"] + b * r2["sum"], rtol=0, atol=1e-5)


def test_bf16_features_widen_exactly():
    g = graphgen.workload("uniform-10k", seed=2, bf16=True)
    rp, col, _, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    rb = oracle.spmm(rp, col, x_bf16=g.x_bf16)
    rf = oracle.spmm(rp, col, x=graphgen.bf16_to_f32(g.x_bf16))
    for k in ("sum", "mean", "max", "argmax", "scale"):
        assert np.array_equal(rb[k], rf[k]), k


def test_row_subset_and_coo_rows_agree():
    g = graphgen.workload("powerlaw-1.2M", seed=3, scale=0.1)
    rp, col, _, wc = csr_with_w(g.src, g.dst, g.n_dst, g.w)
    rows = np.unique(np.random.default_rng(0).integers(0, g.n_dst, 500))
    deg = np.diff(rp)
    rows = np.unique(np.concatenate([rows, [int(np.argmax(deg))], np.nonzero(deg == 0)[0][:5]]))
    full = oracle.spmm(rp, col, x=g.x, w=wc)
    sub = oracle.spmm(rp, col, x=g.x, w=wc, rows=rows)
    coo = oracle.spmm_coo_rows(g.src, g.dst, g.n_dst, rows, x=g.x, w_coo=g.w)
    shuffled = rows[np.argsort(graphgen.uniform_ints(1, 9, rows.shape[0], 10**9))]
    below = np.concatenate([[0], np.cumsum(np.bincount(g.dst, minlength=g.n_dst))])[shuffled]
    coo2 = oracle.spmm_coo_rows(g.src, g.dst, g.n_dst, shuffled, x=g.x, w_coo=g.w,
                                row_start=below)
    for k in ("sum", "mean", "max", "argmax", "scale"):
        assert np.array_equal(sub[k], full[k][rows]), k
        assert np.array_equal(coo[k], full[k][rows]), k
        assert np.array_equal(coo2[k], full[k][shuffled]), k


def test_thread_count_does_not_change_results():
    g = graphgen.workload("uniform-10k", seed=4)
    rp, col, _, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    a = oracle.spmm(rp, col, x=g.x, nthreads=1)
    b = oracle.spmm(rp, col, x=g.x, nthreads=8)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
