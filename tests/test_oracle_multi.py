"""Pins for the oracle's further aggregators (Sec. 2.2, "Aggregations as a
First-Class Principle": min, variance and standard deviation next to sum,
mean and max, stacked, in message passing and in global readouts).

Pins used: numpy's per-row var/std/min/argmin (library routines), the duality
min(x) = -max(-x) against the already pinned max/argmax, closed forms
(constant rows, two-point rows), and numpy segment reductions for a global
readout over a sorted batch vector.
"""
import numpy as np
import pytest

import graphgen
import oracle


def rows_of_messages(rp, col, x, w=None):
    """Per row, the [deg, F] array of fp32 messages in CSR order."""
    out = []
    for r in range(rp.size - 1):
        m = x[col[rp[r]:rp[r + 1]]].astype(np.float32)
        if w is not None:
            m = (w[rp[r]:rp[r + 1], None].astype(np.float64) * m.astype(np.float64)).astype(np.float32)
        out.append(m)
    return out


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("weighted", [False, True])
def test_against_numpy(seed, weighted):
    g = graphgen.mixed_graph(seed, n=600, e=6000, f=6, signed_weights=True)
    rp, col, _, wc = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    w = wc if weighted else None
    r = oracle.spmm_multi(rp, col, x=g.x, w=w)
    msgs = rows_of_messages(rp, col, g.x, w)
    for i, m in enumerate(msgs):
        if m.shape[0] == 0:
            assert np.all(r["argmin"][i] == -1) and np.all(r["min"][i] == 0)
            assert np.all(r["var"][i] == 0) and np.all(r["std"][i] == 0)
            continue
        am = np.argmin(m, axis=0)  # first occurrence, as the CSR order
        assert np.array_equal(r["argmin"][i], rp[i] + am)
        assert np.array_equal(r["min"][i], m.min(axis=0))
        m64 = m.astype(np.float64)
        np.testing.assert_allclose(r["var"][i], m64.var(axis=0), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(r["std"][i], m64.std(axis=0), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("seed", range(3))
def test_min_is_minus_max_of_negated(seed):
    g = graphgen.mixed_graph(seed, n=1500, e=20_000, f=8)
    rp, col, _, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    a = oracle.spmm_multi(rp, col, x=g.x)
    b = oracle.spmm(rp, col, x=-g.x, want=("max",))
    assert np.array_equal(a["argmin"], b["argmax"])
    nonempty = b["argmax"] >= 0
    assert np.array_equal(a["min"][nonempty], -b["max"][nonempty])


def test_closed_forms():
    # row 0: constant messages (var 0); row 1: two points a, b (var (a-b)^2/4);
    # row 2: empty; row 3: duplicates of one edge (min at the first copy)
    src = np.array([0, 0, 0, 1, 2, 3, 3, 3], np.int32)
    dst = np.array([0, 0, 0, 1, 1, 3, 3, 3], np.int32)
    x = np.array([[0.75, -1.0], [2.0, 5.0], [-6.0, 1.0], [3.0, -0.0]], np.float32)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 4)
    r = oracle.spmm_multi(rp, col, x=x)
    assert r["var"][0].tolist() == [0.0, 0.0] and r["std"][0].tolist() == [0.0, 0.0]
    assert r["var"][1].tolist() == [16.0, 4.0] and r["std"][1].tolist() == [4.0, 2.0]
    assert r["argmin"][1].tolist() == [4, 4] and r["min"][1].tolist() == [-6.0, 1.0]
    assert r["argmin"][2].tolist() == [-1, -1] and r["var"][2].tolist() == [0.0, 0.0]
    assert r["argmin"][3].tolist() == [5, 5]


@pytest.mark.parametrize("seed", range(3))
def test_readout_over_sorted_batch(seed):
    # a global readout: nodes grouped by a sorted batch vector, col = identity
    rng = np.random.default_rng(seed)
    sizes = rng.integers(0, 40, 25)
    batch = np.repeat(np.arange(25), sizes).astype(np.int32)
    n = batch.size
    x = rng.standard_normal((n, 5)).astype(np.float32)
    rp, col, _, _ = oracle.coo_to_csr(np.arange(n, dtype=np.int32), batch, 25, n_src=n)
    assert np.array_equal(col, np.arange(n))
    fw = oracle.spmm(rp, col, x=x)
    mu = oracle.spmm_multi(rp, col, x=x)
    for b in range(25):
        seg = x[rp[b]:rp[b + 1]].astype(np.float64)
        if seg.shape[0] == 0:
            continue
        np.testing.assert_allclose(fw["sum"][b], seg.sum(axis=0), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(fw["mean"][b], seg.mean(axis=0), rtol=1e-12, atol=1e-12)
        assert np.array_equal(fw["max"][b], x[rp[b]:rp[b + 1]].max(axis=0))
        assert np.array_equal(mu["min"][b], x[rp[b]:rp[b + 1]].min(axis=0))
        np.testing.assert_allclose(mu["std"][b], seg.std(axis=0), rtol=1e-12, atol=1e-14)
