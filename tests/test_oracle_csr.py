"""Pins for the oracle's COO -> CSR conversion (Sec. 2.2, the sorted
edge_index behind the CSR/CSC cache).

Library pin: numpy's stable argsort of dst gives the permutation; col =
src[perm]; rowptr = [0, cumsum(bincount(dst))].  Invariant pins: see
checks.check_csr_invariants.
"""
import json
import os

import numpy as np
import pytest

import graphgen
import oracle
from checks import check_csr_invariants

HERE = os.path.dirname(os.path.abspath(__file__))


def numpy_csr(src, dst, n):
    perm = np.argsort(dst, kind="stable")
    rowptr = np.concatenate([[0], np.cumsum(np.bincount(dst, minlength=n))])
    return rowptr, src[perm], perm


def random_graph(seed, n, e):
    rng = np.random.default_rng(seed)
    src = rng.integers(0, n, e).astype(np.int32)
    dst = rng.integers(0, n, e).astype(np.int32)
    return src, dst


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("n,e", [(1, 0), (1, 5), (7, 0), (7, 40), (64, 300), (1000, 200),
                                 (300, 5000)])
def test_matches_numpy_stable_argsort(seed, n, e):
    src, dst = random_graph(seed, n, e)
    rp, col, perm, _ = oracle.coo_to_csr(src, dst, n)
    rp2, col2, perm2 = numpy_csr(src, dst, n)
    assert np.array_equal(rp, rp2)
    assert np.array_equal(col, col2)
    assert np.array_equal(perm, perm2)
    check_csr_invariants(src, dst, n, rp, col, perm)


def test_payload_follows_perm():
    src, dst = random_graph(3, 50, 700)
    val = np.random.default_rng(3).standard_normal(700).astype(np.float32)
    rp, col, perm, vout = oracle.coo_to_csr(src, dst, 50, val=val)
    assert np.array_equal(vout.view(np.uint32), val[perm].view(np.uint32))


@pytest.mark.parametrize("name", ["uniform-10k", "powerlaw-1.2M"])
def test_workloads_match_numpy(name):
    g = graphgen.workload(name, seed=1)
    rp, col, perm, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    rp2, col2, perm2 = numpy_csr(g.src, g.dst, g.n_dst)
    assert np.array_equal(rp, rp2) and np.array_equal(col, col2) and np.array_equal(perm, perm2)


def test_structured_cases():
    n = 9
    # already sorted, reverse sorted, all into one row, all self-loops
    cases = [
        (np.arange(20, dtype=np.int32) % n, np.sort(np.arange(20, dtype=np.int32) % n)),
        (np.arange(20, dtype=np.int32) % n, np.sort(np.arange(20, dtype=np.int32) % n)[::-1].copy()),
        (np.arange(20, dtype=np.int32) % n, np.full(20, 4, np.int32)),
        (np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int32)),
    ]
    for src, dst in cases:
        rp, col, perm, _ = oracle.coo_to_csr(src, dst, n)
        rp2, col2, perm2 = numpy_csr(src, dst, n)
        assert np.array_equal(rp, rp2) and np.array_equal(col, col2) and np.array_equal(perm, perm2)


def test_bipartite_sizes():
    rng = np.random.default_rng(0)
    src = rng.integers(0, 13, 400).astype(np.int32)
    dst = rng.integers(0, 5, 400).astype(np.int32)
    rp, col, perm, _ = oracle.coo_to_csr(src, dst, 5, n_src=13)
    rp2, col2, perm2 = numpy_csr(src, dst, 5)
    assert np.array_equal(rp, rp2) and np.array_equal(col, col2)


def test_rejects_out_of_range():
    with pytest.raises(ValueError):
        oracle.coo_to_csr(np.array([0, 1], np.int32), np.array([0, 5], np.int32), 5)
    with pytest.raises(ValueError):
        oracle.coo_to_csr(np.array([0, -1], np.int32), np.array([0, 1], np.int32), 5)


def test_golden_worked_example():
    g = json.load(open(os.path.join(HERE, "golden", "worked_example.json")))
    src = np.array(g["src"], np.int32)
    dst = np.array(g["dst"], np.int32)
    w = np.array(g["w"], np.float32)
    rp, col, perm, wc = oracle.coo_to_csr(src, dst, g["N"], val=w)
    assert rp.tolist() == g["rowptr"]
    assert col.tolist() == g["col"]
    assert perm.tolist() == g["perm"]
    assert wc.tolist() == g["w_csr"]


def test_csr_rows_matches_full_conversion():
    src, dst = random_graph(11, 500, 20_000)
    rp, col, _, _ = oracle.coo_to_csr(src, dst, 500)
    rows = np.array([499, 3, 0, 250, 17, 64, 63, 65, 128], np.int64)
    seg, cols = oracle.csr_rows(src, dst, 500, rows)
    for k, r in enumerate(rows):
        assert np.array_equal(cols[seg[k]:seg[k + 1]], col[rp[r]:rp[r + 1]])
