"""Pins for the oracle's heterogeneous sum (Sec. 2.2, Heterogeneous Message
Passing: the nested Eq. (1), summing per-relation aggregations into each
destination node type).

Pins: (1) the identity that a sum of per-relation sums is one homogeneous sum
over the union graph whose node ids are offset by type; (2) per-relation
scipy.sparse products added up; (3) a hand-checked two-type example.
"""
import numpy as np
import scipy.sparse as sp

import graphgen
import oracle
from checks import scaled_error


def small_hetero(seed):
    return graphgen.hetero_graph(seed, [300, 120, 7],
                                 [(0, 0, 900), (0, 1, 1100), (1, 0, 1000), (1, 2, 400)], 16)


def test_union_graph_identity():
    g = small_hetero(0)
    outs, scs = oracle.hetero_sum(g.n_per_type, g.x_bf16, g.rel_src_type, g.rel_dst_type,
                                  g.rel_src, g.rel_dst)
    off = np.concatenate([[0], np.cumsum(g.n_per_type)])
    xall = np.concatenate([graphgen.bf16_to_f32(x) for x in g.x_bf16])
    for t in range(len(g.n_per_type)):
        rs = [r for r in range(len(g.rel_src)) if g.rel_dst_type[r] == t]
        if not rs:
            assert np.all(outs[t] == 0)
            continue
        src = np.concatenate([g.rel_src[r] + off[g.rel_src_type[r]] for r in rs]).astype(np.int32)
        dst = np.concatenate([g.rel_dst[r] for r in rs]).astype(np.int32)
        rp, col, _, _ = oracle.coo_to_csr(src, dst, g.n_per_type[t], n_src=xall.shape[0])
        r = oracle.spmm(rp, col, x=xall, want=("sum", "scale"))
        # same terms in the same order (relations ascending, COO order within)
        assert np.array_equal(r["sum"], outs[t])
        assert np.array_equal(r["scale"], scs[t])


def test_per_relation_scipy():
    g = small_hetero(1)
    outs, scs = oracle.hetero_sum(g.n_per_type, g.x_bf16, g.rel_src_type, g.rel_dst_type,
                                  g.rel_src, g.rel_dst)
    for t in range(len(g.n_per_type)):
        ref = np.zeros((g.n_per_type[t], g.F))
        for r in range(len(g.rel_src)):
            if g.rel_dst_type[r] != t:
                continue
            st = g.rel_src_type[r]
            A = sp.csr_matrix((np.ones(g.rel_src[r].shape[0]), (g.rel_dst[r], g.rel_src[r])),
                              shape=(g.n_per_type[t], g.n_per_type[st]))
            ref += A @ graphgen.bf16_to_f32(g.x_bf16[st]).astype(np.float64)
        assert scaled_error(outs[t], ref, scs[t]) < 1e-14


def test_hand_example():
    # types: 0 with 2 nodes, 1 with 1 node; relations r0: 0->1, r1: 1->0, r2: 0->0
    x0 = graphgen.f32_to_bf16(np.array([[1.0], [2.0]], np.float32))
    x1 = graphgen.f32_to_bf16(np.array([[10.0]], np.float32))
    outs, _ = oracle.hetero_sum([2, 1], [x0, x1], [0, 1, 0], [1, 0, 0],
                                [np.array([0, 1, 1], np.int32), np.array([0], np.int32),
                                 np.array([1], np.int32)],
                                [np.array([0, 0, 0], np.int32), np.array([1], np.int32),
                                 np.array([0], np.int32)])
    # node 0 of type 1 receives x0[0] + 2 * x0[1] = 5 over r0
    assert outs[1].tolist() == [[5.0]]
    # type 0: node 1 gets x1[0] = 10 over r1; node 0 gets x0[1] = 2 over r2
    assert outs[0].tolist() == [[2.0], [10.0]]
