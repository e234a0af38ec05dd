"""Pins for the oracle's segment matmul (Sec. 2.2, heterogeneous GNNs: the
projections {H_T W_T} with a weight tensor of shape [|T|, F, F'], and their
gradients with respect to H_T and W).

Pins used: brute-force triple loops in Python on tiny shapes, the identity
weight (out = X), the block-diagonal identity (the whole product equals one
dense matmul of X against the block-diagonal stack, numpy), reverse-mode
differentiation by torch autograd in float64, and the adjoint identity
<XW, G> = <X, G W^T> = <W, X^T G>.
"""
import numpy as np
import pytest
import torch

import graphgen
import oracle


def bf16_of(a):
    return graphgen.f32_to_bf16(np.asarray(a, np.float32))


def wide(b):
    return graphgen.bf16_to_f32(b).astype(np.float64)


def case(seed, sizes, F, Fo):
    rng = np.random.default_rng(seed)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    x = bf16_of(rng.standard_normal((seg[-1], F)))
    w = bf16_of(rng.standard_normal((len(sizes), F, Fo)))
    return seg, x, w


def test_brute_force_tiny():
    seg, x, w = case(0, [3, 0, 2], 4, 5)
    out, sc = oracle.segment_matmul(seg, x, w)
    X, W = wide(x), wide(w)
    for t in range(3):
        for r in range(seg[t], seg[t + 1]):
            for o in range(5):
                s = a = 0.0
                for f in range(4):
                    s += X[r, f] * W[t, f, o]
                    a += abs(X[r, f] * W[t, f, o])
                assert out[r, o] == pytest.approx(s, rel=1e-15, abs=1e-15)
                assert sc[r, o] == pytest.approx(a, rel=1e-15, abs=1e-15)


def test_identity_weight():
    seg, x, _ = case(1, [50, 7, 20], 16, 16)
    w = bf16_of(np.broadcast_to(np.eye(16), (3, 16, 16)))
    out, _ = oracle.segment_matmul(seg, x, w)
    assert np.array_equal(out, wide(x))


@pytest.mark.parametrize("seed", range(3))
def test_block_diagonal_equivalence(seed):
    sizes = [40, 0, 13, 64]
    F, Fo = 24, 16
    seg, x, w = case(seed, sizes, F, Fo)
    out, _ = oracle.segment_matmul(seg, x, w)
    # one dense product: each row's features placed in its type's block
    T = len(sizes)
    big = np.zeros((seg[-1], T * F))
    for t in range(T):
        big[seg[t]:seg[t + 1], t * F:(t + 1) * F] = wide(x)[seg[t]:seg[t + 1]]
    np.testing.assert_allclose(out, big @ wide(w).reshape(T * F, Fo), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_gradients_match_autograd(seed):
    sizes = [30, 5, 0, 17]
    F, Fo = 12, 20
    seg, x, w = case(seed, sizes, F, Fo)
    d = bf16_of(np.random.default_rng(seed + 9).standard_normal((seg[-1], Fo)))
    dx, _, dw, _ = oracle.segment_matmul_backward(seg, x, w, d)
    X = torch.from_numpy(wide(x)).requires_grad_(True)
    W = torch.from_numpy(wide(w)).requires_grad_(True)
    outs = [X[seg[t]:seg[t + 1]] @ W[t] for t in range(len(sizes))]
    (torch.cat(outs) * torch.from_numpy(wide(d))).sum().backward()
    np.testing.assert_allclose(dx, X.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, W.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_adjoint_identity():
    seg, x, w = case(5, [300, 200, 1], 32, 48)
    d = bf16_of(np.random.default_rng(1).standard_normal((seg[-1], 48)))
    out, _ = oracle.segment_matmul(seg, x, w)
    dx, _, dw, _ = oracle.segment_matmul_backward(seg, x, w, d)
    lhs = float(np.sum(out * wide(d)))
    assert lhs == pytest.approx(float(np.sum(dx * wide(x))), rel=1e-10)
    assert lhs == pytest.approx(float(np.sum(dw * wide(w))), rel=1e-10)
