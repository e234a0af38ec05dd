"""Parity of the segment matmul on the matrix cores (through the C ABI) with
the CPU oracle.

Inputs are bf16, exact in fp32, and every product of two bf16 values is exact
in fp32, so the only error is fp32 accumulation: |y - y_ref| <= 1e-5 * sum
|x w| per output element (the summand-scaled bound of the other sums); a bf16
output adds one rounding, 2^-8 of |y_ref|.
"""
import sys

import numpy as np
import pytest
import torch

import graphgen
import oracle
import paper_2507_16991_amd as mp

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
TOL = 1e-5


@pytest.fixture(autouse=True)
def _announce(request):
    sys.stderr.write(f"\n[gpu-case] {request.node.nodeid}\n")
    sys.stderr.flush()
    yield
    torch.cuda.synchronize()


def bf16_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def inputs(seed, sizes, F, Fo):
    seg = [0] + list(np.cumsum(sizes))
    N, T = int(seg[-1]), len(sizes)
    x = graphgen.f32_to_bf16(graphgen.normal_f32(seed, 3, N * F).reshape(N, F))
    w = graphgen.f32_to_bf16((graphgen.normal_f32(seed, 5, T * F * Fo) / np.sqrt(F))
                             .astype(np.float32).reshape(T, F, Fo))
    d = graphgen.f32_to_bf16(graphgen.normal_f32(seed, 11, N * Fo).reshape(N, Fo))
    return seg, x, w, d


def check(y, ref, scale, bf16_out=False):
    y = y.float().cpu().numpy().astype(np.float64)
    bound = TOL * scale + (2.0 ** -8 * np.abs(ref) if bf16_out else 0.0)
    bad = np.abs(y - ref) > bound
    assert not bad.any(), f"{bad.sum()} elements off; worst {np.max(np.abs(y - ref) - bound)}"


SHAPES = [([1000, 0, 257], 128, 128), ([5], 8, 8), ([3000, 129, 4100], 64, 136),
          ([300, 1], 256, 520), ([127, 128, 129], 24, 40)]


@pytest.mark.parametrize("sizes,F,Fo", SHAPES)
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_forward(sizes, F, Fo, out_dtype):
    seg, x, w, _ = inputs(len(sizes) + F, sizes, F, Fo)
    out = mp.segment_matmul(seg, bf16_dev(x), bf16_dev(w), out_dtype=out_dtype)
    torch.cuda.synchronize()
    ref, sc = oracle.segment_matmul(seg, x, w)
    check(out, ref, sc, out_dtype == torch.bfloat16)


@pytest.mark.parametrize("sizes,F,Fo", SHAPES)
def test_backward(sizes, F, Fo):
    seg, x, w, d = inputs(len(sizes) + Fo, sizes, F, Fo)
    dx, dW = mp.segment_matmul_backward(seg, bf16_dev(x), bf16_dev(w), bf16_dev(d))
    torch.cuda.synchronize()
    rdx, sdx, rdw, sdw = oracle.segment_matmul_backward(seg, x, w, d)
    check(dx, rdx, sdx)
    check(dW, rdw, sdw)


def test_backward_single_outputs_and_bf16_dx():
    seg, x, w, d = inputs(2, [700, 2100], 32, 64)
    dx, dW = mp.segment_matmul_backward(seg, bf16_dev(x), bf16_dev(w), bf16_dev(d),
                                        want_dw=False, dx_dtype=torch.bfloat16)
    assert dW is None
    dx2, dW2 = mp.segment_matmul_backward(seg, bf16_dev(x), bf16_dev(w), bf16_dev(d),
                                          want_dx=False)
    assert dx2 is None
    torch.cuda.synchronize()
    rdx, sdx, rdw, sdw = oracle.segment_matmul_backward(seg, x, w, d)
    check(dx, rdx, sdx, bf16_out=True)
    check(dW2, rdw, sdw)


def test_deterministic():
    seg, x, w, d = inputs(4, [5000, 3000], 128, 128)
    X, W, D = bf16_dev(x), bf16_dev(w), bf16_dev(d)
    a = mp.segment_matmul(seg, X, W)
    b = mp.segment_matmul(seg, X, W)
    _, g1 = mp.segment_matmul_backward(seg, X, W, D, want_dx=False)
    _, g2 = mp.segment_matmul_backward(seg, X, W, D, want_dx=False)
    assert torch.equal(a, b) and torch.equal(g1, g2)


def test_typed_projection_full_size_sampled():
    """The typed graph's node tables (1.9M, 736k, 8.7k rows, F = F' = 128):
    forward and input gradient on sampled rows of every type; the weight
    gradient on the first 150,000 rows of each type."""
    sizes = [1_900_000, 736_000, 8_700]
    seg, x, w, d = inputs(7, sizes, 128, 128)
    X, W, D = bf16_dev(x), bf16_dev(w), bf16_dev(d)
    out = mp.segment_matmul(seg, X, W).cpu().numpy()
    dx, _ = mp.segment_matmul_backward(seg, X, W, D, want_dw=False)
    dx = dx.cpu().numpy()
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    pick = [np.sort(rng.choice(n, size=min(n, 2000), replace=False)) + seg[t]
            for t, n in enumerate(sizes)]
    sub_seg = [0] + list(np.cumsum([len(p) for p in pick]))
    rows = np.concatenate(pick)
    ref, sc = oracle.segment_matmul(sub_seg, x[rows], w)
    check(torch.from_numpy(out[rows]), ref, sc)
    rdx, sdx, _, _ = oracle.segment_matmul_backward(sub_seg, x[rows], w, d[rows])
    check(torch.from_numpy(dx[rows]), rdx, sdx)
    print("[note] forward and dx sampled rows ok", file=sys.stderr, flush=True)
    head = [np.arange(seg[t], seg[t] + min(n, 150_000)) for t, n in enumerate(sizes)]
    hseg = [0] + list(np.cumsum([len(h) for h in head]))
    hrows = np.concatenate(head)
    _, dW = mp.segment_matmul_backward(hseg, bf16_dev(x[hrows]), W, bf16_dev(d[hrows]),
                                       want_dx=False)
    torch.cuda.synchronize()
    _, _, rdw, sdw = oracle.segment_matmul_backward(hseg, x[hrows], w, d[hrows])
    check(dW, rdw, sdw)
