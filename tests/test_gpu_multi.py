"""Parity of the stacked aggregations and the global readout (through the C
ABI) with the CPU oracle.

max/argmax and min/argmin must be bit-exact; sum and mean are held to the
summand-scaled bound of the forward tests (1e-5 for fp32 features, 1e-2 for
bf16).  The variance is a sum of the non-negative terms (m - mean)^2 / deg,
so its summand-scaled error is its relative error: |v - v_ref| <= 1e-5 v_ref
(v_ref == 0 must be matched exactly), for both feature dtypes, since bf16
widens to fp32 exactly and both accumulate in fp32.  The standard deviation
is held to the same bound relative to itself.
"""
import sys

import numpy as np
import pytest
import torch

import graphgen
import oracle
import paper_2507_16991_amd as mp
from checks import scaled_error

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
TOL = {torch.float32: 1e-5, torch.bfloat16: 1e-2}
VAR_TOL = 1e-5  # relative, both feature dtypes (fp32 accumulation)
ALL = ["sum", "mean", "max", "min", "var", "std"]


@pytest.fixture(autouse=True)
def _announce(request):
    sys.stderr.write(f"\n[gpu-case] {request.node.nodeid}\n")
    sys.stderr.flush()
    yield
    torch.cuda.synchronize()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def x_pair(g, dtype):
    if dtype == torch.float32:
        return dev(g.x), {"x": g.x}
    return dev(g.x_bf16.view(np.int16)).view(torch.bfloat16), {"x_bf16": g.x_bf16}


def compare(res, rp_o, col_o, w_o, xkw, names, dtype, rows=None):
    ref = oracle.spmm(rp_o, col_o, w=w_o, rows=rows, **xkw)
    mul = oracle.spmm_multi(rp_o, col_o, w=w_o, rows=rows, **xkw)
    sel = (lambda a: a) if rows is None else (lambda a: a[rows])
    deg = np.diff(rp_o) if rows is None else rp_o[rows + 1] - rp_o[rows]
    tol = TOL[dtype]
    errs = {}
    for n in names:
        y = sel(res[n].cpu().numpy())
        if n == "sum":
            errs[n] = scaled_error(y, ref["sum"], ref["scale"])
        elif n == "mean":
            errs[n] = scaled_error(y, ref["mean"], ref["scale"] / np.maximum(deg, 1)[:, None])
        elif n == "var":
            errs[n] = scaled_error(y, mul["var"], mul["var"])
            assert errs[n] <= VAR_TOL, f"var relative error {errs[n]}"
            continue
        elif n == "std":
            errs[n] = scaled_error(y, mul["std"], mul["std"])
            assert errs[n] <= VAR_TOL, f"std relative error {errs[n]}"
            continue
        elif n == "max":
            a = sel(res["argmax"].cpu().numpy()).astype(np.int64)
            assert np.array_equal(a, ref["argmax"]), "argmax"
            assert np.array_equal(y.view(np.uint32), ref["max"].view(np.uint32)), "max bits"
            continue
        elif n == "min":
            a = sel(res["argmin"].cpu().numpy()).astype(np.int64)
            assert np.array_equal(a, mul["argmin"]), "argmin"
            assert np.array_equal(y.view(np.uint32), mul["min"].view(np.uint32)), "min bits"
            continue
        assert errs[n] <= tol, f"{n} error {errs[n]}"
    return errs


@pytest.fixture(scope="module")
def mixed():
    g = graphgen.mixed_graph(0, f=64, signed_weights=True)
    rp_o, col_o, _, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    return g, rp_o, col_o, w_o


def run_multi(g, rp_o, col_o, w_o, names, dtype, weighted, use_plan, opts=None):
    rp, col = dev(rp_o.astype(np.int32)), dev(col_o)
    x, xkw = x_pair(g, dtype)
    plan = mp.Plan(rp, g.E, g.F, dtype, opts=opts) if use_plan else None
    res = mp.spmm_multi(rp, col, x, names, w=dev(w_o) if weighted else None, plan=plan)
    torch.cuda.synchronize()
    return compare(res, rp_o, col_o, w_o if weighted else None, xkw, names, dtype)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("use_plan", [False, True])
def test_multi_all(mixed, dtype, weighted, use_plan):
    run_multi(*mixed, ALL, dtype, weighted, use_plan)


@pytest.mark.parametrize("names", [["min"], ["var", "mean"], ["std", "max"], ["min", "sum"],
                                   ["std"], ["max", "min", "mean", "std"]])
def test_multi_subsets(mixed, names):
    run_multi(*mixed, names, torch.float32, True, True)


@pytest.mark.parametrize("thresholds", [(8, 64, 16), (1, 2, 1)])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_multi_plan_regimes(mixed, thresholds, dtype):
    run_multi(*mixed, ALL, dtype, True, True, opts=thresholds)


@pytest.mark.parametrize("F", [1, 3, 8, 24, 100, 300, 520])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_multi_feature_widths(F, dtype):
    g = graphgen.mixed_graph(F, n=700, e=9000, f=F)
    rp_o, col_o, _, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    run_multi(g, rp_o, col_o, w_o, ALL, dtype, False, True, opts=(0, 128, 32))


def test_multi_ties_and_signed_zero():
    # duplicates (equal messages) and -0.0 / +0.0: first CSR position wins
    src = np.array([1, 1, 0, 2, 3, 0], np.int32)
    dst = np.array([0, 0, 0, 1, 1, 2], np.int32)
    x = np.array([[0.0, 1.0], [-2.0, 3.0], [-0.0, 1.0], [0.0, 1.0]], np.float32)
    rp_o, col_o, _, _ = oracle.coo_to_csr(src, dst, 4)
    res = mp.spmm_multi(dev(rp_o.astype(np.int32)), dev(col_o), dev(x), ALL)
    torch.cuda.synchronize()
    compare(res, rp_o, col_o, None, {"x": x}, ALL, torch.float32)
    assert res["argmin"].cpu().tolist()[1] == [3, 3]  # -0.0 ties +0.0: first edge


@pytest.mark.parametrize("use_plan", [False, True])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_readout(use_plan, dtype):
    rng = np.random.default_rng(3)
    sizes = rng.integers(0, 3000, 64)
    sizes[[5, 40]] = 0  # empty graphs in the batch
    batch = np.repeat(np.arange(64), sizes).astype(np.int32)
    n = int(batch.size)
    xf = graphgen.normal_f32(4, 3, n * 40).reshape(n, 40)
    xb = graphgen.f32_to_bf16(xf)
    rp_o, col_o, _, _ = oracle.coo_to_csr(np.arange(n, dtype=np.int32), batch, 64, n_src=n)
    ptr = dev(rp_o.astype(np.int32))
    x = dev(xf) if dtype == torch.float32 else dev(xb.view(np.int16)).view(torch.bfloat16)
    xkw = {"x": xf} if dtype == torch.float32 else {"x_bf16": xb}
    plan = mp.Plan(ptr, n, 40, dtype) if use_plan else None
    res = mp.readout(ptr, x, ALL, plan=plan)
    torch.cuda.synchronize()
    compare(res, rp_o, col_o, None, xkw, ALL, dtype)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_row_strided_features(mixed, dtype):
    """Stacked aggregation and readout over a feature table whose rows are
    F + 28 elements apart (a view of a wider table)."""
    g, rp_o, col_o, w_o = mixed
    F = g.F
    x = dev(g.x) if dtype == torch.float32 else dev(g.x_bf16.view(np.int16)).view(torch.bfloat16)
    xkw = {"x": g.x} if dtype == torch.float32 else {"x_bf16": g.x_bf16}
    xs = torch.zeros(g.n_src, F + 28, dtype=dtype, device=DEV)[:, :F]
    xs.copy_(x)
    rp = dev(rp_o.astype(np.int32))
    plan = mp.Plan(rp, g.E, F, dtype)
    res = mp.spmm_multi(rp, dev(col_o), xs, ALL, plan=plan)
    torch.cuda.synchronize()
    compare(res, rp_o, col_o, None, xkw, ALL, dtype)
    # readout of the same rows in 7 consecutive segments
    n = g.n_src
    cuts = np.linspace(0, n, 8).astype(np.int64)
    ptr = dev(cuts.astype(np.int32))
    res = mp.readout(ptr, xs, ALL)
    torch.cuda.synchronize()
    compare(res, cuts, np.arange(n, dtype=np.int32), None, xkw, ALL, dtype)


def test_readout_from_sorted_batch_vector():
    # ptr from the batch vector with the sorted-COO fast path, then the readout
    rng = np.random.default_rng(5)
    batch = np.sort(rng.integers(0, 300, 50_000)).astype(np.int32)
    n = batch.size
    xf = graphgen.normal_f32(6, 3, n * 16).reshape(n, 16)
    nodes = dev(np.arange(n, dtype=np.int32))
    ptr, _, _, _ = mp.sorted_coo_to_csr(nodes, dev(batch), 300)
    res = mp.readout(ptr, dev(xf), ["mean", "max", "std"], plan=mp.Plan(ptr, n, 16))
    torch.cuda.synchronize()
    rp_o, col_o, _, _ = oracle.coo_to_csr(np.arange(n, dtype=np.int32), batch, 300, n_src=n)
    assert np.array_equal(ptr.cpu().numpy(), rp_o)
    compare(res, rp_o, col_o, None, {"x": xf}, ["mean", "max", "std"], torch.float32)


def large_mean_features(g):
    """Features whose rows are far from zero against their spread, where a
    one-pass E[m^2] - E[m]^2 in fp32 would lose every digit: columns 0..15
    are 1000 + N(0,1), 16..23 the constant 3.7 (every row's messages equal:
    variance exactly 0), 24..31 1e4 + 0.01 N(0,1), the rest N(0,1)."""
    x = g.x.astype(np.float64).copy()
    x[:, :16] += 1000.0
    x[:, 16:24] = 3.7
    x[:, 24:32] = 1e4 + 0.01 * x[:, 24:32]
    return x.astype(np.float32)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("opts", [None, (8, 64, 16), (1, 2, 1)])
def test_multi_large_mean_and_constant_rows(mixed, dtype, opts):
    """Variance and std held to 1e-5 of themselves on rows with large means
    and on constant rows (exactly 0), through every row class (the small
    thresholds send rows through the hub chunks and their fix-up)."""
    g, rp_o, col_o, w_o = mixed
    xf = large_mean_features(g)
    xb = graphgen.f32_to_bf16(xf)
    x = dev(xf) if dtype == torch.float32 else dev(xb.view(np.int16)).view(torch.bfloat16)
    xkw = {"x": xf} if dtype == torch.float32 else {"x_bf16": xb}
    rp = dev(rp_o.astype(np.int32))
    for use_plan in (False, True):
        plan = mp.Plan(rp, g.E, g.F, dtype, opts=opts) if use_plan else None
        res = mp.spmm_multi(rp, dev(col_o), x, ALL, plan=plan)
        torch.cuda.synchronize()
        errs = compare(res, rp_o, col_o, None, xkw, ALL, dtype)
        assert not res["var"][:, 16:24].any(), "constant messages: variance exactly 0"
        print(f"[note] large-mean multi errors {errs}", file=sys.stderr, flush=True)
    # the readout over the same rows (segments of consecutive rows)
    cuts = np.linspace(0, g.n_src, 9).astype(np.int64)
    res = mp.readout(dev(cuts.astype(np.int32)), x, ["mean", "var", "std"])
    torch.cuda.synchronize()
    compare(res, cuts, np.arange(g.n_src, dtype=np.int32), None, xkw, ["mean", "var", "std"],
            dtype)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_multi_chunglu_full_sampled(dtype):
    """Full-size power-law graph in the benchmark's configuration: one
    stacked call (mean, min, max, std) on fp32 features, and on bf16
    features laid out in 256-byte rows; checked on all hub rows plus random
    rows."""
    g = graphgen.workload("chunglu-124M", seed=0, bf16=dtype == torch.bfloat16)
    rp_o, col_o, _, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    rp, col = dev(rp_o.astype(np.int32)), dev(col_o)
    names = ["mean", "min", "max", "std"]
    if dtype == torch.float32:
        x, xkw = dev(g.x), {"x": g.x}
    else:
        x = mp.pad_rows(dev(g.x_bf16.view(np.int16)).view(torch.bfloat16))
        assert x.stride(0) == 128
        xkw = {"x_bf16": g.x_bf16}
    res = mp.spmm_multi(rp, col, x, names, plan=mp.Plan(rp, g.E, g.F, dtype))
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([np.argsort(np.diff(rp_o))[-64:],
                                     rng.integers(0, g.n_dst, 3000)]))
    errs = compare(res, rp_o, col_o, None, xkw, names, dtype, rows=rows)
    print(f"[note] chunglu multi errors {errs}", file=sys.stderr, flush=True)
