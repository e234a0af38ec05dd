"""Parity of the stacked aggregations and the global readout (through the C
ABI) with the CPU oracle.

max/argmax and min/argmin must be bit-exact; sum and mean are held to the
summand-scaled bound of the forward tests (1e-5 for fp32 features, 1e-2 for
bf16); the variance, computed in one pass as E[m^2] - E[m]^2, to the same
bound relative to var_scale = sum m^2 / deg + (sum |m| / deg)^2, and the
standard deviation to the square root of that bound (|sqrt a - sqrt b| <=
sqrt |a - b|).
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
            errs[n] = scaled_error(y, mul["var"], mul["var_scale"])
        elif n == "std":
            d = np.abs(y.astype(np.float64) - mul["std"])
            bound = np.sqrt(tol * mul["var_scale"])
            assert np.all((d <= bound) | (d == 0)), f"std off by {np.max(d - bound)}"
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
