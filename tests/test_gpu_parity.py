"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Integer outputs (rowptr, col, perm, argmax) and max values must be bit-exact.
Sums and means must satisfy max |y - y_ref| / sum_p |m_p| <= 1e-5 for fp32
features and <= 1e-2 for bf16 features (fp32 accumulation in both cases; the
second bound is the stated one for bf16 features, and bf16 outputs add one
bf16 rounding).  Mean uses the same scale divided by the in-degree.
"""
import os
import sys

import numpy as np
import pytest
import torch

import graphgen
import oracle
import paper_2507_16991_amd as mp
from checks import check_csr_invariants, scaled_error

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
TOL = {torch.float32: 1e-5, torch.bfloat16: 1e-2}


@pytest.fixture(autouse=True)
def _announce(request):
    sys.stderr.write(f"\n[gpu-case] {request.node.nodeid}\n")
    sys.stderr.flush()
    yield
    torch.cuda.synchronize()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def x_of(g, dtype):
    if dtype == torch.float32:
        return dev(g.x)
    return dev(g.x_bf16.view(np.int16)).view(torch.bfloat16)


def x_f32_host(g, dtype):
    return g.x if dtype == torch.float32 else graphgen.bf16_to_f32(g.x_bf16)


# ---- COO -> CSR ------------------------------------------------------------------

def check_csr(src, dst, n, rowptr_dtype=torch.int32, val=None):
    s, d = dev(src), dev(dst)
    v = None if val is None else dev(val)
    rp, col, perm, vout = mp.coo_to_csr(s, d, n, rowptr_dtype=rowptr_dtype, want_perm=True, val=v)
    rp_o, col_o, perm_o, v_o = oracle.coo_to_csr(src, dst, n, val=val)
    assert np.array_equal(rp.cpu().numpy().astype(np.int64), rp_o), "rowptr"
    assert np.array_equal(col.cpu().numpy(), col_o), "col"
    assert np.array_equal(perm.cpu().numpy().astype(np.int64), perm_o), "perm"
    if val is not None:
        assert np.array_equal(vout.cpu().numpy().view(np.uint32), v_o.view(np.uint32)), "val"
    return rp, col


def test_csr_worked_example():
    import json
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")))
    rp, col = check_csr(np.array(g["src"], np.int32), np.array(g["dst"], np.int32), g["N"],
                        val=np.array(g["w"], np.float32))
    assert rp.cpu().tolist() == g["rowptr"] and col.cpu().tolist() == g["col"]


@pytest.mark.parametrize("n,e", [(1, 0), (1, 7), (5, 0), (2, 4096), (255, 4095), (256, 4097),
                                 (257, 10000), (1 << 16, 70_001), (70_000, 12_289),
                                 ((1 << 20) + 3, 50_000), (3, 200_000)])
@pytest.mark.parametrize("itype", [torch.int32, torch.int64])
def test_csr_shapes(n, e, itype):
    src = graphgen.uniform_ints(n + e, 1, e, n)
    dst = graphgen.uniform_ints(n + e, 2, e, n)
    val = graphgen.uniform_f32(n + e, 3, e)
    check_csr(src, dst, n, itype, val)


@pytest.mark.parametrize("want_perm", [False, True])
def test_csr_four_passes(want_perm):
    """Keys of 29 bits (N = 2^28 + 5): four radix passes (7/7/7/8 bits), with
    and without the COO-id payload, int64 rowptr."""
    n, e = (1 << 28) + 5, 300_000
    src = graphgen.uniform_ints(11, 1, e, n)
    dst = graphgen.uniform_ints(11, 2, e, n)
    dst[:1000] = n - 1 - np.arange(1000, dtype=np.int32)  # the top digits are used too
    if want_perm:
        check_csr(src, dst, n, torch.int64)
        return
    rp, col, _, _ = mp.coo_to_csr(dev(src), dev(dst), n, rowptr_dtype=torch.int64)
    rp_o, col_o, _, _ = oracle.coo_to_csr(src, dst, n)
    assert np.array_equal(rp.cpu().numpy(), rp_o), "rowptr"
    assert np.array_equal(col.cpu().numpy(), col_o), "col"


@pytest.mark.parametrize("name,scale", [("uniform-10k", 1.0), ("powerlaw-1.2M", 1.0),
                                        ("chunglu-124M", 0.05)])
def test_csr_workloads(name, scale):
    g = graphgen.workload(name, seed=1, scale=scale, **({} if name != "chunglu-124M" else
                                                         {"bf16": False}))
    check_csr(g.src, g.dst, g.n_dst, val=g.w)


def test_csr_sorted_and_single_row():
    n = 1000
    dst = np.sort(graphgen.uniform_ints(5, 2, 30_000, n))
    src = graphgen.uniform_ints(5, 1, 30_000, n)
    check_csr(src, dst, n)
    check_csr(src, np.full(30_000, 999, np.int32), n)  # every edge into the last row


@pytest.mark.parametrize("n,e", [(1, 0), (7, 0), (1, 9), (300, 4095), (70_000, 12_289),
                                 ((1 << 20) + 3, 50_001), (3, 200_000)])
@pytest.mark.parametrize("itype", [torch.int32, torch.int64])
@pytest.mark.parametrize("offset", [0, 1])
def test_sorted_coo_to_csr(n, e, itype, offset):
    # destination-sorted input: no sort runs and the result equals the stable sort's;
    # offset 1 starts dst one element into its buffer (4-byte, not 16-byte, aligned)
    dst = np.sort(graphgen.uniform_ints(n + e, 2, e, n))
    src = graphgen.uniform_ints(n + e, 1, e, n)
    val = graphgen.uniform_f32(n + e, 3, e)
    pad = lambda a: dev(np.concatenate([np.zeros(offset, a.dtype), a]))[offset:]
    s, d, v = pad(src), pad(dst), pad(val)
    rp, col, perm, vout = mp.sorted_coo_to_csr(s, d, n, rowptr_dtype=itype, want_perm=True, val=v)
    rp_o, col_o, perm_o, v_o = oracle.coo_to_csr(src, dst, n, val=val)
    assert np.array_equal(rp.cpu().numpy().astype(np.int64), rp_o), "rowptr"
    assert np.array_equal(col.cpu().numpy(), col_o), "col"
    assert np.array_equal(perm.cpu().numpy().astype(np.int64), perm_o), "perm"
    assert np.array_equal(vout.cpu().numpy().view(np.uint32), v_o.view(np.uint32)), "val"
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    mp.mp_validate_sorted(d, e, cnt)
    assert int(cnt.item()) == 0


def test_sorted_coo_to_csr_unsorted_input_is_bounded():
    """dst that is not sorted (a caller's broken promise): the outputs are
    unspecified but in bounds, and the call finishes (rowptr by one binary
    search per row, not by fills between consecutive keys)."""
    n, e = 100_000, 1_000_000
    dst = graphgen.uniform_ints(7, 2, e, n)  # random order
    src = graphgen.uniform_ints(7, 1, e, n)
    rp, col, _, _ = mp.sorted_coo_to_csr(dev(src), dev(dst), n)
    torch.cuda.synchronize()
    r = rp.cpu().numpy().astype(np.int64)
    assert r[0] == 0 and r[-1] == e and r.min() >= 0 and r.max() <= e
    assert np.array_equal(col.cpu().numpy(), src)


def test_validate_sorted_counts_descents():
    dst = np.sort(graphgen.uniform_ints(4, 2, 5000, 100))
    bad = dst.copy()
    bad[[0, 1]] = bad[[1, 0]]   # a descent at 1 unless the two are equal
    bad[2500], bad[2501] = 99, 0  # a descent at 2501
    expect = int(np.count_nonzero(bad[1:] < bad[:-1]))
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    mp.mp_validate_sorted(dev(bad), 5000, cnt)
    assert int(cnt.item()) == expect and expect >= 1


# ---- aggregation ---------------------------------------------------------------------

REDUCES = {"sum": mp.MP_SUM, "mean": mp.MP_MEAN, "max": mp.MP_MAX,
           "sum+max": mp.MP_SUM | mp.MP_MAX, "mean+max": mp.MP_MEAN | mp.MP_MAX}


def compare_spmm(rp_o, col_o, w_csr, x_host_f32, out, out_max, argout, reduce, dtype,
                 rows=None):
    """Compare device outputs (full arrays, or the listed rows) with the oracle."""
    ref = oracle.spmm(rp_o, col_o, x=x_host_f32, w=w_csr, rows=rows)
    sel = (lambda a: a) if rows is None else (lambda a: a[rows])
    errs = {}
    deg = np.diff(rp_o) if rows is None else (rp_o[rows + 1] - rp_o[rows])
    if reduce & mp.MP_SUM:
        y = sel(out.float().cpu().numpy())
        errs["sum"] = scaled_error(y, ref["sum"], ref["scale"])
    if reduce & mp.MP_MEAN:
        y = sel(out.float().cpu().numpy())
        errs["mean"] = scaled_error(y, ref["mean"], ref["scale"] / np.maximum(deg, 1)[:, None])
    # a bf16 output adds one bf16 rounding (relative 2^-9 <= 2^-8 of the scale)
    tol = TOL[dtype] + (2.0 ** -8 if out is not None and out.dtype == torch.bfloat16 else 0.0)
    for k, e in errs.items():
        assert e <= tol, f"{k} error {e}"
    if reduce & mp.MP_MAX:
        a = sel(argout.cpu().numpy()).astype(np.int64)
        bad = np.argwhere(a != ref["argmax"])
        assert bad.size == 0, f"argmax differs at {bad[:3].tolist()}: " \
                              f"{a[tuple(bad[0])]} vs {ref['argmax'][tuple(bad[0])]}"
        m = sel(out_max.float().cpu().numpy())
        assert np.array_equal(m.view(np.uint32), ref["max"].view(np.uint32)), "max bits"
    return errs


@pytest.fixture(scope="module")
def mixed():
    g = graphgen.mixed_graph(0, f=64)
    rp_o, col_o, perm_o, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    return g, rp_o, col_o, w_o


def run_case(g, rp_o, col_o, w_o, dtype, reduce, weighted, use_plan, out_dtype=torch.float32,
             max_dtype=torch.float32, itype=torch.int32, opts=None):
    rp = dev(rp_o.astype(np.int32 if itype == torch.int32 else np.int64))
    col = dev(col_o)
    x = x_of(g, dtype)
    w = dev(w_o) if weighted else None
    plan = mp.Plan(rp, g.E, g.F, dtype, opts=opts) if use_plan else None
    out, out_max, argout = mp.spmm(rp, col, x, reduce, w=w, plan=plan, out_dtype=out_dtype,
                                   max_dtype=max_dtype)
    torch.cuda.synchronize()
    return compare_spmm(rp_o, col_o, w_o if weighted else None, x_f32_host(g, dtype), out,
                        out_max, argout, reduce, dtype)


@pytest.mark.parametrize("reduce", list(REDUCES))
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("use_plan", [False, True])
def test_spmm_mixed(mixed, reduce, dtype, weighted, use_plan):
    g, rp_o, col_o, w_o = mixed
    run_case(g, rp_o, col_o, w_o, dtype, REDUCES[reduce], weighted, use_plan)


@pytest.mark.parametrize("thresholds", [(8, 64, 16), (1, 2, 1), (64, 256, 64)])
@pytest.mark.parametrize("reduce", ["sum", "mean+max"])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_spmm_plan_regimes(mixed, thresholds, reduce, dtype):
    """Push rows through every code path: small groups, mid rows, hub chunks
    (with tiny chunks, so hubs have many chunks) and the chunk fix-up."""
    g, rp_o, col_o, w_o = mixed
    run_case(g, rp_o, col_o, w_o, dtype, REDUCES[reduce], True, True, opts=thresholds)


@pytest.mark.parametrize("F", [1, 2, 3, 5, 8, 24, 100, 128, 300, 520])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_spmm_feature_widths(F, dtype):
    g = graphgen.mixed_graph(F, n=700, e=9000, f=F)
    rp_o, col_o, _, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    for reduce in (mp.MP_SUM, mp.MP_MEAN | mp.MP_MAX):
        for use_plan in (False, True):
            run_case(g, rp_o, col_o, w_o, dtype, reduce, True, use_plan, opts=(0, 128, 32))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("pad", [0, 1, 4, 28])
def test_spmm_row_stride(mixed, dtype, pad):
    """Feature rows F + pad elements apart (a view of a wider table): an odd
    stride forces narrower vector loads, a stride of whole cache lines is the
    aligned layout; results equal the contiguous table's, and the oracle's."""
    g, rp_o, col_o, w_o = mixed
    F = g.F
    rp, col, w = dev(rp_o.astype(np.int32)), dev(col_o), dev(w_o)
    x = x_of(g, dtype)
    wide = torch.zeros(g.n_src, F + pad, dtype=dtype, device=DEV)
    xs = wide[:, :F]
    xs.copy_(x)
    plan = mp.Plan(rp, g.E, F, dtype)
    for reduce in (mp.MP_SUM | mp.MP_MAX, mp.MP_MEAN):
        a = mp.spmm(rp, col, xs, reduce, w=w, plan=plan)
        b = mp.spmm(rp, col, x, reduce, w=w, plan=plan)
        torch.cuda.synchronize()
        compare_spmm(rp_o, col_o, w_o, x_f32_host(g, dtype), *a, reduce, dtype)
        eb = x.element_size()
        vec = lambda n: next(v for v in (16, 8, 4, 2, 1) if n % v == 0)
        if vec((F + pad) * eb) >= vec(F * eb):  # same lane-chunks: same order, same bits
            for u, v in zip(a, b):
                if u is not None:
                    assert torch.equal(u, v)


@pytest.mark.parametrize("F,ld,dtype", [(100, 128, torch.bfloat16), (3, 4, torch.float32),
                                        (5, 8, torch.bfloat16), (300, 320, torch.bfloat16),
                                        (522, 528, torch.bfloat16), (50, 64, torch.float32),
                                        (7, 9, torch.float32)])
@pytest.mark.parametrize("use_plan", [False, True])
def test_spmm_padded_rows(F, ld, dtype, use_plan):
    """Tables whose row padding holds NaN: whatever vector width the row
    stride allows, no padding element may reach an output row or a hub
    partial."""
    g = graphgen.mixed_graph(F, n=700, e=9000, f=F)
    rp_o, col_o, _, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    rp, col, w = dev(rp_o.astype(np.int32)), dev(col_o), dev(w_o)
    x = x_of(g, dtype)
    xs = mp.pad_rows(x, ld)
    # poison the padding: it is read but must never reach an output
    wide = xs.as_strided((g.n_src, ld), (ld, 1))
    wide[:, F:] = float("nan")
    plan = mp.Plan(rp, g.E, F, dtype, opts=(0, 128, 32)) if use_plan else None
    for reduce, wt in ((mp.MP_SUM | mp.MP_MAX, False), (mp.MP_MEAN, True), (mp.MP_MAX, True)):
        res = mp.spmm(rp, col, xs, reduce, w=w if wt else None, plan=plan)
        torch.cuda.synchronize()
        compare_spmm(rp_o, col_o, w_o if wt else None, x_f32_host(g, dtype), *res, reduce, dtype)
    stats = mp.spmm_multi(rp, col, xs, ["sum", "min", "std"], plan=plan)
    torch.cuda.synchronize()
    for k in ("sum", "min", "std"):
        assert bool(torch.isfinite(stats[k]).all())


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("F,ld", [(100, 128), (3, 5), (64, 64), (300, 320)])
def test_pad_rows(dtype, F, ld):
    rng = np.random.default_rng(F)
    x = torch.from_numpy(rng.standard_normal((777, F)).astype(np.float32)).to(DEV).to(dtype)
    xp = mp.pad_rows(x, ld)
    torch.cuda.synchronize()
    assert xp.shape == (777, F) and xp.stride(0) == ld
    assert torch.equal(xp, x)
    back = mp.pad_rows(xp, F)  # strided in, contiguous out
    torch.cuda.synchronize()
    assert torch.equal(back, x)


def test_spmm_signed_weights_and_ties():
    g = graphgen.mixed_graph(3, f=16, signed_weights=True)
    g.x = (np.round(g.x * 2) / 2).astype(np.float32)  # coarse values: many ties
    g.x_bf16 = graphgen.f32_to_bf16(g.x)
    rp_o, col_o, _, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    for dtype in (torch.float32, torch.bfloat16):
        for weighted in (False, True):
            run_case(g, rp_o, col_o, w_o, dtype, mp.MP_SUM | mp.MP_MAX, weighted, True,
                     opts=(0, 256, 64))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("use_plan", [False, True])
def test_spmm_infinite_messages(mixed, dtype, use_plan):
    """Infinities are ordinary values: a row whose messages of a feature are
    all -inf has max -inf at its FIRST edge (the empty pair is always
    replaced by the first message), and +inf wins wherever it occurs.
    Feature 0 is -inf in every source row, feature 1 +inf in every source
    row, feature 2 -inf in every other source row; the rest stay finite."""
    g, rp_o, col_o, w_o = mixed
    x = g.x.copy()
    x[:, 0] = -np.inf
    x[:, 1] = np.inf
    x[::2, 2] = -np.inf
    xb = graphgen.f32_to_bf16(x)
    xh = x if dtype == torch.float32 else graphgen.bf16_to_f32(xb)
    xd = dev(x) if dtype == torch.float32 else dev(xb.view(np.int16)).view(torch.bfloat16)
    rp, col = dev(rp_o.astype(np.int32)), dev(col_o)
    plan = mp.Plan(rp, g.E, g.F, dtype, opts=(8, 64, 16)) if use_plan else None
    _, out_max, argout = mp.spmm(rp, col, xd, mp.MP_MAX, plan=plan)
    torch.cuda.synchronize()
    ref = oracle.spmm(rp_o, col_o, x=xh, want=("max",))
    assert np.array_equal(argout.cpu().numpy().astype(np.int64), ref["argmax"])
    assert np.array_equal(out_max.cpu().numpy().view(np.uint32), ref["max"].view(np.uint32))
    deg = np.diff(rp_o)
    first = np.where(deg > 0, rp_o[:-1], -1)
    assert np.array_equal(ref["argmax"][:, 0], first), "oracle: all -inf -> first edge"
    # the stacked statistics: min of the +inf feature at the first edge too
    res = mp.spmm_multi(rp, col, xd, ["max", "min"], plan=plan)
    torch.cuda.synchronize()
    assert np.array_equal(res["argmax"].cpu().numpy().astype(np.int64), ref["argmax"])
    mref = oracle.spmm_multi(rp_o, col_o, x=xh)
    assert np.array_equal(res["argmin"].cpu().numpy().astype(np.int64), mref["argmin"])
    assert np.array_equal(res["min"].cpu().numpy().view(np.uint32),
                          mref["min"].view(np.uint32))
    assert np.array_equal(mref["argmin"][:, 1], first), "oracle: all +inf -> first edge"


def test_spmm_output_dtypes(mixed):
    g, rp_o, col_o, w_o = mixed
    run_case(g, rp_o, col_o, w_o, torch.bfloat16, mp.MP_SUM | mp.MP_MAX, False, True,
             out_dtype=torch.bfloat16, max_dtype=torch.bfloat16)
    run_case(g, rp_o, col_o, w_o, torch.float32, mp.MP_MEAN, True, True, out_dtype=torch.bfloat16)
    run_case(g, rp_o, col_o, w_o, torch.float32, mp.MP_MEAN | mp.MP_MAX, True, True,
             itype=torch.int64)


def test_spmm_empty_and_degenerate():
    # no edges at all: every row empty
    n = 300
    x = torch.randn(n, 12, device=DEV)
    rp = torch.zeros(n + 1, dtype=torch.int32, device=DEV)
    col = torch.zeros(1, dtype=torch.int32, device=DEV)
    for use_plan in (False, True):
        plan = mp.Plan(rp, 0, 12) if use_plan else None
        out, m, a = mp.spmm(rp, col, x, mp.MP_SUM | mp.MP_MAX, plan=plan)
        assert torch.all(out == 0) and torch.all(a == -1)
        assert torch.all(m.view(torch.int32) == 0)
    # bipartite: N_dst != N_src, a single destination row
    src = graphgen.uniform_ints(9, 1, 5000, 4000)
    dst = np.zeros(5000, np.int32)
    xs = graphgen.normal_f32(9, 3, 4000 * 4).reshape(4000, 4)
    rp_o, col_o, _, _ = oracle.coo_to_csr(src, dst, 1, n_src=4000)
    for use_plan in (False, True):
        rpd = dev(rp_o.astype(np.int32))
        plan = mp.Plan(rpd, 5000, 4) if use_plan else None
        out, m, a = mp.spmm(rpd, dev(col_o), dev(xs), mp.MP_SUM | mp.MP_MAX, plan=plan)
        torch.cuda.synchronize()
        compare_spmm(rp_o, col_o, None, xs, out, m, a, mp.MP_SUM | mp.MP_MAX, torch.float32)


def test_plan_mismatch_rejected_and_dtype_shared(mixed):
    g, rp_o, col_o, w_o = mixed
    rp = dev(rp_o.astype(np.int32))
    plan = mp.Plan(rp, g.E, g.F, torch.float32)
    # a plan serves both feature dtypes
    out, _, _ = mp.spmm(rp, dev(col_o), x_of(g, torch.bfloat16), mp.MP_SUM, plan=plan)
    torch.cuda.synchronize()
    compare_spmm(rp_o, col_o, None, x_f32_host(g, torch.bfloat16), out, None, None, mp.MP_SUM,
                 torch.bfloat16)
    # a different feature width or rowptr does not
    x8 = torch.zeros(g.n_src, 8, device=DEV)
    with pytest.raises(mp.MPError) as e:
        mp.spmm(rp, dev(col_o), x8, mp.MP_SUM, plan=plan)
    assert e.value.status == -6
    with pytest.raises(mp.MPError) as e:
        mp.spmm(rp.clone(), dev(col_o), x_of(g, torch.float32), mp.MP_SUM, plan=plan)
    assert e.value.status == -6


def test_determinism_across_runs_and_streams(mixed):
    g, rp_o, col_o, w_o = mixed
    rp, col, x, w = dev(rp_o.astype(np.int32)), dev(col_o), x_of(g, torch.float32), dev(w_o)
    plan = mp.Plan(rp, g.E, g.F, opts=(0, 256, 64))
    outs = []
    for k in range(3):
        s = torch.cuda.Stream() if k == 2 else torch.cuda.current_stream()
        with torch.cuda.stream(s):
            outs.append(mp.spmm(rp, col, x, mp.MP_SUM | mp.MP_MAX, w=w, plan=plan))
        torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o[0].view(torch.int32), outs[0][0].view(torch.int32))
        assert torch.equal(o[2], outs[0][2])


def test_validate_kernels():
    src = graphgen.uniform_ints(2, 1, 1000, 50)
    dst = graphgen.uniform_ints(2, 2, 1000, 50)
    cnt = torch.zeros(1, dtype=torch.int64, device=DEV)
    mp.mp_validate_coo(dev(src), dev(dst), 1000, 50, 50, cnt)
    assert int(cnt.item()) == 0
    bad = dst.copy()
    bad[[3, 500]] = [50, -1]
    mp.mp_validate_coo(dev(src), dev(bad), 1000, 50, 50, cnt)
    assert int(cnt.item()) == 2
    rp_o, col_o, _, _ = oracle.coo_to_csr(src, dst, 50)
    rp = dev(rp_o.astype(np.int32))
    mp.mp_validate_csr(rp, mp.MP_I32, dev(col_o), 50, 50, 1000, cnt)
    assert int(cnt.item()) == 0
    rp2 = rp.clone()
    rp2[10] = rp2[11] + 1  # one decreasing step (10 -> 11)
    mp.mp_validate_csr(rp2, mp.MP_I32, dev(col_o), 50, 50, 1000, cnt)
    assert int(cnt.item()) == 1


# ---- workloads -------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["uniform-10k", "powerlaw-1.2M"])
def test_workload_small_full(name):
    g = graphgen.workload(name, seed=0)
    s, d = dev(g.src), dev(g.dst)
    rp, col, perm, wc = mp.coo_to_csr(s, d, g.n_dst, want_perm=True,
                                      val=None if g.w is None else dev(g.w))
    rp_o, col_o, perm_o, w_o = oracle.coo_to_csr(g.src, g.dst, g.n_dst, val=g.w)
    assert np.array_equal(col.cpu().numpy(), col_o)
    plan = mp.Plan(rp, g.E, g.F)
    x = dev(g.x)
    cases = [(mp.MP_SUM, None)] if g.w is None else [(mp.MP_MEAN, None), (mp.MP_SUM, wc)]
    for reduce, w in cases:
        out, _, _ = mp.spmm(rp, col, x, reduce, w=w, plan=plan)
        torch.cuda.synchronize()
        errs = compare_spmm(rp_o, col_o, None if w is None else w_o, g.x, out, None, None, reduce,
                            torch.float32)
        print(name, reduce, errs)


@pytest.fixture(scope="module")
def chunglu_full():
    g = graphgen.workload("chunglu-124M", seed=0)
    rp_o, col_o, perm_o, _ = oracle.coo_to_csr(g.src, g.dst, g.n_dst)
    return g, rp_o, col_o, perm_o


def test_chunglu_124M_csr_bit_exact(chunglu_full):
    g, rp_o, col_o, perm_o = chunglu_full
    rp, col, perm, _ = mp.coo_to_csr(dev(g.src), dev(g.dst), g.n_dst, want_perm=True)
    assert np.array_equal(rp.cpu().numpy().astype(np.int64), rp_o)
    assert np.array_equal(col.cpu().numpy(), col_o)
    assert np.array_equal(perm.cpu().numpy().astype(np.int64), perm_o)


def compare_rows_chunked(ref, rp_o, out, out_max, argout, reduce, tol, chunk=1 << 18):
    """Every row of a full-size call against the oracle's outputs for all
    rows, in blocks of rows (bounded host memory).  Returns the worst scaled
    error of the sum or mean."""
    deg = np.diff(rp_o)
    y = out.float().cpu().numpy() if out is not None else None
    m = out_max.float().cpu().numpy() if out_max is not None else None
    a = argout.cpu().numpy() if argout is not None else None
    worst = 0.0
    n = deg.shape[0]
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        if reduce & mp.MP_SUM:
            e = scaled_error(y[r0:r1], ref["sum"][r0:r1], ref["scale"][r0:r1])
            assert e <= tol, f"rows {r0}..{r1}: sum error {e}"
            worst = max(worst, e)
        if reduce & mp.MP_MEAN:
            sc = ref["scale"][r0:r1] / np.maximum(deg[r0:r1], 1)[:, None]
            e = scaled_error(y[r0:r1], ref["mean"][r0:r1], sc)
            assert e <= tol, f"rows {r0}..{r1}: mean error {e}"
            worst = max(worst, e)
        if reduce & mp.MP_MAX:
            bad = np.argwhere(a[r0:r1].astype(np.int64) != ref["argmax"][r0:r1])
            assert bad.size == 0, f"argmax differs at row {r0 + bad[0][0]}, feature {bad[0][1]}"
            assert np.array_equal(m[r0:r1].view(np.uint32),
                                  ref["max"][r0:r1].view(np.uint32)), f"max bits, rows {r0}.."
    return worst


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_chunglu_124M_spmm_all_rows(chunglu_full, dtype):
    """Full-size run in the benchmark's configuration (bf16 features laid
    out in 256-byte rows, as the benchmark's step does), compared with the
    oracle on EVERY one of the 2,449,029 rows: sum, mean, max + argmax and
    the fused sum|max call.  bf16 features widen to fp32 exactly and are
    accumulated in fp32, so their sums and means are held to the fp32 bound
    (1e-5) as well as the stated 1e-2."""
    g, rp_o, col_o, _ = chunglu_full
    rp = dev(rp_o.astype(np.int32))
    col = dev(col_o)
    x = x_of(g, dtype)
    if dtype == torch.bfloat16:
        x = mp.pad_rows(x)
        assert x.stride(0) == 128
    plan = mp.Plan(rp, g.E, g.F, dtype)
    ref = (oracle.spmm(rp_o, col_o, x=g.x) if dtype == torch.float32
           else oracle.spmm(rp_o, col_o, x_bf16=g.x_bf16))
    for reduce in (mp.MP_SUM, mp.MP_MEAN, mp.MP_MAX, mp.MP_SUM | mp.MP_MAX):
        out, out_max, argout = mp.spmm(rp, col, x, reduce, plan=plan)
        torch.cuda.synchronize()
        worst = compare_rows_chunked(ref, rp_o, out, out_max, argout, reduce, TOL[torch.float32])
        sys.stderr.write(f"chunglu all rows {dtype} reduce {reduce}: worst error {worst:.3e}\n")
        del out, out_max, argout


# ---- heterogeneous -------------------------------------------------------------------------

def run_hetero(g, plan_on=True, one_buffer=False):
    """one_buffer: the per-type tables are consecutive slices of one tensor
    (the library then gathers from it as a single table)."""
    T = len(g.n_per_type)
    rels = [(g.rel_src_type[r], g.rel_dst_type[r], dev(g.rel_src[r]), dev(g.rel_dst[r]))
            for r in range(len(g.rel_src))]
    if one_buffer:
        allx = dev(np.concatenate(g.x_bf16).view(np.int16)).view(torch.bfloat16)
        xs = list(torch.split(allx, g.n_per_type))
    else:
        xs = [dev(x.view(np.int16)).view(torch.bfloat16) for x in g.x_bf16]
    outs_o, scs_o = oracle.hetero_sum(g.n_per_type, g.x_bf16, g.rel_src_type, g.rel_dst_type,
                                      g.rel_src, g.rel_dst)
    per_type = {}
    for t in range(T):
        if t not in g.rel_dst_type:
            continue
        rp, col = mp.hetero_build(g.n_per_type, rels, t)
        E_T = int(col.numel())
        plan = mp.Plan(rp, E_T, g.F, torch.bfloat16) if plan_on else None
        out = mp.hetero_spmm(g.n_per_type, xs, t, rp, col, plan=plan)
        torch.cuda.synchronize()
        per_type[t] = (rp.cpu().numpy().astype(np.int64), col.cpu().numpy())
        err = scaled_error(out.cpu().numpy(), outs_o[t], scs_o[t])
        assert err <= TOL[torch.bfloat16], f"type {t}: error {err}"
        assert err <= 1e-5, f"type {t}: fp32 accumulation error {err}"
    # every destination type at once: one CSR over all nodes (global ids)
    # whose row slices are exactly the per-type CSRs, and one aggregation
    rp, col = mp.hetero_build(g.n_per_type, rels, mp.MP_ALL_TYPES)
    plan = mp.Plan(rp, int(col.numel()), g.F, torch.bfloat16) if plan_on else None
    out = mp.hetero_spmm(g.n_per_type, xs, mp.MP_ALL_TYPES, rp, col, plan=plan)
    torch.cuda.synchronize()
    rp_h, col_h, out_h = rp.cpu().numpy().astype(np.int64), col.cpu().numpy(), out.cpu().numpy()
    offs = np.concatenate([[0], np.cumsum(g.n_per_type)])
    for t in range(T):
        a, b = offs[t], offs[t + 1]
        if t in per_type:
            rp_t, col_t = per_type[t]
            assert np.array_equal(rp_h[a:b + 1] - rp_h[a], rp_t), f"type {t}: rowptr slice"
            assert np.array_equal(col_h[rp_h[a]:rp_h[b]], col_t), f"type {t}: col slice"
            err = scaled_error(out_h[a:b], outs_o[t], scs_o[t])
            assert err <= 1e-5, f"all types, type {t}: error {err}"
        else:
            assert rp_h[b] == rp_h[a] and not out_h[a:b].any(), f"type {t}: no incoming edges"


def test_hetero_small():
    g = graphgen.hetero_graph(4, [3000, 1200, 70],
                              [(0, 0, 9000), (0, 1, 11000), (1, 0, 10000), (1, 2, 4000)], 128)
    run_hetero(g, True)
    run_hetero(g, False)
    run_hetero(g, True, one_buffer=True)


def test_hetero_many_types():
    """More node types than the 4-table kernel variant covers."""
    n = [500, 40, 700, 1, 300, 90, 2000]
    rels = [(a, b, 300 + 97 * (a * 7 + b)) for a in range(7) for b in range(7) if (a + b) % 3 == 0]
    g = graphgen.hetero_graph(8, n, rels, 64)
    run_hetero(g, True)
    run_hetero(g, False)


def test_hetero_20M():
    g = graphgen.workload("hetero-20M", seed=0)
    run_hetero(g, True)
    run_hetero(g, True, one_buffer=True)


# ---- web-scale single-GPU shard ---------------------------------------------------------

def _note(msg):
    sys.stderr.write(f"[web-1.6B] {msg}\n")
    sys.stderr.flush()


def test_web_1_6B_fused_sum_max_sampled():
    """N = 1e8, E = 1.6e9, F = 64 bf16, int64 rowptr, fused sum (fp32) + max
    (bf16, exact) + argmax in one pass, as the benchmark option runs it.
    rowptr is checked in full against numpy's bincount + cumsum; the column
    segments and outputs of sampled rows (the 2 largest rows -- the top one
    holds ~84M edges --, 16 random rows among those with >= 10^4 edges, and
    20k random rows, empty ones included) are checked against the oracle
    computed straight from COO."""
    g = graphgen.workload("web-1.6B", seed=0)
    N, E, F = g.n_dst, g.E, g.F
    _note(f"generated N={N} E={E}")
    s, d = dev(g.src), dev(g.dst)
    rp, col, _, _ = mp.coo_to_csr(s, d, N, rowptr_dtype=torch.int64)
    del s, d
    torch.cuda.synchronize()
    deg = np.bincount(g.dst, minlength=N).astype(np.int64)
    below = np.concatenate([[0], np.cumsum(deg)])
    rp_h = rp.cpu().numpy()
    assert np.array_equal(rp_h, below), "rowptr"
    _note(f"rowptr ok, max degree {deg.max()}")

    top = np.argsort(deg)[-2:]
    hubs = np.nonzero(deg >= 10_000)[0]
    pick = hubs[graphgen.uniform_ints(12, 6, 16, hubs.shape[0])]
    rnd = graphgen.uniform_ints(12, 5, 20_000, N).astype(np.int64)
    rows = np.unique(np.concatenate([top, pick, rnd])).astype(np.int64)
    seg, cols_ref = oracle.csr_rows(g.src, g.dst, N, rows)
    _note(f"oracle column segments of {rows.shape[0]} rows ({cols_ref.shape[0]} edges)")
    idx = np.concatenate([np.arange(rp_h[r], rp_h[r + 1]) for r in rows]).astype(np.int64)
    assert np.array_equal(col[dev(idx)].cpu().numpy(), cols_ref), "col segments"
    del idx, cols_ref
    _note("column segments ok")

    x = dev(g.x_bf16.view(np.int16)).view(torch.bfloat16)
    plan = mp.Plan(rp, E, F, torch.bfloat16)
    out, out_max, argout = mp.spmm(rp, col, x, mp.MP_SUM | mp.MP_MAX, plan=plan,
                                   max_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    rd = dev(rows)
    y = out[rd].cpu().numpy()
    ym = out_max[rd].view(torch.int16).cpu().numpy().view(np.uint16)
    ya = argout[rd].cpu().numpy().astype(np.int64)
    del out, out_max, argout, x
    _note("device aggregation done")
    ref = oracle.spmm_coo_rows(g.src, g.dst, N, rows, x_bf16=g.x_bf16, row_start=below[rows])
    err = scaled_error(y, ref["sum"], ref["scale"])
    _note(f"rows {rows.shape[0]} sum error {err:.3e}")
    assert err <= TOL[torch.bfloat16], f"sum error {err}"
    assert err <= 1e-5, f"fp32 accumulation error {err}"
    assert np.array_equal(ya, ref["argmax"]), "argmax"
    assert np.array_equal(ym, (ref["max"].view(np.uint32) >> 16).astype(np.uint16)), "max bits"
